// Shared device helpers for the gfx950 kernels: element types, conversions,
// 16-byte vector access and wave-wide (64-lane) reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nt {

typedef _Float16 f16;
typedef __bf16 bf16;

constexpr int kWave = 64;

template <typename T> __device__ __forceinline__ float to_f32(T v) { return static_cast<float>(v); }
template <typename T> __device__ __forceinline__ T from_f32(float v) { return static_cast<T>(v); }

// Elements of T in one 16-byte vector.
template <typename T> struct Vec { static constexpr int N = 16 / sizeof(T); };

// Load / store N = 16/sizeof(T) consecutive elements as fp32.
template <typename T>
__device__ __forceinline__ void load16(const T* p, float* out) {
  uint4 raw = *reinterpret_cast<const uint4*>(p);
  const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) out[i] = to_f32(e[i]);
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const float* in) {
  uint4 raw;
  T* e = reinterpret_cast<T*>(&raw);
#pragma unroll
  for (int i = 0; i < Vec<T>::N; ++i) e[i] = from_f32<T>(in[i]);
  *reinterpret_cast<uint4*>(p) = raw;
}

// Load/store EPL contiguous elements (EPL a multiple of 16/sizeof(T), or 2 for tiny rows).
template <typename T, int EPL>
__device__ __forceinline__ void load_row(const T* p, float* out) {
  if constexpr (EPL * sizeof(T) % 16 == 0) {
#pragma unroll
    for (int i = 0; i < EPL; i += Vec<T>::N) load16(p + i, out + i);
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) out[i] = to_f32(p[i]);
  }
}
template <typename T, int EPL>
__device__ __forceinline__ void store_row(T* p, const float* in) {
  if constexpr (EPL * sizeof(T) % 16 == 0) {
#pragma unroll
    for (int i = 0; i < EPL; i += Vec<T>::N) store16(p + i, in + i);
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) p[i] = from_f32<T>(in[i]);
  }
}

// Butterfly reductions: every lane ends with the same bits (each step adds a pair that
// its partner adds in the other order, and fp addition is commutative).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// LayerNorm of one row held as EPL fp32 values per lane (row length 64*EPL):
// biased variance, two passes over registers, fp32 throughout.
template <int EPL>
__device__ __forceinline__ void wave_layernorm(const float* x, float* y, const float* gamma,
                                               const float* beta, int col0, float inv_d, float eps) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) s += x[i];
  const float mean = wave_sum(s) * inv_d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const float c = x[i] - mean;
    q += c * c;
  }
  const float var = wave_sum(q) * inv_d;
  const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
  for (int i = 0; i < EPL; ++i) y[i] = (x[i] - mean) * rstd * gamma[col0 + i] + beta[col0 + i];
}

}  // namespace nt
