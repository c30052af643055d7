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

// One MFMA step over a 16-byte fragment per lane: 16x16 fp32 accumulator C += A.B^T
// with lane l supplying row (l % 16) of A and of B^T at k-chunk (l / 16); only the two
// operands' agreement on which k a lane element carries matters.  fp16/bf16 use
// v_mfma_f32_16x16x32_{f16,bf16} (k = 32); fp32 uses four v_mfma_f32_16x16x4_f32 (true
// fp32 products, k = 16).  Lane l receives C[4*(l/16) + r][l % 16] in element r.
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bhalf8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;
template <> struct Mfma<f16> {
  static __device__ __forceinline__ floatx4 step(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c,
                                                  0, 0, 0);
  }
};
template <> struct Mfma<bf16> {
  static __device__ __forceinline__ floatx4 step(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bhalf8, a), __builtin_bit_cast(bhalf8, b),
                                                   c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static __device__ __forceinline__ floatx4 step(u32x4 a, u32x4 b, floatx4 c) {
    const floatx4 av = __builtin_bit_cast(floatx4, a);
    const floatx4 bv = __builtin_bit_cast(floatx4, b);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, c, 0, 0, 0);
    return c;
  }
};

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
