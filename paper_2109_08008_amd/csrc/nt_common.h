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

// Code of the OCP FP8 E4M3 value (exponent bias 7, 3 mantissa bits, subnormals in steps
// of 2^-9, largest finite 448) nearest to x, ties to even; magnitudes beyond 448
// saturate to 448 and NaN gives 0x7F.  On the fp32 bits: below 2^-6 the value is a
// multiple of 2^-9 (code 8 is 2^-6 itself), found by an exact scaling and a rounding to
// the nearest even integer; above, the 23-bit mantissa is rounded to 3 bits (a carry
// moves into the exponent) and the exponent is rebiased from 127 to 7.  The host
// quantizer of FP8 weights and the projection that writes an FP8 key/value cache both
// use it.
__host__ __device__ inline uint8_t e4m3_rne(float x) {
  const uint32_t bits = __builtin_bit_cast(uint32_t, x);
  const uint32_t sign = (bits >> 24) & 0x80u, u = bits & 0x7FFFFFFFu;
  if (u > 0x7F800000u) return 0x7F;
  uint32_t code;
  if (u < 0x3C800000u) {
    code = (uint32_t)__builtin_rintf(__builtin_bit_cast(float, u) * 512.0f);
  } else {
    code = ((u + 0x7FFFFu + ((u >> 20) & 1u)) >> 20) - (120u << 3);
    if (code > 0x7Eu) code = 0x7Eu;
  }
  return (uint8_t)(sign | code);
}

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

// Whole-wave reductions without an LDS round trip per step.  Inside each row of 16
// lanes four DPP butterfly steps: lane^1 and lane^2 by quad permutes, then the mirrored
// half of each 8 and of each 16 lanes, which after the earlier steps holds the partial of
// lane^4 and lane^8.  The four row results are then read as scalars and combined as
// (r0 op r1) op (r2 op r3).  Each step pairs partials symmetrically and fp addition is
// commutative, so every lane ends with the same bits: the xor butterfly's result taken
// over the offsets 1, 2, ..., 32 in that order.  All 64 lanes must be active (every
// caller reduces across a whole wave).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_mov_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ float readlane_f(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
__device__ __forceinline__ int readlane_i(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
constexpr int DPP_XOR1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane 7-j of each 8
constexpr int DPP_MIRROR = 0x140;       // lane 15-j of each 16
constexpr int DPP_XOR8 = 0x128;         // row_ror:8, lane j^8 of each 16
// Sum over aligned groups of N consecutive lanes (N = 1, 2, 4, 8 or 16), by the same
// steps: every lane of a group ends with the group's sum, the xor butterfly's bits.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "a power-of-two group inside a row");
  if constexpr (N >= 2) v += dpp_mov<DPP_XOR1>(v);
  if constexpr (N >= 4) v += dpp_mov<DPP_XOR2>(v);
  if constexpr (N >= 8) v += dpp_mov<DPP_HALF_MIRROR>(v);
  if constexpr (N >= 16) v += dpp_mov<DPP_MIRROR>(v);
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<DPP_XOR1>(v);
  v += dpp_mov<DPP_XOR2>(v);
  v += dpp_mov<DPP_HALF_MIRROR>(v);
  v += dpp_mov<DPP_MIRROR>(v);
  return (readlane_f(v, 0) + readlane_f(v, 16)) + (readlane_f(v, 32) + readlane_f(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<DPP_XOR1>(v));
  v = fmaxf(v, dpp_mov<DPP_XOR2>(v));
  v = fmaxf(v, dpp_mov<DPP_HALF_MIRROR>(v));
  v = fmaxf(v, dpp_mov<DPP_MIRROR>(v));
  return fmaxf(fmaxf(readlane_f(v, 0), readlane_f(v, 16)), fmaxf(readlane_f(v, 32), readlane_f(v, 48)));
}

// LayerNorm of one row held as EPL fp32 values per lane (row length 64*EPL):
// biased variance, two passes over registers, fp32 throughout.
template <int EPL>
struct LnCols {   // the lane's gain and bias columns
  float g[EPL], b[EPL];
};
template <int EPL>
__device__ __forceinline__ void load_ln_cols(const float* gamma, const float* beta, int col0, LnCols<EPL>& c) {
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    c.g[i] = gamma[col0 + i];
    c.b[i] = beta[col0 + i];
  }
}
template <int EPL>
__device__ __forceinline__ void wave_layernorm(const float* x, float* y, const LnCols<EPL>& c, float inv_d,
                                               float eps) {
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
  for (int i = 0; i < EPL; ++i) y[i] = (x[i] - mean) * rstd * c.g[i] + c.b[i];
}
// The same with the gain and bias read at the call (their loads overlap the reductions).
template <int EPL>
__device__ __forceinline__ void wave_layernorm(const float* x, float* y, const float* gamma,
                                               const float* beta, int col0, float inv_d, float eps) {
  LnCols<EPL> c;
  load_ln_cols<EPL>(gamma, beta, col0, c);
  wave_layernorm<EPL>(x, y, c, inv_d, eps);
}

}  // namespace nt
