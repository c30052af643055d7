// Dense projections of the encoder, the decoder step and the tied output projection
// (the "MM" that dominates the paper's GPU profile, Sec. 4.4) as one MFMA GEMM for
// gfx950:  C[M,N] = A[M,K] . Bt[N,K]^T with fp32 accumulation and a fused epilogue.
//
// Tiling: 128x128 output tile per 256-thread workgroup, four waves in a 2x2 grid, each
// owning 64x64 = 4x4 MFMA blocks of 16x16.  K advances 128 bytes per step (64 halves or
// 32 floats), double-buffered through LDS (2 x 32 KB) with an XOR swizzle of the
// 16-byte chunks so that both the cooperative stores and the fragment reads are free of
// bank conflicts.  fp16/bf16 use v_mfma_f32_16x16x32_{f16,bf16}; fp32 uses four
// v_mfma_f32_16x16x4_f32 per 16-byte fragment (true fp32 products, no reduced-precision
// inputs).  Because the two operands of an MFMA only need to agree on which k each
// lane supplies, lane l feeds A[row l%16][k-chunk l/16] and Bt[col l%16][same chunk].
//
// Tiles are numbered so that neighbouring tiles (which share A rows or B columns) run
// on the same XCD: workgroup ids are dealt round-robin over the 8 XCDs, so id -> tile
// is remapped to give each XCD a contiguous range, then grouped 8 tile-rows at a time.
//
// Every output element is reduced over K in the same order whatever M is, so a row's
// result does not depend on how many other rows share the launch (batch invariance).
#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

constexpr int BM = 128, BN = 128;
constexpr int ROWB = 128;           // bytes of K per tile row per step
constexpr int CH = ROWB / 16;       // 16-byte chunks per tile row
constexpr int NTHR = 256;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bhalf8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;
template <> struct Mfma<f16> {
  static __device__ __forceinline__ floatx4 step(const uint4& a, const uint4& b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a), __builtin_bit_cast(half8, b), c,
                                                  0, 0, 0);
  }
};
template <> struct Mfma<bf16> {
  static __device__ __forceinline__ floatx4 step(const uint4& a, const uint4& b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bhalf8, a), __builtin_bit_cast(bhalf8, b),
                                                   c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static __device__ __forceinline__ floatx4 step(const uint4& a, const uint4& b, floatx4 c) {
    const float4 av = __builtin_bit_cast(float4, a);
    const float4 bv = __builtin_bit_cast(float4, b);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, c, 0, 0, 0);
    return c;
  }
};

// Byte offset of 16-byte chunk `ch` of tile row `row` in a swizzled LDS tile.
__device__ __forceinline__ int swz(int row, int ch) { return row * ROWB + ((ch ^ (row & 7)) << 4); }

// Applies the epilogue to up to 4 consecutive columns n..n+3 of row m (n % 4 == 0).
// d, dh and ldc are multiples of 4 in every mode that scatters, so the 4 columns never
// straddle a head or a K/V boundary and land on 4 consecutive destination elements.
template <typename T>
__device__ __forceinline__ void epilogue4(const GemmEpi& e, int m, int n, int N, float4 v4) {
  float v[4] = {v4.x, v4.y, v4.z, v4.w};
  const int cnt = min(4, N - n);
  if (e.bias) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (k < cnt) v[k] += e.bias[n + k];
  }
  const bool vec = cnt == 4 && (e.ldc & 3) == 0;
  if (e.out_f32) {
    float* o = static_cast<float*>(e.out) + (size_t)m * e.ldc + n;
    if (vec) {
      *reinterpret_cast<float4*>(o) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (k < cnt) o[k] = v[k];
    }
    return;
  }
  T* o = nullptr;
  switch (e.mode) {
    case EPI_STORE:
      o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
      break;
    case EPI_RELU:
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = fmaxf(v[k], 0.f);
      o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
      break;
    case EPI_RESID: {
      const T* r = static_cast<const T*>(e.resid) + (size_t)m * e.ldc + n;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (k < cnt) v[k] += to_f32(r[k]);
      o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
      break;
    }
    case EPI_SELF_QKV: {
      if (n < e.d) {
        o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
      } else {
        int c = n - e.d;
        const int kv = c >= e.d;
        c -= kv * e.d;
        const int h = c / e.dh, x = c - h * e.dh;
        const int p = e.sent_list[m / e.beam] * e.beam + m % e.beam;
        o = static_cast<T*>(kv ? e.vcache : e.kcache) + ((size_t)(p * e.H + h) * e.Tcap + e.t) * e.dh + x;
      }
      break;
    }
    case EPI_CROSS_KV: {
      const int j = n / (2 * e.d);
      int c = n - j * 2 * e.d;
      const int kv = c >= e.d;
      c -= kv * e.d;
      const int h = c / e.dh, x = c - h * e.dh;
      const int b = m / e.S, s = m - b * e.S;
      o = static_cast<T*>(e.cross) + ((((size_t)j * 2 + kv) * e.B + b) * e.H + h) * (size_t)e.S * e.dh +
          (size_t)s * e.dh + x;
      break;
    }
  }
  if (vec || (e.mode >= EPI_SELF_QKV && cnt == 4)) {
    if constexpr (sizeof(T) == 2) {
      T t4[4] = {from_f32<T>(v[0]), from_f32<T>(v[1]), from_f32<T>(v[2]), from_f32<T>(v[3])};
      *reinterpret_cast<uint2*>(o) = *reinterpret_cast<const uint2*>(t4);
    } else {
      *reinterpret_cast<float4*>(o) = make_float4(v[0], v[1], v[2], v[3]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (k < cnt) o[k] = from_f32<T>(v[k]);
  }
}

template <typename T, int ROLE>
__global__ __launch_bounds__(NTHR) void gemm_kernel(const T* __restrict__ A, int lda, const T* __restrict__ Bt,
                                                    int M, int N, int K, GemmEpi epi, int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][(BM + BN) * ROWB];

  // --- tile assignment: XCD-contiguous, then grouped by 8 tile-rows ---
  const int ntiles = tiles_m * tiles_n;
  int pid = blockIdx.x;
  {
    const int q = ntiles / 8, r = ntiles % 8, xcd = pid % 8, idx = pid / 8;
    pid = xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  }
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int first_m = (pid / per_group) * GROUP;
  const int gsize = min(tiles_m - first_m, GROUP);
  const int tm = first_m + (pid % per_group) % gsize;
  const int tn = (pid % per_group) / gsize;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const char* Ab = reinterpret_cast<const char*>(A);
  const char* Bb = reinterpret_cast<const char*>(Bt);

  // --- global -> register staging: 4 chunks of A and 4 of Bt per thread per step ---
  // Rows past the edge re-read the last valid row; their results are never stored.
  const int row0 = tid / CH, ch0 = tid % CH;      // chunk i covers tile row row0 + 32*i
  constexpr int RSTEP = NTHR / CH;
  const size_t lda_b = (size_t)lda * sizeof(T), ldb_b = (size_t)K * sizeof(T);
  const char* const pa0 = Ab + (size_t)min(m0 + row0 + 0 * RSTEP, M - 1) * lda_b + ch0 * 16;
  const char* const pa1 = Ab + (size_t)min(m0 + row0 + 1 * RSTEP, M - 1) * lda_b + ch0 * 16;
  const char* const pa2 = Ab + (size_t)min(m0 + row0 + 2 * RSTEP, M - 1) * lda_b + ch0 * 16;
  const char* const pa3 = Ab + (size_t)min(m0 + row0 + 3 * RSTEP, M - 1) * lda_b + ch0 * 16;
  const char* const pb0 = Bb + (size_t)min(n0 + row0 + 0 * RSTEP, N - 1) * ldb_b + ch0 * 16;
  const char* const pb1 = Bb + (size_t)min(n0 + row0 + 1 * RSTEP, N - 1) * ldb_b + ch0 * 16;
  const char* const pb2 = Bb + (size_t)min(n0 + row0 + 2 * RSTEP, N - 1) * ldb_b + ch0 * 16;
  const char* const pb3 = Bb + (size_t)min(n0 + row0 + 3 * RSTEP, N - 1) * ldb_b + ch0 * 16;
  const int lo0 = swz(row0 + 0 * RSTEP, ch0), lo1 = swz(row0 + 1 * RSTEP, ch0);
  const int lo2 = swz(row0 + 2 * RSTEP, ch0), lo3 = swz(row0 + 3 * RSTEP, ch0);
  uint4 ra0, ra1, ra2, ra3, rb0, rb1, rb2, rb3;
#define NT_GLOAD(kt)                                                 \
  {                                                                  \
    const size_t kb_ = (size_t)(kt) * ROWB;                          \
    ra0 = *reinterpret_cast<const uint4*>(pa0 + kb_);                \
    ra1 = *reinterpret_cast<const uint4*>(pa1 + kb_);                \
    ra2 = *reinterpret_cast<const uint4*>(pa2 + kb_);                \
    ra3 = *reinterpret_cast<const uint4*>(pa3 + kb_);                \
    rb0 = *reinterpret_cast<const uint4*>(pb0 + kb_);                \
    rb1 = *reinterpret_cast<const uint4*>(pb1 + kb_);                \
    rb2 = *reinterpret_cast<const uint4*>(pb2 + kb_);                \
    rb3 = *reinterpret_cast<const uint4*>(pb3 + kb_);                \
  }
#define NT_LSTORE(buf)                                               \
  {                                                                  \
    unsigned char* la_ = lds[buf];                                   \
    unsigned char* lb_ = lds[buf] + BM * ROWB;                       \
    *reinterpret_cast<uint4*>(la_ + lo0) = ra0;                      \
    *reinterpret_cast<uint4*>(la_ + lo1) = ra1;                      \
    *reinterpret_cast<uint4*>(la_ + lo2) = ra2;                      \
    *reinterpret_cast<uint4*>(la_ + lo3) = ra3;                      \
    *reinterpret_cast<uint4*>(lb_ + lo0) = rb0;                      \
    *reinterpret_cast<uint4*>(lb_ + lo1) = rb1;                      \
    *reinterpret_cast<uint4*>(lb_ + lo2) = rb2;                      \
    *reinterpret_cast<uint4*>(lb_ + lo3) = rb3;                      \
  }

  const int wave = tid / kWave, lane = tid % kWave;
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 15, fc = lane >> 4;   // fragment row / 16-byte chunk within a k-slice
  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = (int)((size_t)K * sizeof(T) / ROWB);
  NT_GLOAD(0);
  NT_LSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) NT_GLOAD(kt + 1);
    const unsigned char* As = lds[buf];
    const unsigned char* Bs = lds[buf] + BM * ROWB;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      uint4 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        af[i] = *reinterpret_cast<const uint4*>(As + swz(wm * 64 + i * 16 + fr, kk * 4 + fc));
        bf[i] = *reinterpret_cast<const uint4*>(Bs + swz(wn * 64 + i * 16 + fr, kk * 4 + fc));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = Mfma<T>::step(af[i], bf[j], acc[i][j]);
    }
    if (kt + 1 < nk) NT_LSTORE(buf ^ 1);
    __syncthreads();
  }

#undef NT_GLOAD
#undef NT_LSTORE

  // --- epilogue through LDS, 64 rows at a time: fragments -> [64][132] fp32 tile (the
  // 132-float row stride keeps the fragment writes conflict-free) -> 4 consecutive
  // columns per thread for coalesced stores ---
  constexpr int CS = 132;
  float* cs = reinterpret_cast<float*>(&lds[0][0]);
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (half) __syncthreads();
    if (wm == half) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) cs[(i * 16 + fc * 4 + r) * CS + wn * 64 + j * 16 + fr] = acc[i][j][r];
    }
    __syncthreads();
    for (int g = tid; g < 64 * 32; g += NTHR) {
      const int row = g >> 5, c4 = g & 31;
      const int m = m0 + half * 64 + row, n = n0 + c4 * 4;
      if (m < M && n < N) epilogue4<T>(epi, m, n, N, *reinterpret_cast<const float4*>(&cs[row * CS + c4 * 4]));
    }
  }
}

template <typename T, int ROLE>
hipError_t launch(const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const int tm = (M + BM - 1) / BM, tn = (N + BN - 1) / BN;
  hipLaunchKernelGGL((gemm_kernel<T, ROLE>), dim3(tm * tn), dim3(NTHR), 0, s, static_cast<const T*>(A), lda,
                     static_cast<const T*>(Bt), M, N, K, epi, tm, tn);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_role(const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                       hipStream_t s, int role) {
  switch (role) {
    case 1: return launch<T, 1>(A, lda, Bt, M, N, K, epi, s);
    case 2: return launch<T, 2>(A, lda, Bt, M, N, K, epi, s);
    default: return launch<T, 0>(A, lda, Bt, M, N, K, epi, s);
  }
}

}  // namespace

hipError_t gemm(DT dt, const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                hipStream_t s, int role) {
  switch (dt) {
    case DT::F32: return launch_role<float>(A, lda, Bt, M, N, K, epi, s, role);
    case DT::F16: return launch_role<f16>(A, lda, Bt, M, N, K, epi, s, role);
    case DT::BF16: return launch_role<bf16>(A, lda, Bt, M, N, K, epi, s, role);
  }
  return hipErrorInvalidValue;
}

}  // namespace nt
