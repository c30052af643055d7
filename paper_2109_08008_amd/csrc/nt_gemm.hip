// Dense projections of the encoder, the decoder step and the tied output projection
// (the "MM" that dominates the paper's GPU profile, Sec. 4.4) as one MFMA GEMM for
// gfx950:  C[M,N] = A[M,K] . Bt[N,K]^T with fp32 accumulation and a fused epilogue.
//
// Tiling: BMxBN output tile (128x128, 128x64 or 64x32) per 256-thread workgroup, four
// waves in a 2x2 grid of 16x16 MFMA blocks.  K advances 128 bytes per step (64 halves or 32
// floats) through a ring of STAGES LDS slots filled by direct global->LDS loads
// (global_load_lds_dwordx4), so STAGES-1 k-tiles are in flight while one is multiplied;
// one barrier per k-step.  The loop body is kept compact (no unrolling over k): every
// workgroup of a small decode-step GEMM starts on a cold instruction cache.  The 16-byte chunks of each tile row are XOR-swizzled so that
// the fragment reads are free of bank conflicts.  fp16/bf16 use v_mfma_f32_16x16x32_{f16,bf16}; fp32 uses four
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
#include <limits.h>

#include <type_traits>

#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

constexpr int BM = 128, BN = 128;
constexpr int ROWB = 128;           // bytes of K per tile row per step
constexpr int CH = ROWB / 16;       // 16-byte chunks per tile row
constexpr int NTHR = 256;

// Byte offset of 16-byte chunk `ch` of tile row `row` in a swizzled LDS tile.
__device__ __forceinline__ int swz(int row, int ch) { return row * ROWB + ((ch ^ (row & 7)) << 4); }
// Same for the 64-byte rows of an FP8 weight tile (64 k-values per step): rows r, r+4,
// r+8, r+12 fall on the same banks, so the chunk position is XORed with bits 2..3 of
// the row and 16 consecutive rows read at one chunk hit 16 distinct bank groups.
constexpr int ROWB8 = 64;
__device__ __forceinline__ int swz8(int row, int ch) { return row * ROWB8 + ((ch ^ ((row >> 2) & 3)) << 4); }

// Eight FP8 E4M3 weights (two 32-bit words, k in byte order) as eight fp16 values of an
// MFMA operand.  Every E4M3 value is exact in fp16, so the conversion loses nothing.
template <bool HI>
__device__ __forceinline__ unsigned f8x2(unsigned w) {
  return __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, HI));
}
__device__ __forceinline__ u32x4 f8_to_f16x8(unsigned w0, unsigned w1) {
  return u32x4{f8x2<false>(w0), f8x2<true>(w0), f8x2<false>(w1), f8x2<true>(w1)};
}

// Sum and sum of squares of the eight (fp16/bf16) or four (fp32) values of one 16-byte
// operand fragment, each taken relative to the row's shift c (one of the row's own
// values), added into s and q in fp32: the row statistics of a folded LayerNorm.  With
// the shift, the variance (q/K - (s/K)^2) no longer cancels when the row's mean is large
// against its spread: the deviations from c are of the size of the spread.  For fp16 the
// deviation is formed in fp16 (exact whenever x and c are within a factor of two, which is
// where cancellation would matter), then squared and summed by fdot2 in fp32.
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
template <typename T>
__device__ __forceinline__ void frag_stats(const u32x4& a, T c, float& s, float& q) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if constexpr (std::is_same<T, f16>::value) {
      // the word is copied out first: a bit_cast of the vector element itself read word 0
      const unsigned u = a[w];
      const half2v h = __builtin_bit_cast(half2v, u) - half2v{c, c};
      s = __builtin_amdgcn_fdot2(h, half2v{(_Float16)1.0f, (_Float16)1.0f}, s, false);
      q = __builtin_amdgcn_fdot2(h, h, q, false);
    } else if constexpr (std::is_same<T, bf16>::value) {
      const float cf = to_f32(c);
      const float lo = __uint_as_float(a[w] << 16) - cf, hi = __uint_as_float(a[w] & 0xffff0000u) - cf;
      s += lo;
      s += hi;
      q = fmaf(lo, lo, q);
      q = fmaf(hi, hi, q);
    } else {
      const float x = __uint_as_float(a[w]) - to_f32(c);
      s += x;
      q = fmaf(x, x, q);
    }
  }
}

// Four consecutive elements of the model dtype as loaded (raw bits: converted only where
// they are used, so the load does not have to complete where it is issued).
template <typename T> struct Raw4 { using type = uint2; };
template <> struct Raw4<float> { using type = float4; };
template <typename T>
__device__ __forceinline__ float4 raw4_to_f32(typename Raw4<T>::type r) {
  if constexpr (std::is_same<T, float>::value) {
    return r;
  } else {
    // pins the conversion here: the compiler would otherwise move it up to the load and
    // wait for the data there
    asm volatile("" : "+v"(r.x), "+v"(r.y));
    const T* h = reinterpret_cast<const T*>(&r);
    return make_float4(to_f32(h[0]), to_f32(h[1]), to_f32(h[2]), to_f32(h[3]));
  }
}

// Applies the epilogue MODE to up to 4 consecutive columns n..n+3 of row m (n % 4 == 0).
// With OPS, it adds the bias (if any) and, for EPI_RESID, the residual itself; without,
// the caller has added both (an EPI_RESID group is then a plain store).  The mode is a
// template argument so that a tile's unrolled groups carry only their own mode's code.
// fp32 output (out_f32) goes with EPI_STORE only.  d, dh and ldc are multiples of 4 in
// every mode that scatters, so the 4 columns never straddle a head or a K/V boundary and
// land on 4 consecutive destination elements.
template <typename T, int MODE, bool OPS>
__device__ __forceinline__ void epilogue4(const GemmEpi& e, int m, int n, int N, float4 v4, int t_slot) {
  float v[4] = {v4.x, v4.y, v4.z, v4.w};
  const int cnt = min(4, N - n);
  if constexpr (OPS) {
    if (e.bias) {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (k < cnt) v[k] += e.bias[n + k];
    }
  }
  const bool vec = cnt == 4 && (e.ldc & 3) == 0;
  if constexpr (MODE == EPI_STORE) {
    if (e.out_f32) {
      const int mo = e.out_map ? e.sent_list[m / e.beam] * e.beam + m % e.beam : m;
      float* o = static_cast<float*>(e.out) + (size_t)mo * e.ldc + n;
      if (vec) {
        *reinterpret_cast<float4*>(o) = make_float4(v[0], v[1], v[2], v[3]);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (k < cnt) o[k] = v[k];
      }
      return;
    }
  }
  T* o = nullptr;
  if constexpr (MODE == EPI_STORE) {
    o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
  } else if constexpr (MODE == EPI_RELU) {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = fmaxf(v[k], 0.f);
    o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
  } else if constexpr (MODE == EPI_RESID) {
    if constexpr (OPS) {
      const T* r = static_cast<const T*>(e.resid) + (size_t)m * e.ldc + n;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (k < cnt) v[k] += to_f32(r[k]);
    }
    o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
  } else if constexpr (MODE == EPI_SELF_QKV) {
    if (n < e.d) {
      o = static_cast<T*>(e.out) + (size_t)m * e.ldc + n;
    } else {
      int c = n - e.d;
      const int kv = c >= e.d;
      c -= kv * e.d;
      const int h = c / e.dh, x = c - h * e.dh;
      const int p = e.sent_list[m / e.beam] * e.beam + m % e.beam;
      const size_t idx = ((size_t)(p * e.H + h) * e.Tcap + t_slot) * e.dh + x;
      if (e.kv_f8) {   // E4M3 cache: the 4 columns as 4 bytes, one 32-bit store (idx % 4 == 0)
        uint8_t* o8 = static_cast<uint8_t*>(kv ? e.vcache : e.kcache) + idx;
        if (cnt == 4) {
          *reinterpret_cast<uint32_t*>(o8) = (uint32_t)e4m3_rne(v[0]) | ((uint32_t)e4m3_rne(v[1]) << 8) |
                                             ((uint32_t)e4m3_rne(v[2]) << 16) | ((uint32_t)e4m3_rne(v[3]) << 24);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (k < cnt) o8[k] = e4m3_rne(v[k]);
        }
        return;
      }
      o = static_cast<T*>(kv ? e.vcache : e.kcache) + idx;
    }
  } else {
    static_assert(MODE == EPI_CROSS_KV, "epilogue mode");
    const int j = n / (2 * e.d);
    int c = n - j * 2 * e.d;
    const int kv = c >= e.d;
    c -= kv * e.d;
    const int h = c / e.dh, x = c - h * e.dh;
    const int b = m / e.S, s = m - b * e.S;
    o = static_cast<T*>(e.cross) + ((((size_t)j * 2 + kv) * e.B + b) * e.H + h) * (size_t)e.S * e.dh +
        (size_t)s * e.dh + x;
  }
  if (vec || (MODE >= EPI_SELF_QKV && cnt == 4)) {
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

// s_waitcnt immediate that waits until at most `vm` vector-memory operations of this wave
// are outstanding (expcnt / lgkmcnt left unconstrained).
__host__ __device__ constexpr int vmcnt_imm(int vm) { return (vm & 0xF) | ((vm >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

#define NT_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// Fragment reads are issued as inline ds_read_b128 so that the compiler does not place a
// wait for every in-flight direct global->LDS load in front of them (it cannot tell them
// apart from the loads still filling other slots).  Completion is then made explicit:
// lds_wait() waits for the reads and names the fragments as operands, so no use of a
// fragment can be scheduled before it.
__device__ __forceinline__ u32x4 lds_read16(const unsigned char* p) {
  u32x4 v;
  const unsigned a = (unsigned)(uintptr_t)NT_LDS(p);
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}
// LdsWait<FM, FN>::run<N>(a, b): wait until at most N LDS operations of this wave are
// outstanding (reads complete in order, so every read issued before the last N has
// landed), naming the fragments a and b as its operands.
// Bias and residual of the 4-column group (row m, columns n..n+3), fetched ahead of the
// group's epilogue as raw vectors.  Both loads are issued unconditionally, without any
// branch: a per-thread branch makes the compiler wait for the loads at its join, and even
// a uniform one per group becomes a jump to out-of-line code, an instruction-cache miss
// per group in these large unrolled kernels.  An operand the epilogue does not have, and
// a group that is out of range, ragged or not vector-aligned, read `safe` (any readable
// 16-byte aligned address; always the same cached line) instead; such a group reports
// false and its epilogue then loads for itself.
template <typename T>
__device__ __forceinline__ bool fetch_group(const GemmEpi& e, bool has_b, bool has_r, const char* safe, int m,
                                            int n, int M, int N, float4& b, typename Raw4<T>::type& r) {
  using R4 = typename Raw4<T>::type;
  const char* bp = has_b ? reinterpret_cast<const char*>(e.bias + n) : safe;
  const char* rp = has_r ? reinterpret_cast<const char*>(static_cast<const T*>(e.resid) + (size_t)m * e.ldc + n) : safe;
  const bool ok = m < M && n + 4 <= N && (!has_b || (reinterpret_cast<uintptr_t>(bp) & 15) == 0) &&
                  (!has_r || (reinterpret_cast<uintptr_t>(rp) & (sizeof(R4) - 1)) == 0);
  b = *reinterpret_cast<const float4*>(ok ? bp : safe);
  r = *reinterpret_cast<const R4*>(ok ? rp : safe);
  return ok;
}

// The epilogue of one group: with its operands fetched (ok), adds bias, then residual --
// the order epilogue4 adds them in -- and stores; otherwise epilogue4 loads them itself.
template <typename T, int MODE>
__device__ __forceinline__ void finish_group(const GemmEpi& e, bool ok, int m, int n, int N, float4 v,
                                             const float4& b, const typename Raw4<T>::type& r, int t_slot) {
  if (__builtin_expect(ok, 1)) {
    if (e.bias) { v.x += b.x; v.y += b.y; v.z += b.z; v.w += b.w; }
    if constexpr (MODE == EPI_RESID) {
      const float4 rf = raw4_to_f32<T>(r);
      v.x += rf.x; v.y += rf.y; v.z += rf.z; v.w += rf.w;
    }
    epilogue4<T, MODE, false>(e, m, n, N, v, t_slot);
  } else {
    epilogue4<T, MODE, true>(e, m, n, N, v, t_slot);
  }
}

template <int FM, int FN> struct LdsWait;
template <> struct LdsWait<1, 1> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[1], u32x4 (&b)[1]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(b[0]) : [n] "i"(N));
  }
};
template <> struct LdsWait<1, 2> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[1], u32x4 (&b)[2]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(b[0]), "+v"(b[1]) : [n] "i"(N));
  }
};
template <> struct LdsWait<2, 1> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[2], u32x4 (&b)[1]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]) : [n] "i"(N));
  }
};
template <> struct LdsWait<2, 2> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[2], u32x4 (&b)[2]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]) : [n] "i"(N));
  }
};
template <> struct LdsWait<2, 4> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[2], u32x4 (&b)[4]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]) : [n] "i"(N));
  }
};
template <> struct LdsWait<4, 2> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[4], u32x4 (&b)[2]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]) : [n] "i"(N));
  }
};
template <> struct LdsWait<4, 4> {
  template <int N = 0>
  static __device__ __forceinline__ void run(u32x4 (&a)[4], u32x4 (&b)[4]) {
    asm volatile("s_waitcnt lgkmcnt(%[n])" : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]) : [n] "i"(N));
  }
};

// Fused selection epilogue: the rows of an LDS-staged fp32 tile (ER rows x BN columns,
// row stride CS) are reduced to one record per row: the max, the sum of exp(x - max),
// and for K2 = 1 the best (value, column) -- the max at its lowest column.  TPR
// consecutive lanes share a row; each scans its columns in increasing order.  Two
// passes: the max (and its column), then one exponential per logit.  Both searches take
// K2 = 1: greedy needs nothing else, beam ranks the tiles by their best entries.
__device__ __forceinline__ bool topk_better(float v1, int i1, float v2, int i2) {
  return v1 > v2 || (v1 == v2 && i1 < i2);
}

template <int ER, int BN_, int K2>
__device__ __forceinline__ void topk_tile_rows(const float* cs, int CS, int mrow0, int n0, int M, int N, int tn,
                                               const GemmEpi& e) {
  static_assert(K2 == 0 || K2 == 1, "records carry at most the best entry");
  constexpr int TPR = NTHR / ER;            // threads per row (2, 4 or 8)
  static_assert(TPR >= 1 && TPR <= kWave && (TPR & (TPR - 1)) == 0, "row group inside a wave");
  const int row = threadIdx.x / TPR, sub = threadIdx.x % TPR;
  const int m = mrow0 + row;
  float mx = -INFINITY;
  int bi = INT_MAX;   // lowest column holding mx (K2 = 1)
  for (int g4 = sub; g4 < BN_ / 4; g4 += TPR) {
    const float4 q = *reinterpret_cast<const float4*>(&cs[row * CS + g4 * 4]);
    const float xs[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int n = n0 + g4 * 4 + u;
      const float x = n < N ? xs[u] : -INFINITY;
      if constexpr (K2 == 1) {
        if (x > mx) { mx = x; bi = n; }   // columns rise within a lane: ties keep the lowest
      } else {
        mx = fmaxf(mx, x);
      }
    }
  }
#pragma unroll
  for (int o = TPR / 2; o > 0; o >>= 1) {
    const float om = __shfl_xor(mx, o, kWave);
    if constexpr (K2 == 1) {
      const int oi = __shfl_xor(bi, o, kWave);
      if (topk_better(om, oi, mx, bi)) { mx = om; bi = oi; }
    } else {
      mx = fmaxf(mx, om);
    }
  }
  float sum = 0.f;
  if (mx != -INFINITY) {
    for (int g4 = sub; g4 < BN_ / 4; g4 += TPR) {
      const float4 q = *reinterpret_cast<const float4*>(&cs[row * CS + g4 * 4]);
      const float xs[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) sum += __expf((n0 + g4 * 4 + u < N ? xs[u] : -INFINITY) - mx);
    }
  }
#pragma unroll
  for (int o = TPR / 2; o > 0; o >>= 1) sum += __shfl_xor(sum, o, kWave);
  if (sub == 0 && m < M) {
    float* rec = e.part + ((size_t)m * e.n_tiles + tn) * topk_record(e.k2);
    rec[0] = mx;
    rec[1] = sum;
    if constexpr (K2 == 1) {
      rec[2] = mx;
      rec[3] = __int_as_float(bi);
    }
  }
}

// F8: Bt holds FP8 E4M3 weights ([N][K] bytes) with one fp32 scale per output column
// (epi.wscale); A stays fp16.  The weight tile then takes 64-byte rows in LDS (a 1 KB
// wave load moves 16 of them), each lane's 16-byte B fragment carries the 16 k-values
// of both half-steps, and lane l supplies A k-values 16*(l/16) .. +7 and +8 .. +15 (the
// two operands agree on the k each lane carries, which is all the MFMA needs).
template <typename T, int BM_, int BN_, int STAGES, int ROLE, bool F8 = false, bool LNF = false>
__global__ __launch_bounds__(NTHR) void gemm_kernel(const T* __restrict__ A, int lda, const void* __restrict__ Bt,
                                                    int M, int N, int K, GemmEpi epi, int tiles_m, int tiles_n) {
  static_assert(!F8 || std::is_same<T, f16>::value, "FP8 weights pair with fp16 activations");
  constexpr int ROWB_B = F8 ? ROWB8 : ROWB;
  constexpr int STAGE_BYTES = BM_ * ROWB + BN_ * ROWB_B;
  constexpr int GROUPS_A = BM_ / 8;                 // 8 A rows = one 1 KB wave load
  constexpr int GROUPS = GROUPS_A + BN_ * ROWB_B / 1024;
  constexpr int LPW = GROUPS / 4;                   // loads per wave per stage
  constexpr int WM = BM_ / 2, WN = BN_ / 2;         // 2x2 waves
  constexpr int FM = WM / 16, FN = WN / 16;         // 16x16 blocks per wave
  static_assert(GROUPS % 4 == 0, "tile rows must split evenly over 4 waves");
  static_assert(STAGES >= 2 && STAGES <= 8, "1..7 k-tiles in flight");
  static_assert((STAGES - 2) * LPW <= 63, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) unsigned char lds[STAGES * STAGE_BYTES];

  // live rows of a decode step: the grid covers the whole batch, and the workgroups past
  // the live tiles exit.  Live tiles take the lowest workgroup ids, which the dispatcher
  // deals round-robin over the 8 XCDs, so a shrinking batch still spreads over all of them.
  // The arguments span three scalar-cache lines; naming fields from each of them here
  // makes the three misses overlap instead of following one another down the prologue.
  asm volatile("" ::"s"(epi.ctl), "s"(epi.bias), "s"(epi.out), "s"(epi.ldc), "s"(epi.wscale), "s"(epi.part),
               "s"(tiles_n), "s"(M), "s"(Bt));
  if (epi.ctl) {
    M = min(M, epi.ctl[CTL_NLIVE] * epi.ctl_rows);
    tiles_m = (M + BM_ - 1) / BM_;
  }
  // --- tile assignment: XCD-contiguous, then grouped by 8 tile-rows ---
  // (role 3: block pid of the pair list; its rows are pairs of one 128-column tile)
  const int ntiles = ROLE == 3 ? *epi.gnblk : tiles_m * tiles_n;
  int pid = blockIdx.x;
  if (pid >= ntiles) return;
  {
    const int q = ntiles / 8, r = ntiles % 8, xcd = pid % 8, idx = pid / 8;
    pid = xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
  }
  const int* prow = nullptr;   // role 3: the block's pair ids
  int tm = 0, tn = 0;
  if constexpr (ROLE == 3) {
    static_assert(BN_ == 128, "a pair block covers one 128-column tile");
    tn = epi.gblk[3 * pid];
    prow = epi.sorted + epi.gblk[3 * pid + 1];
    M = epi.gblk[3 * pid + 2];
  } else {
    constexpr int GROUP = 8;
    const int per_group = GROUP * tiles_n;
    const int first_m = (pid / per_group) * GROUP;
    const int gsize = min(tiles_m - first_m, GROUP);
    tm = first_m + (pid % per_group) % gsize;
    tn = (pid % per_group) / gsize;
  }
  const int m0 = tm * BM_, n0 = tn * BN_;
  const int t_slot = epi.ctl ? epi.ctl[CTL_T] : epi.t;

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const size_t lda_b = (size_t)lda * sizeof(T), ldb_b = (size_t)K * (F8 ? 1 : sizeof(T));

  // Direct global -> LDS loads: one instruction moves 8 tile rows (64 lanes x 16 B, lane l
  // to LDS byte 16*l of the group).  Lane l fills LDS chunk (l & 7) of row l/8, which
  // holds global chunk (l & 7) ^ (row & 7) under the swizzle; rows past the edge re-read
  // the last valid row (their results are never stored).
  // FP8 weight tile: a wave load moves 16 rows of 64 bytes; lane l fills LDS chunk (l & 3)
  // of row l/4, which holds global chunk (l & 3) ^ ((row >> 2) & 3) = (l & 3) ^ (l >> 4).
  const int lrow = lane >> 3, lchunk = (lane & 7) ^ lrow;
  const int brow8 = lane >> 2, bchunk8 = (lane & 3) ^ (lane >> 4);
  const char* Ab = reinterpret_cast<const char*>(A) + lchunk * 16;
  const char* Bb = reinterpret_cast<const char*>(Bt) + (F8 ? bchunk8 : lchunk) * 16;
  // byte offset of A row `row_` of the tile (load i_ of this wave): role 3 gathers the
  // rows of its pairs, read once here
  size_t aoff3[ROLE == 3 ? LPW : 1];
  if constexpr (ROLE == 3) {
#pragma unroll
    for (int i_ = 0; i_ < LPW; ++i_) {
      const int g_ = wave * LPW + i_;
      aoff3[i_] = g_ < GROUPS_A ? (size_t)(prow[min(g_ * 8 + lrow, M - 1)] / epi.pair_k) * lda_b : 0;
    }
  }
  auto a_off = [&](int i_, int row_) -> size_t {
    if constexpr (ROLE == 3) return aoff3[i_];
    else return (size_t)min(m0 + row_, M - 1) * lda_b;
  };
#define NT_ISSUE(kt, SL)                                                                          \
  {                                                                                               \
    unsigned char* sb_ = lds + (SL) * STAGE_BYTES;                                                \
    _Pragma("unroll") for (int i_ = 0; i_ < LPW; ++i_) {                                          \
      const int g_ = wave * LPW + i_;                                                             \
      const char* src_;                                                                           \
      unsigned char* dst_;                                                                        \
      if (!F8 || g_ < GROUPS_A) {                                                                 \
        const int row_ = g_ * 8 + lrow;                                                           \
        const size_t kb_ = (size_t)(kt) * ROWB;                                                   \
        src_ = row_ < BM_ ? Ab + a_off(i_, row_) + kb_                                            \
                          : Bb + (size_t)min(n0 + row_ - BM_, N - 1) * ldb_b + kb_;               \
        dst_ = sb_ + g_ * 1024;                                                                   \
      } else {                                                                                    \
        const int b_ = g_ - GROUPS_A;                                                             \
        src_ = Bb + (size_t)min(n0 + b_ * 16 + brow8, N - 1) * ldb_b + (size_t)(kt) * ROWB8;      \
        dst_ = sb_ + BM_ * ROWB + b_ * 1024;                                                      \
      }                                                                                           \
      __builtin_amdgcn_global_load_lds(src_, NT_LDS(dst_), 16, 0, 0);                             \
    }                                                                                             \
  }

  const int fr = lane & 15, fc = lane >> 4;   // fragment row / 16-byte chunk within a k-slice
  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int wm = wave >> 1, wn = wave & 1;

  // epilogue geometry (see the epilogue below)
  constexpr int CS = BN_ + 4;
  constexpr int LDSB = STAGES * STAGE_BYTES;
  constexpr int ER = (BM_ * CS * 4 <= LDSB) ? BM_ : (WM * CS * 4 <= LDSB) ? WM : WM / 2;
  constexpr int PASSES = BM_ / ER;
  constexpr int EPG = ER * (BN_ / 4);           // 4-column output groups per pass
  // The epilogue operands that do not depend on the product -- bias and residual -- are
  // fetched before the k-loop when each thread owns at most 4 output groups (the small
  // decode-step tiles), so their latency hides behind it.  They stay as loaded until the
  // epilogue: converting them, or loading them under a per-thread branch (whose join
  // copies the registers), would make the prologue wait for them before the first tile
  // loads issue.  So every thread loads unconditionally, and a group that is ragged or not
  // vector-aligned reads the (16-byte aligned) base of A instead and is left to the
  // epilogue's own loads.  The epilogue adds them in its own order (bias, then residual),
  // so results are bitwise unchanged.
  constexpr bool PRE = ROLE < 2 && EPG % NTHR == 0 && PASSES * (EPG / NTHR) <= 4;
  constexpr int NPRE = PRE ? PASSES * (EPG / NTHR) : 1;
  using R4 = typename Raw4<T>::type;
  float4 pre_b[NPRE];
  R4 pre_r[NPRE];
  unsigned pre_ok = 0;   // bit q: group q was fetched here
  const bool has_b = epi.bias != nullptr, has_r = epi.mode == EPI_RESID;   // the same in every thread
  const char* safe = reinterpret_cast<const char*>(A);
  if constexpr (PRE) {
#pragma unroll
    for (int q = 0; q < NPRE; ++q) {
      const int pass = q / (EPG / NTHR), g = tid + (q % (EPG / NTHR)) * NTHR;
      const int m = m0 + pass * ER + g / (BN_ / 4), n = n0 + (g % (BN_ / 4)) * 4;
      pre_ok |= (unsigned)fetch_group<T>(epi, has_b, has_r, safe, m, n, M, N, pre_b[q], pre_r[q]) << q;
    }
  }

  // folded LayerNorm: lane (fr, fc) sums the k-chunks fc and 4+fc of its fragment rows
  // over every k-step; the four lanes of a row together see each of its K values once.
  // The lane's column sums (its output column is fixed per 16x16 block) and its rows'
  // shifts (each row's first value, the same for the four lanes of a row) are fetched
  // here, so their latency hides behind the k-loop instead of stalling it.
  float lsum[LNF ? FM : 1], lsq[LNF ? FM : 1], lcs[LNF ? FN : 1];
  T lsh[LNF ? FM : 1];
#pragma unroll
  for (int i = 0; i < (LNF ? FM : 1); ++i) lsum[i] = lsq[i] = 0.f;
  if constexpr (LNF) {
#pragma unroll
    for (int j = 0; j < FN; ++j) lcs[j] = epi.lnf_colsum[min(n0 + wn * WN + j * 16 + fr, N - 1)];
#pragma unroll
    for (int i = 0; i < FM; ++i) lsh[i] = A[(size_t)min(m0 + wm * WM + i * 16 + fr, M - 1) * lda];
  }

  const int nk = (int)((size_t)K * sizeof(T) / ROWB);
  for (int st = 0; st < STAGES - 1 && st < nk; ++st) NT_ISSUE(st, st)
  int slot = 0;   // slot of k-step kt
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + STAGES - 2 <= nk - 1) __builtin_amdgcn_s_waitcnt(vmcnt_imm((STAGES - 2) * LPW));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_s_barrier();   // tile kt is in LDS for every wave; slot kt-1 is free
    if (kt + STAGES - 1 < nk) NT_ISSUE(kt + STAGES - 1, slot == 0 ? STAGES - 1 : slot - 1)
    const unsigned char* As = lds + slot * STAGE_BYTES;
    const unsigned char* Bs = As + BM_ * ROWB;
    // both halves of the k-step are read back to back; the second half's reads land
    // while the first half's MFMAs run
    u32x4 af0[FM], bf0[FN], af1[FM], bf1[FN];
    if constexpr (F8) {
      u32x4 bq[FN];   // 16 FP8 weights: k 16*fc .. 16*fc+15
#pragma unroll
      for (int i = 0; i < FM; ++i) af0[i] = lds_read16(As + swz(wm * WM + i * 16 + fr, 2 * fc));
#pragma unroll
      for (int j = 0; j < FN; ++j) bq[j] = lds_read16(Bs + swz8(wn * WN + j * 16 + fr, fc));
#pragma unroll
      for (int i = 0; i < FM; ++i) af1[i] = lds_read16(As + swz(wm * WM + i * 16 + fr, 2 * fc + 1));
      LdsWait<FM, FN>::template run<FM>(af0, bq);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        bf0[j] = f8_to_f16x8(bq[j].x, bq[j].y);
        bf1[j] = f8_to_f16x8(bq[j].z, bq[j].w);
      }
    } else {
#pragma unroll
      for (int i = 0; i < FM; ++i) af0[i] = lds_read16(As + swz(wm * WM + i * 16 + fr, fc));
#pragma unroll
      for (int j = 0; j < FN; ++j) bf0[j] = lds_read16(Bs + swz(wn * WN + j * 16 + fr, fc));
#pragma unroll
      for (int i = 0; i < FM; ++i) af1[i] = lds_read16(As + swz(wm * WM + i * 16 + fr, 4 + fc));
#pragma unroll
      for (int j = 0; j < FN; ++j) bf1[j] = lds_read16(Bs + swz(wn * WN + j * 16 + fr, 4 + fc));
      LdsWait<FM, FN>::template run<FM + FN>(af0, bf0);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::step(af0[i], bf0[j], acc[i][j]);
    if constexpr (LNF) {
#pragma unroll
      for (int i = 0; i < FM; ++i) frag_stats<T>(af0[i], lsh[i], lsum[i], lsq[i]);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep the second wait behind the first half's MFMAs
    LdsWait<FM, FN>::template run<0>(af1, bf1);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::step(af1[i], bf1[j], acc[i][j]);
    if constexpr (LNF) {
#pragma unroll
      for (int i = 0; i < FM; ++i) frag_stats<T>(af1[i], lsh[i], lsum[i], lsq[i]);
    }
    slot = slot == STAGES - 1 ? 0 : slot + 1;
  }
#undef NT_ISSUE
  // folded LayerNorm: each row's mean and 1/sqrt(biased variance + eps) from the sums of
  // its deviations from the shift c (mean = c + s/K, variance = q/K - (s/K)^2, fp32),
  // kept per tile row for the epilogue (the accumulators become
  // rstd * (acc - mean * colsum[n]) as they enter the epilogue)
  float* ln_mu = nullptr;
  float* ln_rs = nullptr;
  if constexpr (LNF) {
    __shared__ __attribute__((aligned(16))) float ln_stat[2 * BM_];
    ln_mu = ln_stat;
    ln_rs = ln_stat + BM_;
    const float inv_k = 1.0f / (float)K;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      float s = lsum[i], q = lsq[i];
      s += __shfl_xor(s, 16, kWave);
      q += __shfl_xor(q, 16, kWave);
      s += __shfl_xor(s, 32, kWave);
      q += __shfl_xor(q, 32, kWave);
      if (wn == 0 && fc == 0) {
        const float ms = s * inv_k;
        const float var = fmaxf(q * inv_k - ms * ms, 0.f);
        ln_mu[wm * WM + i * 16 + fr] = to_f32(lsh[i]) + ms;
        ln_rs[wm * WM + i * 16 + fr] = 1.0f / sqrtf(var + epi.lnf_eps);
      }
    }
  }
  __syncthreads();

  // --- epilogue through the LDS ring in passes of ER rows: fragments -> [ER][BN+4] fp32
  // tile (the BN+4 stride keeps the fragment writes conflict-free) -> 4 consecutive
  // columns per thread for coalesced stores ---
  static_assert(ER * CS * 4 <= LDSB && ER % 16 == 0, "epilogue tile fits the LDS ring");
  float* cs = reinterpret_cast<float*>(lds);
  // FP8 weights: each output column carries its weight scale (a lane's column is fixed
  // per 16x16 block), applied as the accumulators enter the tile so every epilogue sees
  // the scaled products
  float wsc[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn * WN + j * 16 + fr;
    wsc[j] = F8 ? (n < N ? epi.wscale[n] : 0.f) : 1.f;
  }
  // Tiles without the prologue prefetch fetch each pass's bias and residual before staging
  // the pass through LDS, so the loads are in flight while it is staged; and all of them
  // before any store: a load issued after a store waits for it (the output may alias the
  // residual), one round trip per group.  Groups are disjoint between threads, and each
  // residual element is read by the thread that overwrites it, so reading them all first
  // is the same computation.
  constexpr bool BATCH = !PRE && EPG % NTHR == 0 && ROLE < 2;   // the projection has no operands to fetch
  constexpr int GPT = BATCH ? EPG / NTHR : 1;
#pragma unroll
  for (int pass = 0; pass < PASSES; ++pass) {
    if (pass) __syncthreads();
    float4 eb[GPT];
    R4 er[GPT];
    unsigned eok = 0;
    if constexpr (BATCH) {
      if (!(ROLE == 2 && epi.mode == EPI_TOPK)) {
#pragma unroll
        for (int u = 0; u < GPT; ++u) {
          const int g = tid + u * NTHR;
          const int m = m0 + pass * ER + g / (BN_ / 4), n = n0 + (g % (BN_ / 4)) * 4;
          eok |= (unsigned)fetch_group<T>(epi, has_b, has_r, safe, m, n, M, N, eb[u], er[u]) << u;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int rb = wm * WM + i * 16;            // first tile row of this block
      if (rb >= pass * ER && rb < pass * ER + ER) {
        float4 mu4{0.f, 0.f, 0.f, 0.f}, rs4{1.f, 1.f, 1.f, 1.f};   // lane rows rb + 4*fc + r
        if constexpr (LNF) {
          mu4 = *reinterpret_cast<const float4*>(ln_mu + rb + fc * 4);
          rs4 = *reinterpret_cast<const float4*>(ln_rs + rb + fc * 4);
        }
        const float mur[4] = {mu4.x, mu4.y, mu4.z, mu4.w}, rsr[4] = {rs4.x, rs4.y, rs4.z, rs4.w};
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float v = F8 ? acc[i][j][r] * wsc[j] : acc[i][j][r];
            if constexpr (LNF) v = (v - mur[r] * lcs[j]) * rsr[r];
            cs[(rb - pass * ER + fc * 4 + r) * CS + wn * WN + j * 16 + fr] = v;
          }
      }
    }
    __syncthreads();
    if constexpr (ROLE == 3) {   // the pairs' logits, row = pair id
      for (int g = tid; g < EPG; g += NTHR) {
        const int row = g / (BN_ / 4), c4 = g % (BN_ / 4);
        if (pass * ER + row < M) {
          float4 v = *reinterpret_cast<const float4*>(&cs[row * CS + c4 * 4]);
          const int n = n0 + c4 * 4;
          if (n + 0 >= N) v.x = -INFINITY;
          if (n + 1 >= N) v.y = -INFINITY;
          if (n + 2 >= N) v.z = -INFINITY;
          if (n + 3 >= N) v.w = -INFINITY;
          *reinterpret_cast<float4*>(static_cast<float*>(epi.out) + (size_t)prow[pass * ER + row] * BN_ + c4 * 4) = v;
        }
      }
      continue;
    }
    if (ROLE == 2 && epi.mode == EPI_TOPK) {
      topk_tile_rows<ER, BN_, 1>(cs, CS, m0 + pass * ER, n0, M, N, tn, epi);
      if (!epi.out) continue;   // the records are all the selection needs; else the logits too
    }
    // The mode is the same for every thread: one branch per pass, then that mode's groups.
    auto finish_pass = [&](auto mode_c) {
      constexpr int MODE = decltype(mode_c)::value;
      if constexpr (PRE) {
#pragma unroll
        for (int u = 0; u < EPG / NTHR; ++u) {
          const int g = tid + u * NTHR, q = pass * (EPG / NTHR) + u;
          const int row = g / (BN_ / 4), c4 = g % (BN_ / 4);
          const int m = m0 + pass * ER + row, n = n0 + c4 * 4;
          if (m < M && n < N)
            finish_group<T, MODE>(epi, (pre_ok >> q) & 1u, m, n, N,
                                  *reinterpret_cast<const float4*>(&cs[row * CS + c4 * 4]), pre_b[q], pre_r[q], t_slot);
        }
      } else if constexpr (BATCH) {
#pragma unroll
        for (int u = 0; u < GPT; ++u) {
          const int g = tid + u * NTHR;
          const int row = g / (BN_ / 4), c4 = g % (BN_ / 4);
          const int m = m0 + pass * ER + row, n = n0 + c4 * 4;
          if (m < M && n < N)
            finish_group<T, MODE>(epi, (eok >> u) & 1u, m, n, N,
                                  *reinterpret_cast<const float4*>(&cs[row * CS + c4 * 4]), eb[u], er[u], t_slot);
        }
      } else {
        for (int g = tid; g < EPG; g += NTHR) {
          const int row = g / (BN_ / 4), c4 = g % (BN_ / 4);
          const int m = m0 + pass * ER + row, n = n0 + c4 * 4;
          if (m < M && n < N)
            epilogue4<T, MODE, true>(epi, m, n, N, *reinterpret_cast<const float4*>(&cs[row * CS + c4 * 4]), t_slot);
        }
      }
    };
    switch (epi.mode) {
      case EPI_RELU: finish_pass(std::integral_constant<int, EPI_RELU>{}); break;
      case EPI_RESID: finish_pass(std::integral_constant<int, EPI_RESID>{}); break;
      case EPI_SELF_QKV: finish_pass(std::integral_constant<int, EPI_SELF_QKV>{}); break;
      case EPI_CROSS_KV: finish_pass(std::integral_constant<int, EPI_CROSS_KV>{}); break;
      default: finish_pass(std::integral_constant<int, EPI_STORE>{}); break;
    }
  }
}

template <typename T, int BM_, int BN_, int STAGES, int ROLE, bool F8 = false, bool LNF = false>
hipError_t launch_tile(const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                       hipStream_t s) {
  const int tm = (M + BM_ - 1) / BM_, tn = (N + BN_ - 1) / BN_;
  NT_LAUNCH((gemm_kernel<T, BM_, BN_, STAGES, ROLE, F8, LNF>), dim3(tm * tn), dim3(NTHR), 0, s,
                     static_cast<const T*>(A), lda, Bt, M, N, K, epi, tm, tn);
  return hipGetLastError();
}

// Tile choice by problem size, measured on MI355X with four batches' GEMMs in flight at
// once (how nt_translate runs them).  LDS footprint matters more than pipeline depth, so
// the big tiles use two stages.
//   M >= 4096 (encoder, big batches): 128x64 for N <= 2048, else 128x128; and
//                      128x128 for the FFN's second GEMM (K >= 2048) from 8M outputs up
//                      (16384x512x2048: 40.6 us against 52.1; 16384x1024x4096: 135.4
//                      against 161.4; 8192x512x2048 stays: 26.0 against 31.0);
//   M*N < 1M outputs:  64x32, 3 stages (skinny decode-step shapes; 4 stages for the
//                      decoder's K >= 2048);
//   M*N < 3M outputs:  64x128, 2 stages (1300x1536: 5.6 us against 6.8 at 64x32;
//                      2160x1024x1024: 8.6 against 12.0);
//   larger:            128x128, 2 stages (2160x1024x4096: 27.8 us against 43.8 at 64x32),
//                      except in decoder steps, which take 64x128 there (below).
// All reduce each output over K in the same order, so the choice never changes a result.
template <typename T, int ROLE>
hipError_t launch(const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi, hipStream_t s,
                  int tile) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (tile == 0) {
    const long long mn = (long long)M * N;
    if (M >= 4096) tile = N <= 2048 && (K < 2048 || mn < (8ll << 20)) ? 3 : 2;
    else tile = mn < (1ll << 20) ? 1 : mn < (3ll << 20) ? 4 : 2;
  }
  // FP8 weights (fp16 activations only).  A 64-byte weight row moves 16 rows per wave
  // load, so the narrow tiles change: measured at decode shapes with four GEMMs in flight,
  // 32x64 (3 stages) is the best small tile (650x512x512: 5.1 us against 6.2 at 64x64;
  // 1300x512x2048: 13.0 against 15.9).  Alone, 64x64 is the faster middle tile
  // (1300x1536x512: 8.2 against 9.1 us at 64x128), but inside whole translations the
  // decoder's projections run best at 64x128 above the smallest shapes.
  // folded LayerNorm: decoder-step launches with weights in the model dtype
  if (epi.lnf_colsum) {
    if constexpr (ROLE != 1) {
      return hipErrorInvalidValue;
    } else {
      // (128x128 would hold the row statistics at one wave per SIMD: 64x128 instead)
      if (epi.wscale) {   // FP8 weights with the gain folded in: the FP8 tile map
        if constexpr (!std::is_same<T, f16>::value) {
          return hipErrorInvalidValue;
        } else {
          // 64x128 for every tile above the smallest, as for the decoder's FP8 residual
          // projections below (measured on wide-30-6-fp8 with four batches in flight:
          // 264.6k -> 278.4k tok/s against 128x64 / 64x64; base-6-6-fp8 648.9k -> 655.7k)
          switch (tile) {
            case 2:
            case 3:
            case 4: return launch_tile<T, 64, 128, 2, ROLE, true, true>(A, lda, Bt, M, N, K, epi, s);
            default: return launch_tile<T, 32, 64, 3, ROLE, true, true>(A, lda, Bt, M, N, K, epi, s);
          }
        }
      }
      switch (tile) {
        case 2:
        case 4: return launch_tile<T, 64, 128, 2, ROLE, false, true>(A, lda, Bt, M, N, K, epi, s);
        case 3: return launch_tile<T, 128, 64, 2, ROLE, false, true>(A, lda, Bt, M, N, K, epi, s);
        default: return launch_tile<T, 64, 32, 3, ROLE, false, true>(A, lda, Bt, M, N, K, epi, s);
      }
    }
  }
  if (epi.wscale) {
    if constexpr (!std::is_same<T, f16>::value || ROLE == 2) {
      return hipErrorInvalidValue;
    } else {
      if (ROLE == 1 && tile != 1)   // decoder steps: 64x128 (see the folded map above)
        return launch_tile<T, 64, 128, 2, ROLE, true>(A, lda, Bt, M, N, K, epi, s);
      switch (tile) {
        case 2: return launch_tile<T, 128, 128, 2, ROLE, true>(A, lda, Bt, M, N, K, epi, s);
        case 3: return launch_tile<T, 128, 64, 2, ROLE, true>(A, lda, Bt, M, N, K, epi, s);
        case 4: return launch_tile<T, 64, 64, 3, ROLE, true>(A, lda, Bt, M, N, K, epi, s);
        default: return launch_tile<T, 32, 64, 3, ROLE, true>(A, lda, Bt, M, N, K, epi, s);
      }
    }
  }
  // decoder steps keep to 64-row tiles where the shape picks 128x128: alone, 3172x1024x4096
  // takes 40.7 us at 64x128 against 47.5 us, 3172x1024x1024 13.2 against 18.3 (the
  // 128x128 choice was measured against 64x32 only)
  if (ROLE == 1 && tile == 2) tile = 4;
  switch (tile) {
    case 2: return launch_tile<T, 128, 128, 2, ROLE>(A, lda, Bt, M, N, K, epi, s);
    case 3: return launch_tile<T, 128, 64, 2, ROLE>(A, lda, Bt, M, N, K, epi, s);
    case 4: return launch_tile<T, 64, 128, 2, ROLE>(A, lda, Bt, M, N, K, epi, s);
    default:
      // the decoder's FFN2 (K = 4d) runs the longest k-loop of the step: a fourth stage
      // in flight (48 KB of LDS) cut its kernel time 4% on base-6-6, 2% on wide-30-6
      if (ROLE == 1 && K >= 2048) return launch_tile<T, 64, 32, 4, ROLE>(A, lda, Bt, M, N, K, epi, s);
      return launch_tile<T, 64, 32, 3, ROLE>(A, lda, Bt, M, N, K, epi, s);
  }
}

template <typename T>
hipError_t launch_role(const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                       hipStream_t s, int role, int tile) {
  switch (role) {
    case 1: return launch<T, 1>(A, lda, Bt, M, N, K, epi, s, tile);
    case 2: return launch<T, 2>(A, lda, Bt, M, N, K, epi, s, tile);
    default: return launch<T, 0>(A, lda, Bt, M, N, K, epi, s, tile);
  }
}

template <typename T>
hipError_t launch_pairs(const void* A, int lda, const void* Bt, int N, int K, const GemmEpi& epi, int max_blocks,
                        hipStream_t s) {
  NT_LAUNCH((gemm_kernel<T, PAIR_BM, 128, 2, 3>), dim3(max_blocks), dim3(NTHR), 0, s, static_cast<const T*>(A), lda,
            Bt, PAIR_BM, N, K, epi, 1, 1);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_pairs(DT dt, const void* A, int lda, const void* Bt, int N, int K, const GemmEpi& epi,
                      int max_blocks, hipStream_t s) {
  if (max_blocks <= 0) return hipSuccess;
  if (!epi.gblk || !epi.gnblk || !epi.sorted || !epi.out || epi.wscale || epi.lnf_colsum || epi.pair_k < 1)
    return hipErrorInvalidValue;
  if (((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(Bt)) & 15) != 0) return hipErrorInvalidValue;
  switch (dt) {
    case DT::F32: return launch_pairs<float>(A, lda, Bt, N, K, epi, max_blocks, s);
    case DT::F16: return launch_pairs<f16>(A, lda, Bt, N, K, epi, max_blocks, s);
    case DT::BF16: return launch_pairs<bf16>(A, lda, Bt, N, K, epi, max_blocks, s);
  }
  return hipErrorInvalidValue;
}

hipError_t gemm(DT dt, const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                hipStream_t s, int role, int tile) {
  if (epi.wscale && dt != DT::F16) return hipErrorInvalidValue;   // FP8 weights pair with fp16
  // operand rows move in 16-byte pieces, and the kernel reads A's base as a stand-in
  if (((reinterpret_cast<uintptr_t>(A) | reinterpret_cast<uintptr_t>(Bt)) & 15) != 0) return hipErrorInvalidValue;
  switch (dt) {
    case DT::F32: return launch_role<float>(A, lda, Bt, M, N, K, epi, s, role, tile);
    case DT::F16: return launch_role<f16>(A, lda, Bt, M, N, K, epi, s, role, tile);
    case DT::BF16: return launch_role<bf16>(A, lda, Bt, M, N, K, epi, s, role, tile);
  }
  return hipErrorInvalidValue;
}

}  // namespace nt
