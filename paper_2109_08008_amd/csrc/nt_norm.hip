// Row-wise kernels: the fused history-LayerNorm + DLCL combination of the encoder
// (Sec. 2.1 Eq. 2), plain LayerNorm, the decoder-step embedding, and weight packing.
//
// One 64-lane wave owns one token row of d = 64*EPL elements; lane l holds columns
// [l*EPL, (l+1)*EPL), so every row access is one contiguous, coalesced 64*EPL*b-byte
// transaction.  All statistics and sums are fp32 (Sec. 4.2: reductions are done in a
// wider type than the 16-bit storage).  These kernels are HBM-bound.
#include <algorithm>

#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

// Holds v as a rounded fp32 register value, so that its conversion to the model dtype is a
// rounding of its own.  Left alone, the compiler fuses the last multiply-add before a
// 16-bit store with the conversion (one rounding instead of two) in some instantiations
// and not in others, which would make the low bits depend on the instantiation.
__device__ __forceinline__ void fp32_pin(float& v) { asm volatile("" : "+v"(v)); }

constexpr int ROWS_PER_BLOCK = 4;

// Eq. 2 at the end of encoder layer l-1:
//   h_{l-1} = LN_{hist,l-1}(y_{l-1})            (written into the history, once)
//   x_l     = sum_{k=0}^{l-1} W[l,k] h_k          (fp32 accumulation, k ascending)
//   u_l     = LN(x_l)                            (ln1 of layer l, or LN_out for l = L+1)
// For l = 1, y_0 = sqrt(d) E[id] + PE(pos) is formed in registers (PAD positions -> 0).
// Each history entry is read as stored (rounded to the model dtype), including the one
// just produced, so the result does not depend on whether it came from memory.
// NP: most partial sums this instantiation carries (n_part <= NP; 0 for rows that carry
// none).  With partials and at most eight elements a lane, the kernel is held to 64 VGPRs
// so that eight waves share a SIMD, as for the other rows.
template <typename T, int EPL, int NP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NP > 0 && EPL <= 8 ? 8 : 1)))
void dlcl_kernel(DlclArgs a) {
  const int row = blockIdx.x * ROWS_PER_BLOCK + threadIdx.x / kWave;
  if (row >= a.rows) return;
  const int lane = threadIdx.x % kWave;
  const int d = a.d, c0 = lane * EPL;
  const float inv_d = 1.0f / (float)d;
  T* hist = static_cast<T*>(a.hist);

  float y[EPL];
  if (a.l == 1) {
    const int b = row / a.S, pos = row - b * a.S;
    if (pos < a.lens[b]) {
      const int id = min(max(a.ids[row], 0), a.V - 1);
      load_row<T, EPL>(static_cast<const T*>(a.E) + (size_t)id * d + c0, y);
      const float* pe = a.pe + (size_t)pos * d + c0;
#pragma unroll
      for (int i = 0; i < EPL; ++i) y[i] = a.emb_scale * y[i] + pe[i];
    } else {
#pragma unroll
      for (int i = 0; i < EPL; ++i) y[i] = 0.f;
    }
  } else {
    load_row<T, EPL>(static_cast<const T*>(a.y_prev) + (size_t)row * d + c0, y);
  }

  float h[EPL];
  if (a.hist_norm) {
    wave_layernorm<EPL>(y, h, a.hist_ln, a.hist_ln + d, c0, inv_d, a.eps);
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) h[i] = y[i];
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) fp32_pin(h[i]);
  store_row<T, EPL>(hist + (size_t)(a.l - 1) * a.hist_stride + (size_t)row * d + c0, h);
#pragma unroll
  for (int i = 0; i < EPL; ++i) h[i] = to_f32(from_f32<T>(h[i]));

  float acc[EPL];
  if (a.part_in) {   // this row's sum of entries 0 .. k_start-1, from the block start
    const float* pr = a.part_in + (size_t)row * d + c0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = pr[i];
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
  }
  float pacc[NP > 0 ? NP : 1][EPL];
#pragma unroll
  for (int j = 0; j < NP; ++j)
#pragma unroll
    for (int i = 0; i < EPL; ++i) pacc[j][i] = 0.f;
  const T* hrow = hist + (size_t)row * d + c0;
#pragma unroll 2
  for (int k = a.k_start; k < a.l - 1; ++k) {
    float e[EPL];
    load_row<T, EPL>(hrow + (size_t)k * a.hist_stride, e);
    const float w = a.w[k];
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += w * e[i];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      if (j < a.n_part) {
        const int rj = a.l + 1 + j;
        const float wj = a.w_all[(size_t)rj * (rj - 1) / 2 + k];
#pragma unroll
        for (int i = 0; i < EPL; ++i) pacc[j][i] += wj * e[i];
      }
    }
  }
  {
    const float w = a.w[a.l - 1];
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] += w * h[i];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      if (j < a.n_part) {
        const int rj = a.l + 1 + j;
        const float wj = a.w_all[(size_t)rj * (rj - 1) / 2 + a.l - 1];
        float* po = a.part_out + j * a.part_stride + (size_t)row * d + c0;
#pragma unroll
        for (int i = 0; i < EPL; ++i) po[i] = pacc[j][i] + wj * h[i];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    fp32_pin(acc[i]);
    acc[i] = to_f32(from_f32<T>(acc[i]));
  }
  if (a.x_out) store_row<T, EPL>(static_cast<T*>(a.x_out) + (size_t)row * d + c0, acc);
  float u[EPL];
  wave_layernorm<EPL>(acc, u, a.ln, a.ln + d, c0, inv_d, a.eps);
#pragma unroll
  for (int i = 0; i < EPL; ++i) fp32_pin(u[i]);
  store_row<T, EPL>(static_cast<T*>(a.u_out) + (size_t)row * d + c0, u);
}

template <typename T, int EPL>
__global__ __launch_bounds__(256) void ln_kernel(const T* __restrict__ x, const float* __restrict__ ln,
                                                 T* __restrict__ y, int rows, int d, float eps, const int* ctl,
                                                 int ctl_rows) {
  asm volatile("" ::"s"(x), "s"(ln), "s"(y), "s"(ctl), "s"(rows), "s"(d), "s"(ctl_rows));   // one wait for all arguments
  const int row = blockIdx.x * ROWS_PER_BLOCK + threadIdx.x / kWave;
  if (row >= rows) return;
  // Every row of the grid is allocated, so the row and the gain/bias are read before the
  // live-row count arrives: the count (just written, often by another XCD) gates only
  // the store, and its latency overlaps the row's.
  const int c0 = (threadIdx.x % kWave) * EPL;
  LnCols<EPL> lc;
  load_ln_cols<EPL>(ln, ln + d, c0, lc);
  float v[EPL], o[EPL];
  load_row<T, EPL>(x + (size_t)row * d + c0, v);
  const int live = ctl ? min(rows, ctl[CTL_NLIVE] * ctl_rows) : rows;
  wave_layernorm<EPL>(v, o, lc, 1.0f / (float)d, eps);
  if (row < live) store_row<T, EPL>(y + (size_t)row * d + c0, o);
}

// Decoder input of step t for live row r: z = sqrt(d) E[tok] + PE(t), u = LN(z) (u and ln
// null when the first layer's projection normalises its input itself).
// Every row of the grid computes (its list entry and token are valid IDs whether or not
// the row is live), and the live-row count gates only the stores: so the count, the list
// entry and the gain/bias are in flight together instead of one after another.
template <typename T, int EPL>
__global__ __launch_bounds__(256) void dec_embed_kernel(const int* __restrict__ cur_tok,
                                                        const int* __restrict__ sent_list, int beam,
                                                        const T* __restrict__ E, const float* __restrict__ pe,
                                                        const int* __restrict__ ctl, float scale,
                                                        const float* __restrict__ ln, T* __restrict__ z,
                                                        T* __restrict__ u, int rows, int d, float eps) {
  asm volatile("" ::"s"(cur_tok), "s"(sent_list), "s"(E), "s"(pe), "s"(ctl), "s"(ln), "s"(rows), "s"(beam),
               "s"(d));
  const int row = blockIdx.x * ROWS_PER_BLOCK + threadIdx.x / kWave;
  if (row >= rows) return;
  const int c0 = (threadIdx.x % kWave) * EPL;
  LnCols<EPL> lc;
  if (u) load_ln_cols<EPL>(ln, ln + d, c0, lc);
  const int sent = sent_list[row / beam], t = ctl[CTL_T], nlive = ctl[CTL_NLIVE];
  asm volatile("" ::"v"(sent), "v"(t), "v"(nlive));   // both loads issued before either is waited on
  const int p = sent * beam + row % beam;
  const bool live = row < min(rows, nlive * beam);
  float v[EPL], o[EPL];
  load_row<T, EPL>(E + (size_t)cur_tok[p] * d + c0, v);
  const float* pr = pe + (size_t)t * d + c0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) v[i] = to_f32(from_f32<T>(scale * v[i] + pr[i]));
  if (live) store_row<T, EPL>(z + (size_t)row * d + c0, v);
  if (!u) return;
  wave_layernorm<EPL>(v, o, lc, 1.0f / (float)d, eps);
  if (live) store_row<T, EPL>(u + (size_t)row * d + c0, o);
}

// dst[n][k] = src[k][n] through a 32x33 LDS tile.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const float* __restrict__ src, T* __restrict__ dst, int K,
                                                        int N) {
  __shared__ float tile[32][33];
  const int k0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
  const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;
  for (int r = ty; r < 32; r += 8) {
    const int k = k0 + r, n = n0 + tx;
    tile[r][tx] = (k < K && n < N) ? src[(size_t)k * N + n] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int n = n0 + r, k = k0 + tx;
    if (n < N && k < K) dst[(size_t)n * K + k] = from_f32<T>(tile[tx][r]);
  }
}

template <typename T>
__global__ void convert_kernel(const float* __restrict__ src, T* __restrict__ dst, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = from_f32<T>(src[i]);
}

#define NT_EPL_SWITCH(d, CALL) \
  switch ((d) / 64) {          \
    case 1: CALL(1); break;    \
    case 2: CALL(2); break;    \
    case 4: CALL(4); break;    \
    case 6: CALL(6); break;    \
    case 8: CALL(8); break;    \
    case 12: CALL(12); break;  \
    case 16: CALL(16); break;  \
    default: return hipErrorInvalidValue; \
  }

template <typename T>
hipError_t dlcl_t(const DlclArgs& a, hipStream_t s) {
  const dim3 grid((a.rows + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK);
  if (a.n_part < 0 || a.n_part > DLCL_PARTS) return hipErrorInvalidValue;
#define NT_CALL(E)                                                                    \
  if (a.n_part > 0) NT_LAUNCH((dlcl_kernel<T, E, DLCL_PARTS>), grid, dim3(256), 0, s, a); \
  else NT_LAUNCH((dlcl_kernel<T, E, 0>), grid, dim3(256), 0, s, a)
  NT_EPL_SWITCH(a.d, NT_CALL)
#undef NT_CALL
  return hipGetLastError();
}

template <typename T>
hipError_t ln_t(const void* x, const float* ln, void* y, int rows, int d, float eps, hipStream_t s, const int* ctl,
                int ctl_rows) {
  const dim3 grid((rows + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK);
#define NT_CALL(E)                                                                                            \
  NT_LAUNCH((ln_kernel<T, E>), grid, dim3(256), 0, s, static_cast<const T*>(x), ln, static_cast<T*>(y), \
                     rows, d, eps, ctl, ctl_rows)
  NT_EPL_SWITCH(d, NT_CALL)
#undef NT_CALL
  return hipGetLastError();
}

template <typename T>
hipError_t emb_t(const int* cur_tok, const int* sent_list, int beam, const void* E, const float* pe, const int* ctl,
                 float scale, const float* ln, void* z, void* u, int rows, int d, float eps, hipStream_t s) {
  const dim3 grid((rows + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK);
#define NT_CALL(EP)                                                                                            \
  NT_LAUNCH((dec_embed_kernel<T, EP>), grid, dim3(256), 0, s, cur_tok, sent_list, beam,               \
                     static_cast<const T*>(E), pe, ctl, scale, ln, static_cast<T*>(z), static_cast<T*>(u), rows, \
                     d, eps)
  NT_EPL_SWITCH(d, NT_CALL)
#undef NT_CALL
  return hipGetLastError();
}

}  // namespace

#define NT_DT_SWITCH(dt, FN, ...)                          \
  switch (dt) {                                            \
    case DT::F32: return FN<float>(__VA_ARGS__);           \
    case DT::F16: return FN<f16>(__VA_ARGS__);             \
    case DT::BF16: return FN<bf16>(__VA_ARGS__);           \
  }                                                        \
  return hipErrorInvalidValue;

hipError_t dlcl_combine(DT dt, const DlclArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  NT_DT_SWITCH(dt, dlcl_t, a, s)
}

hipError_t layernorm(DT dt, const void* x, const float* ln, void* y, int rows, int d, float eps, hipStream_t s,
                     const int* ctl, int ctl_rows) {
  if (rows <= 0) return hipSuccess;
  NT_DT_SWITCH(dt, ln_t, x, ln, y, rows, d, eps, s, ctl, ctl_rows)
}

hipError_t dec_embed_ln(DT dt, const int* cur_tok, const int* sent_list, int beam, const void* E, const float* pe,
                        const int* ctl, float emb_scale, const float* ln, void* z, void* u, int rows, int d,
                        float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  NT_DT_SWITCH(dt, emb_t, cur_tok, sent_list, beam, E, pe, ctl, emb_scale, ln, z, u, rows, d, eps, s)
}

namespace {
template <typename T>
hipError_t transpose_t(const float* src, void* dst, int K, int N, hipStream_t s) {
  NT_LAUNCH(transpose_kernel<T>, dim3((N + 31) / 32, (K + 31) / 32), dim3(256), 0, s, src,
                     static_cast<T*>(dst), K, N);
  return hipGetLastError();
}
template <typename T>
hipError_t convert_t(const float* src, void* dst, size_t n, hipStream_t s) {
  const size_t blocks = std::min<size_t>((n + 255) / 256, 65536);
  NT_LAUNCH(convert_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, src, static_cast<T*>(dst), n);
  return hipGetLastError();
}
// One wave per packed row: the row's K values summed in fp32 (lanes stride over k).
template <typename T>
__global__ __launch_bounds__(256) void row_sums_kernel(const T* __restrict__ Bt, int N, int K,
                                                       float* __restrict__ out) {
  const int n = blockIdx.x * 4 + threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (n >= N) return;
  float s = 0.f;
  for (int k = lane; k < K; k += kWave) s += to_f32(Bt[(size_t)n * K + k]);
  s = wave_sum(s);
  if (lane == 0) out[n] = s;
}

template <typename T>
hipError_t row_sums_t(const void* Bt, int N, int K, float* out, hipStream_t s) {
  NT_LAUNCH(row_sums_kernel<T>, dim3((N + 3) / 4), dim3(256), 0, s, static_cast<const T*>(Bt), N, K, out);
  return hipGetLastError();
}
}  // namespace

hipError_t packed_row_sums(DT dt, const void* Bt, int N, int K, float* out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  NT_DT_SWITCH(dt, row_sums_t, Bt, N, K, out, s)
}

hipError_t pack_transpose(DT dt, const float* src, void* dst, int K, int N, hipStream_t s) {
  NT_DT_SWITCH(dt, transpose_t, src, dst, K, N, s)
}

hipError_t pack_convert(DT dt, const float* src, void* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  NT_DT_SWITCH(dt, convert_t, src, dst, n, s)
}

}  // namespace nt
