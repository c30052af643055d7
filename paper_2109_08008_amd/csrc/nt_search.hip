// Search kernels: greedy and beam selection over the fp32 logits, the per-sentence
// search update, batch compaction and the final backtrack.
//
// Greedy (Sec. 4.4): argmax of the logits (ties -> lowest ID) in the same pass as an
// online log-sum-exp, so the chosen token's log-prob is logit - LSE without a
// log_softmax over the vocabulary (Sec. 4.4 drops it for greedy search).
// Beam: each live row keeps its 2K largest logits and its LSE; per sentence the K*2K
// candidates c = score_h + logit - LSE_h are ranked by (c desc, h*V + w asc), the first
// 2K walked: EOS candidates finish (score c / ((5+n)/6)^alpha, n tokens incl. EOS), the
// first K others form the next beam.  A sentence stops once its best finished score is
// at least every live score (Sec. 4.1 "Faster Beam Search") or at its length limit.
// Finished sentences leave the batch by compaction (Sec. 4.1 "Batch Pruning"): the
// list of live sentences is rebuilt and every per-row kernel indexes through it, so
// no cache row is ever copied.
#include <limits.h>

#include <mutex>
#include <vector>

#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

constexpr int SEL_THREADS = 256;
constexpr int SEL_BATCH = 8;      // row loads in flight per thread

struct MaxSum {
  float m, s;
};
__device__ __forceinline__ MaxSum ms_merge(MaxSum a, MaxSum b) {
  if (b.m == -INFINITY) return a;
  if (a.m == -INFINITY) return b;
  const float m = fmaxf(a.m, b.m);
  return {m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}
// (value desc, index asc)
__device__ __forceinline__ bool better(float v1, int i1, float v2, int i2) {
  return v1 > v2 || (v1 == v2 && i1 < i2);
}

// Whole-wave reductions on the DPP network, by the steps of wave_sum.  wave_best keeps
// the best entry under (value desc, index asc) with empty entries (index INT_MAX) last, a
// strict total order, so its result does not depend on the order of the steps;
// ms_merge is symmetric in its operands, so both lanes of a pair hold the same bits after
// each step of wave_ms.  Every lane returns the wave's result; all 64 must be active.
__device__ __forceinline__ bool takes(float ov, int oi, float v, int i) {
  return oi != INT_MAX && (i == INT_MAX || better(ov, oi, v, i));
}
template <int CTRL>
__device__ __forceinline__ void best_step(float& v, int& i, float& p) {
  const float ov = dpp_mov<CTRL>(v), op = dpp_mov<CTRL>(p);
  const int oi = dpp_mov_i<CTRL>(i);
  if (takes(ov, oi, v, i)) { v = ov; i = oi; p = op; }
}
__device__ __forceinline__ void wave_best(float& v, int& i, float& p) {
  best_step<DPP_XOR1>(v, i, p);
  best_step<DPP_XOR2>(v, i, p);
  best_step<DPP_HALF_MIRROR>(v, i, p);
  best_step<DPP_MIRROR>(v, i, p);
  float bv = readlane_f(v, 0), bp = readlane_f(p, 0);
  int bi = readlane_i(i, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const float rv = readlane_f(v, 16 * r), rp = readlane_f(p, 16 * r);
    const int ri = readlane_i(i, 16 * r);
    if (takes(rv, ri, bv, bi)) { bv = rv; bi = ri; bp = rp; }
  }
  v = bv;
  i = bi;
  p = bp;
}
__device__ __forceinline__ void wave_best(float& v, int& i) {
  float p = 0.f;   // no payload: the compiler drops its moves
  wave_best(v, i, p);
}
template <int CTRL>
__device__ __forceinline__ MaxSum ms_step(MaxSum a) {
  return ms_merge(a, MaxSum{dpp_mov<CTRL>(a.m), dpp_mov<CTRL>(a.s)});
}
__device__ __forceinline__ MaxSum wave_ms(MaxSum a) {
  a = ms_step<DPP_XOR1>(a);
  a = ms_step<DPP_XOR2>(a);
  a = ms_step<DPP_HALF_MIRROR>(a);
  a = ms_step<DPP_MIRROR>(a);
  const MaxSum r0{readlane_f(a.m, 0), readlane_f(a.s, 0)}, r1{readlane_f(a.m, 16), readlane_f(a.s, 16)};
  const MaxSum r2{readlane_f(a.m, 32), readlane_f(a.s, 32)}, r3{readlane_f(a.m, 48), readlane_f(a.s, 48)};
  return ms_merge(ms_merge(r0, r1), ms_merge(r2, r3));
}

// Per-thread online max/sum and argmax over a row; returns block-wide results in
// every thread.  Elements are visited in increasing index per thread.
__device__ void row_lse_argmax(const float* __restrict__ x, int V, float& lse, float& best, int& bidx) {
  __shared__ float sm[SEL_THREADS / kWave], ss[SEL_THREADS / kWave], sb[SEL_THREADS / kWave];
  __shared__ int si[SEL_THREADS / kWave];
  const int tid = threadIdx.x;
  MaxSum acc{-INFINITY, 0.f};
  float bv = -INFINITY;
  int bi = INT_MAX;
  const bool vec = (V % 4) == 0 && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
  if (vec) {
    const float4* x4 = reinterpret_cast<const float4*>(x);
    for (int i = tid; i < V / 4; i += SEL_THREADS) {
      const float4 v = x4[i];
      const float mx = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
      if (mx > acc.m) {
        acc.s = acc.m == -INFINITY ? 0.f : acc.s * __expf(acc.m - mx);
        acc.m = mx;
      }
      acc.s += __expf(v.x - acc.m) + __expf(v.y - acc.m) + __expf(v.z - acc.m) + __expf(v.w - acc.m);
      if (v.x > bv) { bv = v.x; bi = 4 * i; }
      if (v.y > bv) { bv = v.y; bi = 4 * i + 1; }
      if (v.z > bv) { bv = v.z; bi = 4 * i + 2; }
      if (v.w > bv) { bv = v.w; bi = 4 * i + 3; }
    }
  } else {
    for (int i = tid; i < V; i += SEL_THREADS) {
      const float v = x[i];
      if (v > acc.m) {
        acc.s = acc.m == -INFINITY ? 0.f : acc.s * __expf(acc.m - v);
        acc.m = v;
      }
      acc.s += __expf(v - acc.m);
      if (v > bv) { bv = v; bi = i; }
    }
  }
  // wave reduction
  acc = wave_ms(acc);
  wave_best(bv, bi);
  const int wave = tid / kWave, lane = tid % kWave;
  if (lane == 0) { sm[wave] = acc.m; ss[wave] = acc.s; sb[wave] = bv; si[wave] = bi; }
  __syncthreads();
  MaxSum tot{sm[0], ss[0]};
  float fb = sb[0];
  int fi = si[0];
#pragma unroll
  for (int w = 1; w < SEL_THREADS / kWave; ++w) {
    tot = ms_merge(tot, MaxSum{sm[w], ss[w]});
    if (better(sb[w], si[w], fb, fi)) { fb = sb[w]; fi = si[w]; }
  }
  lse = tot.m + logf(tot.s);
  best = fb;
  bidx = fi;
}

// Greedy update of sentence b (beam 1: physical row = sentence) with the emitted token
// and its log-prob: EOS finishes the sentence (its log-prob counts in the score), as does
// reaching the length limit.
__device__ void greedy_update(const SearchState& st, int b, int tok, float lp, int t) {
  const int p = b;
  const int R = st.B;
  st.score[p] += lp;
  if (tok == st.eos) {
    st.done[b] = 1;
    st.best_score[b] = st.score[p];
    st.best_raw[b] = st.score[p];
    st.best_nout[b] = t;
    st.best_step[b] = t - 1;
    st.best_row[b] = p;
    return;
  }
  st.tok_hist[(size_t)t * R + p] = tok;
  st.lp_hist[(size_t)t * R + p] = lp;
  st.cur_tok[p] = tok;
  if (t + 1 >= st.maxlen[b]) {
    st.done[b] = 1;
    st.best_score[b] = st.score[p];
    st.best_raw[b] = st.score[p];
    st.best_nout[b] = t + 1;
    st.best_step[b] = t;
    st.best_row[b] = p;
  }
}

__global__ __launch_bounds__(SEL_THREADS) void greedy_kernel(const float* __restrict__ logits,
                                                             const int* __restrict__ forced, SearchState st) {
  const int r = blockIdx.x;
  if (r >= st.ctl[CTL_NLIVE]) return;           // block-uniform; beam 1: rows = live sentences
  const int t = st.ctl[CTL_T];
  const int b = st.sent_list[r];
  const float* x = logits + (size_t)r * st.V;
  float lse, best;
  int bidx;
  row_lse_argmax(x, st.V, lse, best, bidx);
  if (threadIdx.x != 0 || st.done[b]) return;
  int tok = forced ? forced[b] : bidx;
  if (tok < 0 || tok >= st.V) tok = st.eos;   // out-of-range forced ID or an all-NaN row: end the sentence
  greedy_update(st, b, tok, st.logp_input ? x[tok] : x[tok] - lse, t);
}

// Ensemble combination of one member's logits into the per-token scores (see
// ens_combine): the row's log-sum-exp first, then one coalesced pass over the row.
__global__ __launch_bounds__(SEL_THREADS) void ens_combine_kernel(const float* __restrict__ logits,
                                                                  float* __restrict__ comb,
                                                                  const int* __restrict__ ctl, int beam, int V,
                                                                  int member, int n_members, int rule) {
  const int r = blockIdx.x;
  if (r >= ctl[CTL_NLIVE] * beam) return;   // block-uniform
  const float* x = logits + (size_t)r * V;
  float* c = comb + (size_t)r * V;
  float lse, best;
  int bidx;
  row_lse_argmax(x, V, lse, best, bidx);
  const bool first = member == 0, last = member == n_members - 1;
  const float inv_m = 1.0f / (float)n_members, log_m = logf((float)n_members);
  for (int v = threadIdx.x; v < V; v += SEL_THREADS) {
    const float lp = x[v] - lse;
    float o;
    if (rule == 0) {
      o = first ? lp : c[v] + lp;
      if (last) o *= inv_m;
    } else {
      o = lp;
      if (!first) {
        const float a = c[v], hi = fmaxf(a, lp), lo = fminf(a, lp);
        o = hi == -INFINITY ? -INFINITY : hi + log1pf(expf(lo - hi));
      }
      if (last) o -= log_m;
    }
    c[v] = o;
  }
}

// Greedy selection from the projection's per-tile partials [rows][n_tiles][4]
// (max, sum exp, best value, best index): merged in tile order, then the update.
__global__ __launch_bounds__(SEL_THREADS) void greedy_fused_kernel(const float* __restrict__ part, int n_tiles,
                                                                   SearchState st) {
  __shared__ float sm[SEL_THREADS / kWave], ss[SEL_THREADS / kWave], sb[SEL_THREADS / kWave];
  __shared__ int si[SEL_THREADS / kWave];
  asm volatile("" ::"s"(part), "s"(n_tiles), "s"(st.sent_list), "s"(st.ctl));   // one wait for the arguments
  const int r = blockIdx.x;   // every row of the grid has records and a list entry
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const float4* rec = reinterpret_cast<const float4*>(part + (size_t)r * n_tiles * 4);
  // The thread's first record, the list entry and the step counters are read together;
  // the live-row check waits for them all at once.
  float4 q0 = rec[min(tid, n_tiles - 1)];
  const int b = st.sent_list[r], nlive = st.ctl[CTL_NLIVE], t = st.ctl[CTL_T];
  asm volatile("" ::"v"(q0.x), "v"(q0.y), "v"(q0.z), "v"(q0.w), "v"(b), "s"(nlive), "s"(t));
  if (r >= nlive) return;
  if (tid >= n_tiles) q0 = float4{-INFINITY, 0.f, -INFINITY, __int_as_float(INT_MAX)};   // merges as nothing
  MaxSum acc{-INFINITY, 0.f};
  float bv = -INFINITY;
  int bi = INT_MAX;
  for (int i = tid; i < n_tiles; i += SEL_THREADS) {
    const float4 q = i == tid ? q0 : rec[i];
    acc = ms_merge(acc, MaxSum{q.x, q.y});
    const int qi = __float_as_int(q.w);
    if (qi != INT_MAX && better(q.z, qi, bv, bi)) { bv = q.z; bi = qi; }
  }
  acc = wave_ms(acc);
  wave_best(bv, bi);
  if (lane == 0) { sm[wave] = acc.m; ss[wave] = acc.s; sb[wave] = bv; si[wave] = bi; }
  __syncthreads();
  if (tid != 0 || st.done[b]) return;
  MaxSum tot{sm[0], ss[0]};
  float fb = sb[0];
  int fi = si[0];
  for (int w = 1; w < SEL_THREADS / kWave; ++w) {
    tot = ms_merge(tot, MaxSum{sm[w], ss[w]});
    if (better(sb[w], si[w], fb, fi)) { fb = sb[w]; fi = si[w]; }
  }
  const float lse = tot.m + logf(tot.s);
  int tok = fi;
  float lp = fb - lse;
  if (tok < 0 || tok >= st.V) { tok = st.eos; lp = 0.f; }   // an all-NaN row: end the sentence
  greedy_update(st, b, tok, lp, t);
}

// ---- beam: per-row LSE and top-2K logits -----------------------------------------------
template <int K2>
__device__ __forceinline__ void list_insert(float (&v)[K2], int (&ix)[K2], float x, int i) {
  if (!(x > v[K2 - 1])) return;       // equal values keep the earlier (lower) index
  v[K2 - 1] = x;
  ix[K2 - 1] = i;
#pragma unroll
  for (int j = K2 - 1; j > 0; --j) {
    if (v[j] > v[j - 1]) {
      const float tv = v[j]; v[j] = v[j - 1]; v[j - 1] = tv;
      const int ti = ix[j]; ix[j] = ix[j - 1]; ix[j - 1] = ti;
    }
  }
}

template <int K2>
__global__ __launch_bounds__(SEL_THREADS) void beam_select_kernel(const float* __restrict__ logits,
                                                                  const int* __restrict__ ctl, int beam, int V, int k2,
                                                                  float* __restrict__ topv, int* __restrict__ topi,
                                                                  float* __restrict__ lse_out) {
  __shared__ float wv[SEL_THREADS / kWave][K2];
  __shared__ int wi[SEL_THREADS / kWave][K2];
  __shared__ float sm[SEL_THREADS / kWave], ss[SEL_THREADS / kWave];
  const int r = blockIdx.x;
  if (ctl && r >= ctl[CTL_NLIVE] * beam) return;
  const float* x = logits + (size_t)r * V;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;

  // one pass over the row: online max/sum for the LSE and a sorted list of this
  // thread's K2 largest logits (elements visited in increasing index)
  MaxSum acc{-INFINITY, 0.f};
  float v[K2];
  int ix[K2];
#pragma unroll
  for (int j = 0; j < K2; ++j) { v[j] = -INFINITY; ix[j] = INT_MAX; }
  const bool vec = (V % 4) == 0 && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
  if (vec) {
    // SEL_BATCH loads of a thread are issued together before any is used (one memory
    // latency per batch instead of per element group)
    const float4* x4 = reinterpret_cast<const float4*>(x);
    const int nv = V / 4;
    for (int i0 = tid; i0 < nv; i0 += SEL_THREADS * SEL_BATCH) {
      float4 qs[SEL_BATCH];
#pragma unroll
      for (int u = 0; u < SEL_BATCH; ++u) {
        const int i = i0 + u * SEL_THREADS;
        qs[u] = i < nv ? x4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
#pragma unroll
      for (int u = 0; u < SEL_BATCH; ++u) {
        const int i = i0 + u * SEL_THREADS;
        const float4 q = qs[u];
        const float mx = fmaxf(fmaxf(q.x, q.y), fmaxf(q.z, q.w));
        if (mx > acc.m) {
          acc.s = acc.m == -INFINITY ? 0.f : acc.s * __expf(acc.m - mx);
          acc.m = mx;
        }
        if (i < nv) acc.s += __expf(q.x - acc.m) + __expf(q.y - acc.m) + __expf(q.z - acc.m) + __expf(q.w - acc.m);
        if (mx > v[K2 - 1]) {
          list_insert<K2>(v, ix, q.x, 4 * i);
          list_insert<K2>(v, ix, q.y, 4 * i + 1);
          list_insert<K2>(v, ix, q.z, 4 * i + 2);
          list_insert<K2>(v, ix, q.w, 4 * i + 3);
        }
      }
    }
  } else {
    for (int i = tid; i < V; i += SEL_THREADS) {
      const float q = x[i];
      if (q > acc.m) {
        acc.s = acc.m == -INFINITY ? 0.f : acc.s * __expf(acc.m - q);
        acc.m = q;
      }
      acc.s += __expf(q - acc.m);
      list_insert<K2>(v, ix, q, i);
    }
  }
  acc = wave_ms(acc);
  if (lane == 0) { sm[wave] = acc.m; ss[wave] = acc.s; }

  // each wave merges its 64 lists: K2 rounds of a wave-wide (value desc, index asc) argmax;
  // the winning lane drops its head
  for (int round = 0; round < K2; ++round) {
    float bv = v[0];
    int bi = ix[0];
    wave_best(bv, bi);
    if (lane == 0) { wv[wave][round] = bv; wi[wave][round] = bi; }
    if (ix[0] == bi && v[0] == bv && bi != INT_MAX) {
#pragma unroll
      for (int j = 0; j < K2 - 1; ++j) { v[j] = v[j + 1]; ix[j] = ix[j + 1]; }
      v[K2 - 1] = -INFINITY;
      ix[K2 - 1] = INT_MAX;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int head[SEL_THREADS / kWave] = {0, 0, 0, 0};
    for (int j = 0; j < k2; ++j) {
      int w = 0;
      float bv = -INFINITY;
      int bi = INT_MAX;
      for (int q = 0; q < SEL_THREADS / kWave; ++q) {
        if (head[q] >= K2 || wi[q][head[q]] == INT_MAX) continue;     // list exhausted
        if (bi == INT_MAX || better(wv[q][head[q]], wi[q][head[q]], bv, bi)) {
          bv = wv[q][head[q]]; bi = wi[q][head[q]]; w = q;
        }
      }
      head[w]++;
      topv[(size_t)r * k2 + j] = bv;
      topi[(size_t)r * k2 + j] = bi;
    }
    MaxSum tot{sm[0], ss[0]};
#pragma unroll
    for (int w = 1; w < SEL_THREADS / kWave; ++w) tot = ms_merge(tot, MaxSum{sm[w], ss[w]});
    lse_out[r] = tot.m + logf(tot.s);
  }
}

// Beam selection for rows of at most SEL_THREADS * 4 * SEL_REG logits, held in registers:
// pass 1 forms the online (max, sum exp) and each thread's maximum; the K2-th largest
// thread maximum is a threshold that every one of the row's K2 best logits reaches (the
// K2 largest thread maxima are K2 distinct logits at or above it); pass 2 inserts only
// logits at or above it into the thread lists, which are then merged as in
// beam_select_kernel.  Same result, without a list insertion for most logits.
constexpr int SEL_REG = 32;        // float4 per thread -> rows up to 32768 logits
template <int K2>
__global__ __launch_bounds__(SEL_THREADS) void beam_select_reg_kernel(const float* __restrict__ logits,
                                                                      const int* __restrict__ ctl, int beam, int V,
                                                                      int k2, float* __restrict__ topv,
                                                                      int* __restrict__ topi,
                                                                      float* __restrict__ lse_out) {
  __shared__ float wv[SEL_THREADS / kWave][K2];
  __shared__ int wi[SEL_THREADS / kWave][K2];
  __shared__ float sm[SEL_THREADS / kWave], ss[SEL_THREADS / kWave];
  __shared__ float wmax[SEL_THREADS / kWave][K2];
  __shared__ float thr_s;
  const int r = blockIdx.x;
  if (ctl && r >= ctl[CTL_NLIVE] * beam) return;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const float4* x4 = reinterpret_cast<const float4*>(logits + (size_t)r * V);
  const int nv = V / 4;
  float4 q[SEL_REG];
#pragma unroll
  for (int u = 0; u < SEL_REG; ++u) {
    const int i = tid + u * SEL_THREADS;
    q[u] = i < nv ? x4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
  // pass 1: thread maximum, then the sum of exp against it
  float tmax = -INFINITY;
#pragma unroll
  for (int u = 0; u < SEL_REG; ++u) tmax = fmaxf(tmax, fmaxf(fmaxf(q[u].x, q[u].y), fmaxf(q[u].z, q[u].w)));
  MaxSum acc{tmax, 0.f};
  if (tmax != -INFINITY) {
#pragma unroll
    for (int u = 0; u < SEL_REG; ++u)
      acc.s += (__expf(q[u].x - tmax) + __expf(q[u].y - tmax)) + (__expf(q[u].z - tmax) + __expf(q[u].w - tmax));
  }
  acc = wave_ms(acc);
  if (lane == 0) { sm[wave] = acc.m; ss[wave] = acc.s; }
  // the K2 largest thread maxima of each wave (K2 rounds of a wave max; one lane drops out)
  {
    float mine = tmax;
    for (int j = 0; j < K2; ++j) {
      float best = mine;
      int bl = lane;
      wave_best(best, bl);
      if (lane == 0) wmax[wave][j] = best;
      if (lane == bl) mine = -INFINITY;
    }
  }
  __syncthreads();
  if (tid == 0) {
    // K2-th largest of the per-wave sorted lists
    int head[SEL_THREADS / kWave] = {0, 0, 0, 0};
    float t = -INFINITY;
    for (int j = 0; j < K2; ++j) {
      int w = 0;
      float bv = -INFINITY;
      for (int q2 = 0; q2 < SEL_THREADS / kWave; ++q2)
        if (head[q2] < K2 && (wmax[q2][head[q2]] > bv || w < 0)) { bv = wmax[q2][head[q2]]; w = q2; }
      head[w]++;
      t = bv;
    }
    thr_s = t;
  }
  __syncthreads();
  const float thr = thr_s;
  // pass 2: bit masks of the logits at or above the threshold (bit 4*(u%8)+c of word u/8),
  // then the few candidates go into the thread list in increasing index order, re-read
  // from memory (the register copy cannot be indexed by a run-time position)
  unsigned cand[SEL_REG / 8] = {};
#pragma unroll
  for (int u = 0; u < SEL_REG; ++u) {
    const float4 x = q[u];
    const unsigned bits = (x.x >= thr ? 1u : 0u) | (x.y >= thr ? 2u : 0u) | (x.z >= thr ? 4u : 0u) |
                          (x.w >= thr ? 8u : 0u);
    if (tid + u * SEL_THREADS < nv) cand[u / 8] |= bits << (4 * (u % 8));   // padding never re-read
  }
  float v[K2];
  int ix[K2];
#pragma unroll
  for (int j = 0; j < K2; ++j) { v[j] = -INFINITY; ix[j] = INT_MAX; }
  const float* row = logits + (size_t)r * V;
#pragma unroll
  for (int wd = 0; wd < SEL_REG / 8; ++wd) {
    unsigned m = cand[wd];
    while (m) {
      const int b = __builtin_ctz(m);
      m &= m - 1;
      const int idx = 4 * (tid + (wd * 8 + b / 4) * SEL_THREADS) + (b & 3);
      list_insert<K2>(v, ix, row[idx], idx);
    }
  }
  // merge: per wave K2 rounds of a (value desc, index asc) argmax, then thread 0 over waves
  for (int round = 0; round < K2; ++round) {
    float bv = v[0];
    int bi = ix[0];
    wave_best(bv, bi);
    if (lane == 0) { wv[wave][round] = bv; wi[wave][round] = bi; }
    if (ix[0] == bi && v[0] == bv && bi != INT_MAX) {
#pragma unroll
      for (int j = 0; j < K2 - 1; ++j) { v[j] = v[j + 1]; ix[j] = ix[j + 1]; }
      v[K2 - 1] = -INFINITY;
      ix[K2 - 1] = INT_MAX;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int head[SEL_THREADS / kWave] = {0, 0, 0, 0};
    for (int j = 0; j < k2; ++j) {
      int w = 0;
      float bv = -INFINITY;
      int bi = INT_MAX;
      for (int q2 = 0; q2 < SEL_THREADS / kWave; ++q2) {
        if (head[q2] >= K2 || wi[q2][head[q2]] == INT_MAX) continue;
        if (bi == INT_MAX || better(wv[q2][head[q2]], wi[q2][head[q2]], bv, bi)) {
          bv = wv[q2][head[q2]]; bi = wi[q2][head[q2]]; w = q2;
        }
      }
      head[w]++;
      topv[(size_t)r * k2 + j] = bv;
      topi[(size_t)r * k2 + j] = bi;
    }
    MaxSum tot{sm[0], ss[0]};
#pragma unroll
    for (int w = 1; w < SEL_THREADS / kWave; ++w) tot = ms_merge(tot, MaxSum{sm[w], ss[w]});
    lse_out[r] = tot.m + logf(tot.s);
  }
}

// Beam selection from the output projection's per-tile records.  The projection's
// epilogue leaves, for every row and 128-column tile, the tile row's (max, sum of
// exp(x - max)); the logits are written as well.  Let tau be the k2-th largest of a row's
// tile maxima.  Every logit among the row's k2 largest lies in a tile whose maximum is at
// least tau: a logit x in a tile of maximum below tau is smaller than at least k2 logits
// (one per tile of maximum >= tau).  Equal values are covered too: a tile whose maximum
// is below tau holds nothing equal to the k2-th largest logit, which is >= tau.  So only
// the candidate tiles are read back -- usually k2 of them -- and the log-sum-exp comes
// from merging the records.  One wave per row; the result equals a scan of the whole row
// in (value desc, index asc) order.
constexpr int TILE_COLS = 128;
constexpr int SEL_TPL = 8;          // tile records per lane: up to 512 tiles (V <= 65536)

template <int K2>
__global__ __launch_bounds__(256) void beam_select_tiles_kernel(const float* __restrict__ part, int n_tiles,
                                                                const float* __restrict__ logits,
                                                                const int* __restrict__ ctl, int beam, int rows,
                                                                int V, int k2, float* __restrict__ topv,
                                                                int* __restrict__ topi,
                                                                float* __restrict__ lse_out) {
  constexpr int REC = 4;            // record floats (max, sum, best value, best index)
  constexpr int SEL_CAND = K2 < 8 ? 8 : K2 > 16 ? 16 : K2;   // candidate tiles per batch (usually all)
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  asm volatile("" ::"s"(part), "s"(n_tiles), "s"(logits), "s"(ctl), "s"(beam), "s"(rows), "s"(V), "s"(k2));
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows) return;            // grid tail
  const float* rec = part + (size_t)r * n_tiles * REC;
  // The row's records (every row of the grid has them) and the live count are read
  // together; the live-row check waits for them all at once.
  float2 rq[SEL_TPL];
#pragma unroll
  for (int j = 0; j < SEL_TPL; ++j)
    rq[j] = *reinterpret_cast<const float2*>(rec + (size_t)min(lane + j * kWave, n_tiles - 1) * REC);
  const int live = ctl ? min(rows, ctl[CTL_NLIVE] * beam) : rows;
#pragma unroll
  for (int j = 0; j < SEL_TPL; ++j) asm volatile("" ::"v"(rq[j].x), "v"(rq[j].y));
  asm volatile("" ::"s"(live));
  if (r >= live) return;            // whole wave; no block barrier below
  // the lane's tile maxima, and the row's (max, sum) merged over every record
  float tm[SEL_TPL];
  MaxSum acc{-INFINITY, 0.f};
#pragma unroll
  for (int j = 0; j < SEL_TPL; ++j) {
    const int t = lane + j * kWave;
    tm[j] = t < n_tiles ? rq[j].x : -INFINITY;
    if (t < n_tiles) acc = ms_merge(acc, MaxSum{rq[j].x, rq[j].y});
  }
  acc = wave_ms(acc);
  // tau: k2 rounds of a wave max over the tile maxima, each winner giving up that entry
  float tau = -INFINITY;
  {
    float rest[SEL_TPL];
#pragma unroll
    for (int j = 0; j < SEL_TPL; ++j) rest[j] = tm[j];
    for (int round = 0; round < k2; ++round) {
      float mine = -INFINITY;
#pragma unroll
      for (int j = 0; j < SEL_TPL; ++j) mine = fmaxf(mine, rest[j]);
      float best = mine;
      int bl = lane;
      wave_best(best, bl);
      tau = best;
      if (lane == bl) {
        bool gone = false;
#pragma unroll
        for (int j = 0; j < SEL_TPL; ++j)
          if (!gone && rest[j] == best) { rest[j] = -INFINITY; gone = true; }
      }
    }
  }
  // candidate tiles in increasing order, read SEL_CAND at a time with every load issued
  // before any use; each lane inserts its columns in increasing index order
  float v[K2];
  int ix[K2];
#pragma unroll
  for (int j = 0; j < K2; ++j) { v[j] = -INFINITY; ix[j] = INT_MAX; }
  const float* row = logits + (size_t)r * V;
  int j = 0;
  unsigned long long mask = __ballot(lane < n_tiles && tm[0] >= tau);
  bool more = true;
  while (more) {
    int ct[SEL_CAND];
#pragma unroll
    for (int c = 0; c < SEL_CAND; ++c) {
      ct[c] = -1;
      while (more && mask == 0) {
        if (++j >= SEL_TPL) {
          more = false;
        } else {
          float tj = -INFINITY;
#pragma unroll
          for (int q = 0; q < SEL_TPL; ++q) tj = q == j ? tm[q] : tj;
          mask = __ballot(lane + j * kWave < n_tiles && tj >= tau);
        }
      }
      if (more) {
        const int l = __builtin_ctzll(mask);
        mask &= mask - 1;
        ct[c] = l + j * kWave;
      }
    }
    float xs[SEL_CAND][2];
#pragma unroll
    for (int c = 0; c < SEL_CAND; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = ct[c] * TILE_COLS + h * kWave + lane;
        const bool ok = ct[c] >= 0 && n < V;
        const float x = row[ok ? n : 0];
        xs[c][h] = ok ? x : -INFINITY;
      }
#pragma unroll
    for (int c = 0; c < SEL_CAND; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float x = xs[c][h];
        if (x >= tau) list_insert<K2>(v, ix, x, ct[c] * TILE_COLS + h * kWave + lane);
      }
  }
  // k2 rounds of a (value desc, index asc) wave argmax
  for (int round = 0; round < k2; ++round) {
    float bv = v[0];
    int bi = ix[0];
    wave_best(bv, bi);
    if (lane == 0) {
      topv[(size_t)r * k2 + round] = bi == INT_MAX ? -INFINITY : bv;
      topi[(size_t)r * k2 + round] = bi;
    }
    if (ix[0] == bi && bi != INT_MAX) {
#pragma unroll
      for (int q = 0; q < K2 - 1; ++q) { v[q] = v[q + 1]; ix[q] = ix[q + 1]; }
      v[K2 - 1] = -INFINITY;
      ix[K2 - 1] = INT_MAX;
    }
  }
  if (lane == 0) lse_out[r] = acc.m + logf(acc.s);
}

// Beam selection without stored logits.  The projection leaves only the per-tile records
// (max, sum of exp(x - max), best value, best column).  Order a row's tiles by their best
// entries under (value desc, column asc) and take the first k2: the j-th largest logit x
// of the row (same order) lies in some tile T, and every tile ranked before T has a best
// entry ranked before T's, which is at or before x -- j - 1 entries at most -- so T is
// among the first k2.  Only those tiles' logits are formed again (gemm_pairs, bitwise the
// projection's values), and the row's k2 largest come from them.
template <int TPL>
__global__ __launch_bounds__(256) void beam_pick_tiles_kernel(const float* __restrict__ part, int n_tiles,
                                                              const int* __restrict__ ctl, int beam, int rows,
                                                              int k2, int* __restrict__ ptile,
                                                              float* __restrict__ tau_out,
                                                              float* __restrict__ lse_out) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  asm volatile("" ::"s"(part), "s"(n_tiles), "s"(ctl), "s"(beam), "s"(rows), "s"(k2));
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows) return;            // grid tail
  const float* rec = part + (size_t)r * n_tiles * 4;
  float4 rq[TPL];
#pragma unroll
  for (int j = 0; j < TPL; ++j)
    rq[j] = *reinterpret_cast<const float4*>(rec + (size_t)min(lane + j * kWave, n_tiles - 1) * 4);
  const int live = ctl ? min(rows, ctl[CTL_NLIVE] * beam) : rows;
#pragma unroll
  for (int j = 0; j < TPL; ++j) asm volatile("" ::"v"(rq[j].x), "v"(rq[j].y), "v"(rq[j].z), "v"(rq[j].w));
  asm volatile("" ::"s"(live));
  if (r >= live) return;            // whole wave; no block barrier below
  float tv[TPL];                    // the lane's tiles' best entries; taken ones become empty
  int tc[TPL];
  MaxSum acc{-INFINITY, 0.f};
#pragma unroll
  for (int j = 0; j < TPL; ++j) {
    const bool ok = lane + j * kWave < n_tiles;
    tv[j] = ok ? rq[j].z : -INFINITY;
    tc[j] = ok ? __float_as_int(rq[j].w) : INT_MAX;
    if (ok) acc = ms_merge(acc, MaxSum{rq[j].x, rq[j].y});
  }
  acc = wave_ms(acc);
  float tau = -INFINITY;
  int mine = -1;                    // lane j2 keeps the row's j2-th tile
  for (int j2 = 0; j2 < k2; ++j2) {
    float bv = -INFINITY;
    int bc = INT_MAX;
#pragma unroll
    for (int j = 0; j < TPL; ++j)
      if (takes(tv[j], tc[j], bv, bc)) { bv = tv[j]; bc = tc[j]; }
    wave_best(bv, bc);
    const int tile = bc == INT_MAX ? -1 : bc / TILE_COLS;
    tau = bv;                       // -inf once the row has fewer than k2 tiles
    if (lane == j2) mine = tile;
    if (tile >= 0 && lane == (tile & (kWave - 1))) {   // the owner gives the tile up
#pragma unroll
      for (int j = 0; j < TPL; ++j)
        if (j == tile / kWave) { tv[j] = -INFINITY; tc[j] = INT_MAX; }
    }
  }
  if (lane < k2) ptile[(size_t)r * k2 + lane] = mine;
  if (lane == 0) {
    tau_out[r] = tau;
    lse_out[r] = acc.m + logf(acc.s);
  }
}

// Counting sort of the live rows' pairs by tile in one workgroup, in LDS: the counts, an
// exclusive scan for each tile's first position, the blocks, then every pair placed in
// its tile's run.  Consecutive pairs belong to one row's distinct tiles, so the lanes of
// one LDS atomic meet on an address only across rows (64 / k2 at most).  Up to
// BUCKET_LDS pairs the runs are assembled in LDS and copied out in order (coalesced);
// beyond, each pair is stored to its place directly.  Global memory sees no atomics:
// device-wide atomics on one address serialise.
constexpr int BUCKET_THREADS = 1024, BUCKET_BATCH = 8, BUCKET_LDS = 36864;
__global__ __launch_bounds__(BUCKET_THREADS) void pair_bucket_kernel(const int* __restrict__ ptile,
                                                                     const int* __restrict__ ctl, int beam,
                                                                     int rows, int k2, int n_tiles,
                                                                     int* __restrict__ sorted,
                                                                     int* __restrict__ gblk,
                                                                     int* __restrict__ gnblk) {
  __shared__ int cnt[512], cur[512], nbs[512];
  __shared__ int runs[BUCKET_LDS];
  const int t = threadIdx.x;
  if (t < 512) cnt[t] = 0;
  const int live = ctl ? min(rows, ctl[CTL_NLIVE] * beam) : rows;
  const int np = live * k2;
  __syncthreads();
  // each pass reads BUCKET_BATCH entries a thread before using any: one load round trip per batch
  for (int i0 = t; i0 < np; i0 += BUCKET_THREADS * BUCKET_BATCH) {
    int tl[BUCKET_BATCH];
#pragma unroll
    for (int b = 0; b < BUCKET_BATCH; ++b) {
      const int i = i0 + b * BUCKET_THREADS;
      tl[b] = i < np ? ptile[i] : -1;
    }
#pragma unroll
    for (int b = 0; b < BUCKET_BATCH; ++b)
      if (tl[b] >= 0) atomicAdd(&cnt[tl[b]], 1);
  }
  __syncthreads();
  // exclusive scans of the counts (positions) and of the blocks per tile
  const int c = t < n_tiles ? cnt[t] : 0;
  const int nb = (c + PAIR_BM - 1) / PAIR_BM;
  if (t < 512) { cur[t] = c; nbs[t] = nb; }
  __syncthreads();
  for (int o = 1; o < 512; o <<= 1) {   // inclusive, Hillis-Steele
    const int v1 = t < 512 && t >= o ? cur[t - o] : 0;
    const int v2 = t < 512 && t >= o ? nbs[t - o] : 0;
    __syncthreads();
    if (t < 512) { cur[t] += v1; nbs[t] += v2; }
    __syncthreads();
  }
  const int total = cur[511];
  if (t < n_tiles) {
    const int first = cur[t] - c, fb = nbs[t] - nb;
    for (int b = 0; b < nb; ++b) {
      int* g = gblk + 3 * (size_t)(fb + b);
      g[0] = t;
      g[1] = first + b * PAIR_BM;
      g[2] = min(PAIR_BM, c - b * PAIR_BM);
    }
  }
  if (t == 0) *gnblk = nbs[511];
  __syncthreads();
  if (t < n_tiles) cur[t] -= c;          // each tile's next free position
  __syncthreads();
  const bool in_lds = total <= BUCKET_LDS;   // the same in every thread
  for (int i0 = t; i0 < np; i0 += BUCKET_THREADS * BUCKET_BATCH) {
    int tl[BUCKET_BATCH];
#pragma unroll
    for (int b = 0; b < BUCKET_BATCH; ++b) {
      const int i = i0 + b * BUCKET_THREADS;
      tl[b] = i < np ? ptile[i] : -1;
    }
#pragma unroll
    for (int b = 0; b < BUCKET_BATCH; ++b)
      if (tl[b] >= 0) {
        const int pos = atomicAdd(&cur[tl[b]], 1);
        if (in_lds) runs[pos] = i0 + b * BUCKET_THREADS;
        else sorted[pos] = i0 + b * BUCKET_THREADS;
      }
  }
  if (in_lds) {
    __syncthreads();
    for (int i = t; i < total; i += BUCKET_THREADS) sorted[i] = runs[i];
  }
}

// One wave per live row: the lanes scan the row's recomputed tiles (column h*64 + lane of
// each, both halves), keep the logits at or above tau in sorted lists, and k2 rounds of a
// wave argmax under (value desc, index asc) emit them in order.
template <int K2>
__global__ __launch_bounds__(256) void beam_select_pairs_kernel(const float* __restrict__ logp,
                                                                const int* __restrict__ ptile,
                                                                const float* __restrict__ tau_in,
                                                                const int* __restrict__ ctl, int beam, int rows,
                                                                int V, int k2, float* __restrict__ topv,
                                                                int* __restrict__ topi) {
  constexpr int CB = 8;             // tiles read per batch, every load issued before any use
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  asm volatile("" ::"s"(logp), "s"(ptile), "s"(tau_in), "s"(ctl), "s"(beam), "s"(rows), "s"(V), "s"(k2));
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows) return;
  const int live = ctl ? min(rows, ctl[CTL_NLIVE] * beam) : rows;
  if (r >= live) return;
  const float tau = tau_in[r];
  float v[K2];
  int ix[K2];
#pragma unroll
  for (int j = 0; j < K2; ++j) { v[j] = -INFINITY; ix[j] = INT_MAX; }
  for (int c0 = 0; c0 < k2; c0 += CB) {
    int tl[CB];
    float xs[CB][2];
#pragma unroll
    for (int c = 0; c < CB; ++c) tl[c] = c0 + c < k2 ? ptile[(size_t)r * k2 + c0 + c] : -1;
#pragma unroll
    for (int c = 0; c < CB; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float* src = logp + ((size_t)r * k2 + (tl[c] >= 0 ? c0 + c : 0)) * TILE_COLS + h * kWave + lane;
        xs[c][h] = *src;
      }
#pragma unroll
    for (int c = 0; c < CB; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = tl[c] * TILE_COLS + h * kWave + lane;
        if (tl[c] >= 0 && n < V && xs[c][h] >= tau) list_insert<K2>(v, ix, xs[c][h], n);
      }
  }
  for (int round = 0; round < k2; ++round) {
    float bv = v[0];
    int bi = ix[0];
    wave_best(bv, bi);
    if (lane == 0) {
      topv[(size_t)r * k2 + round] = bi == INT_MAX ? -INFINITY : bv;
      topi[(size_t)r * k2 + round] = bi;
    }
    if (ix[0] == bi && bi != INT_MAX) {
#pragma unroll
      for (int q = 0; q < K2 - 1; ++q) { v[q] = v[q + 1]; ix[q] = ix[q + 1]; }
      v[K2 - 1] = -INFINITY;
      ix[K2 - 1] = INT_MAX;
    }
  }
}

// The per-tile records of a logits matrix, as the projection's epilogue forms them: one
// wave per (row, tile), (max, sum of exp(x - max)) over the tile's columns.  For tests.
__global__ __launch_bounds__(256) void tile_records_kernel(const float* __restrict__ logits, int rows, int V,
                                                           int n_tiles, float* __restrict__ part) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const long long task = (long long)blockIdx.x * 4 + wave;
  if (task >= (long long)rows * n_tiles) return;
  const int r = (int)(task / n_tiles), t = (int)(task % n_tiles);
  MaxSum acc{-INFINITY, 0.f};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int n = t * TILE_COLS + h * kWave + lane;
    const float x = n < V ? logits[(size_t)r * V + n] : -INFINITY;
    if (x != -INFINITY) acc = ms_merge(acc, MaxSum{x, 1.f});
  }
  acc = wave_ms(acc);
  if (lane == 0) {
    float* q = part + ((size_t)r * n_tiles + t) * 4;
    q[0] = acc.m;
    q[1] = acc.s;
    q[2] = acc.m;
    q[3] = 0.f;
  }
}

// ---- beam: per-sentence update (one wave per live sentence) ----------------------------
constexpr int MAXC = 8;       // candidates per lane: K * 2K <= 512 = 64 * 8

__global__ __launch_bounds__(256) void beam_update_kernel(const float* __restrict__ topv,
                                                          const int* __restrict__ topi,
                                                          const float* __restrict__ lse, SearchState st) {
  __shared__ float sel_c[4][32], sel_lp[4][32];
  __shared__ int sel_key[4][32];
  __shared__ int nk_par[4][16], nk_cnt[4];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  asm volatile("" ::"s"(topv), "s"(topi), "s"(lse), "s"(st.B), "s"(st.beam), "s"(st.V), "s"(st.sent_list),
               "s"(st.ctl), "s"(st.score), "s"(st.done));
  const int bl = blockIdx.x * 4 + wave;
  if (bl >= st.B) return;                           // grid tail
  const int K = st.beam, K2 = 2 * K, V = st.V;
  const int ncand = K * K2;
  // The candidates of list entry bl (every entry of the grid has them), the entry and the
  // live count are read together, then the sentence's flag and scores: two dependent
  // round trips before the merge instead of four.
  float rv[MAXC], rl[MAXC], rs[MAXC];
  int rw[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    rv[c] = -INFINITY;
    rl[c] = 0.f;
    rw[c] = INT_MAX;
    if (c * kWave < ncand) {                // the same in every lane
      const int q = min(lane + c * kWave, ncand - 1), k = q / K2, i = q - k * K2, r = bl * K + k;
      rv[c] = topv[(size_t)r * K2 + i];
      rw[c] = topi[(size_t)r * K2 + i];
      rl[c] = lse[r];
    }
  }
  const int b0 = st.sent_list[bl], nlive = st.ctl[CTL_NLIVE];
  asm volatile("" ::"v"(b0), "s"(nlive));
  if (bl >= nlive) return;                          // whole wave leaves; no block barrier below
  const int b = b0;
  const int t = st.ctl[CTL_T], asel = st.ctl[CTL_ANC];
  const int* anc_cur = st.anc + (size_t)asel * st.anc_stride;
  int* anc_next = st.anc + (size_t)(asel ^ 1) * st.anc_stride;
  const int n = t + 1;
  const int done = st.done[b];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    rs[c] = 0.f;
    if (c * kWave < ncand) rs[c] = st.score[b * K + min(lane + c * kWave, ncand - 1) / K2];
  }
  // the sentence's best finished hypothesis and length limit arrive with the flag and
  // the scores; the serial update below keeps them in registers and stores them once
  int bf_nout = st.best_nout[b], bf_step = st.best_step[b], bf_row = st.best_row[b];
  float bf_score = st.best_score[b], bf_raw = st.best_raw[b];
  const int maxlen_b = st.maxlen[b];
  asm volatile("" ::"v"(done));
  if (done) return;

  float cv[MAXC], clp[MAXC];
  int ck[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int q = lane + c * kWave;
    cv[c] = -INFINITY;
    clp[c] = 0.f;
    ck[c] = INT_MAX;
    if (q < ncand) {
      const int k = q / K2;
      const float v = rv[c];
      const int w = rw[c];
      if (w == INT_MAX) continue;           // fewer than 2K words in the vocabulary
      const float lp = st.logp_input ? v : v - rl[c];
      cv[c] = rs[c] + lp;
      clp[c] = lp;
      ck[c] = k * V + w;
    }
  }
  // top-2K by (c desc, key asc): 2K rounds of a wave argmax; the winner is consumed
  for (int j = 0; j < K2; ++j) {
    float bv = -INFINITY, blp = 0.f;
    int bk = INT_MAX;
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
      if (ck[c] != INT_MAX && (better(cv[c], ck[c], bv, bk) || bk == INT_MAX)) { bv = cv[c]; bk = ck[c]; blp = clp[c]; }
    wave_best(bv, bk, blp);
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
      if (ck[c] == bk) ck[c] = INT_MAX;     // keys are unique: exactly one lane consumes it
    if (lane == 0) { sel_c[wave][j] = bv; sel_key[wave][j] = bk; sel_lp[wave][j] = blp; }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");

  const size_t R = (size_t)st.B * K;
  if (lane == 0) {
    const float lpn = powf((5.0f + (float)n) / 6.0f, st.alpha);
    int nk = 0;
    float nk_score[16];
    int nk_tok[16];
    float nk_lp[16];
    for (int j = 0; j < K2; ++j) {
      const int key = sel_key[wave][j];
      if (key == INT_MAX) continue;
      const float c = sel_c[wave][j];
      const int k = key / V, w = key - k * V;
      const int ppar = b * K + k;
      if (w == st.eos) {
        const float s = c / lpn;
        if (bf_nout < 0 || s > bf_score) {
          bf_score = s;
          bf_raw = c;
          bf_step = t - 1;
          bf_row = ppar;
          bf_nout = t;
        }
      } else if (nk < K) {
        nk_score[nk] = c;
        nk_tok[nk] = w;
        nk_lp[nk] = sel_lp[wave][j];
        nk_par[wave][nk] = ppar;
        ++nk;
      }
    }
    float mx = -INFINITY;
    for (int k = 0; k < K; ++k) {
      const int p = b * K + k;
      if (k < nk) {
        st.score[p] = nk_score[k];
        st.cur_tok[p] = nk_tok[k];
        st.tok_hist[(size_t)t * R + p] = nk_tok[k];
        st.par_hist[(size_t)t * R + p] = nk_par[wave][k];
        st.lp_hist[(size_t)t * R + p] = nk_lp[k];
        mx = fmaxf(mx, nk_score[k]);
      } else {
        st.score[p] = -INFINITY;
      }
    }
    int done = 0;
    if (n >= maxlen_b) {
      for (int k = 0; k < nk; ++k) {
        const float s = nk_score[k] / lpn;
        if (bf_nout < 0 || s > bf_score) {
          bf_score = s;
          bf_raw = nk_score[k];
          bf_step = t;
          bf_row = b * K + k;
          bf_nout = t + 1;
        }
      }
      done = 1;
    } else if (st.early_stop && bf_nout >= 0 && bf_score >= mx / lpn) {
      done = 1;
    } else if (nk == 0) {
      done = 1;
    }
    st.best_score[b] = bf_score;
    st.best_raw[b] = bf_raw;
    st.best_step[b] = bf_step;
    st.best_row[b] = bf_row;
    st.best_nout[b] = bf_nout;
    st.done[b] = done;
    nk_cnt[wave] = done ? 0 : nk;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  // ancestor table of the new beam: slot s < t lives where the parent's slot s lives;
  // slot t is the parent's own row (written this step)
  // (k, s) pairs spread over the lanes; each lane's reads are issued together
  const int nk = nk_cnt[wave], n_pairs = nk * (t + 1);
  constexpr int AB = 4;
  for (int i0 = lane; i0 < n_pairs; i0 += kWave * AB) {
    int val[AB];
#pragma unroll
    for (int u = 0; u < AB; ++u) {
      const int i = i0 + u * kWave;
      const int k = i / (t + 1), s = i - k * (t + 1);
      val[u] = 0;
      if (i < n_pairs) val[u] = s < t ? anc_cur[(size_t)nk_par[wave][k] * st.Tcap + s] : nk_par[wave][k];
    }
#pragma unroll
    for (int u = 0; u < AB; ++u) {
      const int i = i0 + u * kWave;
      const int k = i / (t + 1), s = i - k * (t + 1);
      if (i < n_pairs) anc_next[(size_t)(b * K + k) * st.Tcap + s] = val[u];
    }
  }
}

// ---- end of step: order-preserving in-place filter of the live list ----------------------
// Every entry of a 1024-chunk is read before the chunk's first barrier and written after
// it, at a position no larger than its own, so the filter can run in place.
__global__ __launch_bounds__(1024) void step_end_kernel(int* __restrict__ list, const int* __restrict__ done,
                                                        int* __restrict__ ctl, int* __restrict__ host_ctl,
                                                        int prune, int beam, int Tcap) {
  __shared__ int wsum[1024 / kWave];
  __shared__ int base;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int n = ctl[CTL_NLIVE], t = ctl[CTL_T];
  if (n == 0) return;                                // nothing was live: the step did nothing
  if (tid == 0) base = 0;
  __syncthreads();
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int i = c0 + tid;
    const int b = i < n ? list[i] : 0;
    const int keep = (i < n && !done[b]) ? 1 : 0;
    int x = keep;                                    // inclusive wave scan
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int y = __shfl_up(x, o, kWave);
      if (lane >= o) x += y;
    }
    if (lane == kWave - 1) wsum[wave] = x;
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += wsum[w];
    if (prune && keep) list[off + x - 1] = b;
    __syncthreads();
    if (tid == 0) {
      int tot = 0;
      for (int w = 0; w < 1024 / kWave; ++w) tot += wsum[w];
      base += tot;
    }
    __syncthreads();
  }
  if (tid == 0) {
    const int alive = base;
    int c[CTL_WORDS];
    c[CTL_T] = t + 1;
    // every sentence stops by its length limit (<= Tcap); the second test only guarantees
    // that no step can ever write a cache slot >= Tcap
    c[CTL_NLIVE] = (alive == 0 || t + 1 >= Tcap) ? 0 : (prune ? alive : n);
    c[CTL_NALIVE] = alive;
    c[CTL_ANC] = beam > 1 ? ctl[CTL_ANC] ^ 1 : 0;
#pragma unroll
    for (int j = 0; j < CTL_WORDS; ++j) ctl[j] = c[j];
    if (host_ctl) {
      // the mirror slot of step t, in pinned host memory, for the host to read once the step is done
#pragma unroll
      for (int j = 0; j < CTL_WORDS; ++j) host_ctl[(t % CTL_MIRROR_SLOTS) * CTL_WORDS + j] = c[j];
    }
  }
}

__global__ void finalize_kernel(SearchState st, int* __restrict__ out_tok, float* __restrict__ out_lp,
                                int* __restrict__ out_len, float* __restrict__ out_score) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= st.B) return;
  const size_t R = (size_t)st.B * st.beam;
  const int n = st.best_nout[b];
  int s = st.best_step[b], p = st.best_row[b];
  for (int i = n - 1; i >= 0; --i, --s) {
    out_tok[(size_t)b * st.Tcap + i] = st.tok_hist[(size_t)s * R + p];
    out_lp[(size_t)b * st.Tcap + i] = st.lp_hist[(size_t)s * R + p];
    if (st.beam > 1) p = st.par_hist[(size_t)s * R + p];
  }
  out_len[b] = n < 0 ? 0 : n;
  out_score[b] = st.best_score[b];
}

__global__ void init_kernel(SearchState st, int* __restrict__ list, int* __restrict__ ctl, int bos) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int R = st.B * st.beam;
  if (i == 0) {
    ctl[CTL_T] = 0;
    ctl[CTL_NLIVE] = st.B;
    ctl[CTL_NALIVE] = st.B;
    ctl[CTL_ANC] = 0;
  }
  if (i < R) {
    st.score[i] = (i % st.beam == 0) ? 0.f : -INFINITY;
    st.cur_tok[i] = bos;
  }
  if (i < st.B) {
    st.done[i] = 0;
    st.best_score[i] = -INFINITY;
    st.best_raw[i] = -INFINITY;
    st.best_step[i] = -1;
    st.best_row[i] = -1;
    st.best_nout[i] = -1;
    list[i] = i;
  }
}

__global__ void scatter_logits_kernel(const float* __restrict__ src, const int* __restrict__ sent_list,
                                      const int* __restrict__ ctl, int beam, int V, float* __restrict__ dst) {
  const int r = blockIdx.y;
  if (r >= ctl[CTL_NLIVE] * beam) return;
  const int p = sent_list[r / beam] * beam + r % beam;
  for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x)
    dst[(size_t)p * V + v] = src[(size_t)r * V + v];
}

}  // namespace

hipError_t greedy_step(const float* logits, const int* forced, const SearchState& st, hipStream_t s) {
  const int rows = st.B * st.beam;
  if (rows <= 0) return hipSuccess;
  NT_LAUNCH(greedy_kernel, dim3(rows), dim3(SEL_THREADS), 0, s, logits, forced, st);
  return hipGetLastError();
}

hipError_t ens_combine(const float* logits, float* comb, const int* ctl, int beam, int rows, int V, int member,
                       int n_members, int rule, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (member < 0 || member >= n_members || (rule != 0 && rule != 1)) return hipErrorInvalidValue;
  NT_LAUNCH(ens_combine_kernel, dim3(rows), dim3(SEL_THREADS), 0, s, logits, comb, ctl, beam, V, member, n_members,
            rule);
  return hipGetLastError();
}

hipError_t greedy_step_fused(const float* part, int n_tiles, const SearchState& st, hipStream_t s) {
  const int rows = st.B * st.beam;
  if (rows <= 0) return hipSuccess;
  NT_LAUNCH(greedy_fused_kernel, dim3(rows), dim3(SEL_THREADS), 0, s, part, n_tiles, st);
  return hipGetLastError();
}

hipError_t beam_select(const float* logits, const int* ctl, int beam, int rows, int V, int k2, float* topv, int* topi,
                       float* lse, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const bool reg = (V % 4) == 0 && V <= SEL_THREADS * 4 * SEL_REG && (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  if (reg && k2 <= 8) {
    if (k2 <= 4) NT_LAUNCH(beam_select_reg_kernel<4>, dim3(rows), dim3(SEL_THREADS), 0, s, logits, ctl, beam, V, k2,
                           topv, topi, lse);
    else NT_LAUNCH(beam_select_reg_kernel<8>, dim3(rows), dim3(SEL_THREADS), 0, s, logits, ctl, beam, V, k2, topv,
                   topi, lse);
    return hipGetLastError();
  }
#define NT_SEL(K2)                                                                                          \
  NT_LAUNCH(beam_select_kernel<K2>, dim3(rows), dim3(SEL_THREADS), 0, s, logits, ctl, beam, V, k2, topv, \
                     topi, lse)
  if (k2 <= 4) NT_SEL(4);
  else if (k2 <= 8) NT_SEL(8);
  else if (k2 <= 16) NT_SEL(16);
  else if (k2 <= 32) NT_SEL(32);
  else return hipErrorInvalidValue;
#undef NT_SEL
  return hipGetLastError();
}

hipError_t beam_select_tiles(const float* part, int n_tiles, const float* logits, const int* ctl, int beam, int rows,
                             int V, int k2, float* topv, int* topi, float* lse, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (n_tiles != (V + TILE_COLS - 1) / TILE_COLS || n_tiles > SEL_TPL * kWave || k2 < 1 || k2 > 32 || k2 > V)
    return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
#define NT_SEL(K2) \
  NT_LAUNCH(beam_select_tiles_kernel<K2>, grid, dim3(256), 0, s, part, n_tiles, logits, ctl, beam, rows, V, k2, topv, topi, lse)
  if (k2 <= 4) NT_SEL(4);
  else if (k2 <= 8) NT_SEL(8);
  else if (k2 <= 16) NT_SEL(16);
  else NT_SEL(32);
#undef NT_SEL
  return hipGetLastError();
}

hipError_t beam_pick_tiles(const float* part, int n_tiles, const int* ctl, int beam, int rows, int k2, int* ptile,
                           float* tau, float* lse, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (n_tiles < 1 || n_tiles > SEL_TPL * kWave || k2 < 1 || k2 > 32) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
  if (n_tiles <= 4 * kWave)
    NT_LAUNCH(beam_pick_tiles_kernel<4>, grid, dim3(256), 0, s, part, n_tiles, ctl, beam, rows, k2, ptile, tau, lse);
  else
    NT_LAUNCH(beam_pick_tiles_kernel<SEL_TPL>, grid, dim3(256), 0, s, part, n_tiles, ctl, beam, rows, k2, ptile, tau,
              lse);
  return hipGetLastError();
}

hipError_t pair_bucket(const int* ptile, const int* ctl, int beam, int rows, int k2, int n_tiles, int* sorted,
                       int* gblk, int* gnblk, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (n_tiles < 1 || n_tiles > 512 || k2 < 1 || k2 > 32) return hipErrorInvalidValue;
  NT_LAUNCH(pair_bucket_kernel, dim3(1), dim3(BUCKET_THREADS), 0, s, ptile, ctl, beam, rows, k2, n_tiles, sorted,
            gblk, gnblk);
  return hipGetLastError();
}

hipError_t beam_select_pairs(const float* logp, const int* ptile, const float* tau, const int* ctl, int beam,
                             int rows, int V, int k2, float* topv, int* topi, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (k2 < 1 || k2 > 32) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
#define NT_SEL(K2) \
  NT_LAUNCH(beam_select_pairs_kernel<K2>, grid, dim3(256), 0, s, logp, ptile, tau, ctl, beam, rows, V, k2, topv, topi)
  if (k2 <= 4) NT_SEL(4);
  else if (k2 <= 8) NT_SEL(8);
  else if (k2 <= 16) NT_SEL(16);
  else NT_SEL(32);
#undef NT_SEL
  return hipGetLastError();
}

// ---- records of the allocation-free tiled selection ----------------------------------------
// A file-scope device array stands in for the per-call records buffer of the tiled
// selection, for callers that cannot allocate device memory.  Every GPU holds its own
// copy until the process ends.  In host code the array's name is not a device address:
// each device's copy is located once, with that device current, by hipGetSymbolAddress,
// and only that address is handed to kernels.
constexpr size_t SCRATCH_FLOATS = (size_t)SELECT_NOALLOC_MAX_RECORDS * 4;   // 4 floats a record
static __device__ __align__(256) float scratch[SCRATCH_FLOATS];

hipError_t select_scratch(float** out, size_t* records) {
  static std::mutex mu;
  static std::vector<float*> per_device;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  if ((size_t)dev >= per_device.size()) per_device.resize(dev + 1, nullptr);
  if (!per_device[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    per_device[dev] = static_cast<float*>(p);
  }
  *out = per_device[dev];
  if (records) *records = SCRATCH_FLOATS / 4;
  return hipSuccess;
}

hipError_t tile_records(const float* logits, int rows, int V, float* part, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int n_tiles = (V + TILE_COLS - 1) / TILE_COLS;
  const long long tasks = (long long)rows * n_tiles;
  NT_LAUNCH(tile_records_kernel, dim3((unsigned)((tasks + 3) / 4)), dim3(256), 0, s, logits, rows, V, n_tiles, part);
  return hipGetLastError();
}

hipError_t beam_update(const float* topv, const int* topi, const float* lse, const SearchState& st, hipStream_t s) {
  if (st.B <= 0) return hipSuccess;
  if (st.beam * 2 * st.beam > MAXC * kWave || st.beam > 16) return hipErrorInvalidValue;
  NT_LAUNCH(beam_update_kernel, dim3((st.B + 3) / 4), dim3(256), 0, s, topv, topi, lse, st);
  return hipGetLastError();
}

hipError_t step_end(int* list, const int* done, int* ctl, int* host_ctl, int prune, int beam, int Tcap,
                    hipStream_t s) {
  NT_LAUNCH(step_end_kernel, dim3(1), dim3(1024), 0, s, list, done, ctl, host_ctl, prune, beam, Tcap);
  return hipGetLastError();
}

hipError_t finalize(const SearchState& st, int* out_tok, float* out_lp, int* out_len, float* out_score,
                    hipStream_t s) {
  NT_LAUNCH(finalize_kernel, dim3((st.B + 127) / 128), dim3(128), 0, s, st, out_tok, out_lp, out_len,
                     out_score);
  return hipGetLastError();
}

hipError_t search_init(const SearchState& st, int* list, int* ctl, int bos, hipStream_t s) {
  const int n = st.B * st.beam;
  NT_LAUNCH(init_kernel, dim3((n + 255) / 256), dim3(256), 0, s, st, list, ctl, bos);
  return hipGetLastError();
}

hipError_t scatter_logits(const float* logits, const int* sent_list, const int* ctl, int beam, int rows, int V,
                          float* dst, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  NT_LAUNCH(scatter_logits_kernel, dim3((V + 255) / 256 < 64 ? (V + 255) / 256 : 64, rows), dim3(256), 0,
                     s, logits, sent_list, ctl, beam, V, dst);
  return hipGetLastError();
}

}  // namespace nt
