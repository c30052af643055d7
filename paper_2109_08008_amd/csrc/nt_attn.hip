// Attention kernels for gfx950.
//
// attn_mfma_kernel: groups of queries that share one set of keys, on the matrix cores --
// encoder self-attention (a group is a sentence and its tokens are the queries) and the
// decoder's encoder-decoder attention (a group is a live sentence and its beam rows are
// the queries; the sentence's cross keys/values, computed once per batch, are read once
// for all of its hypotheses, Sec. 4.1 "Caching").  Keys past the group's length are
// masked (padding is inert).
//
// self_attn_kernel: one wave per (live row, head) attends over the row's cached
// self-attention slots 0..t; with beam search a slot may live in the row of an
// ancestor hypothesis (anc table), so beams never copy caches when they reorder.  With
// a single query per row this is a streaming kernel, not a contraction, so it stays on
// the vector units.
#include <type_traits>

#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

// Grouped attention on the matrix cores: one wave per (group, head, block of 16 queries).
// Scores are formed transposed, S^T = K.Q^T, so lane l holds the scores of query l%16
// for keys 4*(l/16)+r of each 16-key block; those are exactly the key slots the lane
// supplies as the A operand of the P.V product (an MFMA only needs its two operands to
// agree on which k each lane element carries), so P never leaves registers.  Values are
// staged through a per-wave LDS tile and read key-major for the B operand.  Softmax is
// exact within chunks of 128 keys (64 in the decoder; scores kept in registers) with an
// online rescale between chunks; exponentials and sums are fp32, P enters P.V in the
// model dtype.  Keys past the group's length get -inf scores (their value rows are
// clamped to a valid one).
//
// RPR (relative positions, self-attention): before the keys, the wave forms
// qa[i][m] = q_i . table_k[m] for its 16 queries in fp32, and each score gains
// qa[i][clip(j - i) + k] before the scale.  The value rows' share,
// sum_j p_ij table_v[clip(j - i) + k], is sum_m B_i[m] table_v[m] with B_i[m] the
// probability mass of query i at relative row m: per chunk the probabilities go through
// LDS and each (query, row) pair sums its keys in increasing order (rows inside the
// clip have one key, the two edge rows every key beyond it); B is rescaled with O.
constexpr int RPR_MAX = 33;     // 2k+1 for k <= 16
template <typename T, int DH, int ROLE, bool RPR>
__global__ __launch_bounds__(256) void attn_mfma_kernel(MhaArgs a) {
  constexpr int EB = sizeof(T);
  constexpr int FE = 16 / EB;            // elements per 16-byte fragment
  constexpr int KSTEP = 4 * FE;          // reduction length of one MFMA step (32 or 16)
  constexpr int QK = DH / KSTEP;         // steps over the head dimension
  constexpr int SB = KSTEP / 16;         // 16-key score blocks per P.V step
  constexpr int CB = DH / 16;            // 16-channel output blocks
  // score blocks per softmax chunk: 128 keys for the encoder; 64 for the decoder's
  // cross-attention, whose 16-query blocks carry only the beam's rows (112 VGPRs at fp16
  // d_head 64 against 144, four waves a SIMD against three; 0.8% faster on base-6-6)
  constexpr int NSB = ROLE == 1 ? 4 : 8;
  constexpr int ROWP = DH * EB / 16;     // 16-byte pieces per key row
  constexpr int VSTR = DH * EB / 4 + (EB == 2 ? 2 : 4);   // LDS row stride (dwords), spreads banks
  constexpr int VPL = KSTEP * ROWP / kWave;   // 16-byte value pieces per lane per P.V step
  static_assert(DH % KSTEP == 0 && NSB % SB == 0, "head dim must fill whole MFMA steps");
  static_assert(KSTEP * ROWP % kWave == 0, "value rows of a P.V step split evenly over the lanes");
  constexpr bool KALL = ROLE == 1;   // the chunk's key blocks all loaded before its scores
  __shared__ __attribute__((aligned(16))) unsigned Vs[4][KSTEP][VSTR];
  constexpr int RW = RPR ? 4 : 1;   // per-wave RPR buffers (1 placeholder when unused)
  constexpr int RQ = RPR ? 16 : 1;
  __shared__ float rp_qa[RW][RQ][RPR ? RPR_MAX : 1];        // q_i . table_k[m]
  __shared__ float rp_p[RW][RQ][RPR ? NSB * 16 : 1];        // this chunk's probabilities
  __shared__ float rp_b[RW][RQ][RPR ? RPR_MAX : 1];         // B_i[m]
  __shared__ float rp_alpha[RW][RQ];

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int grp = lane >> 4, ln = lane & 15;
  // every argument of the common path named at entry: their scalar-cache misses overlap
  asm volatile("" ::"s"(a.q), "s"(a.q_ld), "s"(a.k), "s"(a.v), "s"(a.kb), "s"(a.kh), "s"(a.ks), "s"(a.out),
               "s"(a.out_ld), "s"(a.group_map), "s"(a.lens), "s"(a.q_per_group), "s"(a.self_queries),
               "s"(a.n_groups), "s"(a.H), "s"(a.scale), "s"(a.ctl));
  const int qblocks = (a.q_per_group + 15) / 16;
  const int task = blockIdx.x * 4 + wave;
  if (task >= a.n_groups * a.H * qblocks) return;   // grid tail
  const int qb = task % qblocks, gh = task / qblocks;
  const int h = gh % a.H, g = gh / a.H;
  // the group's entry (valid for every group of the grid) and the live count together
  const int b = a.group_map ? a.group_map[g] : g;
  const int nlive = a.ctl ? a.ctl[CTL_NLIVE] : a.n_groups;
  asm volatile("" ::"v"(b), "s"(nlive));
  if (g >= min(a.n_groups, nlive)) return;   // whole wave; wave-local sync only below
  const int len = a.lens[b];
  const int nq = a.self_queries ? min(len, a.q_per_group) : a.q_per_group;
  const int q0 = qb * 16;
  T* out = static_cast<T*>(a.out);
  auto out_at = [&](int i, int ch) -> T* { return out + (size_t)(g * a.q_per_group + i) * a.out_ld + h * DH + ch; };

  if (q0 >= nq) {                                  // a block of padding queries: zero rows
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = q0 + 4 * grp + r;
      if (i < a.q_per_group)
#pragma unroll
        for (int c = 0; c < CB; ++c) *out_at(i, c * 16 + ln) = from_f32<T>(0.f);
    }
    return;
  }

  const size_t ks_b = (size_t)a.ks * EB;
  const char* Kb = reinterpret_cast<const char*>(static_cast<const T*>(a.k) + (size_t)b * a.kb + (size_t)h * a.kh);
  const char* Vb = reinterpret_cast<const char*>(static_cast<const T*>(a.v) + (size_t)b * a.kb + (size_t)h * a.kh);
  const char* qrow = reinterpret_cast<const char*>(static_cast<const T*>(a.q) +
                                                   (size_t)(g * a.q_per_group + min(q0 + ln, nq - 1)) * a.q_ld +
                                                   h * DH);
  u32x4 qf[QK];
#pragma unroll
  for (int st = 0; st < QK; ++st) qf[st] = *reinterpret_cast<const u32x4*>(qrow + st * 64 + grp * 16);

  const int RT = RPR ? 2 * a.rel_k + 1 : 0;
  constexpr int RITEMS = RPR ? (16 * RPR_MAX + kWave - 1) / kWave : 1;   // (query, row) pairs per lane
  float bacc[RITEMS];
  if constexpr (RPR) {
    // qa[i][m] = q_{q0+i} . table_k[m] over the full head, one pair per lane at a time
    for (int it = lane; it < 16 * RT; it += kWave) {
      const int i = it / RT, m = it - i * RT;
      const T* qr = static_cast<const T*>(a.q) + (size_t)(g * a.q_per_group + min(q0 + i, nq - 1)) * a.q_ld + h * DH;
      const float* tk = a.relk + (size_t)m * DH;
      float dot = 0.f;
#pragma unroll 8
      for (int e = 0; e < DH; ++e) dot += to_f32(qr[e]) * tk[e];
      rp_qa[wave][i][m] = dot;
    }
#pragma unroll
    for (int t2 = 0; t2 < RITEMS; ++t2) bacc[t2] = 0.f;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  }

  float m = -INFINITY, lsum = 0.f;   // running max / sum of query q0+ln (same in all 4 groups)
  floatx4 o[CB];                     // O[q0 + 4*grp + r][c*16 + ln]
#pragma unroll
  for (int c = 0; c < CB; ++c) o[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  const unsigned short* vh = reinterpret_cast<const unsigned short*>(&Vs[wave][0][0]);

  // value rows key0 .. key0 + KSTEP - 1 of this head (rows past len clamped) into registers
  auto load_v = [&](int key0, u32x4 (&dst)[VPL]) {
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
      const int pc = lane + u * kWave, row = pc / ROWP, col = pc % ROWP;
      dst[u] = *reinterpret_cast<const u32x4*>(Vb + (size_t)min(key0 + row, len - 1) * ks_b + col * 16);
    }
  };

  for (int c0 = 0; c0 < len; c0 += NSB * 16) {
    const int nb = min(NSB, (len - c0 + 15) / 16);
    // the chunk's first P.V values are fetched now, so their latency overlaps the scores
    u32x4 vcur[VPL];
    load_v(c0, vcur);
    floatx4 sc[NSB];
    float cmax = -INFINITY;
    // decoder: every key block of the chunk is fetched before the first score, so the
    // blocks' loads are in flight together (rows past len re-read the last key, and
    // their scores are masked below)
    u32x4 kf[KALL ? NSB : 1][KALL ? QK : 1];
    if constexpr (KALL) {
#pragma unroll
      for (int kb = 0; kb < NSB; ++kb) {
        const char* krow = Kb + (size_t)min(c0 + kb * 16 + ln, len - 1) * ks_b;
#pragma unroll
        for (int st = 0; st < QK; ++st) kf[kb][st] = *reinterpret_cast<const u32x4*>(krow + st * 64 + grp * 16);
      }
      __builtin_amdgcn_sched_barrier(0);   // the value and key loads all issue before the scores
    }
#pragma unroll
    for (int kb = 0; kb < NSB; ++kb) {
      sc[kb] = floatx4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      if (KALL || kb < nb) {
        const char* krow = Kb + (size_t)min(c0 + kb * 16 + ln, len - 1) * ks_b;
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < QK; ++st)
          acc = Mfma<T>::step(KALL ? kf[kb % (KALL ? NSB : 1)][st % (KALL ? QK : 1)]
                                   : *reinterpret_cast<const u32x4*>(krow + st * 64 + grp * 16),
                              qf[st], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = c0 + kb * 16 + 4 * grp + r;
          float raw = acc[r];
          if constexpr (RPR) raw += rp_qa[wave][ln][min(max(key - (q0 + ln), -a.rel_k), a.rel_k) + a.rel_k];
          sc[kb][r] = key < len ? raw * a.scale : -INFINITY;
          cmax = fmaxf(cmax, sc[kb][r]);
        }
      }
    }
    cmax = fmaxf(cmax, __shfl_xor(cmax, 16, kWave));
    cmax = fmaxf(cmax, __shfl_xor(cmax, 32, kWave));
    const float mn = fmaxf(m, cmax);
    const float alpha = __expf(m - mn);              // 0 on the first chunk
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NSB; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc[kb][r] = __expf(sc[kb][r] - mn);
        psum += sc[kb][r];
      }
    psum += __shfl_xor(psum, 16, kWave);
    psum += __shfl_xor(psum, 32, kWave);
    lsum = lsum * alpha + psum;
    m = mn;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ar = __shfl(alpha, 4 * grp + r, kWave);   // alpha of query q0 + 4*grp + r
#pragma unroll
      for (int c = 0; c < CB; ++c) o[c][r] *= ar;
    }
    if constexpr (RPR) {
      // this chunk's probability mass of every (query, relative row) pair
#pragma unroll
      for (int kb = 0; kb < NSB; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) rp_p[wave][ln][kb * 16 + 4 * grp + r] = sc[kb][r];
      if (grp == 0) rp_alpha[wave][ln] = alpha;
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
#pragma unroll
      for (int t2 = 0; t2 < RITEMS; ++t2) {
        const int it = lane + t2 * kWave;
        if (it >= 16 * RT) continue;
        const int i = it / RT, rel = it - i * RT - a.rel_k;
        const int jq = q0 + i - c0;                 // the query's own position in chunk coordinates
        int lo, hi;                                 // chunk keys of this row: [lo, hi)
        if (rel == -a.rel_k) { lo = 0; hi = jq - a.rel_k + 1; }
        else if (rel == a.rel_k) { lo = jq + a.rel_k; hi = NSB * 16; }
        else { lo = jq + rel; hi = lo + 1; }
        lo = max(lo, 0);
        hi = min(hi, NSB * 16);
        float sum = 0.f;
        for (int j = lo; j < hi; ++j) sum += rp_p[wave][i][j];
        bacc[t2] = bacc[t2] * rp_alpha[wave][i] + sum;
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    }

    for (int kb = 0; kb < nb; kb += SB) {
      // the next step's values are fetched while this step's go through LDS (8-byte
      // writes) into the P.V product
      const bool more = kb + SB < nb;
      u32x4 vnext[VPL];
      if (more) load_v(c0 + (kb + SB) * 16, vnext);
#pragma unroll
      for (int u = 0; u < VPL; ++u) {
        const int pc = lane + u * kWave, row = pc / ROWP, col = pc % ROWP;
        unsigned* dst = &Vs[wave][row][col * 4];
        *reinterpret_cast<uint2*>(dst) = make_uint2(vcur[u].x, vcur[u].y);
        *reinterpret_cast<uint2*>(dst + 2) = make_uint2(vcur[u].z, vcur[u].w);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      // A operand: P of query ln at keys 16*(kb+j) + 4*grp + r, in the model dtype
      u32x4 pf;
      if constexpr (EB == 2) {
        T pe[8];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) pe[4 * j + r] = from_f32<T>(sc[kb + j][r]);
        pf = __builtin_bit_cast(u32x4, pe);
      } else {
        pf = __builtin_bit_cast(u32x4, sc[kb]);
      }
#pragma unroll
      for (int c = 0; c < CB; ++c) {
        // B operand: V[key 16*j + 4*grp + r][channel c*16 + ln], same key order as pf
        u32x4 vf;
        if constexpr (EB == 2) {
          unsigned short e[8];
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) e[4 * j + r] = vh[(16 * j + 4 * grp + r) * (VSTR * 2) + c * 16 + ln];
          vf = __builtin_bit_cast(u32x4, e);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) vf[r] = Vs[wave][4 * grp + r][c * 16 + ln];
        }
        o[c] = Mfma<T>::step(pf, vf, o[c]);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      if (more) {
#pragma unroll
        for (int u = 0; u < VPL; ++u) vcur[u] = vnext[u];
      }
    }
  }

  if constexpr (RPR) {
    // the value tables' share: O[i][ch] += sum_m B_i[m] table_v[m][ch]
#pragma unroll
    for (int t2 = 0; t2 < RITEMS; ++t2) {
      const int it = lane + t2 * kWave;
      if (it < 16 * RT) rp_b[wave][it / RT][it % RT] = bacc[t2];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    for (int m = 0; m < RT; ++m) {
      const float* tv = a.relv + (size_t)m * DH;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float bm = rp_b[wave][4 * grp + r][m];
#pragma unroll
        for (int c = 0; c < CB; ++c) o[c][r] += bm * tv[c * 16 + ln];
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = q0 + 4 * grp + r;
    const float inv = 1.0f / __shfl(lsum, 4 * grp + r, kWave);
    if (i >= a.q_per_group) continue;
#pragma unroll
    for (int c = 0; c < CB; ++c) *out_at(i, c * 16 + ln) = from_f32<T>(i < nq ? o[c][r] * inv : 0.f);
  }
}

// Decoder self-attention: one wave per (live row, head) over the row's cached slots
// 0..t.  Slot s of a beam hypothesis lives in the physical row of its ancestor at step s
// (anc), so reordering beams never copies the cache.
//
// With one query this is a stream over the cache, kept on the vector units and laid out
// for coalescing: the CPR = 16-byte chunks of a key's row sit on CPR consecutive lanes,
// so one load instruction of the wave reads whole rows (8 keys of 128 bytes at d_head
// 64).  Each lane carries KPL = 4 keys of a chunk of GPW * KPL keys (lane group g holds
// keys g*KPL .. g*KPL+3).  A key's score is its lanes' partial dot products summed by a
// butterfly inside the group; P.V accumulates per lane over its keys for its 16-byte
// slice of channels and is summed over the lane groups once, after the last chunk.  The
// softmax is online across chunks, in fp32.  No LDS, so occupancy is set by registers:
// four keys a lane (80 VGPRs at fp16, six waves a SIMD) measured 4% faster on base-6-6
// than eight (91 VGPRs, five waves), and two (66 VGPRs) no faster than four.
//
// KV is the cache's element type: the model dtype, or E4M3 bytes (uint8_t) in FP8 mode,
// where a 16-byte chunk carries 16 channels (64-byte keys at d_head 64 on 4 lanes), the
// query and the output stay fp16, and the codes are widened exactly (through fp16).
template <typename KV> struct KvChunk {
  static __device__ __forceinline__ void get(const uint4& r, float* out) {
    const KV* e = reinterpret_cast<const KV*>(&r);
#pragma unroll
    for (int i = 0; i < 16 / (int)sizeof(KV); ++i) out[i] = to_f32(e[i]);
  }
};
template <> struct KvChunk<uint8_t> {
  static __device__ __forceinline__ void get(const uint4& r, float* out) {
    const unsigned w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w[i], 1.0f, false);   // bytes 0, 1
      const auto hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w[i], 1.0f, true);    // bytes 2, 3
      out[4 * i] = (float)lo[0];
      out[4 * i + 1] = (float)lo[1];
      out[4 * i + 2] = (float)hi[0];
      out[4 * i + 3] = (float)hi[1];
    }
  }
};
template <typename T, int DH, typename KV>
__global__ __launch_bounds__(256) void self_attn_kernel(SelfAttnArgs a) {
  // KPL keys a lane: 4 of 2-byte (or wider) elements, 2 of E4M3 bytes -- the same 128 bytes
  // of keys and values in flight per lane and 32 keys per wave (118 VGPRs with 4 E4M3 keys)
  constexpr int VEC = 16 / (int)sizeof(KV), CPR = DH / VEC, GPW = kWave / CPR;
  constexpr int KPL = sizeof(KV) == 1 ? 2 : 4, KCH = GPW * KPL;
  static_assert(CPR >= 1 && CPR <= kWave && (CPR & (CPR - 1)) == 0, "a key's chunks fit in a wave");
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  // every argument the wave uses, named at entry: their scalar-cache misses overlap
  asm volatile("" ::"s"(a.q), "s"(a.kcache), "s"(a.vcache), "s"(a.sent_list), "s"(a.beam), "s"(a.anc),
               "s"(a.anc_stride), "s"(a.out), "s"(a.rows), "s"(a.H), "s"(a.Tcap), "s"(a.scale), "s"(a.ctl));
  const int pair = blockIdx.x * 4 + wave;
  if (pair >= a.rows * a.H) return;            // grid tail
  const int row = pair / a.H, h = pair % a.H;
  const int c = lane % CPR, g = lane / CPR;    // channel chunk and key group of this lane
  // The list entry, the query and the step counters are read together (every row of the
  // grid is allocated and its list entry names a valid sentence); only the cache stream
  // waits for the live-row check.
  const int sent = a.sent_list[row / a.beam];
  float q[VEC];
  load_row<T, VEC>(static_cast<const T*>(a.q) + (size_t)row * a.H * DH + h * DH + c * VEC, q);
  const int nlive = a.ctl[CTL_NLIVE], t = a.ctl[CTL_T], asel = a.ctl[CTL_ANC];
  asm volatile("" ::"v"(sent), "s"(nlive), "s"(t), "s"(asel));
  if (row >= min(a.rows, nlive * a.beam)) return;   // whole wave exits; no block barrier below
  const int p = sent * a.beam + row % a.beam;
#pragma unroll
  for (int x = 0; x < VEC; ++x) q[x] *= a.scale;
  const int n = t + 1;
  const int* anc = a.anc ? a.anc + (size_t)asel * a.anc_stride + (size_t)p * a.Tcap : nullptr;
  const size_t head = (size_t)h * a.Tcap * DH + c * VEC;
  const KV* K = static_cast<const KV*>(a.kcache) + head;
  const KV* Vc = static_cast<const KV*>(a.vcache) + head;
  const size_t row_stride = (size_t)a.H * a.Tcap * DH;
  float m = -INFINITY, lsum = 0.f, o[VEC];
#pragma unroll
  for (int x = 0; x < VEC; ++x) o[x] = 0.f;
  // the physical row of each of the lane's slots of a chunk (slot t was just written by
  // this row; slots past the end re-read the last one, their scores are masked)
  int ph[KPL];
  auto anc_rows = [&](int c0) {
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const int s = min(c0 + g * KPL + j, t);
      ph[j] = (anc && s < t) ? anc[s] : p;
    }
  };
  anc_rows(0);
  for (int c0 = 0; c0 < n; c0 += KCH) {
    // all key/value loads with no branch between them, then the next chunk's ancestor
    // rows, in flight with them: one dependent round trip per chunk
    uint4 kr[KPL], vr[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const size_t off = (size_t)ph[j] * row_stride + (size_t)min(c0 + g * KPL + j, t) * DH;
      kr[j] = *reinterpret_cast<const uint4*>(K + off);
      vr[j] = *reinterpret_cast<const uint4*>(Vc + off);
    }
    if (anc && c0 + KCH < n) anc_rows(c0 + KCH);
    float sc[KPL], cmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      float ke[VEC];
      KvChunk<KV>::get(kr[j], ke);
      float dot = 0.f;
#pragma unroll
      for (int x = 0; x < VEC; ++x) dot += q[x] * ke[x];
      if constexpr (CPR <= 16) {
        dot = group_sum<CPR>(dot);
      } else {
        dot = group_sum<16>(dot);
        dot += __shfl_xor(dot, 16, kWave);
      }
      sc[j] = c0 + g * KPL + j < n ? dot : -INFINITY;
      cmax = fmaxf(cmax, sc[j]);
    }
    const float mn = fmaxf(m, wave_max(cmax));   // finite: slot 0 is in the first chunk
    const float alpha = __expf(m - mn);
    float ps = 0.f;
#pragma unroll
    for (int x = 0; x < VEC; ++x) o[x] *= alpha;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const float pj = __expf(sc[j] - mn);
      float ve[VEC];
      KvChunk<KV>::get(vr[j], ve);
      ps += pj;
#pragma unroll
      for (int x = 0; x < VEC; ++x) o[x] += pj * ve[x];
    }
    lsum = lsum * alpha + (c == 0 ? ps : 0.f);   // one lane per key group counts its keys
    m = mn;
  }
#pragma unroll
  for (int ofs = CPR; ofs < kWave; ofs <<= 1)
#pragma unroll
    for (int x = 0; x < VEC; ++x) o[x] += ofs == 8 ? dpp_mov<DPP_XOR8>(o[x]) : __shfl_xor(o[x], ofs, kWave);
  const float inv = 1.0f / wave_sum(lsum);
  if (g == 0) {
#pragma unroll
    for (int x = 0; x < VEC; ++x) o[x] *= inv;
    store_row<T, VEC>(static_cast<T*>(a.out) + (size_t)row * a.H * DH + h * DH + c * VEC, o);
  }
}

template <typename T, int ROLE, bool RPR>
hipError_t mha_launch(const MhaArgs& a, hipStream_t s) {
  const long long tasks = (long long)a.n_groups * a.H * ((a.q_per_group + 15) / 16);
  const dim3 grid((unsigned)((tasks + 3) / 4));
  switch (a.dh) {
    case 32: NT_LAUNCH((attn_mfma_kernel<T, 32, ROLE, RPR>), grid, dim3(256), 0, s, a); break;
    case 64: NT_LAUNCH((attn_mfma_kernel<T, 64, ROLE, RPR>), grid, dim3(256), 0, s, a); break;
    case 128: NT_LAUNCH((attn_mfma_kernel<T, 128, ROLE, RPR>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int ROLE>
hipError_t mha_t(const MhaArgs& a, hipStream_t s) {
  if (ROLE == 0 && a.rel_k > 0) {
    if (!a.relk || !a.relv || a.rel_k > (RPR_MAX - 1) / 2 || !a.self_queries) return hipErrorInvalidValue;
    return mha_launch<T, 0, true>(a, s);
  }
  return mha_launch<T, ROLE, false>(a, s);
}

template <typename T, int DH>
void self_launch(const SelfAttnArgs& a, hipStream_t s) {
  const dim3 grid((a.rows * a.H + 3) / 4);
  if constexpr (std::is_same<T, f16>::value) {
    if (a.kv_f8) {
      NT_LAUNCH((self_attn_kernel<T, DH, uint8_t>), grid, dim3(4 * kWave), 0, s, a);
      return;
    }
  }
  NT_LAUNCH((self_attn_kernel<T, DH, T>), grid, dim3(4 * kWave), 0, s, a);
}

template <typename T>
hipError_t self_t(const SelfAttnArgs& a, hipStream_t s) {
  switch (a.dh) {
    case 32: self_launch<T, 32>(a, s); break;
    case 64: self_launch<T, 64>(a, s); break;
    case 128: self_launch<T, 128>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t mha(DT dt, const MhaArgs& a, hipStream_t s, int role) {
  if (a.n_groups <= 0 || a.q_per_group <= 0) return hipSuccess;
  switch (dt) {
    case DT::F32: return role ? mha_t<float, 1>(a, s) : mha_t<float, 0>(a, s);
    case DT::F16: return role ? mha_t<f16, 1>(a, s) : mha_t<f16, 0>(a, s);
    case DT::BF16: return role ? mha_t<bf16, 1>(a, s) : mha_t<bf16, 0>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t self_attn(DT dt, const SelfAttnArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.kv_f8 && dt != DT::F16) return hipErrorInvalidValue;   // the FP8 cache pairs with fp16
  switch (dt) {
    case DT::F32: return self_t<float>(a, s);
    case DT::F16: return self_t<f16>(a, s);
    case DT::BF16: return self_t<bf16>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace nt
