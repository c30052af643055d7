// Attention kernels for gfx950.
//
// mha_kernel: groups of queries that share one set of keys -- encoder self-attention
// (a group is a sentence and its tokens are the queries) and the decoder's
// encoder-decoder attention (a group is a live sentence and its beam rows are the
// queries; the sentence's cross keys/values, computed once per batch, are read once per
// workgroup and shared by every hypothesis, Sec. 4.1 "Caching").  Keys stream through
// LDS in chunks of 64; each wave carries 8 queries with an online (running max / sum)
// fp32 softmax, so any key length works with a fixed LDS footprint.  Keys past the
// group's length are masked (padding is inert).
//
// cross_attn_kernel: the decoder's encoder-decoder attention with one wave per (live
// sentence, head); the sentence's beam rows are the wave's queries.
//
// self_attn_kernel: one wave per (live row, head) attends over the row's cached
// self-attention slots 0..t; with beam search a slot may live in the row of an
// ancestor hypothesis (anc table), so beams never copy caches when they reorder.
#include "nt_common.h"
#include "nt_kernels.h"

namespace nt {
namespace {

constexpr int QW = 8;        // queries per wave
constexpr int KC = 64;       // keys per chunk
constexpr int NW = 4;        // waves per workgroup

template <typename T, int DH, int ROLE>
__global__ __launch_bounds__(256) void mha_kernel(MhaArgs a) {
  constexpr int CPL = DH > 64 ? DH / 64 : 1;   // channels per lane in the P.V phase
  __shared__ float Ks[KC][DH + 1];
  __shared__ float Vs[KC][DH];
  __shared__ float Qs[NW * QW][DH];
  __shared__ float Ps[NW][KC][QW];

  const int qblocks = (a.q_per_group + NW * QW - 1) / (NW * QW);
  const int g = blockIdx.x / qblocks, qb = blockIdx.x % qblocks;
  const int h = blockIdx.y;
  const int b = a.group_map ? a.group_map[g] : g;
  const int len = a.lens[b];
  const int nq = a.self_queries ? min(len, a.q_per_group) : a.q_per_group;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;

  const T* Q = static_cast<const T*>(a.q);
  const T* Kp = static_cast<const T*>(a.k) + (size_t)b * a.kb + (size_t)h * a.kh;
  const T* Vp = static_cast<const T*>(a.v) + (size_t)b * a.kb + (size_t)h * a.kh;

  // queries of this workgroup -> LDS, pre-scaled by 1/sqrt(dh)
  for (int idx = tid; idx < NW * QW * DH; idx += 256) {
    const int qi = idx / DH, e = idx % DH;
    const int i = qb * NW * QW + qi;
    float v = 0.f;
    if (i < nq) v = to_f32(Q[(size_t)(g * a.q_per_group + i) * a.q_ld + h * DH + e]) * a.scale;
    Qs[qi][e] = v;
  }

  float m[QW], l[QW], o[QW][CPL];
#pragma unroll
  for (int j = 0; j < QW; ++j) {
    m[j] = -INFINITY;
    l[j] = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[j][c] = 0.f;
  }

  for (int c0 = 0; c0 < len; c0 += KC) {
    __syncthreads();
    for (int idx = tid; idx < KC * DH; idx += 256) {
      const int r = idx / DH, e = idx % DH;
      const int s = c0 + r;
      float kv = 0.f, vv = 0.f;
      if (s < len) {
        kv = to_f32(Kp[(size_t)s * a.ks + e]);
        vv = to_f32(Vp[(size_t)s * a.ks + e]);
      }
      Ks[r][e] = kv;
      Vs[r][e] = vv;
    }
    __syncthreads();

    // scores: lane = key
    const bool valid = c0 + lane < len;
    float sc[QW];
#pragma unroll
    for (int j = 0; j < QW; ++j) sc[j] = 0.f;
#pragma unroll 8
    for (int e = 0; e < DH; ++e) {
      const float kv = Ks[lane][e];
#pragma unroll
      for (int j = 0; j < QW; ++j) sc[j] += Qs[wave * QW + j][e] * kv;
    }
#pragma unroll
    for (int j = 0; j < QW; ++j) {
      const float s = valid ? sc[j] : -INFINITY;
      const float mn = fmaxf(m[j], wave_max(s));
      const float p = valid ? expf(s - mn) : 0.f;
      const float alpha = expf(m[j] - mn);
      l[j] = l[j] * alpha + wave_sum(p);
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[j][c] *= alpha;
      m[j] = mn;
      Ps[wave][lane][j] = p;
    }
    __syncthreads();

    // P.V: lane = channel
    const int kmax = min(KC, len - c0);
    for (int k = 0; k < kmax; ++k) {
      const float4 p0 = *reinterpret_cast<const float4*>(&Ps[wave][k][0]);
      const float4 p1 = *reinterpret_cast<const float4*>(&Ps[wave][k][4]);
      const float pk[QW] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int e = lane * CPL + c;
        const float v = e < DH ? Vs[k][e] : 0.f;
#pragma unroll
        for (int j = 0; j < QW; ++j) o[j][c] += pk[j] * v;
      }
    }
  }

  T* out = static_cast<T*>(a.out);
#pragma unroll
  for (int j = 0; j < QW; ++j) {
    const int i = qb * NW * QW + wave * QW + j;
    if (i >= a.q_per_group) continue;
    const size_t row = (size_t)(g * a.q_per_group + i) * a.out_ld + h * DH;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int e = lane * CPL + c;
      if (e < DH) out[row + e] = from_f32<T>(i < nq ? o[j][c] / l[j] : 0.f);
    }
  }
}

// One wave attends KQ queries (held in LDS, pre-scaled) over n keys, streaming the
// keys in chunks of 64 with an online fp32 softmax.  Lane s loads the key and value
// rows of key c0+s itself (16-byte loads, all in flight together); the value rows go
// to LDS so that the P.V product (lane = channel) reads them without waiting on HBM
// once per key.  row_of(s) maps a key index to the start of its key/value row.
template <typename T, int DH, int KQ, typename RowFn>
__device__ __forceinline__ void wave_attend(const float (&Qs)[KQ][DH], float (&Ps)[KQ][KC], T (&Vs)[KC][DH + 8],
                                            int n, const T* __restrict__ Kbase, const T* __restrict__ Vbase,
                                            RowFn row_of, float (&o)[KQ][DH > 64 ? DH / 64 : 1], float (&l)[KQ]) {
  constexpr int CPL = DH > 64 ? DH / 64 : 1;
  const int lane = threadIdx.x % kWave;
  float m[KQ];
#pragma unroll
  for (int i = 0; i < KQ; ++i) {
    m[i] = -INFINITY;
    l[i] = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[i][c] = 0.f;
  }
  for (int c0 = 0; c0 < n; c0 += KC) {
    const int s = c0 + lane;
    const bool valid = s < n;
    float sc[KQ];
#pragma unroll
    for (int i = 0; i < KQ; ++i) sc[i] = 0.f;
    if (valid) {
      const size_t r = row_of(s);
      const T* kr = Kbase + r;
      const T* vr = Vbase + r;
      uint4 kv[DH * sizeof(T) / 16], vv[DH * sizeof(T) / 16];
#pragma unroll
      for (int j = 0; j < DH * (int)sizeof(T) / 16; ++j) {
        kv[j] = reinterpret_cast<const uint4*>(kr)[j];
        vv[j] = reinterpret_cast<const uint4*>(vr)[j];
      }
#pragma unroll
      for (int j = 0; j < DH * (int)sizeof(T) / 16; ++j) *reinterpret_cast<uint4*>(&Vs[lane][j * Vec<T>::N]) = vv[j];
#pragma unroll
      for (int j = 0; j < DH * (int)sizeof(T) / 16; ++j) {
        const T* ke = reinterpret_cast<const T*>(&kv[j]);
#pragma unroll
        for (int x = 0; x < Vec<T>::N; ++x) {
          const float k = to_f32(ke[x]);
#pragma unroll
          for (int i = 0; i < KQ; ++i) sc[i] += Qs[i][j * Vec<T>::N + x] * k;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < KQ; ++i) {
      const float v = valid ? sc[i] : -INFINITY;
      const float mn = fmaxf(m[i], wave_max(v));
      const float p = valid ? __expf(v - mn) : 0.f;
      const float alpha = __expf(m[i] - mn);
      l[i] = l[i] * alpha + wave_sum(p);
#pragma unroll
      for (int c = 0; c < CPL; ++c) o[i][c] *= alpha;
      m[i] = mn;
      Ps[i][lane] = p;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    const int kmax = min(KC, n - c0);
    for (int k = 0; k < kmax; ++k) {
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const int e = lane * CPL + c;
        const float v = e < DH ? to_f32(Vs[k][e]) : 0.f;
#pragma unroll
        for (int i = 0; i < KQ; ++i) o[i][c] += Ps[i][k] * v;
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  }
}

// Encoder-decoder attention of the decoder step: one wave per (live sentence, head).
// The KQ beam rows of a sentence share its cross keys/values, so the wave reads each
// key and value of the sentence once for all of them.
// Waves per workgroup for the one-wave-per-task attention kernels: as many as fit in
// 64 KB of LDS (so two workgroups share a CU), at most 4.
template <typename T, int DH, int KQ>
constexpr int attn_waves() {
  constexpr int per_wave = KQ * DH * 4 + KQ * KC * 4 + KC * (DH + 8) * (int)sizeof(T);
  return per_wave * 4 <= 65536 ? 4 : per_wave * 2 <= 65536 ? 2 : 1;
}

template <typename T, int DH, int KQ>
__global__ __launch_bounds__(256) void cross_attn_kernel(MhaArgs a) {
  constexpr int CPL = DH > 64 ? DH / 64 : 1;
  constexpr int NWV = attn_waves<T, DH, KQ>();
  __shared__ float Qs[NWV][KQ][DH];
  __shared__ float Ps[NWV][KQ][KC];
  __shared__ __attribute__((aligned(16))) T Vs[NWV][KC][DH + 8];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int pair = blockIdx.x * NWV + wave;
  if (pair >= a.n_groups * a.H) return;          // whole wave exits; no block barrier below
  const int g = pair / a.H, h = pair % a.H;
  const int b = a.group_map ? a.group_map[g] : g;
  const int len = a.lens[b];
  const int nq = a.q_per_group;                  // <= KQ
  const T* Q = static_cast<const T*>(a.q);
  for (int idx = lane; idx < KQ * DH; idx += kWave) {
    const int i = idx / DH, e = idx % DH;
    Qs[wave][i][e] = i < nq ? to_f32(Q[(size_t)(g * nq + i) * a.q_ld + h * DH + e]) * a.scale : 0.f;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  const T* Kp = static_cast<const T*>(a.k) + (size_t)b * a.kb + (size_t)h * a.kh;
  const T* Vp = static_cast<const T*>(a.v) + (size_t)b * a.kb + (size_t)h * a.kh;
  const long long ks = a.ks;
  float o[KQ][CPL], l[KQ];
  wave_attend<T, DH, KQ>(Qs[wave], Ps[wave], Vs[wave], len, Kp, Vp, [&](int s) { return (size_t)s * ks; }, o, l);
  T* out = static_cast<T*>(a.out);
#pragma unroll
  for (int i = 0; i < KQ; ++i) {
    if (i >= nq) continue;
    const float inv = 1.0f / l[i];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int e = lane * CPL + c;
      if (e < DH) out[(size_t)(g * nq + i) * a.out_ld + h * DH + e] = from_f32<T>(o[i][c] * inv);
    }
  }
}

// Decoder self-attention: one wave per (live row, head) over the row's cached slots
// 0..t.  Slot s of a beam hypothesis lives in the physical row of its ancestor at step s
// (anc), so reordering beams never copies the cache.
template <typename T, int DH>
__global__ __launch_bounds__(256) void self_attn_kernel(SelfAttnArgs a) {
  constexpr int CPL = DH > 64 ? DH / 64 : 1;
  constexpr int NWV = attn_waves<T, DH, 1>();
  __shared__ float Qs[NWV][1][DH];
  __shared__ float Ps[NWV][1][KC];
  __shared__ __attribute__((aligned(16))) T Vs[NWV][KC][DH + 8];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int pair = blockIdx.x * NWV + wave;
  if (pair >= a.rows * a.H) return;            // whole wave exits; no block barrier below
  const int row = pair / a.H, h = pair % a.H;
  const int p = a.sent_list[row / a.beam] * a.beam + row % a.beam;
  const T* q = static_cast<const T*>(a.q) + (size_t)row * a.H * DH + h * DH;
  for (int e = lane; e < DH; e += kWave) Qs[wave][0][e] = to_f32(q[e]) * a.scale;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  const size_t head = (size_t)h * a.Tcap * DH;
  const size_t row_stride = (size_t)a.H * a.Tcap * DH;
  const int* anc = a.anc ? a.anc + (size_t)p * a.Tcap : nullptr;
  const int t = a.t;
  auto row_of = [&](int s) {
    const int ph = (anc && s < t) ? anc[s] : p;
    return (size_t)ph * row_stride + (size_t)s * DH;
  };
  float o[1][CPL], l[1];
  wave_attend<T, DH, 1>(Qs[wave], Ps[wave], Vs[wave], t + 1, static_cast<const T*>(a.kcache) + head,
                        static_cast<const T*>(a.vcache) + head, row_of, o, l);
  T* out = static_cast<T*>(a.out) + (size_t)row * a.H * DH + h * DH;
  const float inv = 1.0f / l[0];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int e = lane * CPL + c;
    if (e < DH) out[e] = from_f32<T>(o[0][c] * inv);
  }
}

template <typename T, int DH, int KQ>
void cross_launch(const MhaArgs& a, hipStream_t s) {
  constexpr int NWV = attn_waves<T, DH, KQ>();
  const dim3 grid((a.n_groups * a.H + NWV - 1) / NWV);
  hipLaunchKernelGGL((cross_attn_kernel<T, DH, KQ>), grid, dim3(NWV * kWave), 0, s, a);
}

template <typename T, int DH>
hipError_t cross_t(const MhaArgs& a, hipStream_t s) {
  const int q = a.q_per_group;
  if (q <= 1) cross_launch<T, DH, 1>(a, s);
  else if (q <= 2) cross_launch<T, DH, 2>(a, s);
  else if (q <= 4) cross_launch<T, DH, 4>(a, s);
  else if (q <= 8) cross_launch<T, DH, 8>(a, s);
  else if (q <= 16) cross_launch<T, DH, 16>(a, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename T, int ROLE>
hipError_t mha_t(const MhaArgs& a, hipStream_t s) {
  if (ROLE == 1 && !a.self_queries) {
    switch (a.dh) {
      case 32: return cross_t<T, 32>(a, s);
      case 64: return cross_t<T, 64>(a, s);
      case 128: return cross_t<T, 128>(a, s);
      default: return hipErrorInvalidValue;
    }
  }
  const int qblocks = (a.q_per_group + NW * QW - 1) / (NW * QW);
  const dim3 grid(a.n_groups * qblocks, a.H);
  switch (a.dh) {
    case 32: hipLaunchKernelGGL((mha_kernel<T, 32, ROLE>), grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((mha_kernel<T, 64, ROLE>), grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((mha_kernel<T, 128, ROLE>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int DH>
void self_launch(const SelfAttnArgs& a, hipStream_t s) {
  constexpr int NWV = attn_waves<T, DH, 1>();
  const dim3 grid((a.rows * a.H + NWV - 1) / NWV);
  hipLaunchKernelGGL((self_attn_kernel<T, DH>), grid, dim3(NWV * kWave), 0, s, a);
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
  switch (dt) {
    case DT::F32: return self_t<float>(a, s);
    case DT::F16: return self_t<f16>(a, s);
    case DT::BF16: return self_t<bf16>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace nt
