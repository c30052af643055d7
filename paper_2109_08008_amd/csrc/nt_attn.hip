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

constexpr int MAX_SLOTS = 1024;

template <typename T, int DH>
__global__ __launch_bounds__(256) void self_attn_kernel(SelfAttnArgs a) {
  constexpr int CPL = DH > 64 ? DH / 64 : 1;
  __shared__ float Qs[NW][DH];
  __shared__ float Ss[NW][MAX_SLOTS];
  __shared__ int Rs[NW][MAX_SLOTS];

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int pair = blockIdx.x * NW + wave;
  if (pair >= a.rows * a.H) return;            // whole wave exits; no block barrier below
  const int row = pair / a.H, h = pair % a.H;
  const int p = a.sent_list[row / a.beam] * a.beam + row % a.beam;
  const int ns = a.t + 1;

  const T* q = static_cast<const T*>(a.q) + (size_t)row * a.H * DH + h * DH;
  for (int e = lane; e < DH; e += kWave) Qs[wave][e] = to_f32(q[e]) * a.scale;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");

  const T* Kc = static_cast<const T*>(a.kcache);
  const T* Vc = static_cast<const T*>(a.vcache);
  float mx = -INFINITY;
  for (int s = lane; s < ns; s += kWave) {
    const int ph = (a.anc && s < a.t) ? a.anc[(size_t)p * a.Tcap + s] : p;
    const T* kr = Kc + ((size_t)(ph * a.H + h) * a.Tcap + s) * DH;
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < DH; e += Vec<T>::N) {
      float kv[Vec<T>::N];
      load16(kr + e, kv);
#pragma unroll
      for (int i = 0; i < Vec<T>::N; ++i) acc += Qs[wave][e + i] * kv[i];
    }
    Ss[wave][s] = acc;
    Rs[wave][s] = ph;
    mx = fmaxf(mx, acc);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int s = lane; s < ns; s += kWave) {
    const float pr = expf(Ss[wave][s] - mx);
    Ss[wave][s] = pr;
    sum += pr;
  }
  sum = wave_sum(sum);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");

  float o[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) o[c] = 0.f;
#pragma unroll 4
  for (int s = 0; s < ns; ++s) {
    const float pr = Ss[wave][s];
    const T* vr = Vc + ((size_t)(Rs[wave][s] * a.H + h) * a.Tcap + s) * DH;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int e = lane * CPL + c;
      if (e < DH) o[c] += pr * to_f32(vr[e]);
    }
  }
  T* out = static_cast<T*>(a.out) + (size_t)row * a.H * DH + h * DH;
  const float inv = 1.0f / sum;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int e = lane * CPL + c;
    if (e < DH) out[e] = from_f32<T>(o[c] * inv);
  }
}

template <typename T, int ROLE>
hipError_t mha_t(const MhaArgs& a, hipStream_t s) {
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

template <typename T>
hipError_t self_t(const SelfAttnArgs& a, hipStream_t s) {
  if (a.t + 1 > MAX_SLOTS) return hipErrorInvalidValue;
  const dim3 grid((a.rows * a.H + NW - 1) / NW);
  switch (a.dh) {
    case 32: hipLaunchKernelGGL((self_attn_kernel<T, 32>), grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL((self_attn_kernel<T, 64>), grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((self_attn_kernel<T, 128>), grid, dim3(256), 0, s, a); break;
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
