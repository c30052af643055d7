// Host runtime of the translation library: the C ABI declared in include/nt.h.
//
//  * model: validates the shape, lays the weights out on the device (matrices
//    transposed to [out][in] in the model dtype, vectors fp32, a sinusoidal position
//    table) and converts the caller's fp32 blob there with packing kernels;
//  * workspace arena: one caller-owned device buffer per batch is carved into every
//    tensor the encoder and decoder need (the memory pool of Sec. 4.4; nothing is
//    allocated during decoding); encoder temporaries and decoder buffers share space,
//    since the encoder is finished before the first decoder step;
//  * encoder (Eq. 1-2), decoder steps with cached keys/values (Sec. 4.1), greedy and
//    beam search, batch pruning (Sec. 4.1) and dynamic batching (Sec. 4.2);
//  * optional per-kernel-class event timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <mutex>
#include <numeric>
#include <string>
#include <deque>
#include <vector>

#include "../../include/nt.h"
#include "nt_common.h"
#include "nt_kernels.h"

using nt::DT;

namespace nt {
thread_local LaunchEvents g_launch_events;
}

// --------------------------------------------------------------------------------------
// errors
namespace {
thread_local std::string g_err;

nt_status fail(nt_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define NT_HIP(expr)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess) return fail(NT_E_DEVICE, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, __LINE__); \
  } while (0)

#define NT_TRY(expr)                    \
  do {                                  \
    nt_status s_ = (expr);              \
    if (s_ != NT_OK) return s_;         \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// --------------------------------------------------------------------------------------
// kernel timing: each timed launch records its dispatch's start / stop into an event pair
struct ProfRec {
  int cls;
  hipEvent_t a, b;
  double bytes, flops;
};
std::mutex g_prof_mu;
uint32_t g_prof_mask = 0;
int g_prof_stride = 1;
int64_t g_prof_seen[NT_K_COUNT] = {};
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// How launches of enabled classes are timed on this thread: every stride-th launch of a
// class (the step-level entry points), never (nt_translate outside its samples, and
// graph capture), or every launch (a sampled unit of nt_translate).
enum ProfMode { PROF_STRIDE = 0, PROF_NONE = 1, PROF_ALL = 2 };
thread_local int g_prof_mode = PROF_STRIDE;
int64_t g_prof_enc_units = 0, g_prof_step_units = 0;   // nt_translate units seen while profiling
std::atomic<bool> g_use_graphs{true};   // nt_translate replays a captured decode step
std::atomic<bool> g_beam_fused{true};   // beam selection without stored logits (nt_set_beam_fused)
std::atomic<int> g_streams{4};          // batches nt_translate decodes concurrently

struct ProfModeScope {
  int saved;
  explicit ProfModeScope(int m) : saved(g_prof_mode) { g_prof_mode = m; }
  ~ProfModeScope() { g_prof_mode = saved; }
};

// Whether the next nt_translate unit (a batch encode, or a decoder step) is a timing
// sample: every stride-th unit of its kind while a class that kind launches is enabled.
// A sample runs alone on the GPU (the other batches' streams are drained first), so its
// kernel times are those of the kernels by themselves.
constexpr uint32_t kEncClasses = (1u << NT_K_GEMM_ENC) | (1u << NT_K_DLCL) | (1u << NT_K_LN) | (1u << NT_K_ATTN_ENC);
constexpr uint32_t kStepClasses = (1u << NT_K_GEMM_DEC) | (1u << NT_K_GEMM_VOCAB) | (1u << NT_K_LN) |
                                  (1u << NT_K_ATTN_SELF) | (1u << NT_K_ATTN_CROSS) | (1u << NT_K_SELECT) |
                                  (1u << NT_K_SEARCH);
bool prof_unit_sampled(bool encode) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!(g_prof_mask & (encode ? kEncClasses : kStepClasses))) return false;
  int64_t& n = encode ? g_prof_enc_units : g_prof_step_units;
  return n++ % g_prof_stride == 0;
}

template <typename F>
hipError_t timed(int cls, hipStream_t s, double bytes, double flops, F&& launch) {
  if (g_prof_mode == PROF_NONE || !(g_prof_mask & (1u << cls))) return launch();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (g_prof_mode == PROF_STRIDE && g_prof_seen[cls]++ % g_prof_stride != 0) return launch();
  hipEvent_t a = prof_event(), b = prof_event();
  if (!a || !b) return hipErrorOutOfMemory;
  // the launch writes its dispatch's own start / stop times into a and b
  nt::g_launch_events = nt::LaunchEvents{a, b};
  const hipError_t e = launch();
  const bool launched = nt::g_launch_events.start == nullptr;
  nt::g_launch_events = nt::LaunchEvents{};
  if (e != hipSuccess || !launched) {   // nothing was launched (or it failed): no record
    g_prof_pool.push_back(a);
    g_prof_pool.push_back(b);
    return e;
  }
  (void)s;
  g_prof.push_back({cls, a, b, bytes, flops});
  return e;
}

}  // namespace

// --------------------------------------------------------------------------------------
// model
struct EncLayerW {
  const float *ln1, *bqkv, *bo, *ln2, *b1, *b2;
  const void *Wqkv, *Wo, *W1, *W2;
  const float *relk, *relv;   // [2k+1][d_head] relative-position tables, or null
  // FP8 weights: the column scales of Wqkv, Wo, W1, W2 (null for weights in the model dtype)
  const float *sqkv = nullptr, *so = nullptr, *s1 = nullptr, *s2 = nullptr;
};
struct DecLayerW {
  const float *ln1, *bqkv, *bo, *ln2, *bq, *boc, *ln3, *b1, *b2;
  const void *Wqkv, *Wo, *Wq, *Woc, *W1, *W2;
  const float *sqkv = nullptr, *so = nullptr, *sq = nullptr, *soc = nullptr, *s1 = nullptr, *s2 = nullptr;
  // Folded pre-norm LayerNorms (weights in the model dtype): Wqkv, Wq and W1 hold
  // diag(gamma) W of ln1, ln2 and ln3, their biases b + beta W, and these the column sums of
  // the packed matrices; null when the LayerNorms run as kernels of their own (FP8).
  const float *cqkv = nullptr, *cq = nullptr, *c1 = nullptr;
};

struct nt_model {
  nt_model_cfg cfg;
  DT dt;
  size_t eb;
  int d, H, dh, F, L, Ld, V;
  const void* E;
  const float* pe;
  const float* hist_ln;   // [L+1][2][d]
  const float* dlcl;      // row l (1-based) at dlcl + l(l-1)/2
  std::vector<EncLayerW> enc;
  const float* enc_out_ln;
  std::vector<DecLayerW> dec;
  const void* Wkv_all;    // [Ld*2d][d]
  const float* bkv_all;   // [Ld*2d]
  const float* skv_all = nullptr;   // FP8 weights: column scales of Wkv_all
  const float* dec_out_ln;
  // an ensemble (nt_ensemble): the member models, borrowed, and the combination rule;
  // empty for a loaded model, whose only member is itself
  std::vector<nt_model*> members;
  int rule = 0;
};

namespace {

int n_members(const nt_model& m) { return m.members.empty() ? 1 : (int)m.members.size(); }
const nt_model& member(const nt_model& m, int i) { return m.members.empty() ? m : *m.members[i]; }

nt_status validate_cfg(const nt_model_cfg* c) {
  if (!c) return fail(NT_E_INVALID, "null model config");
  if (c->d_model <= 0 || c->n_heads <= 0 || c->d_ffn <= 0 || c->n_enc < 0 || c->n_dec <= 0 || c->vocab <= 0 ||
      c->max_positions <= 0)
    return fail(NT_E_INVALID, "model sizes must be positive (n_enc >= 0)");
  if (c->vocab < 4) return fail(NT_E_INVALID, "vocab must hold PAD, BOS, EOS and a word (>= 4)");
  for (int id : {c->pad_id, c->bos_id, c->eos_id})
    if (id < 0 || id >= c->vocab) return fail(NT_E_INVALID, "special token id %d outside [0, %d)", id, c->vocab);
  if (c->dtype < NT_F32 || c->dtype > NT_BF16) return fail(NT_E_INVALID, "unknown dtype %d", c->dtype);
  if (c->d_model % 64 != 0) return fail(NT_E_UNSUPPORTED, "d_model %% 64 != 0 (d_model=%d)", c->d_model);
  const int e = c->d_model / 64;
  if (e != 1 && e != 2 && e != 4 && e != 6 && e != 8 && e != 12 && e != 16)
    return fail(NT_E_UNSUPPORTED, "d_model=%d not in {64,128,256,384,512,768,1024}", c->d_model);
  if (c->d_model % c->n_heads != 0) return fail(NT_E_UNSUPPORTED, "d_model %% n_heads != 0");
  const int dh = c->d_model / c->n_heads;
  if (dh != 32 && dh != 64 && dh != 128) return fail(NT_E_UNSUPPORTED, "head size %d not in {32,64,128}", dh);
  if (c->d_ffn % 64 != 0) return fail(NT_E_UNSUPPORTED, "d_ffn %% 64 != 0 (d_ffn=%d)", c->d_ffn);
  if (c->max_positions > 1024) return fail(NT_E_UNSUPPORTED, "max_positions > 1024");
  if (!(c->ln_eps > 0.f)) return fail(NT_E_INVALID, "ln_eps must be > 0");
  if (c->rel_pos_k < 0 || c->rel_pos_k > 16) return fail(NT_E_UNSUPPORTED, "rel_pos_k %d outside [0, 16]", c->rel_pos_k);
  if (c->fp8_weights != 0 && c->fp8_weights != 1) return fail(NT_E_INVALID, "fp8_weights must be 0 or 1");
  if (c->fp8_weights && c->dtype != NT_F16) return fail(NT_E_UNSUPPORTED, "fp8_weights needs dtype NT_F16");
  if (c->fp8_kv != 0 && c->fp8_kv != 1) return fail(NT_E_INVALID, "fp8_kv must be 0 or 1");
  if (c->fp8_kv && c->dtype != NT_F16) return fail(NT_E_UNSUPPORTED, "fp8_kv needs dtype NT_F16");
  return NT_OK;
}

// Offsets of the device layout (bytes) and of the host blob (floats).
struct ModelLayout {
  size_t total = 0;
  size_t E, pe, hist_ln, dlcl, enc_out_ln, Wkv_all, bkv_all, dec_out_ln;
  struct Enc { size_t ln1, Wqkv, bqkv, Wo, bo, ln2, W1, b1, W2, b2, relk, relv, sqkv, so, s1, s2; };
  struct Dec { size_t ln1, Wqkv, bqkv, Wo, bo, ln2, Wq, bq, Woc, boc, ln3, W1, b1, W2, b2, sqkv, so, sq, soc, s1, s2,
               cqkv, cq, c1; };
  size_t skv_all = 0;
  std::vector<Enc> enc;
  std::vector<Dec> dec;
  // host blob (fp32) offsets
  size_t hE, hhist, hdlcl, henc_out, hdec_out, host_floats;
  struct HEnc { size_t ln1, Wqkv, bqkv, Wo, bo, ln2, W1, b1, W2, b2, relk, relv; };
  struct HDec { size_t ln1, Wqkv, bqkv, Wo, bo, ln2, Wq, bq, Wkv, bkv, Woc, boc, ln3, W1, b1, W2, b2; };
  std::vector<HEnc> henc;
  std::vector<HDec> hdec;
};

ModelLayout layout_of(const nt_model_cfg& c) {
  ModelLayout Lo;
  const size_t d = c.d_model, F = c.d_ffn, V = c.vocab, L = c.n_enc, Ld = c.n_dec;
  const size_t eb = c.dtype == NT_F32 ? 4 : 2;
  const bool f8 = c.fp8_weights != 0;
  const size_t mb = f8 ? 1 : eb;   // bytes per projection weight (E keeps eb)
  const size_t dh = d / c.n_heads, rt = c.rel_pos_k > 0 ? 2 * (size_t)c.rel_pos_k + 1 : 0;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  Lo.E = take(V * d * eb);
  Lo.pe = take((size_t)c.max_positions * d * 4);
  Lo.hist_ln = take((L + 1) * 2 * d * 4);
  Lo.dlcl = take((L + 1) * (L + 2) / 2 * 4);
  for (size_t i = 0; i < L; ++i) {
    ModelLayout::Enc e;
    e.ln1 = take(2 * d * 4);
    e.Wqkv = take(3 * d * d * mb);
    e.bqkv = take(3 * d * 4);
    e.Wo = take(d * d * mb);
    e.bo = take(d * 4);
    e.ln2 = take(2 * d * 4);
    e.W1 = take(F * d * mb);
    e.b1 = take(F * 4);
    e.W2 = take(d * F * mb);
    e.b2 = take(d * 4);
    e.sqkv = f8 ? take(3 * d * 4) : 0;
    e.so = f8 ? take(d * 4) : 0;
    e.s1 = f8 ? take(F * 4) : 0;
    e.s2 = f8 ? take(d * 4) : 0;
    e.relk = rt ? take(rt * dh * 4) : 0;
    e.relv = rt ? take(rt * dh * 4) : 0;
    Lo.enc.push_back(e);
  }
  Lo.enc_out_ln = take(2 * d * 4);
  for (size_t j = 0; j < Ld; ++j) {
    ModelLayout::Dec e;
    e.ln1 = take(2 * d * 4);
    e.Wqkv = take(3 * d * d * mb);
    e.bqkv = take(3 * d * 4);
    e.Wo = take(d * d * mb);
    e.bo = take(d * 4);
    e.ln2 = take(2 * d * 4);
    e.Wq = take(d * d * mb);
    e.bq = take(d * 4);
    e.Woc = take(d * d * mb);
    e.boc = take(d * 4);
    e.ln3 = take(2 * d * 4);
    e.W1 = take(F * d * mb);
    e.b1 = take(F * 4);
    e.W2 = take(d * F * mb);
    e.b2 = take(d * 4);
    e.sqkv = f8 ? take(3 * d * 4) : 0;
    e.so = f8 ? take(d * 4) : 0;
    e.sq = f8 ? take(d * 4) : 0;
    e.soc = f8 ? take(d * 4) : 0;
    e.s1 = f8 ? take(F * 4) : 0;
    e.s2 = f8 ? take(d * 4) : 0;
    e.cqkv = take(3 * d * 4);
    e.cq = take(d * 4);
    e.c1 = take(F * 4);
    Lo.dec.push_back(e);
  }
  Lo.Wkv_all = take(Ld * 2 * d * d * mb);
  Lo.bkv_all = take(Ld * 2 * d * 4);
  Lo.skv_all = f8 ? take(Ld * 2 * d * 4) : 0;
  Lo.dec_out_ln = take(2 * d * 4);
  Lo.total = off;

  // host blob, canonical order (see include/nt.h)
  size_t h = 0;
  Lo.hE = h; h += V * d;
  Lo.hhist = h; h += (L + 1) * 2 * d;
  Lo.hdlcl = h; h += (L + 1) * (L + 2) / 2;
  for (size_t i = 0; i < L; ++i) {
    ModelLayout::HEnc e;
    e.ln1 = h; h += 2 * d;
    e.Wqkv = h; h += d * 3 * d;
    e.bqkv = h; h += 3 * d;
    e.Wo = h; h += d * d;
    e.bo = h; h += d;
    e.ln2 = h; h += 2 * d;
    e.W1 = h; h += d * F;
    e.b1 = h; h += F;
    e.W2 = h; h += F * d;
    e.b2 = h; h += d;
    e.relk = h; h += rt * dh;
    e.relv = h; h += rt * dh;
    Lo.henc.push_back(e);
  }
  Lo.henc_out = h; h += 2 * d;
  for (size_t j = 0; j < Ld; ++j) {
    ModelLayout::HDec e;
    e.ln1 = h; h += 2 * d;
    e.Wqkv = h; h += d * 3 * d;
    e.bqkv = h; h += 3 * d;
    e.Wo = h; h += d * d;
    e.bo = h; h += d;
    e.ln2 = h; h += 2 * d;
    e.Wq = h; h += d * d;
    e.bq = h; h += d;
    e.Wkv = h; h += d * 2 * d;
    e.bkv = h; h += 2 * d;
    e.Woc = h; h += d * d;
    e.boc = h; h += d;
    e.ln3 = h; h += 2 * d;
    e.W1 = h; h += d * F;
    e.b1 = h; h += F;
    e.W2 = h; h += F * d;
    e.b2 = h; h += d;
    Lo.hdec.push_back(e);
  }
  Lo.hdec_out = h; h += 2 * d;
  Lo.host_floats = h;
  return Lo;
}

// --------------------------------------------------------------------------------------
// FP8 weights: OCP E4M3 (sign, 4 exponent bits with bias 7, 3 mantissa bits; subnormals
// of 2^-9; no infinities; 0x7F / 0xFF are NaN, so the largest finite value is 448).

uint8_t e4m3_code(float x) { return nt::e4m3_rne(x); }

// Value of an E4M3 code (finite codes only; the quantizer never produces NaN).
double e4m3_value(uint8_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  const double v = e == 0 ? std::ldexp((double)m, -9) : std::ldexp(8.0 + m, e - 10);
  return (c & 0x80) ? -v : v;
}

// Weight matrix W [in][out] (row-major, y = x W) as FP8 codes q [out][in] (the GEMM's
// K-contiguous layout) with one scale per output column n: scale = max_k |W[k][n]| / 448
// (1 for an all-zero column) and q = e4m3_code(W[k][n] / scale), both in fp32.
void quantize_fp8(const float* W, int in, int out, std::vector<uint8_t>& q, std::vector<float>& scale) {
  std::vector<float> amax(out, 0.f);
  for (int k = 0; k < in; ++k)
    for (int n = 0; n < out; ++n) amax[n] = std::max(amax[n], std::fabs(W[(size_t)k * out + n]));
  scale.resize(out);
  for (int n = 0; n < out; ++n) scale[n] = amax[n] > 0.f ? amax[n] / 448.0f : 1.0f;
  q.resize((size_t)in * out);
  for (int k = 0; k < in; ++k)
    for (int n = 0; n < out; ++n) q[(size_t)n * in + k] = e4m3_code(W[(size_t)k * out + n] / scale[n]);
}

// --------------------------------------------------------------------------------------
// Blocked DLCL: a block start's pass over the old history entries also sums them for the
// next n rows (n <= nt::DLCL_PARTS), which then start from those fp32 partial sums and
// read only the entries after the block start.  The fp32 additions happen in the same
// order, so the result is the same bit for bit.  The blocks are placed to move the fewest
// bytes (history entries read and written, an fp32 partial counting as two entries): a
// row that starts a block at l with n partials costs (l - 1) + 2n, the i-th row inside it
// 2 + (i - 1).  Shallow encoders come out unblocked.
// Returns sched[1..L+1]: the partial count of a row that starts a block (0: a plain row),
// -1 for a row inside a block.
std::vector<int> dlcl_schedule(int L) {
  const int R = L + 1, P = nt::DLCL_PARTS;
  std::vector<long long> f(R + 2, 0);   // f[l]: least cost of rows l..R, row l not in a block
  std::vector<int> best(R + 2, 0);
  for (int l = R; l >= 1; --l) {
    f[l] = -1;
    long long inside = 0;
    for (int n = 0; n <= std::min(P, R - l); ++n) {
      if (n > 0) inside += 2 + (n - 1);
      const long long c = (l - 1) + 2LL * n + inside + f[l + n + 1];
      if (f[l] < 0 || c < f[l]) {
        f[l] = c;
        best[l] = n;
      }
    }
  }
  std::vector<int> sched(R + 1, 0);
  for (int l = 1; l <= R; l += best[l] + 1) {
    sched[l] = best[l];
    for (int i = 1; i <= best[l]; ++i) sched[l + i] = -1;
  }
  return sched;
}
int dlcl_max_parts(int L) {
  const std::vector<int> s = dlcl_schedule(L);
  return *std::max_element(s.begin(), s.end());
}

// --------------------------------------------------------------------------------------
// workspace arena of one batch
struct MemberPlan {
  size_t enc_out, cross, kself, vself;   // one model's encoder output and caches
};
struct WsPlan {
  size_t total = 0;
  // persistent through the batch: inputs, every member's caches, the search state
  size_t src, len, maxlen;
  std::vector<MemberPlan> mem;
  size_t score, cur_tok, tok_hist, par_hist, lp_hist, anc, done, best_score, best_raw, best_step,
      best_row, best_nout, list, ctl, out_tok, out_lp, out_len, out_score;
  // encoder temporaries (union with the decoder buffers below); the members encode and
  // step one after another, so they share both, sized for the largest member
  size_t hist, x, u, qkv, att, a, f, y, dlcl_part;
  // decoder buffers (comb: an ensemble's combined scores)
  size_t z, du, dq, datt, df, logits, comb, topv, topi, lse;
  size_t tparts;   // beam: the projection's per-tile records
  // beam without stored logits: each pair's tile, the pairs sorted by tile, the rows'
  // thresholds, the recomputed tiles and the blocks of the recompute
  bool beam_pairs = false;
  int pair_blocks = 0;
  size_t gptile, gsorted, gtau, glog, gblk, gnblk;
};

WsPlan ws_plan(const nt_model& m, int B, int S, int K, int Tcap) {
  WsPlan p;
  const int M = n_members(m);
  const size_t T = (size_t)B * S, R = (size_t)B * K, eb = m.eb;
  const size_t n_tiles = (m.V + 127) / 128, k2 = 2 * (size_t)K;
  p.beam_pairs = K > 1 && M == 1 && g_beam_fused.load();
  p.pair_blocks = p.beam_pairs ? (int)((R * k2 + nt::PAIR_BM - 1) / nt::PAIR_BM + n_tiles) : 0;
  size_t d = 0, F = 0, hist = 0, dlcl_part = 0;
  for (int i = 0; i < M; ++i) {
    const nt_model& mi = member(m, i);
    d = std::max<size_t>(d, mi.d);
    F = std::max<size_t>(F, mi.F);
    hist = std::max<size_t>(hist, (size_t)(mi.L + 1) * mi.d);
    dlcl_part = std::max<size_t>(dlcl_part, (size_t)dlcl_max_parts(mi.L) * mi.d);
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 1));
    return o;
  };
  p.src = take(T * 4);
  p.len = take(B * 4);
  p.maxlen = take(B * 4);
  p.mem.resize(M);
  for (int i = 0; i < M; ++i) {
    const nt_model& mi = member(m, i);
    const size_t di = mi.d;
    p.mem[i].enc_out = take(T * di * eb);
    p.mem[i].cross = take((size_t)mi.Ld * 2 * T * di * eb);
    const size_t kvb = mi.cfg.fp8_kv ? 1 : eb;   // E4M3 keys and values, or the model dtype
    p.mem[i].kself = take((size_t)mi.Ld * R * Tcap * di * kvb);
    p.mem[i].vself = take((size_t)mi.Ld * R * Tcap * di * kvb);
  }
  p.score = take(R * 4);
  p.cur_tok = take(R * 4);
  p.tok_hist = take((size_t)Tcap * R * 4);
  p.par_hist = take((size_t)Tcap * R * 4);
  p.lp_hist = take((size_t)Tcap * R * 4);
  p.anc = take(K > 1 ? 2 * R * Tcap * 4 : 0);
  p.done = take(B * 4);
  p.best_score = take(B * 4);
  p.best_raw = take(B * 4);
  p.best_step = take(B * 4);
  p.best_row = take(B * 4);
  p.best_nout = take(B * 4);
  p.list = take((size_t)B * 4);
  p.ctl = take(nt::CTL_WORDS * 4);
  p.out_tok = take((size_t)B * Tcap * 4);
  p.out_lp = take((size_t)B * Tcap * 4);
  p.out_len = take(B * 4);
  p.out_score = take(B * 4);
  const size_t base = off;
  // encoder temporaries
  p.hist = take(hist * T * eb);
  p.x = take(T * d * eb);
  p.u = take(T * d * eb);
  p.qkv = take(T * 3 * d * eb);
  p.att = take(T * d * eb);
  p.a = take(T * d * eb);
  p.f = take(T * F * eb);
  p.y = take(T * d * eb);
  p.dlcl_part = take(dlcl_part * T * 4);   // fp32 partial sums of a DLCL block
  const size_t enc_end = off;
  // decoder buffers reuse the same space
  off = base;
  p.z = take(R * d * eb);
  p.du = take(R * d * eb);
  p.dq = take(R * d * eb);
  p.datt = take(R * d * eb);
  p.df = take(R * F * eb);
  // fp32 logits, or (fused greedy selection) the per-tile partial records, whichever is
  // larger; beam without stored logits needs neither
  const size_t recs = R * n_tiles * nt::topk_record(1) * 4;
  p.logits = take(p.beam_pairs ? 0 : std::max(R * m.V * 4, recs));
  p.comb = M > 1 ? take(R * m.V * 4) : 0;
  p.topv = take(R * 2 * K * 4);
  p.topi = take(R * 2 * K * 4);
  p.lse = take(R * 4);
  p.tparts = take(K > 1 ? recs : 0);
  p.gptile = take(p.beam_pairs ? R * k2 * 4 : 0);
  p.gsorted = take(p.beam_pairs ? R * k2 * 4 : 0);
  p.gtau = take(p.beam_pairs ? R * 4 : 0);
  p.glog = take(p.beam_pairs ? R * k2 * 128 * 4 : 0);
  p.gblk = take((size_t)p.pair_blocks * 3 * 4);
  p.gnblk = take(p.beam_pairs ? 4 : 0);
  p.total = std::max(enc_end, off);
  return p;
}

int max_tgt_of(const nt_search_cfg& s, int len) {
  const int n = (int)std::floor((double)s.max_len_a * (double)len) + s.max_len_b;
  return s.max_len_cap > 0 ? std::min(n, s.max_len_cap) : n;
}

nt_status validate_search(const nt_model& m, const nt_search_cfg* s) {
  if (!s) return fail(NT_E_INVALID, "null search config");
  if (s->beam < 1) return fail(NT_E_INVALID, "beam must be >= 1");
  if (s->beam > 16) return fail(NT_E_UNSUPPORTED, "beam %d > 16", s->beam);
  if (s->max_len_a < 0.f || !std::isfinite(s->max_len_a)) return fail(NT_E_INVALID, "max_len_a must be >= 0");
  if (s->token_budget < 0 || s->max_batch_sents < 0) return fail(NT_E_INVALID, "negative budget / sentence cap");
  if (s->max_len_cap < 0) return fail(NT_E_INVALID, "max_len_cap must be >= 0");
  if (!std::isfinite(s->len_penalty)) return fail(NT_E_INVALID, "len_penalty must be finite");
  (void)m;
  return NT_OK;
}

}  // namespace

// --------------------------------------------------------------------------------------
// decoder state
struct nt_dec_state {
  nt_model* m;
  nt_search_cfg sc;
  int B, S, K, Tcap;
  // host copy of the device control block, as of the last step the host has read
  int t = 0;
  int n_live = 0;     // entries of the live list
  int n_alive = 0;    // sentences not finished
  bool finished = false;
  WsPlan plan;
  char* ws;
  int* h_ctl = nullptr;   // pinned mirror [CTL_MIRROR_SLOTS][CTL_WORDS], written by the step-end kernel
  int* d_hctl = nullptr;  // its device-side address
  bool own_ctl = true;    // the mirror was allocated for this state (else borrowed)
  template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  int* list() const { return at<int>(plan.list); }
  int* ctl() const { return at<int>(plan.ctl); }
  size_t anc_stride() const { return (size_t)B * K * Tcap; }
  nt::SearchState search() const {
    nt::SearchState s;
    s.B = B;
    s.beam = K;
    s.V = m->V;
    s.eos = m->cfg.eos_id;
    s.Tcap = Tcap;
    s.alpha = sc.len_penalty;
    s.early_stop = sc.early_stop;
    s.logp_input = n_members(*m) > 1 ? 1 : 0;
    s.sent_list = list();
    s.ctl = ctl();
    s.score = at<float>(plan.score);
    s.cur_tok = at<int>(plan.cur_tok);
    s.tok_hist = at<int>(plan.tok_hist);
    s.par_hist = at<int>(plan.par_hist);
    s.lp_hist = at<float>(plan.lp_hist);
    s.anc = K > 1 ? at<int>(plan.anc) : nullptr;
    s.anc_stride = anc_stride();
    s.done = at<int>(plan.done);
    s.maxlen = at<int>(plan.maxlen);
    s.best_score = at<float>(plan.best_score);
    s.best_raw = at<float>(plan.best_raw);
    s.best_step = at<int>(plan.best_step);
    s.best_row = at<int>(plan.best_row);
    s.best_nout = at<int>(plan.best_nout);
    return s;
  }
};

namespace {

// ---- encoder (Eq. 1-2) ---------------------------------------------------------------
// Encoder of member mi (the model itself unless it is an ensemble) into that member's
// encoder output and cross keys/values.
nt_status run_encoder(nt_dec_state* st, int mi, hipStream_t s) {
  const nt_model& m = member(*st->m, mi);
  const MemberPlan& mp = st->plan.mem[mi];
  const int B = st->B, S = st->S, d = m.d, L = m.L;
  const int T = B * S;
  const double eb = (double)m.eb;
  auto at = [&](size_t o) { return st->ws + o; };
  const WsPlan& p = st->plan;
  const size_t hist_stride = (size_t)T * d;
  const float eps = m.cfg.ln_eps;

  auto gemm_enc = [&](const void* A, int lda, const void* W, int N, int K, const nt::GemmEpi& e) -> hipError_t {
    const double wb = e.wscale ? 1.0 : eb;   // bytes per weight (FP8: one)
    const double bytes = (double)T * K * eb + (double)N * K * wb + (double)T * N * eb * (e.mode == nt::EPI_RESID ? 2 : 1);
    return timed(NT_K_GEMM_ENC, s, bytes, 2.0 * T * N * K, [&] { return nt::gemm(m.dt, A, lda, W, T, N, K, e, s); });
  };

  const std::vector<int> sched = dlcl_schedule(L);
  int blk = 0;   // the row that started the current DLCL block

  for (int l = 1; l <= L + 1; ++l) {
    nt::DlclArgs a{};
    a.l = l;
    a.y_prev = l == 1 ? nullptr : at(p.y);
    a.ids = st->at<int>(p.src);
    a.lens = st->at<int>(p.len);
    a.S = S;
    a.E = m.E;
    a.V = m.V;
    a.pe = m.pe;
    a.emb_scale = std::sqrt((float)d);
    a.hist = at(p.hist);
    a.hist_stride = hist_stride;
    a.hist_ln = m.hist_ln + (size_t)(l - 1) * 2 * d;
    a.hist_norm = m.cfg.dlcl_hist_norm;
    a.w = m.dlcl + (size_t)l * (l - 1) / 2;
    a.x_out = l <= L ? at(p.x) : nullptr;
    a.ln = l <= L ? m.enc[l - 1].ln1 : m.enc_out_ln;
    a.u_out = l <= L ? at(p.u) : at(mp.enc_out);
    a.rows = T;
    a.d = d;
    a.eps = eps;
    a.w_all = m.dlcl;
    double hist_reads = l - 1;   // history entries this row reads (fp32 partials count twice)
    if (sched[l] >= 0) {         // a plain row or a block start
      blk = l;
      if (sched[l] > 0) {
        a.n_part = sched[l];
        a.part_out = reinterpret_cast<float*>(at(p.dlcl_part));
        a.part_stride = (size_t)T * d;
        hist_reads += 2.0 * sched[l];
      }
    } else {                     // inside a block: start from the partial of entries < blk
      a.part_in = reinterpret_cast<const float*>(at(p.dlcl_part)) + (size_t)(l - blk - 1) * T * d;
      a.k_start = blk;
      hist_reads = 2.0 + (l - 1 - blk);
    }
    const double bytes = (double)T * d * eb * (hist_reads + (l <= L ? 4 : 3));
    NT_HIP(timed(NT_K_DLCL, s, bytes, 2.0 * T * d * l, [&] { return nt::dlcl_combine(m.dt, a, s); }));
    if (l > L) break;
    const EncLayerW& w = m.enc[l - 1];

    nt::GemmEpi e{};
    e.mode = nt::EPI_STORE;
    e.bias = w.bqkv;
    e.wscale = w.sqkv;
    e.out = at(p.qkv);
    e.ldc = 3 * d;
    NT_HIP(gemm_enc(at(p.u), d, w.Wqkv, 3 * d, d, e));

    nt::MhaArgs ma{};
    ma.q = at(p.qkv);
    ma.q_ld = 3 * d;
    ma.k = at(p.qkv) + (size_t)d * m.eb;
    ma.v = at(p.qkv) + (size_t)2 * d * m.eb;
    ma.kb = (long long)S * 3 * d;
    ma.kh = m.dh;
    ma.ks = 3 * d;
    ma.out = at(p.att);
    ma.out_ld = d;
    ma.group_map = nullptr;
    ma.lens = st->at<int>(p.len);
    ma.q_per_group = S;
    ma.self_queries = 1;
    ma.n_groups = B;
    ma.H = m.H;
    ma.dh = m.dh;
    ma.scale = 1.0f / std::sqrt((float)m.dh);
    ma.relk = w.relk;
    ma.relv = w.relv;
    ma.rel_k = m.cfg.rel_pos_k;
    NT_HIP(timed(NT_K_ATTN_ENC, s, 4.0 * T * d * eb, 4.0 * B * (double)S * S * d, [&] { return nt::mha(m.dt, ma, s); }));

    e = nt::GemmEpi{};
    e.mode = nt::EPI_RESID;
    e.bias = w.bo;
    e.wscale = w.so;
    e.resid = at(p.x);
    e.out = at(p.a);
    e.ldc = d;
    NT_HIP(gemm_enc(at(p.att), d, w.Wo, d, d, e));

    NT_HIP(timed(NT_K_LN, s, 2.0 * T * d * eb, 8.0 * T * d,
                 [&] { return nt::layernorm(m.dt, at(p.a), w.ln2, at(p.u), T, d, eps, s); }));

    e = nt::GemmEpi{};
    e.mode = nt::EPI_RELU;
    e.bias = w.b1;
    e.wscale = w.s1;
    e.out = at(p.f);
    e.ldc = m.F;
    NT_HIP(gemm_enc(at(p.u), d, w.W1, m.F, d, e));

    e = nt::GemmEpi{};
    e.mode = nt::EPI_RESID;
    e.bias = w.b2;
    e.wscale = w.s2;
    e.resid = at(p.a);
    e.out = at(p.y);
    e.ldc = d;
    NT_HIP(gemm_enc(at(p.f), m.F, w.W2, d, m.F, e));
  }

  // encoder-decoder keys/values of every decoder layer, once per batch (Sec. 4.1)
  nt::GemmEpi e{};
  e.mode = nt::EPI_CROSS_KV;
  e.bias = m.bkv_all;
  e.wscale = m.skv_all;
  e.cross = at(mp.cross);
  e.d = d;
  e.H = m.H;
  e.dh = m.dh;
  e.B = B;
  e.S = S;
  NT_HIP(gemm_enc(at(mp.enc_out), d, m.Wkv_all, 2 * d * m.Ld, d, e));
  return NT_OK;
}

// ---- one decoder step ------------------------------------------------------------------
// Enqueues every kernel of one step.  Grids are sized for the whole batch (Rp = B*K rows,
// B sentences); each kernel reads the live counts and t from the device control block, so
// the same sequence serves every step and can be captured once and replayed.  R and t
// below are the host's copy of the block and only feed the work figures of the timing.
nt_status enqueue_step(nt_dec_state* st, const int32_t* d_forced, float* d_logits, hipStream_t s) {
  const nt_model& top = *st->m;
  const int M = n_members(top);
  const WsPlan& p = st->plan;
  const int K = st->K, R = st->n_live * K, t = st->t;
  const int Rp = st->B * K;
  auto at = [&](size_t o) { return st->ws + o; };
  int* list = st->list();
  int* ctl = st->ctl();
  nt::SearchState ss = st->search();

  // every member's decoder on the shared prefix (one member unless an ensemble)
  for (int mi = 0; mi < M; ++mi) {
    const nt_model& m = member(top, mi);
    const MemberPlan& mp = p.mem[mi];
    const int d = m.d;
    const double eb = (double)m.eb;
    const float eps = m.cfg.ln_eps;
    const int kv8 = m.cfg.fp8_kv ? 1 : 0;     // the self-attention cache holds E4M3 bytes
    const size_t kvb = kv8 ? 1 : m.eb;

    // Algorithmic bytes of a decode-step launch count what the step must move: the
    // weights (read once per step, shared by every row) and, for the vocabulary
    // projection, the logits it stores (fp32, when they are materialised) or its per-tile
    // records; the rows' activations stay out of the count.
    auto gemm_dec = [&](int cls, const void* A, int lda, const void* W, int N, int Kd, const nt::GemmEpi& e) -> hipError_t {
      const double wb = e.wscale ? 1.0 : eb;   // bytes per weight (FP8: one)
      double bytes = (double)N * Kd * wb;
      if (cls == NT_K_GEMM_VOCAB) {
        if (e.out) bytes += (double)R * N * (e.out_f32 ? 4.0 : eb);
        if (e.mode == nt::EPI_TOPK) bytes += (double)R * e.n_tiles * nt::topk_record(e.k2) * 4.0;
      }
      const int role = cls == NT_K_GEMM_VOCAB ? 2 : 1;
      const int tile = e.mode == nt::EPI_TOPK ? 2 : 0;   // the partial records assume 128-column tiles
      nt::GemmEpi ec = e;
      ec.ctl = ctl;
      ec.ctl_rows = K;
      return timed(cls, s, bytes, 2.0 * R * N * Kd, [&] { return nt::gemm(m.dt, A, lda, W, Rp, N, Kd, ec, s, role, tile); });
    };

    // the first layer's ln1 output only when its QKV projection does not normalise itself
    const bool fold0 = m.dec[0].cqkv != nullptr;
    NT_HIP(timed(NT_K_LN, s, (fold0 ? 2.0 : 3.0) * R * d * eb, 8.0 * R * d, [&] {
      return nt::dec_embed_ln(m.dt, st->at<int>(p.cur_tok), list, K, m.E, m.pe, ctl, std::sqrt((float)d),
                              fold0 ? nullptr : m.dec[0].ln1, at(p.z), fold0 ? nullptr : at(p.du), Rp, d, eps, s);
    }));

    for (int j = 0; j < m.Ld; ++j) {
      const DecLayerW& w = m.dec[j];
      char* kc = at(mp.kself) + (size_t)j * Rp * st->Tcap * d * kvb;
      char* vc = at(mp.vself) + (size_t)j * Rp * st->Tcap * d * kvb;

      nt::GemmEpi e{};
      e.mode = nt::EPI_SELF_QKV;
      e.bias = w.bqkv;
      e.wscale = w.sqkv;
      e.out = at(p.dq);
      e.ldc = d;
      e.sent_list = list;
      e.beam = K;
      e.kcache = kc;
      e.vcache = vc;
      e.kv_f8 = kv8;
      e.Tcap = st->Tcap;
      e.d = d;
      e.H = m.H;
      e.dh = m.dh;
      // folded pre-norm LayerNorms: the projection normalises its input rows itself
      const bool fold = w.cqkv != nullptr;
      const void* ln_in = fold ? at(p.z) : at(p.du);
      e.lnf_colsum = w.cqkv;
      e.lnf_eps = eps;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, ln_in, d, w.Wqkv, 3 * d, d, e));

      nt::SelfAttnArgs sa{};
      sa.q = at(p.dq);
      sa.kcache = kc;
      sa.vcache = vc;
      sa.sent_list = list;
      sa.beam = K;
      sa.anc = K > 1 ? st->at<int>(p.anc) : nullptr;
      sa.anc_stride = st->anc_stride();
      sa.out = at(p.datt);
      sa.rows = Rp;
      sa.H = m.H;
      sa.dh = m.dh;
      sa.Tcap = st->Tcap;
      sa.scale = 1.0f / std::sqrt((float)m.dh);
      sa.ctl = ctl;
      sa.kv_f8 = kv8;
      NT_HIP(timed(NT_K_ATTN_SELF, s, (double)R * d * (double)kvb * 2.0 * (t + 1), 4.0 * R * (t + 1) * (double)d,
                   [&] { return nt::self_attn(m.dt, sa, s); }));

      e = nt::GemmEpi{};
      e.mode = nt::EPI_RESID;
      e.bias = w.bo;
      e.wscale = w.so;
      e.resid = at(p.z);
      e.out = at(p.z);
      e.ldc = d;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, at(p.datt), d, w.Wo, d, d, e));

      if (!fold)
        NT_HIP(timed(NT_K_LN, s, 2.0 * R * d * eb, 8.0 * R * d,
                     [&] { return nt::layernorm(m.dt, at(p.z), w.ln2, at(p.du), Rp, d, eps, s, ctl, K); }));

      e = nt::GemmEpi{};
      e.mode = nt::EPI_STORE;
      e.bias = w.bq;
      e.wscale = w.sq;
      e.out = at(p.dq);
      e.ldc = d;
      e.lnf_colsum = w.cq;
      e.lnf_eps = eps;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, ln_in, d, w.Wq, d, d, e));

      const size_t cross_layer = (size_t)2 * st->B * st->S * d;   // elements per layer (K and V)
      nt::MhaArgs ma{};
      ma.q = at(p.dq);
      ma.q_ld = d;
      ma.k = at(mp.cross) + (size_t)j * cross_layer * m.eb;
      ma.v = at(mp.cross) + ((size_t)j * cross_layer + (size_t)st->B * st->S * d) * m.eb;
      ma.kb = (long long)m.H * st->S * m.dh;
      ma.kh = (long long)st->S * m.dh;
      ma.ks = m.dh;
      ma.out = at(p.datt);
      ma.out_ld = d;
      ma.group_map = list;
      ma.lens = st->at<int>(p.len);
      ma.q_per_group = K;
      ma.self_queries = 0;
      ma.n_groups = st->B;
      ma.H = m.H;
      ma.dh = m.dh;
      ma.scale = 1.0f / std::sqrt((float)m.dh);
      ma.ctl = ctl;
      NT_HIP(timed(NT_K_ATTN_CROSS, s, (double)st->n_live * 2 * st->S * d * eb,
                   4.0 * R * (double)st->S * d, [&] { return nt::mha(m.dt, ma, s, 1); }));

      e = nt::GemmEpi{};
      e.mode = nt::EPI_RESID;
      e.bias = w.boc;
      e.wscale = w.soc;
      e.resid = at(p.z);
      e.out = at(p.z);
      e.ldc = d;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, at(p.datt), d, w.Woc, d, d, e));

      if (!fold)
        NT_HIP(timed(NT_K_LN, s, 2.0 * R * d * eb, 8.0 * R * d,
                     [&] { return nt::layernorm(m.dt, at(p.z), w.ln3, at(p.du), Rp, d, eps, s, ctl, K); }));

      e = nt::GemmEpi{};
      e.mode = nt::EPI_RELU;
      e.bias = w.b1;
      e.wscale = w.s1;
      e.out = at(p.df);
      e.ldc = m.F;
      e.lnf_colsum = w.c1;
      e.lnf_eps = eps;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, ln_in, d, w.W1, m.F, d, e));

      e = nt::GemmEpi{};
      e.mode = nt::EPI_RESID;
      e.bias = w.b2;
      e.wscale = w.s2;
      e.resid = at(p.z);
      e.out = at(p.z);
      e.ldc = d;
      NT_HIP(gemm_dec(NT_K_GEMM_DEC, at(p.df), m.F, w.W2, d, m.F, e));

      // the next layer's ln1 (unless folded into its QKV projection), or the output LN
      const float* next_ln = j + 1 < m.Ld ? m.dec[j + 1].ln1 : m.dec_out_ln;
      if (j + 1 == m.Ld || !fold)
        NT_HIP(timed(NT_K_LN, s, 2.0 * R * d * eb, 8.0 * R * d,
                     [&] { return nt::layernorm(m.dt, at(p.z), next_ln, at(p.du), Rp, d, eps, s, ctl, K); }));
    }

    // Tied output projection.  Its epilogue reduces each row to per-tile (max, sum exp,
    // best) records.  Greedy needs nothing else, so its logits never reach HBM.  Beam
    // ranks each row's tiles by their best entries, forms the logits of the first 2K
    // tiles again (the same kernel and k-order, so the same bits), and selects from
    // those: its logits never reach HBM either.  Teacher forcing, greedy copy-out and
    // the plain beam path (nt_set_beam_fused(0)) store the fp32 logits and scan them.
    // An ensemble member writes its logits and folds them into the combined scores.
    if (M > 1) {
      nt::GemmEpi e{};
      e.mode = nt::EPI_STORE;
      e.out = at(p.logits);
      e.ldc = m.V;
      e.out_f32 = 1;
      NT_HIP(gemm_dec(NT_K_GEMM_VOCAB, at(p.du), d, m.E, m.V, d, e));
      NT_HIP(timed(NT_K_SELECT, s, (double)R * m.V * 4 * (mi == 0 ? 2 : 3), 5.0 * R * m.V, [&] {
        return nt::ens_combine(st->at<float>(p.logits), st->at<float>(p.comb), ctl, K, Rp, m.V, mi, M, top.rule, s);
      }));
    } else if (K == 1 && !d_logits && !d_forced) {
      const int n_tiles = (m.V + 127) / 128;
      nt::GemmEpi e{};
      e.mode = nt::EPI_TOPK;
      e.part = st->at<float>(p.logits);
      e.k2 = 1;
      e.n_tiles = n_tiles;
      NT_HIP(gemm_dec(NT_K_GEMM_VOCAB, at(p.du), d, m.E, m.V, d, e));
      const float* part = st->at<float>(p.logits);
      const double pbytes = (double)R * n_tiles * nt::topk_record(1) * 4;
      NT_HIP(timed(NT_K_SELECT, s, pbytes, 0.0, [&] { return nt::greedy_step_fused(part, n_tiles, ss, s); }));
    } else if (!p.beam_pairs) {   // stored logits: teacher forcing, greedy copy-out, plain beam
      nt::GemmEpi e{};
      e.mode = nt::EPI_STORE;
      e.out = at(p.logits);
      e.ldc = m.V;
      e.out_f32 = 1;
      NT_HIP(gemm_dec(NT_K_GEMM_VOCAB, at(p.du), d, m.E, m.V, d, e));
      if (d_logits) NT_HIP(nt::scatter_logits(st->at<float>(p.logits), list, ctl, K, Rp, m.V, d_logits, s));
      if (K == 1) {
        NT_HIP(timed(NT_K_SELECT, s, (double)R * m.V * 4, 3.0 * R * m.V,
                     [&] { return nt::greedy_step(st->at<float>(p.logits), d_forced, ss, s); }));
      } else {
        NT_HIP(timed(NT_K_SELECT, s, (double)R * m.V * 4, 3.0 * R * m.V, [&] {
          return nt::beam_select(st->at<float>(p.logits), ctl, K, Rp, m.V, 2 * K, st->at<float>(p.topv),
                                 st->at<int>(p.topi), st->at<float>(p.lse), s);
        }));
        NT_HIP(timed(NT_K_SEARCH, s, (double)R * 2 * K * 8 + (double)R * t * 8, 0.0, [&] {
          return nt::beam_update(st->at<float>(p.topv), st->at<int>(p.topi), st->at<float>(p.lse), ss, s);
        }));
      }
    } else {
      // Beam without stored logits: records (and, when the caller asks, the logits copied
      // straight to its buffer), the 2K tiles of every row, their blocks, the tiles'
      // logits formed again, the row's 2K largest from them, the update.
      const int n_tiles = (m.V + 127) / 128, k2 = 2 * K;
      nt::GemmEpi e{};
      e.mode = nt::EPI_TOPK;
      e.part = st->at<float>(p.tparts);
      e.k2 = 1;
      e.n_tiles = n_tiles;
      if (d_logits) {
        e.out = d_logits;
        e.ldc = m.V;
        e.out_f32 = 1;
        e.out_map = 1;
        e.sent_list = list;
        e.beam = K;
      }
      NT_HIP(gemm_dec(NT_K_GEMM_VOCAB, at(p.du), d, m.E, m.V, d, e));
      const double rec_bytes = (double)R * n_tiles * nt::topk_record(1) * 4;
      const double pair_bytes = (double)R * k2 * 128 * 4;   // the recomputed tiles' logits
      NT_HIP(timed(NT_K_SELECT, s, rec_bytes, 0.0, [&] {
        return nt::beam_pick_tiles(st->at<float>(p.tparts), n_tiles, ctl, K, Rp, k2, st->at<int>(p.gptile),
                                   st->at<float>(p.gtau), st->at<float>(p.lse), s);
      }));
      NT_HIP(timed(NT_K_SELECT, s, (double)R * k2 * 4 * 3, 0.0, [&] {
        return nt::pair_bucket(st->at<int>(p.gptile), ctl, K, Rp, k2, n_tiles, st->at<int>(p.gsorted),
                               st->at<int>(p.gblk), st->at<int>(p.gnblk), s);
      }));
      nt::GemmEpi g{};
      g.gblk = st->at<int>(p.gblk);
      g.gnblk = st->at<int>(p.gnblk);
      g.sorted = st->at<int>(p.gsorted);
      g.pair_k = k2;
      g.out = st->at<float>(p.glog);
      NT_HIP(timed(NT_K_GEMM_VOCAB, s, pair_bytes, 2.0 * R * k2 * 128 * d,
                   [&] { return nt::gemm_pairs(m.dt, at(p.du), d, m.E, m.V, d, g, p.pair_blocks, s); }));
      NT_HIP(timed(NT_K_SELECT, s, pair_bytes, 0.0, [&] {
        return nt::beam_select_pairs(st->at<float>(p.glog), st->at<int>(p.gptile), st->at<float>(p.gtau), ctl, K,
                                     Rp, m.V, k2, st->at<float>(p.topv), st->at<int>(p.topi), s);
      }));
      NT_HIP(timed(NT_K_SEARCH, s, (double)R * 2 * K * 8 + (double)R * t * 8, 0.0, [&] {
        return nt::beam_update(st->at<float>(p.topv), st->at<int>(p.topi), st->at<float>(p.lse), ss, s);
      }));
    }
  }   // members

  if (M > 1) {   // selection over the ensemble's combined scores
    const float* sc = st->at<float>(p.comb);
    const int V = top.V;
    if (d_logits) NT_HIP(nt::scatter_logits(sc, list, ctl, K, Rp, V, d_logits, s));
    if (K == 1) {
      NT_HIP(timed(NT_K_SELECT, s, (double)R * V * 4, 3.0 * R * V,
                   [&] { return nt::greedy_step(sc, d_forced, ss, s); }));
    } else {
      NT_HIP(timed(NT_K_SELECT, s, (double)R * V * 4, 3.0 * R * V, [&] {
        return nt::beam_select(sc, ctl, K, Rp, V, 2 * K, st->at<float>(p.topv), st->at<int>(p.topi),
                               st->at<float>(p.lse), s);
      }));
      NT_HIP(timed(NT_K_SEARCH, s, (double)R * 2 * K * 8 + (double)R * t * 8, 0.0, [&] {
        return nt::beam_update(st->at<float>(p.topv), st->at<int>(p.topi), st->at<float>(p.lse), ss, s);
      }));
    }
  }
  NT_HIP(timed(NT_K_SEARCH, s, (double)st->n_live * 8, 0.0, [&] {
    return nt::step_end(list, st->at<int>(p.done), ctl, st->d_hctl, st->sc.prune, K, st->Tcap, s);
  }));
  return NT_OK;
}

// Takes in the outcome of step `step` from its mirror slot (the step must have completed).
nt_status absorb_step(nt_dec_state* st, int step) {
  const volatile int* c = st->h_ctl + (step % nt::CTL_MIRROR_SLOTS) * nt::CTL_WORDS;
  if (c[nt::CTL_T] != step + 1)
    return fail(NT_E_STATE, "internal: step %d left t=%d in the control block", step, c[nt::CTL_T]);
  st->t = c[nt::CTL_T];
  st->n_live = c[nt::CTL_NLIVE];
  st->n_alive = c[nt::CTL_NALIVE];
  if (st->n_alive == 0) st->finished = true;
  if (!st->finished && (st->t >= st->Tcap || st->n_live == 0))
    return fail(NT_E_STATE, "internal: %d sentences alive after %d steps", st->n_alive, st->t);
  return NT_OK;
}

// One step issued directly and waited for.
nt_status run_step(nt_dec_state* st, const int32_t* d_forced, float* d_logits, hipStream_t s) {
  const int step = st->t;
  NT_TRY(enqueue_step(st, d_forced, d_logits, s));
  NT_HIP(hipStreamSynchronize(s));
  return absorb_step(st, step);
}

// One step captured into an executable graph (on a private capture stream; nothing runs).
nt_status capture_step(nt_dec_state* st, hipStream_t cs, hipGraphExec_t* exec) {
  hipGraph_t graph = nullptr;
  nt_status r;
  {
    ProfModeScope nop(PROF_NONE);
    NT_HIP(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal));
    r = enqueue_step(st, nullptr, nullptr, cs);
    const hipError_t e = hipStreamEndCapture(cs, &graph);
    if (r == NT_OK && e != hipSuccess) r = fail(NT_E_DEVICE, "hipStreamEndCapture: %s", hipGetErrorString(e));
  }
  if (r != NT_OK) {
    if (graph) (void)hipGraphDestroy(graph);
    return r;
  }
  const hipError_t ie = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  NT_HIP(ie);
  return NT_OK;
}

// Pinned host memory an encode may borrow instead of allocating: with it, nt_encode's work
// is fully asynchronous on the stream (no allocation, no synchronisation).
struct EncodeHost {
  int* maxlen;   // >= B ints; read by a copy on the stream, so left untouched until it ran
  int* h_ctl;    // control-block mirror and its device-side address
  int* d_hctl;
};

nt_status encode_impl(nt_model* m, const int32_t* d_src, const int32_t* d_len, const int32_t* h_len, int B, int S,
                      const nt_search_cfg* sc, void* d_ws, size_t ws_bytes, hipStream_t s, nt_dec_state** out,
                      const EncodeHost* hx = nullptr) {
  if (!m || !d_src || !d_len || !out || !d_ws) return fail(NT_E_INVALID, "null argument to nt_encode");
  NT_TRY(validate_search(*m, sc));
  if (B <= 0 || S <= 0) return fail(NT_E_INVALID, "empty batch (B=%d, S=%d)", B, S);
  if (S > m->cfg.max_positions) return fail(NT_E_INVALID, "S=%d > max_positions=%d", S, m->cfg.max_positions);
  std::vector<int> lens(B);
  if (h_len) {
    std::memcpy(lens.data(), h_len, sizeof(int) * B);
  } else {
    NT_HIP(hipMemcpyAsync(lens.data(), d_len, sizeof(int) * B, hipMemcpyDeviceToHost, s));
    NT_HIP(hipStreamSynchronize(s));
  }
  int Tcap = 0;
  std::vector<int> maxlen_own(hx ? 0 : B);
  int* maxlen = hx ? hx->maxlen : maxlen_own.data();
  for (int b = 0; b < B; ++b) {
    if (lens[b] < 1 || lens[b] > S) return fail(NT_E_INVALID, "sentence %d has length %d outside [1, %d]", b, lens[b], S);
    maxlen[b] = max_tgt_of(*sc, lens[b]);
    if (maxlen[b] < 1) return fail(NT_E_INVALID, "max target length %d < 1", maxlen[b]);
    Tcap = std::max(Tcap, maxlen[b]);
  }
  if (Tcap > m->cfg.max_positions)
    return fail(NT_E_INVALID, "max target length %d > max_positions %d", Tcap, m->cfg.max_positions);
  const WsPlan plan = ws_plan(*m, B, S, sc->beam, Tcap);
  if (ws_bytes < plan.total)
    return fail(NT_E_WORKSPACE, "workspace too small: %zu bytes given, %zu required", ws_bytes, plan.total);
  if ((reinterpret_cast<uintptr_t>(d_ws) & (kAlign - 1)) != 0) return fail(NT_E_INVALID, "workspace must be 256-byte aligned");

  nt_dec_state* st = new nt_dec_state();
  st->m = m;
  st->sc = *sc;
  st->B = B;
  st->S = S;
  st->K = sc->beam;
  st->Tcap = Tcap;
  st->plan = plan;
  st->ws = static_cast<char*>(d_ws);
  st->n_live = B;
  st->n_alive = B;
  if (hx) {
    st->h_ctl = hx->h_ctl;
    st->d_hctl = hx->d_hctl;
    st->own_ctl = false;
  } else if (hipHostMalloc((void**)&st->h_ctl, sizeof(int) * nt::CTL_MIRROR_SLOTS * nt::CTL_WORDS,
                           hipHostMallocCoherent | hipHostMallocMapped) != hipSuccess ||
             hipHostGetDevicePointer((void**)&st->d_hctl, st->h_ctl, 0) != hipSuccess) {
    if (st->h_ctl) (void)hipHostFree(st->h_ctl);
    delete st;
    return fail(NT_E_DEVICE, "pinned control-block mirror: hipHostMalloc / hipHostGetDevicePointer failed");
  }
  auto bail = [&](nt_status code) {
    if (st->own_ctl) (void)hipHostFree(st->h_ctl);
    delete st;
    return code;
  };
  auto chk = [&](hipError_t e, const char* what) -> nt_status {
    if (e == hipSuccess) return NT_OK;
    return bail(fail(NT_E_DEVICE, "%s: %s", what, hipGetErrorString(e)));
  };
  nt_status r;
  if (d_src != st->at<int>(plan.src) &&
      (r = chk(hipMemcpyAsync(st->at<int>(plan.src), d_src, sizeof(int) * (size_t)B * S, hipMemcpyDeviceToDevice, s),
               "copy src")) != NT_OK)
    return r;
  if (d_len != st->at<int>(plan.len) &&
      (r = chk(hipMemcpyAsync(st->at<int>(plan.len), d_len, sizeof(int) * B, hipMemcpyDeviceToDevice, s), "copy len")) != NT_OK)
    return r;
  if ((r = chk(hipMemcpyAsync(st->at<int>(plan.maxlen), maxlen, sizeof(int) * B, hipMemcpyHostToDevice, s),
               "copy maxlen")) != NT_OK)
    return r;
  if (st->K > 1 &&
      (r = chk(hipMemsetAsync(st->at<int>(plan.anc), 0, sizeof(int) * 2 * (size_t)B * st->K * Tcap, s), "clear anc")) != NT_OK)
    return r;
  for (int i = 0; i < n_members(*m); ++i)
    if ((r = run_encoder(st, i, s)) != NT_OK) return bail(r);
  if ((r = chk(nt::search_init(st->search(), st->list(), st->ctl(), m->cfg.bos_id, s), "search init")) != NT_OK) return r;
  // an owned host copy of maxlen must not be freed before the copy has run
  if (!hx && (r = chk(hipStreamSynchronize(s), "sync")) != NT_OK) return r;
  *out = st;
  return NT_OK;
}

nt_status read_impl(nt_dec_state* st, int32_t* h_tokens, int32_t* h_lens, float* h_scores, float* h_token_logp,
                    hipStream_t s) {
  if (!st) return fail(NT_E_INVALID, "null state");
  if (!st->finished) return fail(NT_E_STATE, "%d sentences are still decoding", st->n_alive);
  const WsPlan& p = st->plan;
  NT_HIP(nt::finalize(st->search(), st->at<int>(p.out_tok), st->at<float>(p.out_lp), st->at<int>(p.out_len),
                      st->at<float>(p.out_score), s));
  const size_t n = (size_t)st->B * st->Tcap;
  if (h_tokens) NT_HIP(hipMemcpyAsync(h_tokens, st->at<int>(p.out_tok), n * 4, hipMemcpyDeviceToHost, s));
  if (h_token_logp) NT_HIP(hipMemcpyAsync(h_token_logp, st->at<float>(p.out_lp), n * 4, hipMemcpyDeviceToHost, s));
  if (h_lens) NT_HIP(hipMemcpyAsync(h_lens, st->at<int>(p.out_len), st->B * 4, hipMemcpyDeviceToHost, s));
  if (h_scores) NT_HIP(hipMemcpyAsync(h_scores, st->at<float>(p.out_score), st->B * 4, hipMemcpyDeviceToHost, s));
  NT_HIP(hipStreamSynchronize(s));
  return NT_OK;
}

void free_state(nt_dec_state* st) {
  if (!st) return;
  if (st->own_ctl && st->h_ctl) (void)hipHostFree(st->h_ctl);
  delete st;
}

// ---- dynamic batching (Sec. 4.2) ----------------------------------------------------------
struct Batch {
  int first, count, S, Tcap;   // a run of the length-sorted order
};

std::vector<Batch> plan_batches(const std::vector<int>& order, const std::vector<int>& lens, const nt_search_cfg& sc) {
  std::vector<Batch> out;
  const int n = (int)order.size();
  int i = 0;
  while (i < n) {
    const int S = lens[order[i]];
    int cnt = 1;
    while (i + cnt < n) {
      if (sc.token_budget > 0 && (long long)(cnt + 1) * S > sc.token_budget) break;
      if (sc.max_batch_sents > 0 && cnt + 1 > sc.max_batch_sents) break;
      ++cnt;
    }
    out.push_back({i, cnt, S, max_tgt_of(sc, S)});
    i += cnt;
  }
  return out;
}

nt_status validate_sources(const nt_model& m, const nt_search_cfg& sc, const int32_t* h_src, const int64_t* off,
                           int n_sent, std::vector<int>& lens, bool check_ids) {
  if (!off || n_sent <= 0) return fail(NT_E_INVALID, "n_sent must be > 0 with offsets");
  if (off[0] != 0) return fail(NT_E_INVALID, "h_src_off[0] must be 0");
  lens.resize(n_sent);
  for (int i = 0; i < n_sent; ++i) {
    const int64_t L = off[i + 1] - off[i];
    if (L <= 0) return fail(NT_E_INVALID, "sentence %d is empty", i);
    if (L > m.cfg.max_positions) return fail(NT_E_INVALID, "sentence %d has %lld tokens > max_positions %d", i, (long long)L, m.cfg.max_positions);
    lens[i] = (int)L;
    const int mt = max_tgt_of(sc, (int)L);
    if (mt < 1 || mt > m.cfg.max_positions)
      return fail(NT_E_INVALID, "sentence %d: max target length %d outside [1, max_positions=%d]", i, mt, m.cfg.max_positions);
  }
  if (check_ids) {
    if (!h_src) return fail(NT_E_INVALID, "null h_src");
    for (int64_t k = 0; k < off[n_sent]; ++k)
      if (h_src[k] < 0 || h_src[k] >= m.V)
        return fail(NT_E_INVALID, "token id %d at position %lld outside [0, %d)", h_src[k], (long long)k, m.V);
  }
  return NT_OK;
}

std::vector<int> length_order(const std::vector<int>& lens) {
  std::vector<int> order(lens.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return lens[a] > lens[b]; });
  return order;
}

}  // namespace

// ======================================================================================
// C ABI
extern "C" {

const char* nt_last_error(void) { return g_err.c_str(); }

nt_status nt_weights_size(const nt_model_cfg* cfg, size_t* host_floats, size_t* device_bytes) {
  g_err.clear();
  NT_TRY(validate_cfg(cfg));
  const ModelLayout Lo = layout_of(*cfg);
  if (host_floats) *host_floats = Lo.host_floats;
  if (device_bytes) *device_bytes = Lo.total;
  return NT_OK;
}

nt_status nt_load_weights(const nt_model_cfg* cfg, const float* host_weights, size_t host_floats, void* device_buf,
                          size_t device_bytes, void* stream, nt_model** out) {
  g_err.clear();
  NT_TRY(validate_cfg(cfg));
  if (!host_weights || !device_buf || !out) return fail(NT_E_INVALID, "null argument to nt_load_weights");
  const ModelLayout Lo = layout_of(*cfg);
  if (host_floats != Lo.host_floats)
    return fail(NT_E_INVALID, "weight blob has %zu floats, the model needs %zu", host_floats, Lo.host_floats);
  if (device_bytes < Lo.total) return fail(NT_E_WORKSPACE, "weight buffer too small: %zu bytes given, %zu required", device_bytes, Lo.total);
  if ((reinterpret_cast<uintptr_t>(device_buf) & (kAlign - 1)) != 0) return fail(NT_E_INVALID, "weight buffer must be 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DT dt = static_cast<DT>(cfg->dtype);
  const int d = cfg->d_model, F = cfg->d_ffn, V = cfg->vocab, L = cfg->n_enc, Ld = cfg->n_dec;
  char* base = static_cast<char*>(device_buf);

  float* staging = nullptr;
  NT_HIP(hipMalloc((void**)&staging, Lo.host_floats * sizeof(float)));
  struct Guard {
    float* p;
    ~Guard() { if (p) (void)hipFree(p); }
  } guard{staging};
  NT_HIP(hipMemcpyAsync(staging, host_weights, Lo.host_floats * sizeof(float), hipMemcpyHostToDevice, s));

  auto vec = [&](size_t dev_off, size_t host_off, size_t n) -> hipError_t {
    return hipMemcpyAsync(base + dev_off, staging + host_off, n * 4, hipMemcpyDeviceToDevice, s);
  };
  // a projection matrix: transposed to [out][in] in the model dtype, or quantized to FP8
  // on the host (its codes and column scales copied in; the buffers stay alive until
  // the stream is synchronised below)
  const bool f8 = cfg->fp8_weights != 0;
  std::vector<std::vector<uint8_t>> keep_q;
  std::vector<std::vector<float>> keep_s;
  auto mat = [&](size_t dev_off, size_t host_off, int in, int outn, size_t scale_off) -> hipError_t {
    if (!f8) return nt::pack_transpose(dt, staging + host_off, base + dev_off, in, outn, s);
    keep_q.emplace_back();
    keep_s.emplace_back();
    quantize_fp8(host_weights + host_off, in, outn, keep_q.back(), keep_s.back());
    hipError_t e = hipMemcpyAsync(base + dev_off, keep_q.back().data(), keep_q.back().size(), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
    return hipMemcpyAsync(base + scale_off, keep_s.back().data(), keep_s.back().size() * 4, hipMemcpyHostToDevice, s);
  };
  // A pre-norm LayerNorm folded into the projection it feeds (decoder layers):
  // LN(x) W + b = rstd (x W' - mean colsum(W')) + b' with W' = diag(gamma) W and
  // b' = b + beta W.  W' (fp32 products) replaces W in the staging copy before packing, b'
  // is summed in double, and the column sums come from the packed matrix, so they are
  // those of the values the GEMM multiplies.  With FP8 weights W' is what is quantized
  // (per output column), and the column sums are those of the dequantized codes.
  std::deque<std::vector<float>> keep_f;   // element references stay valid as it grows
  auto folded = [&](size_t dev_w, size_t dev_b, size_t dev_c, size_t hw, size_t hb, size_t hln, int in,
                    int outn, size_t scale_off) -> hipError_t {
    const float* W = host_weights + hw;
    const float* g = host_weights + hln;
    const float* be = host_weights + hln + in;
    keep_f.emplace_back((size_t)in * outn);
    std::vector<float>& Wf = keep_f.back();
    for (int k = 0; k < in; ++k)
      for (int n = 0; n < outn; ++n) Wf[(size_t)k * outn + n] = g[k] * W[(size_t)k * outn + n];
    keep_f.emplace_back(outn);
    std::vector<float>& bf = keep_f.back();
    for (int n = 0; n < outn; ++n) {
      double acc = host_weights[hb + n];
      for (int k = 0; k < in; ++k) acc += (double)be[k] * W[(size_t)k * outn + n];
      bf[n] = (float)acc;
    }
    hipError_t e = hipMemcpyAsync(base + dev_b, bf.data(), bf.size() * 4, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return e;
    if (f8) {
      keep_q.emplace_back();
      keep_s.emplace_back();
      quantize_fp8(Wf.data(), in, outn, keep_q.back(), keep_s.back());
      const std::vector<uint8_t>& q = keep_q.back();
      const std::vector<float>& sc = keep_s.back();
      keep_f.emplace_back(outn);
      std::vector<float>& cs = keep_f.back();
      for (int n = 0; n < outn; ++n) {
        double acc = 0.0;
        for (int k = 0; k < in; ++k) acc += e4m3_value(q[(size_t)n * in + k]);
        cs[n] = (float)(acc * (double)sc[n]);
      }
      e = hipMemcpyAsync(base + dev_w, q.data(), q.size(), hipMemcpyHostToDevice, s);
      if (e == hipSuccess) e = hipMemcpyAsync(base + scale_off, sc.data(), sc.size() * 4, hipMemcpyHostToDevice, s);
      if (e == hipSuccess) e = hipMemcpyAsync(base + dev_c, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, s);
      return e;
    }
    e = hipMemcpyAsync(staging + hw, Wf.data(), Wf.size() * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = nt::pack_transpose(dt, staging + hw, base + dev_w, in, outn, s);
    if (e == hipSuccess) e = nt::packed_row_sums(dt, base + dev_w, outn, in, reinterpret_cast<float*>(base + dev_c), s);
    return e;
  };
  NT_HIP(nt::pack_convert(dt, staging + Lo.hE, base + Lo.E, (size_t)V * d, s));
  NT_HIP(vec(Lo.hist_ln, Lo.hhist, (size_t)(L + 1) * 2 * d));
  NT_HIP(vec(Lo.dlcl, Lo.hdlcl, (size_t)(L + 1) * (L + 2) / 2));
  for (int i = 0; i < L; ++i) {
    const auto& D = Lo.enc[i];
    const auto& Hh = Lo.henc[i];
    NT_HIP(vec(D.ln1, Hh.ln1, 2 * d));
    NT_HIP(mat(D.Wqkv, Hh.Wqkv, d, 3 * d, D.sqkv));
    NT_HIP(vec(D.bqkv, Hh.bqkv, 3 * d));
    NT_HIP(mat(D.Wo, Hh.Wo, d, d, D.so));
    NT_HIP(vec(D.bo, Hh.bo, d));
    NT_HIP(vec(D.ln2, Hh.ln2, 2 * d));
    NT_HIP(mat(D.W1, Hh.W1, d, F, D.s1));
    NT_HIP(vec(D.b1, Hh.b1, F));
    NT_HIP(mat(D.W2, Hh.W2, F, d, D.s2));
    NT_HIP(vec(D.b2, Hh.b2, d));
    if (cfg->rel_pos_k > 0) {
      const size_t rn = (2 * (size_t)cfg->rel_pos_k + 1) * (d / cfg->n_heads);
      NT_HIP(vec(D.relk, Hh.relk, rn));
      NT_HIP(vec(D.relv, Hh.relv, rn));
    }
  }
  NT_HIP(vec(Lo.enc_out_ln, Lo.henc_out, 2 * d));
  const size_t eb = dt == DT::F32 ? 4 : 2;
  for (int j = 0; j < Ld; ++j) {
    const auto& D = Lo.dec[j];
    const auto& Hh = Lo.hdec[j];
    NT_HIP(vec(D.ln1, Hh.ln1, 2 * d));
    NT_HIP(vec(D.ln2, Hh.ln2, 2 * d));
    NT_HIP(vec(D.ln3, Hh.ln3, 2 * d));
    NT_HIP(folded(D.Wqkv, D.bqkv, D.cqkv, Hh.Wqkv, Hh.bqkv, Hh.ln1, d, 3 * d, D.sqkv));
    NT_HIP(folded(D.Wq, D.bq, D.cq, Hh.Wq, Hh.bq, Hh.ln2, d, d, D.sq));
    NT_HIP(folded(D.W1, D.b1, D.c1, Hh.W1, Hh.b1, Hh.ln3, d, F, D.s1));
    NT_HIP(mat(D.Wo, Hh.Wo, d, d, D.so));
    NT_HIP(vec(D.bo, Hh.bo, d));
    NT_HIP(mat(D.Woc, Hh.Woc, d, d, D.soc));
    NT_HIP(vec(D.boc, Hh.boc, d));
    NT_HIP(mat(D.W2, Hh.W2, F, d, D.s2));
    NT_HIP(vec(D.b2, Hh.b2, d));
    // cross K/V projections of all layers stacked into one [Ld*2d][d] matrix
    const size_t mb = f8 ? 1 : eb;
    NT_HIP(mat(Lo.Wkv_all + (size_t)j * 2 * d * d * mb, Hh.Wkv, d, 2 * d, Lo.skv_all + (size_t)j * 2 * d * 4));
    NT_HIP(vec(Lo.bkv_all + (size_t)j * 2 * d * 4, Hh.bkv, 2 * d));
  }
  NT_HIP(vec(Lo.dec_out_ln, Lo.hdec_out, 2 * d));

  // sinusoidal positions, PE(p, 2i) = sin(p / 10000^(2i/d)), PE(p, 2i+1) = cos(same)
  std::vector<float> pe((size_t)cfg->max_positions * d);
  for (int pos = 0; pos < cfg->max_positions; ++pos)
    for (int i = 0; i < d / 2; ++i) {
      const double ang = pos / std::pow(10000.0, 2.0 * i / d);
      pe[(size_t)pos * d + 2 * i] = (float)std::sin(ang);
      pe[(size_t)pos * d + 2 * i + 1] = (float)std::cos(ang);
    }
  NT_HIP(hipMemcpyAsync(base + Lo.pe, pe.data(), pe.size() * 4, hipMemcpyHostToDevice, s));
  NT_HIP(hipStreamSynchronize(s));

  nt_model* m = new nt_model();
  m->cfg = *cfg;
  m->dt = dt;
  m->eb = eb;
  m->d = d;
  m->H = cfg->n_heads;
  m->dh = d / cfg->n_heads;
  m->F = F;
  m->L = L;
  m->Ld = Ld;
  m->V = V;
  auto fp = [&](size_t o) { return reinterpret_cast<const float*>(base + o); };
  m->E = base + Lo.E;
  m->pe = fp(Lo.pe);
  m->hist_ln = fp(Lo.hist_ln);
  m->dlcl = fp(Lo.dlcl);
  for (int i = 0; i < L; ++i) {
    const auto& D = Lo.enc[i];
    m->enc.push_back({fp(D.ln1), fp(D.bqkv), fp(D.bo), fp(D.ln2), fp(D.b1), fp(D.b2), base + D.Wqkv, base + D.Wo,
                      base + D.W1, base + D.W2, cfg->rel_pos_k > 0 ? fp(D.relk) : nullptr,
                      cfg->rel_pos_k > 0 ? fp(D.relv) : nullptr});
    if (f8) {
      EncLayerW& w = m->enc.back();
      w.sqkv = fp(D.sqkv);
      w.so = fp(D.so);
      w.s1 = fp(D.s1);
      w.s2 = fp(D.s2);
    }
  }
  m->enc_out_ln = fp(Lo.enc_out_ln);
  for (int j = 0; j < Ld; ++j) {
    const auto& D = Lo.dec[j];
    m->dec.push_back({fp(D.ln1), fp(D.bqkv), fp(D.bo), fp(D.ln2), fp(D.bq), fp(D.boc), fp(D.ln3), fp(D.b1), fp(D.b2),
                      base + D.Wqkv, base + D.Wo, base + D.Wq, base + D.Woc, base + D.W1, base + D.W2});
    {
      DecLayerW& w = m->dec.back();
      w.cqkv = fp(D.cqkv);
      w.cq = fp(D.cq);
      w.c1 = fp(D.c1);
    }
    if (f8) {
      DecLayerW& w = m->dec.back();
      w.sqkv = fp(D.sqkv);
      w.so = fp(D.so);
      w.sq = fp(D.sq);
      w.soc = fp(D.soc);
      w.s1 = fp(D.s1);
      w.s2 = fp(D.s2);
    }
  }
  m->Wkv_all = base + Lo.Wkv_all;
  m->bkv_all = fp(Lo.bkv_all);
  m->skv_all = f8 ? fp(Lo.skv_all) : nullptr;
  m->dec_out_ln = fp(Lo.dec_out_ln);
  *out = m;
  return NT_OK;
}

void nt_free_model(nt_model* m) { delete m; }

nt_status nt_ensemble(nt_model* const* members, int32_t n_members, int32_t rule, nt_model** out) {
  g_err.clear();
  if (!members || !out) return fail(NT_E_INVALID, "null argument to nt_ensemble");
  if (n_members < 1 || n_members > 8) return fail(NT_E_INVALID, "an ensemble has 1..8 members, not %d", n_members);
  if (rule != NT_ENS_MEAN_LOGP && rule != NT_ENS_LOG_MEAN_P) return fail(NT_E_INVALID, "unknown ensemble rule %d", rule);
  int max_pos = 0;
  for (int i = 0; i < n_members; ++i) {
    const nt_model* mi = members[i];
    if (!mi) return fail(NT_E_INVALID, "ensemble member %d is null", i);
    if (!mi->members.empty()) return fail(NT_E_INVALID, "ensemble member %d is itself an ensemble", i);
    const nt_model_cfg &c = mi->cfg, &c0 = members[0]->cfg;
    if (c.vocab != c0.vocab || c.pad_id != c0.pad_id || c.bos_id != c0.bos_id || c.eos_id != c0.eos_id ||
        c.dtype != c0.dtype)
      return fail(NT_E_INVALID, "ensemble member %d differs from member 0 in vocab, special IDs or dtype", i);
    max_pos = i == 0 ? c.max_positions : std::min(max_pos, c.max_positions);
  }
  nt_model* e = new nt_model();
  *e = *members[0];   // vocabulary, special IDs and dtype; no weights are used through it
  e->cfg.max_positions = max_pos;
  e->enc.clear();
  e->dec.clear();
  e->members.assign(members, members + n_members);
  e->rule = rule;
  *out = e;
  return NT_OK;
}

nt_status nt_workspace_size(const nt_model* m, const nt_search_cfg* search, int32_t max_sents, int32_t max_src,
                            size_t* bytes) {
  g_err.clear();
  if (!m || !bytes) return fail(NT_E_INVALID, "null argument to nt_workspace_size");
  NT_TRY(validate_search(*m, search));
  if (max_sents <= 0 || max_src <= 0) return fail(NT_E_INVALID, "max_sents and max_src must be > 0");
  const int Tcap = std::max(1, max_tgt_of(*search, max_src));
  *bytes = ws_plan(*m, max_sents, max_src, search->beam, Tcap).total;
  return NT_OK;
}

nt_status nt_translate_workspace_size(const nt_model* m, const nt_search_cfg* search, const int64_t* h_src_off,
                                      int32_t n_sent, size_t* bytes) {
  g_err.clear();
  if (!m || !bytes) return fail(NT_E_INVALID, "null argument to nt_translate_workspace_size");
  NT_TRY(validate_search(*m, search));
  std::vector<int> lens;
  NT_TRY(validate_sources(*m, *search, nullptr, h_src_off, n_sent, lens, false));
  const auto order = length_order(lens);
  const auto batches = plan_batches(order, lens, *search);
  size_t slot = 0;
  for (const Batch& b : batches) slot = std::max(slot, align_up(ws_plan(*m, b.count, b.S, search->beam, b.Tcap).total));
  *bytes = slot * (size_t)std::min<int>(g_streams.load(), (int)batches.size());
  return NT_OK;
}

nt_status nt_encode(nt_model* m, const int32_t* d_src, const int32_t* d_len, const int32_t* h_len, int32_t B, int32_t S,
                    const nt_search_cfg* search, void* d_ws, size_t ws_bytes, void* stream, nt_dec_state** st) {
  g_err.clear();
  return encode_impl(m, d_src, d_len, h_len, B, S, search, d_ws, ws_bytes, static_cast<hipStream_t>(stream), st);
}

nt_status nt_decode_step(nt_dec_state* st, const int32_t* d_forced, float* d_logits, int32_t* h_alive, void* stream) {
  g_err.clear();
  if (!st) return fail(NT_E_INVALID, "null state");
  if (st->finished) return fail(NT_E_STATE, "every sentence has finished");
  if (d_forced && st->K != 1) return fail(NT_E_UNSUPPORTED, "teacher forcing needs beam 1");
  NT_TRY(run_step(st, d_forced, d_logits, static_cast<hipStream_t>(stream)));
  if (h_alive) *h_alive = st->n_alive;
  return NT_OK;
}

nt_status nt_dec_state_read(nt_dec_state* st, int32_t* h_tokens, int32_t* h_lens, float* h_scores, float* h_token_logp,
                            void* stream) {
  g_err.clear();
  return read_impl(st, h_tokens, h_lens, h_scores, h_token_logp, static_cast<hipStream_t>(stream));
}

nt_status nt_dec_state_info(const nt_dec_state* st, int32_t* B, int32_t* S, int32_t* beam, int32_t* max_tgt,
                            int32_t* steps, int32_t* alive) {
  g_err.clear();
  if (!st) return fail(NT_E_INVALID, "null state");
  if (B) *B = st->B;
  if (S) *S = st->S;
  if (beam) *beam = st->K;
  if (max_tgt) *max_tgt = st->Tcap;
  if (steps) *steps = st->t;
  if (alive) *alive = st->n_alive;
  return NT_OK;
}

nt_status nt_dec_state_encoder_out(nt_dec_state* st, float* h_enc, void* stream) {
  g_err.clear();
  if (!st || !h_enc) return fail(NT_E_INVALID, "null argument");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const nt_model& m = member(*st->m, 0);
  const size_t n = (size_t)st->B * st->S * m.d;
  std::vector<char> raw(n * m.eb);
  NT_HIP(hipMemcpyAsync(raw.data(), st->ws + st->plan.mem[0].enc_out, raw.size(), hipMemcpyDeviceToHost, s));
  NT_HIP(hipStreamSynchronize(s));
  for (size_t i = 0; i < n; ++i) {
    if (m.dt == DT::F32) {
      h_enc[i] = reinterpret_cast<const float*>(raw.data())[i];
    } else if (m.dt == DT::F16) {
      h_enc[i] = (float)reinterpret_cast<const _Float16*>(raw.data())[i];
    } else {
      uint32_t u = (uint32_t)reinterpret_cast<const uint16_t*>(raw.data())[i] << 16;
      std::memcpy(&h_enc[i], &u, 4);
    }
  }
  return NT_OK;
}

void nt_free_state(nt_dec_state* st) { free_state(st); }

nt_status nt_translate(nt_model* m, const nt_search_cfg* search, const int32_t* h_src, const int64_t* h_src_off,
                       int32_t n_sent, int32_t* h_out, int64_t out_cap, int64_t* h_out_off, float* h_score,
                       float* h_tok_logp, void* d_ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  if (!m || !h_out || !h_out_off || !d_ws) return fail(NT_E_INVALID, "null argument to nt_translate");
  NT_TRY(validate_search(*m, search));
  std::vector<int> lens;
  NT_TRY(validate_sources(*m, *search, h_src, h_src_off, n_sent, lens, true));
  if ((reinterpret_cast<uintptr_t>(d_ws) & (kAlign - 1)) != 0) return fail(NT_E_INVALID, "workspace must be 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const auto order = length_order(lens);
  const auto batches = plan_batches(order, lens, *search);
  const int nb = (int)batches.size();
  size_t slot_bytes = 0;
  int maxB = 0, maxBS = 0, maxBT = 0;
  for (const Batch& b : batches) {
    slot_bytes = std::max(slot_bytes, align_up(ws_plan(*m, b.count, b.S, search->beam, b.Tcap).total));
    maxB = std::max(maxB, b.count);
    maxBS = std::max(maxBS, b.count * b.S);
    maxBT = std::max(maxBT, b.count * b.Tcap);
  }
  if (ws_bytes < slot_bytes)
    return fail(NT_E_WORKSPACE, "workspace too small: %zu bytes given, %zu required", ws_bytes, slot_bytes);
  // batches decoded at once: as many as the setting asks and the workspace holds
  const int NS = (int)std::min<size_t>({(size_t)g_streams.load(), ws_bytes / slot_bytes, (size_t)nb});
  const bool graphs = g_use_graphs;

  // per-slot resources: stream, step events, workspace slice, pinned staging and mirror
  struct Slot {
    hipStream_t s = nullptr;
    hipStream_t cs = nullptr;           // graph capture stream
    hipEvent_t ev[nt::CTL_MIRROR_SLOTS] = {};
    hipGraphExec_t exec = nullptr;
    char* ws = nullptr;
    int *p_src, *p_len, *p_maxlen, *p_olen, *p_otok, *h_ctl, *d_hctl;
    float *p_oscore, *p_olp;
    nt_dec_state* st = nullptr;
    int batch = -1, issued = 0, read = 0;
    bool sampled = false;               // the next step is a timing sample
  };
  struct Res {
    std::vector<Slot> slots;
    void* pin = nullptr;
    int* mirror = nullptr;
    hipEvent_t start = nullptr;
    ~Res() {
      // Every slot's queued work (a replayed step may still be running on an error path)
      // completes before anything it uses is released.
      for (Slot& sl : slots)
        if (sl.s) (void)hipStreamSynchronize(sl.s);
      for (Slot& sl : slots) {
        if (sl.st) free_state(sl.st);
        if (sl.exec) (void)hipGraphExecDestroy(sl.exec);
        for (auto e : sl.ev)
          if (e) (void)hipEventDestroy(e);
        if (sl.cs) (void)hipStreamDestroy(sl.cs);
        if (sl.s) (void)hipStreamDestroy(sl.s);
      }
      if (start) (void)hipEventDestroy(start);
      if (pin) (void)hipHostFree(pin);
      if (mirror) (void)hipHostFree(mirror);
    }
  } res;
  const size_t stage_ints = (size_t)maxBS + 4 * (size_t)maxB + 2 * (size_t)maxBT;
  NT_HIP(hipHostMalloc(&res.pin, stage_ints * 4 * NS, hipHostMallocDefault));
  const size_t mir_ints = (size_t)nt::CTL_MIRROR_SLOTS * nt::CTL_WORDS;
  NT_HIP(hipHostMalloc((void**)&res.mirror, mir_ints * 4 * NS, hipHostMallocCoherent | hipHostMallocMapped));
  int* d_mirror = nullptr;
  NT_HIP(hipHostGetDevicePointer((void**)&d_mirror, res.mirror, 0));
  NT_HIP(hipEventCreateWithFlags(&res.start, hipEventDisableTiming));
  NT_HIP(hipEventRecord(res.start, s));   // work already on the caller's stream comes first
  res.slots.resize(NS);
  for (int i = 0; i < NS; ++i) {
    Slot& sl = res.slots[i];
    NT_HIP(hipStreamCreateWithFlags(&sl.s, hipStreamNonBlocking));
    if (graphs) NT_HIP(hipStreamCreateWithFlags(&sl.cs, hipStreamNonBlocking));
    for (auto& e : sl.ev) NT_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming | hipEventReleaseToSystem));
    NT_HIP(hipStreamWaitEvent(sl.s, res.start, 0));
    sl.ws = static_cast<char*>(d_ws) + (size_t)i * slot_bytes;
    int* q = static_cast<int*>(res.pin) + (size_t)i * stage_ints;
    sl.p_src = q;
    sl.p_len = sl.p_src + maxBS;
    sl.p_maxlen = sl.p_len + maxB;
    sl.p_olen = sl.p_maxlen + maxB;
    sl.p_oscore = reinterpret_cast<float*>(sl.p_olen + maxB);
    sl.p_otok = reinterpret_cast<int*>(sl.p_oscore + maxB);
    sl.p_olp = reinterpret_cast<float*>(sl.p_otok + maxBT);
    sl.h_ctl = res.mirror + (size_t)i * mir_ints;
    sl.d_hctl = d_mirror + (size_t)i * mir_ints;
  }

  std::vector<std::vector<int>> res_tok(n_sent);
  std::vector<std::vector<float>> res_lp(n_sent);
  std::vector<float> res_score(n_sent);

  // inputs of a batch into its slot's staging and workspace, then the (asynchronous) encode
  auto start_batch = [&](Slot& sl, int bi) -> nt_status {
    const Batch& bt = batches[bi];
    const int B = bt.count, S = bt.S;
    for (int i = 0; i < B; ++i) {
      const int sid = order[bt.first + i];
      const int L = lens[sid];
      sl.p_len[i] = L;
      std::memcpy(sl.p_src + (size_t)i * S, h_src + h_src_off[sid], sizeof(int) * L);
      std::fill(sl.p_src + (size_t)i * S + L, sl.p_src + (size_t)(i + 1) * S, m->cfg.pad_id);
    }
    const WsPlan plan = ws_plan(*m, B, S, search->beam, bt.Tcap);
    NT_HIP(hipMemcpyAsync(sl.ws + plan.src, sl.p_src, sizeof(int) * (size_t)B * S, hipMemcpyHostToDevice, sl.s));
    NT_HIP(hipMemcpyAsync(sl.ws + plan.len, sl.p_len, sizeof(int) * B, hipMemcpyHostToDevice, sl.s));
    const EncodeHost hx{sl.p_maxlen, sl.h_ctl, sl.d_hctl};
    NT_TRY(encode_impl(m, reinterpret_cast<int*>(sl.ws + plan.src), reinterpret_cast<int*>(sl.ws + plan.len), sl.p_len,
                       B, S, search, sl.ws, slot_bytes, sl.s, &sl.st, &hx));
    if (graphs) NT_TRY(capture_step(sl.st, sl.cs, &sl.exec));
    sl.batch = bi;
    sl.issued = sl.read = 0;
    sl.sampled = prof_unit_sampled(false);
    return NT_OK;
  };
  // results of a finished batch back to the host, in input order
  auto finish_batch = [&](Slot& sl) -> nt_status {
    const Batch& bt = batches[sl.batch];
    NT_TRY(read_impl(sl.st, sl.p_otok, sl.p_olen, sl.p_oscore, sl.p_olp, sl.s));
    const int Tcap = sl.st->Tcap;
    for (int i = 0; i < bt.count; ++i) {
      const int sid = order[bt.first + i];
      res_tok[sid].assign(sl.p_otok + (size_t)i * Tcap, sl.p_otok + (size_t)i * Tcap + sl.p_olen[i]);
      res_lp[sid].assign(sl.p_olp + (size_t)i * Tcap, sl.p_olp + (size_t)i * Tcap + sl.p_olen[i]);
      res_score[sid] = sl.p_oscore[i];
    }
    free_state(sl.st);
    sl.st = nullptr;
    if (sl.exec) {
      (void)hipGraphExecDestroy(sl.exec);
      sl.exec = nullptr;
    }
    return NT_OK;
  };

  // Outcome of a slot's oldest step in flight (which must have completed or be waited for).
  int finished = 0;
  auto absorb_oldest = [&](Slot& sl) -> nt_status {
    NT_HIP(hipEventSynchronize(sl.ev[sl.read % nt::CTL_MIRROR_SLOTS]));
    NT_TRY(absorb_step(sl.st, sl.st->t));
    ++sl.read;
    if (sl.st->finished) {
      NT_TRY(finish_batch(sl));
      ++finished;
    }
    return NT_OK;
  };
  // Everything queued on every slot completes (before a timing sample runs alone).
  auto drain = [&]() -> nt_status {
    for (Slot& o : res.slots) {
      NT_HIP(hipStreamSynchronize(o.s));
      while (o.st && o.issued > o.read) NT_TRY(absorb_oldest(o));
    }
    return NT_OK;
  };

  // Scheduler: every slot keeps up to two decoder steps in flight on its own stream, so
  // the small kernels of one batch's step overlap those of the others; the host reads a
  // step's outcome (the control-block mirror) while later steps run.  A step issued after
  // its batch's last one finds nothing live and does nothing.  Kernel timing (when
  // enabled) only ever covers sampled units, each run alone.
  ProfModeScope untimed(PROF_NONE);
  constexpr int depth = 2;   // steps in flight per slot (3 or 4 measured the same)
  int next = 0, rr = 0;
  while (finished < nb) {
    bool progressed = false;
    for (Slot& sl : res.slots) {
      if (!sl.st && next < nb) {
        if (prof_unit_sampled(true)) {
          NT_TRY(drain());
          ProfModeScope all(PROF_ALL);
          NT_TRY(start_batch(sl, next++));
          NT_HIP(hipStreamSynchronize(sl.s));
        } else {
          NT_TRY(start_batch(sl, next++));
        }
        progressed = true;
      }
      if (!sl.st || sl.st->finished || sl.issued - sl.read >= depth) continue;
      if (sl.sampled) {
        if (sl.issued != sl.read) continue;          // wait for this slot's steps first
        NT_TRY(drain());
        if (!sl.st || sl.st->finished) continue;
        {
          ProfModeScope all(PROF_ALL);
          NT_TRY(enqueue_step(sl.st, nullptr, nullptr, sl.s));
        }
        NT_HIP(hipEventRecord(sl.ev[sl.issued % nt::CTL_MIRROR_SLOTS], sl.s));
        ++sl.issued;
        NT_TRY(absorb_oldest(sl));
      } else {
        if (graphs) NT_HIP(hipGraphLaunch(sl.exec, sl.s));
        else NT_TRY(enqueue_step(sl.st, nullptr, nullptr, sl.s));
        NT_HIP(hipEventRecord(sl.ev[sl.issued % nt::CTL_MIRROR_SLOTS], sl.s));
        ++sl.issued;
      }
      if (sl.st) sl.sampled = prof_unit_sampled(false);
      progressed = true;
    }
    if (progressed) continue;
    // wait for the oldest step of the next slot (round robin) that has one in flight
    for (int k = 0; k < NS; ++k) {
      Slot& sl = res.slots[(rr + k) % NS];
      if (!sl.st || sl.issued == sl.read) continue;
      rr = (rr + k + 1) % NS;
      NT_TRY(absorb_oldest(sl));
      break;
    }
  }
  for (Slot& sl : res.slots) {
    hipEvent_t e = sl.ev[0];
    NT_HIP(hipEventRecord(e, sl.s));
    NT_HIP(hipStreamWaitEvent(s, e, 0));   // later work on the caller's stream follows ours
  }

  int64_t total = 0;
  for (int i = 0; i < n_sent; ++i) total += (int64_t)res_tok[i].size();
  if (total > out_cap) return fail(NT_E_INVALID, "out_cap %lld too small: %lld output tokens", (long long)out_cap, (long long)total);
  int64_t o = 0;
  h_out_off[0] = 0;
  for (int i = 0; i < n_sent; ++i) {
    std::copy(res_tok[i].begin(), res_tok[i].end(), h_out + o);
    if (h_tok_logp) std::copy(res_lp[i].begin(), res_lp[i].end(), h_tok_logp + o);
    o += (int64_t)res_tok[i].size();
    h_out_off[i + 1] = o;
    if (h_score) h_score[i] = res_score[i];
  }
  return NT_OK;
}

nt_status nt_op_gemm(int32_t dtype, const void* d_A, int32_t lda, const void* d_Bt, int32_t M, int32_t N, int32_t K,
                     const float* d_bias, const void* d_resid, void* d_out, int32_t ldc, int32_t out_f32,
                     int32_t relu, int32_t tile, const float* d_bscale, void* stream) {
  g_err.clear();
  if (!d_A || !d_Bt || !d_out) return fail(NT_E_INVALID, "null argument to nt_op_gemm");
  if (dtype < NT_F32 || dtype > NT_BF16) return fail(NT_E_INVALID, "unknown dtype %d", dtype);
  if (M < 0 || N <= 0 || K <= 0 || K % 64 != 0) return fail(NT_E_UNSUPPORTED, "need N > 0, K > 0, K %% 64 == 0");
  const int eb = dtype == NT_F32 ? 4 : 2;
  if (lda < K || (lda * eb) % 16 != 0 || ldc < N)
    return fail(NT_E_INVALID, "lda must be >= K with 16-byte rows, ldc >= N");
  if (tile < 0 || tile > 4) return fail(NT_E_INVALID, "tile must be 0..4");
  if (relu && (d_resid || out_f32)) return fail(NT_E_UNSUPPORTED, "relu combines with neither resid nor fp32 out");
  if (d_resid && out_f32) return fail(NT_E_UNSUPPORTED, "resid needs a model-dtype output");
  if (d_bscale && dtype != NT_F16) return fail(NT_E_UNSUPPORTED, "FP8 weights (d_bscale) need dtype NT_F16");
  nt::GemmEpi e{};
  e.wscale = d_bscale;
  e.mode = relu ? nt::EPI_RELU : d_resid ? nt::EPI_RESID : nt::EPI_STORE;
  e.bias = d_bias;
  e.resid = d_resid;
  e.out = d_out;
  e.ldc = ldc;
  e.out_f32 = out_f32 ? 1 : 0;
  NT_HIP(nt::gemm(static_cast<DT>(dtype), d_A, lda, d_Bt, M, N, K, e, static_cast<hipStream_t>(stream), 0, tile));
  return NT_OK;
}

nt_status nt_op_gemm_ln(int32_t dtype, const void* d_A, int32_t lda, const void* d_Bt, int32_t M, int32_t N,
                        int32_t K, const float* d_colsum, float ln_eps, const float* d_bias, void* d_out,
                        int32_t ldc, int32_t relu, int32_t tile, const float* d_bscale, void* stream) {
  g_err.clear();
  if (!d_A || !d_Bt || !d_out || !d_colsum) return fail(NT_E_INVALID, "null argument to nt_op_gemm_ln");
  if (dtype < NT_F32 || dtype > NT_BF16) return fail(NT_E_INVALID, "unknown dtype %d", dtype);
  if (M < 0 || N <= 0 || K <= 0 || K % 64 != 0) return fail(NT_E_UNSUPPORTED, "need N > 0, K > 0, K %% 64 == 0");
  const int eb = dtype == NT_F32 ? 4 : 2;
  if (lda < K || (lda * eb) % 16 != 0 || ldc < N)
    return fail(NT_E_INVALID, "lda must be >= K with 16-byte rows, ldc >= N");
  if (tile < 0 || tile > 4) return fail(NT_E_INVALID, "tile must be 0..4");
  if (!(ln_eps > 0.f)) return fail(NT_E_INVALID, "ln_eps must be positive");
  if (d_bscale && dtype != NT_F16) return fail(NT_E_UNSUPPORTED, "FP8 weights (d_bscale) need dtype NT_F16");
  nt::GemmEpi e{};
  e.wscale = d_bscale;
  e.mode = relu ? nt::EPI_RELU : nt::EPI_STORE;
  e.bias = d_bias;
  e.out = d_out;
  e.ldc = ldc;
  e.lnf_colsum = d_colsum;
  e.lnf_eps = ln_eps;
  NT_HIP(nt::gemm(static_cast<DT>(dtype), d_A, lda, d_Bt, M, N, K, e, static_cast<hipStream_t>(stream), 1, tile));
  return NT_OK;
}

nt_status nt_quantize_fp8(const float* h_W, int32_t in, int32_t out, uint8_t* h_q, float* h_scale) {
  g_err.clear();
  if (!h_W || !h_q || !h_scale) return fail(NT_E_INVALID, "null argument to nt_quantize_fp8");
  if (in <= 0 || out <= 0) return fail(NT_E_INVALID, "matrix sizes must be positive");
  std::vector<uint8_t> q;
  std::vector<float> sc;
  quantize_fp8(h_W, in, out, q, sc);
  std::memcpy(h_q, q.data(), q.size());
  std::memcpy(h_scale, sc.data(), sc.size() * 4);
  return NT_OK;
}

nt_status nt_op_select(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv, int32_t* d_topi,
                       float* d_lse, void* stream) {
  g_err.clear();
  if (!d_logits || !d_topv || !d_topi || !d_lse) return fail(NT_E_INVALID, "null argument to nt_op_select");
  if (rows < 0 || V <= 0) return fail(NT_E_INVALID, "rows must be >= 0 and V > 0");
  if (k < 1 || k > 32 || k > V) return fail(NT_E_UNSUPPORTED, "k must be in [1, min(32, V)]");
  NT_HIP(nt::beam_select(d_logits, nullptr, 1, rows, V, k, d_topv, d_topi, d_lse, static_cast<hipStream_t>(stream)));
  return NT_OK;
}

nt_status nt_op_select_tiled(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv,
                             int32_t* d_topi, float* d_lse, void* stream) {
  g_err.clear();
  if (!d_logits || !d_topv || !d_topi || !d_lse) return fail(NT_E_INVALID, "null argument to nt_op_select_tiled");
  if (rows < 0 || V <= 0) return fail(NT_E_INVALID, "rows must be >= 0 and V > 0");
  if (k < 1 || k > 32 || k > V) return fail(NT_E_UNSUPPORTED, "k must be in [1, min(32, V)]");
  if (V > 65536) return fail(NT_E_UNSUPPORTED, "V > 65536");
  if (rows == 0) return NT_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int n_tiles = (V + 127) / 128;
  float* part = nullptr;
  NT_HIP(hipMalloc((void**)&part, (size_t)rows * n_tiles * nt::topk_record(1) * sizeof(float)));
  hipError_t e = nt::tile_records(d_logits, rows, V, part, s);
  if (e == hipSuccess) e = nt::beam_select_tiles(part, n_tiles, d_logits, nullptr, 1, rows, V, k, d_topv, d_topi, d_lse, s);
  const hipError_t se = hipStreamSynchronize(s);   // the records buffer is freed below
  (void)hipFree(part);
  NT_HIP(e);
  NT_HIP(se);
  return NT_OK;
}

nt_status nt_op_select_tiled_noalloc(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv,
                                     int32_t* d_topi, float* d_lse, void* stream) {
  g_err.clear();
  if (!d_logits || !d_topv || !d_topi || !d_lse) return fail(NT_E_INVALID, "null argument to nt_op_select_tiled_noalloc");
  if (rows < 0 || V <= 0) return fail(NT_E_INVALID, "rows must be >= 0 and V > 0");
  if (k < 1 || k > 32 || k > V) return fail(NT_E_UNSUPPORTED, "k must be in [1, min(32, V)]");
  if (V > 65536) return fail(NT_E_UNSUPPORTED, "V > 65536");
  const int n_tiles = (V + 127) / 128;
  if ((long long)rows * n_tiles > NT_SELECT_NOALLOC_MAX_RECORDS)
    return fail(NT_E_UNSUPPORTED, "rows * ceil(V / 128) = %lld records > %d (at most %d rows at V = %d)",
                (long long)rows * n_tiles, NT_SELECT_NOALLOC_MAX_RECORDS, NT_SELECT_NOALLOC_MAX_RECORDS / n_tiles, V);
  if (rows == 0) return NT_OK;
  static_assert(NT_SELECT_NOALLOC_MAX_RECORDS == nt::SELECT_NOALLOC_MAX_RECORDS, "header and kernels agree");
  float* part = nullptr;
  size_t cap = 0;
  NT_HIP(nt::select_scratch(&part, &cap));
  if ((size_t)rows * n_tiles > cap) return fail(NT_E_UNSUPPORTED, "records exceed the static buffer");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  NT_HIP(nt::tile_records(d_logits, rows, V, part, s));
  NT_HIP(nt::beam_select_tiles(part, n_tiles, d_logits, nullptr, 1, rows, V, k, d_topv, d_topi, d_lse, s));
  return NT_OK;
}

nt_status nt_prof_config(uint32_t class_mask, int32_t stride) {
  g_err.clear();
  if (stride < 1) return fail(NT_E_INVALID, "stride must be >= 1");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_mask = class_mask & ((1u << NT_K_COUNT) - 1);
  g_prof_stride = stride;
  for (auto& c : g_prof_seen) c = 0;
  g_prof_enc_units = g_prof_step_units = 0;
  return NT_OK;
}

nt_status nt_prof_units(int64_t* encodes, int64_t* steps) {
  g_err.clear();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (encodes) *encodes = g_prof_enc_units;
  if (steps) *steps = g_prof_step_units;
  return NT_OK;
}

nt_status nt_set_graphs(int32_t enable) {
  g_err.clear();
  g_use_graphs = enable != 0;
  return NT_OK;
}

nt_status nt_set_beam_fused(int32_t enable) {
  g_err.clear();
  g_beam_fused = enable != 0;
  return NT_OK;
}

nt_status nt_set_streams(int32_t n) {
  g_err.clear();
  if (n < 1 || n > 8) return fail(NT_E_INVALID, "stream count %d outside [1, 8]", n);
  g_streams = n;
  return NT_OK;
}

nt_status nt_prof_enable(uint32_t class_mask) { return nt_prof_config(class_mask, 1); }

nt_status nt_prof_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
  }
  g_prof.clear();
  return NT_OK;
}

nt_status nt_prof_get(int32_t kernel_class, int64_t* launches, double* total_ms, double* alg_bytes, double* alg_flops) {
  g_err.clear();
  if (kernel_class < 0 || kernel_class >= NT_K_COUNT) return fail(NT_E_INVALID, "kernel class %d", kernel_class);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  int64_t n = 0;
  double ms = 0, by = 0, fl = 0;
  for (auto& r : g_prof) {
    if (r.cls != kernel_class) continue;
    NT_HIP(hipEventSynchronize(r.b));
    float e = 0.f;
    NT_HIP(hipEventElapsedTime(&e, r.a, r.b));
    ++n;
    ms += e;
    by += r.bytes;
    fl += r.flops;
  }
  if (launches) *launches = n;
  if (total_ms) *total_ms = ms;
  if (alg_bytes) *alg_bytes = by;
  if (alg_flops) *alg_flops = fl;
  return NT_OK;
}

}  // extern "C"
