// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on `s` and
// returns hipGetLastError() of the launch.  Shapes are validated by the runtime
// (nt_runtime.cpp) before any launch; launchers assume them.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace nt {

// Event pair into which the next kernel launch on this thread writes its own start and
// stop times (set by the runtime's kernel timing, cleared by the launch that takes it).
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;

// Every kernel launch of the library: hipExtLaunchKernelGGL with the pending event pair
// (the events then carry the dispatch's own timestamps), else hipLaunchKernelGGL.
#define NT_LAUNCH(kernel, grid, block, shmem, stream, ...)                                        \
  do {                                                                                            \
    if (::nt::g_launch_events.start) {                                                            \
      const ::nt::LaunchEvents ev_ = ::nt::g_launch_events;                                       \
      ::nt::g_launch_events = ::nt::LaunchEvents{};                                               \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev_.start, ev_.stop, 0, __VA_ARGS__); \
    } else {                                                                                      \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                        \
    }                                                                                             \
  } while (0)

enum class DT : int { F32 = 0, F16 = 1, BF16 = 2 };

// Decode-step control block in device memory.  Every decoder-step kernel reads the step
// index and the live counts from it (grids are sized for the whole batch and surplus
// workgroups return at once), and the step-end kernel advances it, so the kernel
// sequence of one step can be captured once and replayed for every step.
enum CtlField : int {
  CTL_T = 0,        // current step t
  CTL_NLIVE = 1,    // entries of the live-sentence list the step works on
  CTL_NALIVE = 2,   // sentences not finished yet
  CTL_ANC = 3,      // which half of the ancestor table is current (beam)
  CTL_WORDS = 4
};
// The step-end kernel also copies the new block into slot (t % CTL_MIRROR_SLOTS) of a
// pinned host mirror, so the host can read step t's outcome while later steps run.
constexpr int CTL_MIRROR_SLOTS = 4;
inline size_t dt_bytes(DT t) { return t == DT::F32 ? 4 : 2; }

// ---------------------------------------------------------------------------------
// GEMM: C[M,N] = A[M,K] . Bt[N,K]^T  (+ epilogue), fp32 accumulation on MFMA.
// A row stride lda (elements), Bt is [N][K] contiguous (weights stored "out x in").
enum EpiMode : int {
  EPI_STORE = 0,      // out = acc + bias
  EPI_RELU = 1,       // out = max(acc + bias, 0)
  EPI_RESID = 2,      // out = resid + acc + bias  (resid may alias out)
  EPI_SELF_QKV = 3,   // decoder: cols [0,d) -> q out; [d,3d) -> K/V cache slot t of phys row
  EPI_CROSS_KV = 4,   // encoder: cols of [Ld][K|V][d] -> cross cache [Ld][2][B][H][S][dh]
  EPI_TOPK = 5,       // output projection: per row and 128-column tile, the (max, sum exp,
                      // largest (value, index)) partials -- instead of the logits, or with
                      // out set, as well as the fp32 logits
};
__host__ __device__ inline int topk_record(int k2) { return 2 + 2 * k2; }   // floats per partial record

struct GemmEpi {
  const int* ctl = nullptr;        // if set, M = ctl[CTL_NLIVE] * ctl_rows (<= the launch M),
  int ctl_rows = 1;                //   and EPI_SELF_QKV writes slot ctl[CTL_T]
  int mode = EPI_STORE;
  const float* bias = nullptr;   // [N] fp32 or null
  const void* resid = nullptr;   // [M][ldc], same type as out
  void* out = nullptr;           // [M][ldc]
  int ldc = 0;
  int out_f32 = 0;               // 1: out is fp32 (logits); else the model dtype
  int out_map = 0;               // fp32 out: row m goes to row sent_list[m / beam] * beam + m % beam
  // EPI_SELF_QKV
  const int* sent_list = nullptr;  // logical sentence -> batch sentence
  int beam = 1;
  void* kcache = nullptr;          // [R][H][Tcap][dh] of this layer
  void* vcache = nullptr;
  int kv_f8 = 0;                   // 1: the caches hold E4M3 bytes (e4m3_rne of the fp32 value)
  int t = 0, Tcap = 0;
  // EPI_SELF_QKV / EPI_CROSS_KV
  int d = 0, H = 0, dh = 0;
  // EPI_CROSS_KV
  void* cross = nullptr;           // [Ld][2][B][H][S][dh]
  int B = 0, S = 0;
  // FP8 weights: Bt is [N][K] FP8 E4M3 bytes and column n of the product is scaled by
  // wscale[n] (fp32); null for weights in the model dtype.  fp16 activations only.
  const float* wscale = nullptr;
  // Pre-norm LayerNorm folded into the product (decoder-step launches, weights in the
  // model dtype, K = the row width): A holds the rows x before normalisation, Bt holds
  // W' = diag(gamma) W, bias holds b + beta W, and lnf_colsum[n] = sum_k Bt[n][k].  The
  // kernel sums each row's x and x^2 from its A fragments during the k-loop, and the
  // epilogue forms rstd * (acc - mean * lnf_colsum[n]) before adding the bias, which is
  // LN(x) W + b up to rounding.
  const float* lnf_colsum = nullptr;
  float lnf_eps = 0.f;
  // EPI_TOPK (the launch uses 128x128 tiles, so n_tiles = ceil(N / 128))
  float* part = nullptr;           // [M][n_tiles][topk_record(k2)]
  int k2 = 1;                      // record layout: 1 (max, sum, best value, best column)
  int n_tiles = 0;
  // Candidate-tile recompute (gemm_pairs): workgroup b takes block gblk[b] = {tile, first,
  // count} (b < *gnblk): the pairs sorted[first + i], i < count, all of that 128-column
  // tile, pair p belonging to row p / pair_k.
  const int* gblk = nullptr;
  const int* gnblk = nullptr;
  const int* sorted = nullptr;
  int pair_k = 1;
};

// role: 0 encoder, 1 decoder step, 2 output projection.  Only the kernel's symbol name
// depends on it, so profiles separate the three uses.  (Role 3 is gemm_pairs below.)
// tile: 0 = chosen by shape, 1 = 64x32, 2 = 128x128, 3 = 128x64, 4 = 64x128 (never changes
// a result).
hipError_t gemm(DT dt, const void* A, int lda, const void* Bt, int M, int N, int K, const GemmEpi& epi,
                hipStream_t s, int role = 0, int tile = 0);

// The output projection's logits of chosen (row, 128-column tile) pairs, recomputed: for
// every block of epi.gblk, the rows of its pairs times the tile's columns of Bt (N = V
// columns in all, K = the row width), written as fp32 to out[pair][128] (columns past N
// get -inf).  The product runs through the same kernel and k-order as gemm(), so each
// value is bitwise the one the projection's EPI_TOPK records were formed from.  The
// grid covers max_blocks blocks; those past *epi.gnblk return.
constexpr int PAIR_BM = 64;      // pair rows per block
hipError_t gemm_pairs(DT dt, const void* A, int lda, const void* Bt, int N, int K, const GemmEpi& epi,
                      int max_blocks, hipStream_t s);

// ---------------------------------------------------------------------------------
// Normalisation / embedding kernels (one wave per row of d = 64*EPL elements).
// Most partial sums a DLCL block start carries.  Two keep the kernel within 64 VGPRs at
// eight elements a lane (eight waves per SIMD); four would save few more reads and cost
// occupancy.
constexpr int DLCL_PARTS = 2;

struct DlclArgs {
  int l;                    // combination row l = 1..L+1; produces history entry l-1
  const void* y_prev;       // [rows][d] model dtype, or null for l = 1 (embedding)
  const int* ids;           // l = 1: [rows] token ids
  const int* lens;          // l = 1: [rows / S] sentence lengths (positions >= len are PAD)
  int S;                    // l = 1: padded length (position = row % S)
  const void* E;            // l = 1: [V][d] embedding
  int V;                    // l = 1: IDs are clamped to [0, V) so bad input cannot read past E
  const float* pe;          // l = 1: [max_pos][d] position table
  float emb_scale;          // sqrt(d)
  void* hist;               // history base; entry k at hist + k*hist_stride elements
  size_t hist_stride;
  const float* hist_ln;     // [2][d] gamma|beta of history entry l-1
  int hist_norm;
  const float* w;           // W[l][0..l-1]
  void* x_out;              // [rows][d] or null
  const float* ln;          // [2][d] LN applied to x (ln1 of layer l, or the output LN)
  void* u_out;              // [rows][d]
  int rows, d;
  float eps;
  // Blocked combination (same sums, fewer history reads): at the start of a block of
  // rows, the pass over the old entries also accumulates the sums of entries 0..l-1 for
  // the next n_part rows l+1 .. l+n_part (their weights in the triangle w_all, row r at
  // w_all + r(r-1)/2), stored in fp32 at part_out + i * part_stride; a later row of the
  // block starts from its partial (part_in) and adds entries k_start..l-1 only.  The fp32
  // additions happen in the same order either way.
  int n_part = 0;                 // 0 .. DLCL_PARTS
  const float* w_all = nullptr;
  float* part_out = nullptr;
  size_t part_stride = 0;
  const float* part_in = nullptr;
  int k_start = 0;
};
hipError_t dlcl_combine(DT dt, const DlclArgs& a, hipStream_t s);

// y = LN(x) row-wise; gamma|beta at ln[0..d), ln[d..2d).  With ctl, the live row count is
// ctl[CTL_NLIVE] * ctl_rows (rows is then the launch maximum).
hipError_t layernorm(DT dt, const void* x, const float* ln, void* y, int rows, int d, float eps, hipStream_t s,
                     const int* ctl = nullptr, int ctl_rows = 1);

// Decoder step input: z[r] = emb_scale*E[tok[phys(r)]] + pe[t]; u[r] = LN(z[r]) unless u is
// null (then ln is not read); rows and t
// from ctl (rows = ctl[CTL_NLIVE] * beam, t = ctl[CTL_T]), `rows` being the launch maximum.
hipError_t dec_embed_ln(DT dt, const int* cur_tok, const int* sent_list, int beam, const void* E,
                        const float* pe, const int* ctl, float emb_scale, const float* ln, void* z, void* u,
                        int rows, int d, float eps, hipStream_t s);

// Weight packing: dst[n][k] = (T) src[k][n] (src fp32 [K][N] row-major).
hipError_t pack_transpose(DT dt, const float* src, void* dst, int K, int N, hipStream_t s);
// dst[i] = (T) src[i].
hipError_t pack_convert(DT dt, const float* src, void* dst, size_t n, hipStream_t s);
// out[n] = sum_k Bt[n][k] in fp32, over a packed [N][K] weight matrix of the model dtype
// (the column sums a folded LayerNorm subtracts, taken from the values the GEMM reads).
hipError_t packed_row_sums(DT dt, const void* Bt, int N, int K, float* out, hipStream_t s);

// ---------------------------------------------------------------------------------
// Attention.
// Grouped multi-head attention over keys stored per (group, head): group g has
// nq(g) queries and len(g) valid keys.  Used for encoder self-attention (group =
// sentence, queries = its tokens) and decoder encoder-decoder attention (group =
// live sentence, queries = its beam rows).
struct MhaArgs {
  const void* q; int q_ld;       // query row r at q + r*q_ld + h*dh
  const void* k; const void* v;  // key (b,h,s) at k + b*kb + h*kh + s*ks
  long long kb, kh, ks;
  void* out; int out_ld;         // out row r at out + r*out_ld + h*dh
  const int* group_map;          // logical group -> b (null: identity)
  const int* lens;               // [b] valid keys (and valid queries for self-attention)
  int q_per_group;               // queries of group g are rows g*q_per_group + i
  int self_queries;              // 1: query i valid only if i < lens[b] (padded rows -> 0)
  int n_groups, H, dh;           // n_groups: launch maximum when ctl is set
  float scale;
  const int* ctl = nullptr;      // if set, the live group count is ctl[CTL_NLIVE]
  // relative positions (self-attention only): tables [2*rel_k+1][dh] fp32 shared by the
  // heads; query i, key j use row clip(j - i, -rel_k, rel_k) + rel_k
  const float* relk = nullptr;
  const float* relv = nullptr;
  int rel_k = 0;
};
// role: 0 encoder self-attention, 1 encoder-decoder attention (symbol name only).
hipError_t mha(DT dt, const MhaArgs& a, hipStream_t s, int role = 0);

// Decoder self-attention of each live row over its cached slots 0..t.
struct SelfAttnArgs {
  const void* q;              // [rows][d]
  const void* kcache; const void* vcache;  // [R][H][Tcap][dh]
  const int* sent_list; int beam;
  const int* anc;             // [2][R][Tcap] physical row holding slot s (null: own row);
  size_t anc_stride;          //   half ctl[CTL_ANC] is current
  void* out;                  // [rows][d]
  int rows, H, dh, Tcap;      // rows: launch maximum; live rows = ctl[CTL_NLIVE] * beam
  float scale;
  const int* ctl;             // step t = ctl[CTL_T]
  int kv_f8;                  // 1: the caches hold E4M3 bytes (q and out stay fp16)
};
hipError_t self_attn(DT dt, const SelfAttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------------
// Search.
struct SearchState {
  int B, beam, V, eos, Tcap;
  float alpha;
  int early_stop;
  int logp_input;         // 1: the selection input already holds per-token scores (an
                          // ensemble's combination), so no log-sum-exp is subtracted
  const int* sent_list;   // live sentences (logical order)
  const int* ctl;         // t = ctl[CTL_T], live list entries = ctl[CTL_NLIVE]
  float* score;           // [R] raw hypothesis scores
  int* cur_tok;           // [R] next input token
  int* tok_hist;          // [Tcap][R]
  int* par_hist;          // [Tcap][R]
  float* lp_hist;         // [Tcap][R]
  int* anc;               // [2][R][Tcap]; half ctl[CTL_ANC] is current, the other is written
  size_t anc_stride;
  int* done;              // [B]
  const int* maxlen;      // [B]
  float* best_score;      // [B] normalised
  float* best_raw;        // [B]
  int* best_step;         // [B]
  int* best_row;          // [B]
  int* best_nout;         // [B]
};

// Greedy: per live row, argmax (lowest ID on ties) and log-sum-exp over V logits, then
// the update (token, log-prob, EOS / length stop).  forced: [R] (by phys row) or null.
// Grids cover the whole batch (st.B * st.beam rows); rows past the live count return.
hipError_t greedy_step(const float* logits, const int* forced, const SearchState& st, hipStream_t s);

// Ensemble decoding: folds member `member` (0-based, of n_members) into the combined
// per-token scores comb [rows][V] of the live rows (ctl-driven, rows = live sentences x
// beam).  With lp = logit - logsumexp(row) of this member's fp32 logits:
//   rule 0: comb = sum of lp over the members so far, divided by n_members after the last;
//   rule 1: comb = logaddexp of lp over the members so far, minus log(n_members) after
//           the last.
// Member 0 initialises comb.  Grid: `rows` blocks (the whole batch); rows past the live
// count return.
hipError_t ens_combine(const float* logits, float* comb, const int* ctl, int beam, int rows, int V, int member,
                       int n_members, int rule, hipStream_t s);

// Beam: per live row, log-sum-exp and the 2K largest logits; then per live sentence the
// candidate ranking, the walk, the stop rule and the ancestor-table update.
// ctl may be null: then all `rows` rows are selected (kernel-level entry point).
hipError_t beam_select(const float* logits, const int* ctl, int beam, int rows, int V, int k2, float* topv, int* topi,
                       float* lse, hipStream_t s);
hipError_t beam_update(const float* topv, const int* topi, const float* lse, const SearchState& st, hipStream_t s);
// The same selection from an EPI_TOPK projection that also wrote the logits: part holds
// each row's per-tile records (k2 = 1 layout, n_tiles = ceil(V / 128) <= 512), and only
// the tiles that can hold one of the row's k2 largest logits are read back.  Same
// results as beam_select (the log-sum-exp merged from the records).
hipError_t beam_select_tiles(const float* part, int n_tiles, const float* logits, const int* ctl, int beam, int rows,
                             int V, int k2, float* topv, int* topi, float* lse, hipStream_t s);
// Beam selection with the logits never stored (three launches around gemm_pairs).
// beam_pick_tiles: per live row, the log-sum-exp merged from its records (lse) and the k2
//   tiles whose best entries rank first under (value desc, column asc); every one of the
//   row's k2 largest logits lies in them.  Pair p = r * k2 + j names the row's j-th tile,
//   ptile[p] (-1 past the row's tiles).  tau[r] is the k2-th best tile maximum, a lower
//   bound of the row's k2-th largest logit.
// pair_bucket (one workgroup, n_tiles <= 512): sorts the live pairs by tile into sorted[]
//   (R * k2 entries) and cuts each tile's run into blocks of at most PAIR_BM pairs,
//   gblk[b] = {tile, first position in sorted, count}, *gnblk = their number.
// beam_select_pairs: per live row, its k2 largest logits (value desc, index asc) from the
//   recomputed tiles logp[p][128] -- the same result as beam_select over the whole row.
hipError_t beam_pick_tiles(const float* part, int n_tiles, const int* ctl, int beam, int rows, int k2, int* ptile,
                           float* tau, float* lse, hipStream_t s);
hipError_t pair_bucket(const int* ptile, const int* ctl, int beam, int rows, int k2, int n_tiles, int* sorted,
                       int* gblk, int* gnblk, hipStream_t s);
hipError_t beam_select_pairs(const float* logp, const int* ptile, const float* tau, const int* ctl, int beam,
                             int rows, int V, int k2, float* topv, int* topi, hipStream_t s);
// Per-tile records of a logits matrix in the projection epilogue's layout (for tests).
hipError_t tile_records(const float* logits, int rows, int V, float* part, hipStream_t s);
// The current device's copy of the library's static records array (room for
// SELECT_NOALLOC_MAX_RECORDS records of the k2 = 1 layout), located on the first call on
// each device and reused after that.
constexpr int SELECT_NOALLOC_MAX_RECORDS = 1 << 20;   // 16 MiB
hipError_t select_scratch(float** out, size_t* records);

// Fused greedy selection after an EPI_TOPK projection (k2 = 1): merges the per-tile
// partials of each live row into the argmax and the LSE, then the greedy update.
hipError_t greedy_step_fused(const float* part, int n_tiles, const SearchState& st, hipStream_t s);

// End of a decode step (one workgroup): counts the unfinished sentences of the live list,
// drops the finished ones in place when pruning, advances t, flips the ancestor half
// (beam) and writes the new block into ctl and, if host_ctl is set (a device-visible
// pointer to pinned host memory of CTL_MIRROR_SLOTS * CTL_WORDS ints), into its mirror
// slot.  Once nothing is alive, or t reaches Tcap, the live count is 0: later steps,
// this kernel included, do nothing.
hipError_t step_end(int* list, const int* done, int* ctl, int* host_ctl, int prune, int beam, int Tcap,
                    hipStream_t s);

// Backtrack every sentence's best hypothesis into out_tok/out_lp [B][Tcap], out_len/out_score [B].
hipError_t finalize(const SearchState& st, int* out_tok, float* out_lp, int* out_len, float* out_score,
                    hipStream_t s);

// Initialise per-batch search state (scores 0 / -inf, BOS, best = -inf, done = 0, identity
// list) and the control block (t = 0, all B sentences live and alive).
hipError_t search_init(const SearchState& st, int* list, int* ctl, int bos, hipStream_t s);

// Scatter the live rows of the compact logits [rows][V] to dst[phys(r)][V].
hipError_t scatter_logits(const float* logits, const int* sent_list, const int* ctl, int beam, int rows, int V,
                          float* dst, hipStream_t s);

}  // namespace nt
