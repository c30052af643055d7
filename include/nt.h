/*
 * nt.h -- C ABI of the MI355X (gfx950) deep-encoder / shallow-decoder translation library.
 *
 * The library translates batches of token-ID sentences with a Transformer whose encoder
 * combines layers dynamically (DLCL, Sec. 2.1 Eq. 1-2: the input of layer l+1 is
 * sum_{k<=l} W_k^(l+1) LN(y_k), y_0 being the embedding) and whose decoder runs one
 * step at a time over cached self-attention keys/values and encoder-decoder
 * keys/values computed once per batch (Sec. 4.1 "Caching").  Around the model sit the
 * decoding optimisations of Sec. 4: greedy search (Sec. 4.4), beam search with the
 * early-stop rule (Sec. 4.1 "Faster Beam Search"), batch pruning (Sec. 4.1), dynamic
 * batching by a token budget (Sec. 4.2), FP16 inference with fp32 reductions (Sec. 4.2)
 * and one memory pool per call (Sec. 4.4 "Profile-guided optimization").
 *
 * Conventions shared by every entry point
 *  - Handles are opaque; device pointers are plain HIP device addresses (for example
 *    torch tensors' data_ptr()); `stream` is a hipStream_t passed as void* (NULL = the
 *    null stream).  All device work is enqueued on that stream.
 *  - The caller owns every buffer it passes in.  The library owns only the small host
 *    structs nt_model and nt_dec_state (freed by nt_free_model / nt_free_state) and never
 *    frees caller memory.
 *  - Every function returns an nt_status and, on failure, sets a thread-local message
 *    readable with nt_last_error().  Nothing throws across the ABI and nothing aborts.
 *  - Special token IDs: PAD = 0, BOS = 1, EOS = 2 (UNK = 3 is an ordinary word).
 *  - Output tokens exclude BOS and EOS.  Outputs of nt_translate are in input order
 *    (Sec. 4.3 and Sec. 5: inputs are sorted by length and the original order restored).
 */
#ifndef NT_H_
#define NT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NT_OK = 0,
  NT_E_INVALID = 1,      /* bad argument: null pointer, empty input, ID out of range, size */
  NT_E_UNSUPPORTED = 2,  /* a shape or option the kernels do not implement */
  NT_E_WORKSPACE = 3,    /* workspace too small; the message states the bytes required */
  NT_E_DEVICE = 4,       /* a HIP runtime error */
  NT_E_STATE = 5,        /* a call that does not fit the state (e.g. a step after the end) */
  NT_E_NUMERIC = 6       /* reserved: NaN/Inf detected by a debug check */
} nt_status;

typedef enum { NT_F32 = 0, NT_F16 = 1, NT_BF16 = 2 } nt_dtype;

typedef struct nt_model nt_model;
typedef struct nt_dec_state nt_dec_state;

/* Model shape and numeric mode.
 *  d_model % n_heads == 0, d_head = d_model / n_heads in {32, 64, 128}, d_model % 64 == 0,
 *  d_ffn % 64 == 0.  max_positions bounds source and target positions (1024 in Sec. 2.2).
 *  dtype: storage type of matrices and activations.  NT_F32 is true fp32 end to end;
 *  NT_F16 / NT_BF16 store weights and activations in 16 bits and keep every
 *  accumulation, LayerNorm, softmax, log-sum-exp, DLCL sum and search score in fp32
 *  (Sec. 4.2 "FP16 Inference": reductions run in a wider type to avoid overflow).
 *  dlcl_hist_norm: 1 = each history entry is LayerNorm'd as in Eq. 2 (the default);
 *  0 = identity, so that one-hot DLCL weights give the plain pre-norm stack.
 *  ln_eps: LayerNorm epsilon (1e-5).
 *  rel_pos_k: 0, or 1..16: relative position representations in encoder self-attention
 *    (the teachers' RPR, Sec. 3.1, maximum relative length 8; Shaw et al. 2018): every
 *    encoder layer then has a key and a value table of 2k+1 rows of d_head (fp32, shared
 *    by the heads, after b_2 in the weight blob); query i and key j use row
 *    clip(j - i, -k, k) + k, added to the key inside the scaled score and to the value
 *    inside the weighted sum.
 *  fp8_weights: 0, or 1 with dtype NT_F16: FP8 weights (the paper leaves lower precision
 *    to future work, Sec. 6).  Every projection matrix of the encoder and the decoder
 *    (W_qkv, W_o, W_1, W_2, W_q, W_kv, W_oc) is stored as OCP FP8 E4M3 with one fp32
 *    scale per output column: scale_n = max_k |W[k,n]| / 448 and q = the E4M3 value
 *    nearest (ties to even) to W[k,n] / scale_n, both computed in fp32 by
 *    nt_load_weights.  The projections multiply fp16 activations by q exactly (every
 *    E4M3 value is an fp16 value) and scale the fp32 sums.  E (embedding and output
 *    projection) stays fp16; activations and every reduction are as for NT_F16.  The
 *    decoder projections that take a pre-norm LayerNorm's output (QKV, cross-Q, FFN1)
 *    quantize the gain-scaled weights diag(gamma) W instead and normalise their input
 *    rows themselves.
 *  fp8_kv: 0, or 1 with dtype NT_F16: the decoder's self-attention key/value cache holds
 *    OCP FP8 E4M3 values, each the E4M3 value nearest (ties to even, saturating at 448)
 *    to the fp32 key or value the QKV projection computes; attention widens them exactly.
 *    Halves the bytes the self-attention streams every step (Sec. 6 leaves lower
 *    precision to future work; this is one reading of it). */
typedef struct {
  int32_t d_model, n_heads, d_ffn, n_enc, n_dec, vocab, max_positions;
  int32_t pad_id, bos_id, eos_id;
  int32_t dtype;
  int32_t dlcl_hist_norm;
  float ln_eps;
  int32_t rel_pos_k;
  int32_t fp8_weights;
  int32_t fp8_kv;
} nt_model_cfg;

/* Search and batching options.
 *  beam: 1 = greedy (Sec. 4.4), 2..16 = beam search (Sec. 4.1).
 *  len_penalty: alpha of lp(n) = ((5+n)/6)^alpha applied to finished/final scores; 0 = raw.
 *  max target tokens of sentence i (EOS counted) = floor(max_len_a * len_i) + max_len_b,
 *    lowered to max_len_cap when max_len_cap > 0 (Sec. 4.4 caps targets at 200 tokens;
 *    0 = no cap).
 *  token_budget: dynamic batching (Sec. 4.2) packs sentences, longest first, while
 *    n_sentences * longest_length <= token_budget (padded source tokens).
 *  max_batch_sents: 0 = no cap; otherwise at most this many sentences per batch.
 *  early_stop: 1 = stop a sentence's beam once its best finished hypothesis scores at
 *    least every live one (Sec. 4.1); 0 = run to the length limit.
 *  prune: 1 = drop finished sentences from the decoder's batch every step (Sec. 4.1
 *    "Batch Pruning"); 0 = keep computing them (results are identical). */
typedef struct {
  int32_t beam;
  float len_penalty;
  float max_len_a;
  int32_t max_len_b;
  int32_t max_len_cap;
  int32_t token_budget;
  int32_t max_batch_sents;
  int32_t early_stop;
  int32_t prune;
} nt_search_cfg;

/* ---- weights --------------------------------------------------------------------------
 * The host weight blob is one fp32 vector in this canonical order (matrices row-major
 * "in x out", y = x W):
 *   E [V,d] (tied: source embedding, target embedding and output projection, Sec. 2.2);
 *   hist_ln[k].{gamma,beta} [d] for k = 0..L  (the LN of Eq. 2, one per history entry);
 *   DLCL W: rows l = 1..L+1, row l holding W[l,0..l-1] (Eq. 2, one scalar per pair);
 *   per encoder layer: ln1.{g,b}, W_qkv [d,3d] (columns Q|K|V, head h at h*dh within
 *     each), b_qkv [3d], W_o [d,d], b_o, ln2.{g,b}, W_1 [d,F], b_1 [F], W_2 [F,d], b_2;
 *   enc_out_ln.{g,b};
 *   per decoder layer: ln1.{g,b}, W_qkv, b_qkv, W_o, b_o, ln2.{g,b}, W_q [d,d], b_q,
 *     W_kv [d,2d] (columns K|V), b_kv, W_oc [d,d], b_oc, ln3.{g,b}, W_1, b_1, W_2, b_2;
 *   dec_out_ln.{g,b}.
 */

/* Sizes for a model: host_floats = length of the fp32 blob; device_bytes = size of the
 * device buffer nt_load_weights needs.  Returns NT_E_INVALID / NT_E_UNSUPPORTED for a
 * shape the library cannot run.
 * Defined by: the model of Sec. 2.1 (pre-norm Transformer whose encoder layers are
 * combined by Eq. 1-2) with tied embeddings (Sec. 2.2); the blob's matrix parameters add
 * up to the counts of Tables 1 and 2 (152M for 35-6, 131M for 35-1, 49M for 9-1). */
nt_status nt_weights_size(const nt_model_cfg* cfg, size_t* host_floats, size_t* device_bytes);

/* Converts the host blob into the device layout: matrices rounded (nearest even) to the
 * model dtype (or, with fp8_weights, the projections quantized to FP8 E4M3 with their
 * column scales) and stored transposed ([out][in]) for the GEMMs, vectors kept in fp32, a
 * sinusoidal position table computed once.  device_buf (>= device_bytes, 256-byte
 * aligned) is borrowed for the model's lifetime.  The host blob may be freed on return.
 * Synchronises `stream` before returning.  Allocates (and frees) one device staging
 * buffer of the blob's size.  NT_E_INVALID for a null pointer, a blob of the wrong length
 * or a misaligned buffer; NT_E_WORKSPACE if device_bytes is too small (the message
 * states the bytes required); NT_E_DEVICE for a HIP error.
 * Defined by: Sec. 4.2 "FP16 Inference" (every model parameter stored in FP16; with
 * NT_F32 they stay fp32), the model of Sec. 2.1-2.2 as for nt_weights_size. */
nt_status nt_load_weights(const nt_model_cfg* cfg, const float* host_weights, size_t host_floats,
                          void* device_buf, size_t device_bytes, void* stream, nt_model** out);
/* Frees the handle (not device_buf, which the caller owns).  NULL is ignored. */
void nt_free_model(nt_model* m);

/* ---- ensembles -------------------------------------------------------------------------
 * Ensemble decoding (the teacher ensemble of Sec. 2.2, Table 1): one model handle over
 * n_members (1..8) loaded models that decode together.  At every step each member runs
 * its own decoder, over its own encoder output and key/value caches, on the shared
 * prefix; the search then ranks words by a combination s(w) of the members'
 * log-probabilities log p_m(w) = logit_m(w) - logsumexp(logit_m), used where one model's
 * log p(w) would be (hypothesis scores, length penalty, stop rule and the reported
 * per-token values are all in s):
 *   NT_ENS_MEAN_LOGP  (0): s(w) = (1/M) sum_m log p_m(w);
 *   NT_ENS_LOG_MEAN_P (1): s(w) = log((1/M) sum_m p_m(w)).
 * The paper names the ensemble but not its combination rule; both common readings are
 * offered.  Members must share vocab, pad/bos/eos IDs and dtype; depth, width, heads,
 * FFN size, DLCL history norm and relative positions may differ.  The handle borrows
 * the members (they must outlive it) and is accepted wherever an nt_model* is taken
 * (workspace sizes, nt_encode, nt_decode_step, nt_translate); nt_free_model frees only
 * the handle.  An ensemble cannot be a member.  For an ensemble, nt_decode_step's
 * d_logits receives s, and nt_dec_state_encoder_out reports the first member's encoder
 * output.  NT_E_INVALID for a null pointer, a member count outside 1..8, an unknown
 * rule, a nested ensemble or members that disagree. */
typedef enum { NT_ENS_MEAN_LOGP = 0, NT_ENS_LOG_MEAN_P = 1 } nt_ensemble_rule;
nt_status nt_ensemble(nt_model* const* members, int32_t n_members, int32_t rule, nt_model** out);

/* ---- workspace (the memory pool)-------------------------------------------------------
 * Bytes of workspace needed to encode and decode one batch of up to max_sents sentences
 * padded to max_src tokens under `search` (beam width and length limits).
 * NT_E_INVALID for a null pointer or a non-positive size; NT_E_UNSUPPORTED for beam > 16.
 * Defined by: the memory pool of Sec. 4.4 ("Profile-guided optimization": blocks are
 * taken from a pool during decoding and given back when the translation is done); here
 * the pool is one caller-owned buffer carved by the library, and nothing is allocated
 * while a batch decodes. */
nt_status nt_workspace_size(const nt_model* m, const nt_search_cfg* search, int32_t max_sents,
                            int32_t max_src, size_t* bytes);

/* Bytes of workspace nt_translate needs for this exact input at the current stream
 * setting (nt_set_streams): one slice per concurrently decoded batch, each the maximum
 * over the batches that dynamic batching forms from it.  A smaller workspace (at least
 * one slice) makes nt_translate decode fewer batches at once.
 * Defined by: the memory pool of Sec. 4.4 and the dynamic batching of Sec. 4.2 (batches
 * hold as many sentences as the token budget allows). */
nt_status nt_translate_workspace_size(const nt_model* m, const nt_search_cfg* search,
                                      const int64_t* h_src_off, int32_t n_sent, size_t* bytes);

/* ---- step-level entry points -----------------------------------------------------------
 * nt_encode runs the DLCL encoder (Eq. 1-2) on a padded batch and computes the
 * encoder-decoder keys/values of every decoder layer once (Sec. 4.1), then sets up the
 * decoder state.  d_src: [B,S] int32 device IDs, row-major, PAD-padded; d_len: [B] int32
 * device lengths (1..S).  IDs must lie in [0, vocab): nt_translate checks them on the
 * host; here an ID outside the range is read as the nearest valid ID.  h_len: NULL, or
 * the same B lengths in host memory (the per-sentence length limits are computed on the
 * host; without h_len the lengths are copied back from d_len, which synchronises the
 * stream).  d_ws / ws_bytes: workspace (256-byte aligned), borrowed until nt_free_state.
 * Asynchronous except for a small host->device copy of the length limits.
 * NT_E_INVALID for a null pointer, an empty batch, a length outside 1..S, S or a target
 * limit beyond max_positions; NT_E_UNSUPPORTED for beam > 16; NT_E_WORKSPACE if ws_bytes
 * is below nt_workspace_size (the message states the bytes required); NT_E_DEVICE.
 * Defined by: Sec. 2.1 Eq. 1-2 (x_{l+1} = sum_{k<=l} W_k^(l+1) LN(y_k)), Sec. 3.2 (the
 * deep encoder), Sec. 4.1 "Caching" (the encoder-decoder keys and values are projected
 * once and kept). */
nt_status nt_encode(nt_model* m, const int32_t* d_src, const int32_t* d_len, const int32_t* h_len,
                    int32_t B, int32_t S, const nt_search_cfg* search, void* d_ws, size_t ws_bytes,
                    void* stream, nt_dec_state** st);

/* One decoder step for every live hypothesis: embedding, Ld pre-norm layers with the
 * cached self-attention keys/values (the new key/value is appended at slot t) and the
 * cached encoder-decoder keys/values, the tied output projection, then selection (greedy
 * argmax with log-sum-exp, or beam top-2K) and the search update; with pruning on, the
 * finished sentences leave the batch.
 * Defined by: Sec. 4.1 "Caching" (keys and values of every earlier step are kept),
 * "Faster Beam Search" (a sentence stops once a candidate has ended with EOS and no
 * live candidate scores higher) and "Batch Pruning" (finished hypotheses leave the
 * batch); Sec. 4.4 "Greedy Search" and the removal of log_softmax for greedy search
 * (the argmax needs no normalisation; the chosen token's log-prob comes from the same
 * pass's log-sum-exp).
 *  d_forced: NULL, or [B*beam] int32 device tokens (greedy only): teacher forcing --
 *    row r emits d_forced[r] instead of its argmax (its log-prob is still recorded);
 *    an ID outside [0, V) is replaced by EOS.
 *  d_logits: NULL, or [B*beam, V] fp32 device buffer receiving this step's logits of
 *    the live rows (rows of finished sentences are left untouched).
 *  h_alive: NULL, or host int32 receiving the number of sentences still decoding; asking
 *    for it synchronises the stream.
 * Returns NT_E_STATE once every sentence has finished. */
nt_status nt_decode_step(nt_dec_state* st, const int32_t* d_forced, float* d_logits, int32_t* h_alive,
                         void* stream);

/* Results of a finished batch, one row per sentence in batch order:
 *  h_tokens [B, max_tgt] int32 (row i valid up to h_lens[i]), h_lens [B],
 *  h_scores [B] (normalised score; with alpha = 0 the sum of log-probs including EOS),
 *  h_token_logp [B, max_tgt] fp32 log-prob of each output token.  Any pointer may be
 *  NULL.  max_tgt is reported by nt_dec_state_info.  NT_E_STATE if a sentence is still
 *  decoding.  Synchronises the stream.
 * Defined by: the result of the search of Sec. 4.1 ("Faster Beam Search": the best
 * finished hypothesis) or of greedy search (Sec. 4.4). */
nt_status nt_dec_state_read(nt_dec_state* st, int32_t* h_tokens, int32_t* h_lens, float* h_scores,
                            float* h_token_logp, void* stream);

/* Shape of a state: batch size, padded source length, beam, max target tokens, steps
 * taken, sentences still decoding (as of the last step that reported it).  Any output
 * pointer may be NULL; NT_E_INVALID for a null state.  Diagnostics (no passage of the
 * paper defines them). */
nt_status nt_dec_state_info(const nt_dec_state* st, int32_t* B, int32_t* S, int32_t* beam,
                            int32_t* max_tgt, int32_t* steps, int32_t* alive);

/* Copies the encoder output LN_out(x_{L+1}) [B,S,d] to host fp32 (rows of padding
 * included).  Synchronises the stream.  For tests.  Defined by: Eq. 2 applied to the
 * last layer's history, then the encoder's output LayerNorm (Sec. 2.1, pre-norm). */
nt_status nt_dec_state_encoder_out(nt_dec_state* st, float* h_enc, void* stream);

/* Frees a state (not its workspace, which the caller owns).  NULL is ignored. */
void nt_free_state(nt_dec_state* st);

/* ---- whole-job entry point -------------------------------------------------------------
 * Translates n_sent sentences given in CSR form on the host (h_src: concatenated IDs,
 * h_src_off: [n_sent+1] offsets, every sentence 1..max_positions IDs in [0, V)).
 * Sentences are sorted by descending length, packed into batches under the token budget,
 * encoded and decoded batch by batch in the workspace, and written back in input order:
 * h_out receives the concatenated output tokens (capacity out_cap; the sum of every
 * sentence's max target length always suffices), h_out_off [n_sent+1] the offsets,
 * h_score [n_sent] (or NULL) the scores, h_tok_logp [out_cap] (or NULL) each output
 * token's log-prob.  Returns when the outputs are in host memory.  Batches run on library
 * streams that wait for the work already queued on `stream`, several at a time
 * (nt_set_streams), each in its own workspace slice, so that the small kernels of one
 * batch's decoder step overlap those of another; results do not depend on it.
 * Every per-step quantity lives in a device-side control block, so the decoder step is
 * one fixed kernel sequence: each batch's step is captured once into a HIP graph and
 * replayed (or, after nt_set_graphs(0), launched kernel by kernel).  Both ways run the
 * same kernels and give bitwise identical results.
 * NT_E_INVALID for a null pointer, n_sent <= 0, an empty sentence, an ID outside
 * [0, V), a source or target limit beyond max_positions, or out_cap below the output
 * size (the message states it); NT_E_UNSUPPORTED for beam > 16; NT_E_WORKSPACE if
 * ws_bytes is below one slice (the message states the bytes required); NT_E_DEVICE.
 * Defined by: Sec. 4.2 "Dynamic Batching" (as many sentences per batch as the token
 * budget allows), Sec. 5 (input sentences sorted by descending length; one memory pool)
 * and Sec. 4.3 "Decoding in Parallel" (parts translated apart, merged back in the
 * original order). */
nt_status nt_translate(nt_model* m, const nt_search_cfg* search, const int32_t* h_src,
                       const int64_t* h_src_off, int32_t n_sent, int32_t* h_out, int64_t out_cap,
                       int64_t* h_out_off, float* h_score, float* h_tok_logp, void* d_ws,
                       size_t ws_bytes, void* stream);

/* ---- kernel-level entry point (diagnostics and tests) ----------------------------------
 * One dense projection as the translation path runs it (the "MM" of the paper's GPU
 * profile, Sec. 4.4): out[M,N] = A[M,K] . Bt[N,K]^T (+ bias[N]) (+ resid[M,N]), then
 * ReLU if relu != 0.  A, Bt, resid and out are device arrays in `dtype` (out is fp32
 * if out_f32); rows of A are lda elements apart, rows of out/resid ldc elements apart;
 * Bt is [N][K] contiguous.  K % 64 == 0; rows of A start 16-byte aligned.  tile: 0 = chosen by
 * shape, 1 = 64x32, 2 = 128x128, 3 = 128x64, 4 = 64x128 output tiles (the choice never
 * changes a result).  d_bscale: NULL, or (dtype NT_F16 only) Bt holds FP8 E4M3 bytes and
 * column n of the product is multiplied by d_bscale[n] (fp32), as for the weights of an
 * fp8_weights model; tiles 1 and 4 are then 32x64 and 64x64.  Asynchronous. */
nt_status nt_op_gemm(int32_t dtype, const void* d_A, int32_t lda, const void* d_Bt, int32_t M, int32_t N, int32_t K,
                     const float* d_bias, const void* d_resid, void* d_out, int32_t ldc, int32_t out_f32,
                     int32_t relu, int32_t tile, const float* d_bscale, void* stream);

/* The same projection with its input's pre-norm LayerNorm folded in (Sec. 2.1: every
 * sublayer normalises its input first), as the decoder step runs it for weights in the
 * model dtype:  out[m][n] = act(rstd_m (A_m . Bt_n - mu_m colsum[n]) + bias[n]), with mu_m
 * the mean of row m of A over its K values, rstd_m = 1/sqrt(var_m + ln_eps) (biased
 * variance), and act = ReLU if relu != 0.  With Bt = (diag(gamma) W)^T, colsum[n] =
 * sum_k Bt[n][k] and bias = b + beta W this is LN(A) W + b.  A, Bt and out (ldc) are
 * device arrays in `dtype`; d_colsum [N] and d_bias [N] fp32 device arrays (bias may be
 * NULL).  K % 64 == 0 and K is the whole row.  tile as for nt_op_gemm (2 runs as 4, which
 * holds the row statistics at a higher occupancy).  d_bscale: NULL, or (dtype NT_F16
 * only) Bt holds FP8 E4M3 bytes and column n of A . Bt is multiplied by d_bscale[n] before
 * the normalisation, as for the decoder projections of an fp8_weights model (colsum then
 * holds the sums of the dequantized columns); tile 1 is then 32x64 and tiles 2-4 are
 * 64x128.  Asynchronous. */
nt_status nt_op_gemm_ln(int32_t dtype, const void* d_A, int32_t lda, const void* d_Bt, int32_t M, int32_t N,
                        int32_t K, const float* d_colsum, float ln_eps, const float* d_bias, void* d_out,
                        int32_t ldc, int32_t relu, int32_t tile, const float* d_bscale, void* stream);

/* The FP8 weight quantization nt_load_weights applies with fp8_weights, on the host: W
 * [in][out] fp32 (row-major, y = x W) -> q [out][in] E4M3 codes (OCP, bias 7, ties to
 * even, saturating at 448) and scale [out] fp32, with scale[n] = max_k |W[k][n]| / 448
 * (1 for an all-zero column) and q[n][k] = E4M3(W[k][n] / scale[n]).  Host pointers;
 * no device work.  For tests. */
nt_status nt_quantize_fp8(const float* h_W, int32_t in, int32_t out, uint8_t* h_q, float* h_scale);

/* One selection step as the beam search runs it (Sec. 4.1, "Faster Beam Search" keeps 2K
 * candidates per hypothesis; Sec. 4.4 drops log_softmax): for each of `rows` rows of
 * d_logits [rows, V] fp32 (rows 16-byte aligned when V % 4 == 0), the k largest logits in
 * (value desc, index asc) order into d_topv / d_topi [rows, k], and the row's log-sum-exp
 * into d_lse [rows].  A logit of -inf is never selected: slots beyond a row's finite
 * logits hold (-inf, INT32_MAX).  1 <= k <= 32 and k <= V.  Device pointers;
 * asynchronous.  For tests. */
nt_status nt_op_select(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv, int32_t* d_topi,
                       float* d_lse, void* stream);

/* The same selection as the beam search runs it from the output projection's per-tile
 * records (the projection's epilogue leaves, per row and 128-column tile, the tile row's
 * max and sum of exp(x - max)): with tau the k-th largest tile maximum of a row, every one
 * of the row's k largest logits lies in a tile whose maximum is >= tau, so only those
 * tiles are read back, and the log-sum-exp is merged from the records.  Here the records
 * are formed from d_logits by a separate kernel, in a device buffer this call allocates
 * and frees.  Same arguments, layout and results as nt_op_select (the log-sum-exp summed
 * in another order); additionally V <= 65536.  For tests. */
nt_status nt_op_select_tiled(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv,
                             int32_t* d_topi, float* d_lse, void* stream);

/* nt_op_select_tiled for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the same kernels, arguments
 * and results, with the per-tile records in a static array that the library holds on
 * each GPU until the process ends (16 MiB: rows * ceil(V / 128) <= 1048576 records, i.e.
 * 4194 rows at V = 32000; larger inputs return NT_E_UNSUPPORTED with the limit in the
 * message).  Nothing is allocated and the stream is not synchronised: the call only
 * enqueues work.  Every call on one GPU shares that GPU's array, which keeps the last
 * call's records (each call writes every record it reads before reading it, so nothing
 * needs clearing); calls that overlap on one GPU -- on different streams, or from
 * different threads -- race on it and must be ordered by the caller.  Runs on the
 * current device. */
#define NT_SELECT_NOALLOC_MAX_RECORDS (1 << 20)
nt_status nt_op_select_tiled_noalloc(const float* d_logits, int32_t rows, int32_t V, int32_t k, float* d_topv,
                                     int32_t* d_topi, float* d_lse, void* stream);

/* Process-wide switch for nt_translate's graph replay of the decoder step (default on;
 * with 0, every step is launched kernel by kernel). */
nt_status nt_set_graphs(int32_t enable);

/* Process-wide choice of the beam selection (default 1).  With 1 the output projection
 * keeps only per-tile records (max, sum of exp, best entry) of each row's 128-column
 * tiles; the 2K tiles whose best entries rank first hold the row's 2K largest logits, and
 * only their logits are formed again, bitwise equal, for the selection -- the R x V
 * logits never reach device memory (Sec. 4.4 drops log_softmax, Sec. 6 names kernel
 * fusion as the way on).  With 0 the projection stores the fp32 logits and the selection
 * scans every row.  Both give bitwise identical results.  It takes effect for workspaces
 * sized and states encoded after the call (the two need different buffers), so set it
 * before nt_workspace_size. */
nt_status nt_set_beam_fused(int32_t enable);

/* Process-wide number of batches nt_translate decodes concurrently, 1..8 (default 4: on
 * MI355X with HIP's default of four hardware queues per process, 4 measured best with
 * graph replay; 3 without it). */
nt_status nt_set_streams(int32_t n);

/* Thread-local message of the last failing call on this thread ("" if none); valid until
 * the next nt_* call on this thread.  A convention of this library, not of the paper. */
const char* nt_last_error(void);

/* ---- kernel timing ---------------------------------------------------------------------
 * When enabled for a kernel class, the library brackets each launch of that class with
 * HIP events on the launch stream and records the launch's algorithmic bytes and flops
 * (the data the method must move or compute, not what the kernel happens to touch). */
typedef enum {
  NT_K_GEMM_ENC = 0,    /* encoder projections (QKV, O, FFN1, FFN2) and the cross-K/V GEMM */
  NT_K_GEMM_DEC = 1,    /* decoder-step projections */
  NT_K_GEMM_VOCAB = 2,  /* tied output projection (logits) */
  NT_K_DLCL = 3,        /* fused history LayerNorm + DLCL combination (+ next LN) */
  NT_K_LN = 4,          /* plain LayerNorm (and the decoder embedding) */
  NT_K_ATTN_ENC = 5,    /* encoder self-attention */
  NT_K_ATTN_SELF = 6,   /* decoder self-attention over the step cache */
  NT_K_ATTN_CROSS = 7,  /* decoder encoder-decoder attention */
  NT_K_SELECT = 8,      /* argmax / top-2K with log-sum-exp */
  NT_K_SEARCH = 9,      /* search update, compaction, finalisation */
  NT_K_COUNT = 10
} nt_kernel_class;

nt_status nt_prof_enable(uint32_t class_mask);   /* bit i enables class i; 0 disables */
/* Like nt_prof_enable, but only every `stride`-th launch of an enabled class is timed
 * (stride >= 1), which keeps the host cost of event recording out of a timed run.
 * nt_translate instead samples whole units -- every stride-th decoder step or batch
 * encode -- and runs each sample alone on the GPU (the other batches' streams drained
 * first) with events on every launch of the enabled classes, so the times are those of
 * the kernels by themselves, as a kernel-trace profiler reports them. */
nt_status nt_prof_config(uint32_t class_mask, int32_t stride);
/* Units nt_translate has counted since the last nt_prof_config, per kind: batch
 * encodes and decoder steps (each counted while a class that kind launches is enabled;
 * stride applies per kind).  Either pointer may be NULL. */
nt_status nt_prof_units(int64_t* encodes, int64_t* steps);
nt_status nt_prof_reset(void);
/* Totals since the last reset for one class; synchronises on the recorded events. */
nt_status nt_prof_get(int32_t kernel_class, int64_t* launches, double* total_ms, double* alg_bytes,
                      double* alg_flops);

#ifdef __cplusplus
}
#endif
#endif /* NT_H_ */
