"""Oracle model: DLCL pre-norm encoder and incremental pre-norm decoder (NumPy).

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, following the paper:

* Encoder, Sec. 2.1 Eq. 1-2 (dynamic linear combination of layers, DLCL): the input
  of layer l+1 is sum_{k<=l} W^(l+1)_k LN(y_k), with y_0 the embedding output and
  y_k the k-th layer's output.  Deep encoder, shallow decoder: Sec. 3.2.
* Tied embeddings: one matrix E is the source embedding, the target embedding and
  the output projection (Sec. 2.2).
* Caching (Sec. 4.1): the decoder keeps the key/value projections of every earlier
  step (self-attention) and of the encoder output (cross-attention, computed once).

Readings of what the paper leaves open (each is also listed in the design notes):

* W is one scalar per (row, entry) pair: a lower-triangular (L+1)x(L+1) matrix.
* Each history entry k has its own LayerNorm, applied once when y_k is produced.
  ``hist_norm=False`` replaces it with the identity (used to check that one-hot W
  reduces to the plain pre-norm stack).
* Every layer (encoder and decoder) is pre-norm; the decoder has no DLCL.
* Encoder output: enc = LN_out(sum_{k<=L} W[L+1,k] h_k).
* Embedding: y_0 = sqrt(d) E[id] + PE(pos), PE interleaved sin/cos from position 0.
* Attention scale 1/sqrt(d_head); ReLU FFN; biases on every projection except the
  tied output projection; LayerNorm with biased variance and eps = 1e-5.
* FP8 key/value cache (with FP8 weights; lower precision is future work in Sec. 6): the
  decoder's self-attention keys and values are kept as the E4M3 values nearest to them
  (ties to even, saturating at 448), quantized as they enter the cache, and attention
  reads them from there, the current step's own key and value included.
* Relative positions (the teachers are "Transformer-DLCL-RPR" with a maximum relative
  length of 8, Sec. 3.1; the method is Shaw et al., 2018), optional and in encoder
  self-attention only: per layer, key and value tables of 2k+1 rows of d_head shared by
  the heads; query i and key j use row clip(j - i, -k, k) + k; the key row is added to
  the key inside the scaled score, the value row to the value inside the weighted sum.
"""
from __future__ import annotations

import math

import numpy as np

import synth


# ---------------------------------------------------------------------------
# Primitives
# ---------------------------------------------------------------------------
def layer_norm(x, gamma, beta, eps=1e-5):
    """LN(u) = gamma * (u - mean) / sqrt(var + eps) + beta over the last axis (biased var)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gamma + beta


def positional_encoding(positions, d, dtype=np.float64):
    """Sinusoidal encoding: PE(p, 2m) = sin(p / 10000^(2m/d)), PE(p, 2m+1) = cos(same)."""
    pos = np.asarray(positions, dtype=np.float64)[:, None]
    m = np.arange(d // 2, dtype=np.float64)[None, :]
    ang = pos / np.power(10000.0, 2.0 * m / d)
    pe = np.empty((pos.shape[0], d), dtype=np.float64)
    pe[:, 0::2] = np.sin(ang)
    pe[:, 1::2] = np.cos(ang)
    return pe.astype(dtype)


def softmax(x, axis=-1):
    m = np.max(x, axis=axis, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=axis, keepdims=True)


def logsumexp(x, axis=-1):
    m = np.max(x, axis=axis, keepdims=True)
    return (m + np.log(np.exp(x - m).sum(axis=axis, keepdims=True))).squeeze(axis)


def rel_index(tq, tk, rel_k):
    """Table row of query i and key j: clip(j - i, -rel_k, rel_k) + rel_k."""
    return np.clip(np.arange(tk)[None, :] - np.arange(tq)[:, None], -rel_k, rel_k) + rel_k


def attention(q, k, v, n_heads, allowed=None, rel=None):
    """Multi-head scaled dot-product attention on already-projected q [Tq,d], k/v [Tk,d].

    Head h uses columns h*dh..(h+1)*dh.  ``allowed`` [Tq,Tk] (bool) masks keys with -inf.
    ``rel`` = (table_k, table_v, rel_k) adds relative position representations (shared
    by the heads): score_ij = q_i . (k_j + table_k[r_ij]) / sqrt(dh) and
    out_i = sum_j p_ij (v_j + table_v[r_ij]), r_ij = rel_index(...)[i, j].
    Returns the concatenated head outputs [Tq, d] (before the output projection).
    """
    tq, d = q.shape
    dh = d // n_heads
    out = np.empty((tq, d), dtype=q.dtype)
    scale = 1.0 / math.sqrt(dh)
    if rel is not None:
        ridx = rel_index(tq, k.shape[0], rel[2])
        ak, av = rel[0][ridx], rel[1][ridx]          # [Tq, Tk, dh]
    for h in range(n_heads):
        sl = slice(h * dh, (h + 1) * dh)
        s = q[:, sl] @ k[:, sl].T
        if rel is not None:
            s = s + np.einsum("id,ijd->ij", q[:, sl], ak)
        s = s * q.dtype.type(scale)
        if allowed is not None:
            s = np.where(allowed, s, -np.inf)
        p = softmax(s, axis=-1)
        out[:, sl] = p @ v[:, sl]
        if rel is not None:
            out[:, sl] += np.einsum("ij,ijd->id", p, av)
    return out


def e4m3_round(x) -> np.ndarray:
    """Nearest FP8 E4M3 value (the OCP "fn" format: 4 exponent bits with bias 7, 3
    mantissa bits, subnormals of 2^-9, no infinities, largest finite 448), ties to even;
    magnitudes beyond 448 saturate to 448.  Returned as float64 values."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    _, E = np.frexp(a)                            # a = f * 2^E with f in [0.5, 1)
    e = np.maximum(E - 1, -6)                     # binade exponent; below 2^-6 the step is 2^-9
    step = np.ldexp(1.0, e - 3)                   # 3 mantissa bits
    q = np.minimum(np.round(a / step) * step, 448.0)   # np.round: half to even
    return np.copysign(q, x)


def quantize_fp8_columns(w):
    """FP8 E4M3 weight quantization with one scale per output column of an [in, out]
    matrix (the lower-precision weights that the paper leaves to future work, Sec. 6):
    scale_n = max_k |w[k, n]| / 448 computed in float32 (1 for an all-zero column), and
    q[k, n] = e4m3_round(float32(w[k, n] / scale_n)), the division in float32 too.
    Returns (q as float64 values, scale as float32); the weight stands for q * scale."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=0)
    scale = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    q = e4m3_round((w / scale[None, :]).astype(np.float32))
    return q, scale


def round_weights(blob: np.ndarray, shape: synth.ModelShape, precision: str) -> np.ndarray:
    """Return a copy of the fp32 blob whose *matrices* (E and every W_*) are rounded as
    the GPU stores them and widened back.  "f16" / "bf16": round to nearest even.
    "f8" (and "f8w", the same weights): the projection matrices W_* become q * scale of :func:`quantize_fp8_columns`
    (exact in float64, which is then the returned dtype) and E is rounded to fp16, as
    an FP8-weight model with fp16 activations stores them; the decoder projections fed by
    a pre-norm LayerNorm quantize the gain-scaled weights instead (see
    :func:`_fp8_fold_layernorm`; their biases change accordingly).  Biases, LayerNorm and DLCL
    scalars keep fp32: that is what a reduced-precision model stores at full precision.
    """
    if precision == "f32":
        return blob.copy()
    if precision in ("f8", "f8w"):
        out = blob.astype(np.float64)
        off = 0
        where = {}
        for e in synth.weight_layout(shape):
            where[e.name] = (off, e)
            seg = blob[off:off + e.size]
            if e.name == "E":
                out[off:off + e.size] = seg.astype(np.float16)
            elif ".W_" in e.name:
                q, sc = quantize_fp8_columns(seg.reshape(e.shape))
                out[off:off + e.size] = (q * sc.astype(np.float64)[None, :]).reshape(-1)
            off += e.size
        for j in range(shape.n_dec):
            for ln, w, b in (("ln1", "W_qkv", "b_qkv"), ("ln2", "W_q", "b_q"), ("ln3", "W_1", "b_1")):
                _fp8_fold_layernorm(blob, out, where, f"dec.{j}.", ln, w, b)
        return out
    out = blob.copy()
    off = 0
    for e in synth.weight_layout(shape):
        if e.name == "E" or ".W_" in e.name:
            seg = out[off:off + e.size]
            if precision == "f16":
                seg[:] = seg.astype(np.float16).astype(np.float32)
            elif precision == "bf16":
                u = seg.view(np.uint32).astype(np.uint64)
                u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
                seg[:] = u.astype(np.uint32).view(np.float32)
            else:
                raise ValueError(precision)
        off += e.size
    return out


def _fp8_fold_layernorm(blob, out, where, p, ln, w, b):
    """FP8 weights of a decoder projection that takes a pre-norm LayerNorm's output.

    Reading (the paper leaves lower precision to future work, Sec. 6): such a projection
    stores its weights with the LayerNorm's gain folded in, Q = fp8(diag(gamma) W) with
    diag(gamma) W formed in float32 and quantized per output column, and computes
    LN0(u) Q + b + beta W, LN0 being the LayerNorm without gain and bias.  The same
    function is written here as weights for the plain form LN(u; gamma, beta) W' + b':
    W' = diag(gamma)^-1 Q and b' = b + beta (W - W'), since
    (LN0(u) * gamma + beta) W' + b' = LN0(u) Q + b + beta W.  A row with gamma = 0 gets
    W' = 0: its LayerNorm output is the constant beta, whose product b' already holds."""
    (og, eg), (ow, ew), (ob, eb) = where[p + ln + ".gamma"], where[p + w], where[p + b]
    gamma = blob[og:og + eg.size]
    beta = blob[og + eg.size:og + 2 * eg.size]
    W = blob[ow:ow + ew.size].reshape(ew.shape)
    q, sc = quantize_fp8_columns((gamma[:, None] * W).astype(np.float32))
    Q = q * sc.astype(np.float64)[None, :]
    g = gamma.astype(np.float64)[:, None]
    W_eff = np.divide(Q, g, out=np.zeros_like(Q), where=g != 0)
    out[ow:ow + ew.size] = W_eff.reshape(-1)
    out[ob:ob + eb.size] = blob[ob:ob + eb.size].astype(np.float64) + beta.astype(np.float64) @ (W.astype(np.float64) - W_eff)


def param_count_formula(V, d, F, L, Ld):
    """Matrix parameters of a tied-embedding Transformer with L encoder / Ld decoder layers:
    V*d + L*(4 d^2 + 2 d F) + Ld*(8 d^2 + 2 d F)."""
    return V * d + L * (4 * d * d + 2 * d * F) + Ld * (8 * d * d + 2 * d * F)


# ---------------------------------------------------------------------------
# Model
# ---------------------------------------------------------------------------
class OracleModel:
    """The full model on one sentence at a time.

    ``blob`` is the canonical fp32 weight vector; ``precision`` rounds its matrices as
    the GPU stores them ("f32", "f16", "bf16", "f8"); arithmetic is done in ``dtype``.
    ``kv_fp8`` keeps the decoder's self-attention keys and values as E4M3 values (by
    default with precision "f8", the FP8 mode; "f8w" is FP8 weights alone).
    """

    def __init__(self, shape: synth.ModelShape, blob: np.ndarray, dtype=np.float64,
                 precision: str = "f32", hist_norm: bool = True, eps: float = 1e-5, kv_fp8=None):
        self.shape = shape
        self.dtype = np.dtype(dtype)
        self.hist_norm = hist_norm
        self.eps = eps
        self.kv_fp8 = precision == "f8" if kv_fp8 is None else bool(kv_fp8)
        named = synth.unpack(shape, round_weights(blob, shape, precision))
        self.p = {k: v.astype(self.dtype) for k, v in named.items()}
        self.d = shape.d_model
        self.H = shape.n_heads
        self.scale_emb = self.dtype.type(math.sqrt(self.d))

    # -- pieces ---------------------------------------------------------------
    def ln(self, x, prefix):
        return layer_norm(x, self.p[prefix + ".gamma"], self.p[prefix + ".beta"], self.eps)

    def embed(self, ids, positions):
        ids = np.asarray(ids, dtype=np.int64)
        return self.scale_emb * self.p["E"][ids] + positional_encoding(positions, self.d, self.dtype)

    def hist_entry(self, y, k):
        """N_k(y_k): the k-th history LayerNorm of Eq. 2, or the identity."""
        return self.ln(y, f"hist_ln.{k}") if self.hist_norm else y

    def dlcl_row(self, l):
        """W[l, 0..l-1] for row l (1-based)."""
        return self.p[f"dlcl.{l}"]

    def enc_layer(self, x, i):
        """One pre-norm encoder layer: a = x + MHA(LN1 x); y = a + FFN(LN2 a)."""
        p = f"enc.{i}."
        d = self.d
        u = self.ln(x, p + "ln1")
        qkv = u @ self.p[p + "W_qkv"] + self.p[p + "b_qkv"]
        rel = (self.p[p + "rel_k"], self.p[p + "rel_v"], self.shape.rel_k) if self.shape.rel_k > 0 else None
        att = attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], self.H, rel=rel)
        a = x + att @ self.p[p + "W_o"] + self.p[p + "b_o"]
        u = self.ln(a, p + "ln2")
        f = np.maximum(u @ self.p[p + "W_1"] + self.p[p + "b_1"], 0)
        return a + f @ self.p[p + "W_2"] + self.p[p + "b_2"]

    # -- encoder (Eq. 1-2) ----------------------------------------------------
    def encode(self, src, return_history=False):
        """DLCL encoder over one unpadded sentence; returns enc [S, d]."""
        L = self.shape.n_enc
        src = np.asarray(src)
        y = self.embed(src, np.arange(len(src)))
        hist = [self.hist_entry(y, 0)]
        for l in range(1, L + 1):
            w = self.dlcl_row(l)
            x = sum(w[k] * hist[k] for k in range(l))
            y = self.enc_layer(x, l - 1)
            hist.append(self.hist_entry(y, l))
        w = self.dlcl_row(L + 1)
        x = sum(w[k] * hist[k] for k in range(L + 1))
        enc = self.ln(x, "enc_out_ln")
        return (enc, hist) if return_history else enc

    def cross_kv(self, enc):
        """Encoder-decoder K/V of every decoder layer, computed once per sentence."""
        d = self.d
        out = []
        for j in range(self.shape.n_dec):
            kv = enc @ self.p[f"dec.{j}.W_kv"] + self.p[f"dec.{j}.b_kv"]
            out.append((kv[:, :d], kv[:, d:]))
        return out

    # -- decoder ----------------------------------------------------------------
    def self_kv(self, k, v):
        """A self-attention key/value as the cache keeps it (E4M3 values with kv_fp8)."""
        if self.kv_fp8:
            return e4m3_round(k).astype(self.dtype), e4m3_round(v).astype(self.dtype)
        return k, v

    def dec_layer_step(self, z, j, cache_k, cache_v, cross):
        """Incremental decoder layer for one row z [d] at the newest position.

        cache_k/cache_v: the row's earlier self-attention keys/values [t, d] of this
        layer (t may be 0).  Returns (z', k_new, v_new)."""
        p = f"dec.{j}."
        d = self.d
        u = self.ln(z[None, :], p + "ln1")
        qkv = u @ self.p[p + "W_qkv"] + self.p[p + "b_qkv"]
        k_new, v_new = self.self_kv(qkv[:, d:2 * d], qkv[:, 2 * d:])
        k_all = np.concatenate([cache_k, k_new], axis=0)
        v_all = np.concatenate([cache_v, v_new], axis=0)
        att = attention(qkv[:, :d], k_all, v_all, self.H)
        z = z + (att @ self.p[p + "W_o"] + self.p[p + "b_o"])[0]
        u = self.ln(z[None, :], p + "ln2")
        q = u @ self.p[p + "W_q"] + self.p[p + "b_q"]
        att = attention(q, cross[j][0], cross[j][1], self.H)
        z = z + (att @ self.p[p + "W_oc"] + self.p[p + "b_oc"])[0]
        u = self.ln(z[None, :], p + "ln3")
        f = np.maximum(u @ self.p[p + "W_1"] + self.p[p + "b_1"], 0)
        z = z + (f @ self.p[p + "W_2"] + self.p[p + "b_2"])[0]
        return z, k_new[0], v_new[0]

    def output_logits(self, z):
        """logits = LN_dec(z) E^T (tied projection, no bias)."""
        return self.ln(z, "dec_out_ln") @ self.p["E"].T

    def decode_full(self, cross, tokens):
        """Full recompute: decoder over [BOS] + tokens with a causal mask.

        Returns logits [len(tokens)+1, V]; row t predicts the token after position t."""
        d, n = self.d, len(tokens) + 1
        inp = np.concatenate([[synth.BOS_ID], np.asarray(tokens, dtype=np.int64)]).astype(np.int64)
        z = self.embed(inp, np.arange(n))
        causal = np.tril(np.ones((n, n), dtype=bool))
        for j in range(self.shape.n_dec):
            p = f"dec.{j}."
            u = self.ln(z, p + "ln1")
            qkv = u @ self.p[p + "W_qkv"] + self.p[p + "b_qkv"]
            k, v = self.self_kv(qkv[:, d:2 * d], qkv[:, 2 * d:])
            att = attention(qkv[:, :d], k, v, self.H, causal)
            z = z + att @ self.p[p + "W_o"] + self.p[p + "b_o"]
            u = self.ln(z, p + "ln2")
            q = u @ self.p[p + "W_q"] + self.p[p + "b_q"]
            z = z + attention(q, cross[j][0], cross[j][1], self.H) @ self.p[p + "W_oc"] + self.p[p + "b_oc"]
            u = self.ln(z, p + "ln3")
            f = np.maximum(u @ self.p[p + "W_1"] + self.p[p + "b_1"], 0)
            z = z + f @ self.p[p + "W_2"] + self.p[p + "b_2"]
        return self.output_logits(z)

    def teacher_forced_logits(self, src, tokens, incremental=True):
        """Logits of every step when the decoder is fed ``tokens`` (BOS first)."""
        cross = self.cross_kv(self.encode(src))
        if not incremental:
            return self.decode_full(cross, tokens)
        sc = IncrementalScorer(self, src, cross=cross)
        rows = []
        prefix: list = []
        for t in range(len(tokens) + 1):
            logits, _ = sc([prefix])
            rows.append(logits[0])
            if t < len(tokens):
                prefix = prefix + [int(tokens[t])]
        return np.stack(rows)


class IncrementalScorer:
    """Next-token logits for a set of target prefixes, with cached keys/values.

    Called once per step with every live prefix of length t (all of the same length);
    the caches of the previous step's prefixes are looked up by the prefix minus its
    last token, extended by one slot, and kept for the next step only.  Returns
    (logits [n, V], lse [n])."""

    def __init__(self, model: OracleModel, src, cross=None):
        self.m = model
        self.cross = cross if cross is not None else model.cross_kv(model.encode(src))
        Ld, d = model.shape.n_dec, model.d
        empty = np.zeros((0, d), dtype=model.dtype)
        self.caches = {(): [(empty, empty) for _ in range(Ld)]}
        self.t = 0

    def __call__(self, prefixes):
        m = self.m
        t = len(prefixes[0]) if prefixes else 0
        new_caches = {}
        logits = []
        for pre in prefixes:
            pre = tuple(int(x) for x in pre)
            assert len(pre) == t
            parent = self.caches[pre[:-1]] if t > 0 else self.caches[()]
            token = pre[-1] if t > 0 else synth.BOS_ID
            z = m.embed([token], [t])[0]
            layer_caches = []
            for j in range(m.shape.n_dec):
                ck, cv = parent[j]
                z, k_new, v_new = m.dec_layer_step(z, j, ck, cv, self.cross)
                layer_caches.append((np.concatenate([ck, k_new[None]]), np.concatenate([cv, v_new[None]])))
            new_caches[pre] = layer_caches
            logits.append(m.output_logits(z[None, :])[0])
        self.caches = new_caches
        logits = np.stack(logits)
        return logits, logsumexp(logits, axis=-1)


class FullRecomputeScorer:
    """Same interface as IncrementalScorer, recomputing the whole prefix every call."""

    def __init__(self, model: OracleModel, src, cross=None):
        self.m = model
        self.cross = cross if cross is not None else model.cross_kv(model.encode(src))

    def __call__(self, prefixes):
        logits = np.stack([self.m.decode_full(self.cross, list(p))[-1] for p in prefixes])
        return logits, logsumexp(logits, axis=-1)
