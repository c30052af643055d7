"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle.

This module only *generates inputs*: model shapes, the canonical weight blob and
token-ID batches.  It holds none of the translation method's arithmetic (no
embedding, normalisation, attention or search), so the oracle and the HIP path
can both consume it without sharing any of the computation they are compared on.

Conventions fixed here (they are interface definitions, not model math):

* Special IDs: PAD = 0, BOS = 1, EOS = 2, UNK = 3; synthetic source IDs are drawn
  from [4, V).
* The weight blob is one fp32 vector in the canonical order returned by
  :func:`weight_layout`; matrices are row-major "in x out" (y = x @ W).
* Random draws use ``numpy.random.default_rng`` (PCG64): weights from seed 0,
  data from seed 1, lengths first and then IDs sentence by sentence.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

PAD_ID, BOS_ID, EOS_ID, UNK_ID = 0, 1, 2, 3
FIRST_WORD_ID = 4
MAX_POSITIONS = 1024  # maximum source/target position of the paper's models (Sec. 2.2)


@dataclass(frozen=True)
class ModelShape:
    d_model: int
    n_heads: int
    d_ffn: int
    n_enc: int
    n_dec: int
    vocab: int
    max_positions: int = MAX_POSITIONS
    rel_k: int = 0          # relative positions in encoder self-attention: clip distance (0 = off)

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclass(frozen=True)
class SearchSetup:
    beam: int = 1
    len_penalty: float = 0.0
    max_len_a: float = 1.5
    max_len_b: int = 10
    max_len_cap: int = 0      # > 0: no target longer than this (0: no cap)
    token_budget: int = 8192
    max_batch_sents: int = 0
    early_stop: int = 1
    prune: int = 1


@dataclass(frozen=True)
class DataSetup:
    n_sent: int
    length_kind: str          # "uniform" or "lognormal"
    length_a: float           # uniform: low (incl.)  | lognormal: mean
    length_b: int             # uniform: high (incl.) | lognormal: max (clip)
    id_kind: str              # "uniform" or "zipf"
    zipf_s: float = 1.1


@dataclass(frozen=True)
class Member:
    """One model of an ensemble workload: its shape, its weights' seed, and whether it is
    a DLCL model (Eq. 2) or a plain pre-norm stack (one-hot DLCL rows with the identity
    in place of the history LayerNorm, which is exactly the plain stack)."""
    model: ModelShape
    weights_seed: int
    dlcl: bool = True


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    data: DataSetup
    search: SearchSetup
    dtype: str                # "f32" | "f16" | "bf16" | "f8" (fp16 activations, FP8 E4M3 weights and
                              # self-attention key/value cache) | "f8w" (FP8 weights alone)
    description: str = ""
    weights_seed: int = 0
    data_seed: int = 1
    members: tuple = ()       # ensemble workloads: the Members (``model`` is the first one's)
    ensemble_rule: int = 0    # 0: mean of the members' log-probs; 1: log of their mean probability


# The five workloads of the benchmark table.  Budgets for the two workloads that
# name none are 8192 padded source tokens.
# The teachers of Sec. 2.2 (Table 1): 35 or 40 encoder layers, with or without DLCL, six
# decoder layers, d = 512, 8 heads, relative positions with maximum distance 8.
_TEACHER = dict(d_model=512, n_heads=8, d_ffn=2048, n_dec=6, vocab=32000, rel_k=8)
_TEACHERS = (
    Member(ModelShape(n_enc=35, **_TEACHER), 10, dlcl=False),
    Member(ModelShape(n_enc=35, **_TEACHER), 11, dlcl=True),
    Member(ModelShape(n_enc=40, **_TEACHER), 12, dlcl=False),
    Member(ModelShape(n_enc=40, **_TEACHER), 13, dlcl=True),
)

WORKLOADS = {
    "tiny": Workload(
        "tiny",
        ModelShape(128, 4, 512, 6, 1, 1000),
        DataSetup(8, "uniform", 8, 16, "uniform"),
        SearchSetup(beam=1, len_penalty=0.0, max_len_a=0.0, max_len_b=24, token_budget=8192),
        "f32",
        "Tiny 6-1, d=128, 8 sentences of 8-16 uniform IDs, greedy, max 24 target tokens, fp32",
    ),
    "base-6-6": Workload(
        "base-6-6",
        ModelShape(512, 8, 2048, 6, 6, 32000),
        DataSetup(2048, "lognormal", 25.0, 100, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=8192),
        "f16",
        "Base 6-6, d=512, 2048 sentences (lognormal mean 25, max 100, Zipf(1.1) IDs), beam 4, fp16",
    ),
    "deep-shallow-greedy": Workload(
        "deep-shallow-greedy",
        ModelShape(512, 8, 2048, 35, 1, 32000),
        DataSetup(8192, "lognormal", 25.0, 150, "zipf"),
        SearchSetup(beam=1, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=8192),
        "f16",
        "Deep-shallow 35-1, d=512, 8192 sentences (mean 25, max 150), greedy, budget 8192, pruning, fp16",
    ),
    "deep-shallow-beam": Workload(
        "deep-shallow-beam",
        ModelShape(512, 8, 2048, 35, 1, 32000),
        DataSetup(8192, "lognormal", 25.0, 150, "zipf"),
        SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.5, max_len_b=10, token_budget=16384),
        "f16",
        "Deep-shallow 35-1, d=512, 8192 sentences, beam 4, length penalty 0.6, budget 16384, fp16",
    ),
    "base-6-6-rpr": Workload(
        "base-6-6-rpr",
        ModelShape(512, 8, 2048, 6, 6, 32000, rel_k=8),
        DataSetup(2048, "lognormal", 25.0, 100, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=8192),
        "f16",
        "Base 6-6 with relative positions (k = 8) in encoder self-attention, as in the DLCL-RPR teachers; "
        "otherwise base-6-6",
    ),
    "teacher-ensemble": Workload(
        "teacher-ensemble",
        _TEACHERS[0].model,
        DataSetup(2998, "lognormal", 25.0, 100, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=8192),
        "f16",
        "Ensemble of the four teachers of Table 1 (35-6 and 40-6, each with and without DLCL, "
        "relative positions k = 8, d=512), 2998 sentences (the size of newstest2018; lognormal mean 25, "
        "max 100, Zipf(1.1) IDs), beam 4, mean of the members' log-probs, fp16",
        members=_TEACHERS,
    ),
    "base-6-6-fp8": Workload(
        "base-6-6-fp8",
        ModelShape(512, 8, 2048, 6, 6, 32000),
        DataSetup(2048, "lognormal", 25.0, 100, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=8192),
        "f8",
        "Base 6-6 with FP8 E4M3 projection weights (column scales), an FP8 E4M3 self-attention key/value "
        "cache and fp16 activations; otherwise base-6-6",
    ),
    "wide-30-6-fp8": Workload(
        "wide-30-6-fp8",
        ModelShape(1024, 16, 4096, 30, 6, 32000),
        DataSetup(4096, "lognormal", 30.0, 200, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=16384),
        "f8",
        "Wide 30-6 with FP8 E4M3 projection weights (column scales), an FP8 E4M3 self-attention key/value "
        "cache and fp16 activations; otherwise wide-30-6",
    ),
    "wide-30-6": Workload(
        "wide-30-6",
        ModelShape(1024, 16, 4096, 30, 6, 32000),
        DataSetup(4096, "lognormal", 30.0, 200, "zipf"),
        SearchSetup(beam=4, len_penalty=0.0, max_len_a=1.5, max_len_b=10, token_budget=16384),
        "f16",
        "Wide 30-6, d=1024, 4096 sentences (mean 30, max 200), beam 4, budget 16384, fp16",
    ),
}


# --------------------------------------------------------------------------
# Weight blob layout
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Entry:
    name: str
    shape: tuple
    init: str            # "normal" | "gamma" | "dlcl"
    dlcl_row: int = 0    # for init == "dlcl": the row index l (1-based)

    @property
    def size(self) -> int:
        return int(np.prod(self.shape))


def weight_layout(m: ModelShape) -> list[Entry]:
    """Canonical order of every parameter in the fp32 weight blob.

    E [V,d] is tied: source embedding, target embedding and output projection.
    The DLCL weights are stored row by row, row l (l = 1..L+1) holding l scalars
    W[l, 0..l-1]; each history entry k = 0..L has its own LayerNorm.
    """
    d, F, V, L, Ld = m.d_model, m.d_ffn, m.vocab, m.n_enc, m.n_dec
    out: list[Entry] = [Entry("E", (V, d), "normal")]
    for k in range(L + 1):
        out += [Entry(f"hist_ln.{k}.gamma", (d,), "gamma"), Entry(f"hist_ln.{k}.beta", (d,), "normal")]
    for l in range(1, L + 2):
        out.append(Entry(f"dlcl.{l}", (l,), "dlcl", l))
    for i in range(L):
        p = f"enc.{i}."
        out += [
            Entry(p + "ln1.gamma", (d,), "gamma"), Entry(p + "ln1.beta", (d,), "normal"),
            Entry(p + "W_qkv", (d, 3 * d), "normal"), Entry(p + "b_qkv", (3 * d,), "normal"),
            Entry(p + "W_o", (d, d), "normal"), Entry(p + "b_o", (d,), "normal"),
            Entry(p + "ln2.gamma", (d,), "gamma"), Entry(p + "ln2.beta", (d,), "normal"),
            Entry(p + "W_1", (d, F), "normal"), Entry(p + "b_1", (F,), "normal"),
            Entry(p + "W_2", (F, d), "normal"), Entry(p + "b_2", (d,), "normal"),
        ]
        if m.rel_k > 0:   # relative key / value tables [2k+1, d_head], shared by the heads
            out += [Entry(p + "rel_k", (2 * m.rel_k + 1, m.d_head), "normal"),
                    Entry(p + "rel_v", (2 * m.rel_k + 1, m.d_head), "normal")]
    out += [Entry("enc_out_ln.gamma", (d,), "gamma"), Entry("enc_out_ln.beta", (d,), "normal")]
    for j in range(Ld):
        p = f"dec.{j}."
        out += [
            Entry(p + "ln1.gamma", (d,), "gamma"), Entry(p + "ln1.beta", (d,), "normal"),
            Entry(p + "W_qkv", (d, 3 * d), "normal"), Entry(p + "b_qkv", (3 * d,), "normal"),
            Entry(p + "W_o", (d, d), "normal"), Entry(p + "b_o", (d,), "normal"),
            Entry(p + "ln2.gamma", (d,), "gamma"), Entry(p + "ln2.beta", (d,), "normal"),
            Entry(p + "W_q", (d, d), "normal"), Entry(p + "b_q", (d,), "normal"),
            Entry(p + "W_kv", (d, 2 * d), "normal"), Entry(p + "b_kv", (2 * d,), "normal"),
            Entry(p + "W_oc", (d, d), "normal"), Entry(p + "b_oc", (d,), "normal"),
            Entry(p + "ln3.gamma", (d,), "gamma"), Entry(p + "ln3.beta", (d,), "normal"),
            Entry(p + "W_1", (d, F), "normal"), Entry(p + "b_1", (F,), "normal"),
            Entry(p + "W_2", (F, d), "normal"), Entry(p + "b_2", (d,), "normal"),
        ]
    out += [Entry("dec_out_ln.gamma", (d,), "gamma"), Entry("dec_out_ln.beta", (d,), "normal")]
    return out


def blob_size(m: ModelShape) -> int:
    return sum(e.size for e in weight_layout(m))


_LIVELY_DEC_ATTN = (".W_qkv", ".W_q", ".W_kv", ".W_oc")


def _lively_std(e: Entry, m: ModelShape, std: float) -> float:
    """Per-entry std of the test-only "lively" recipe (see make_weights)."""
    r = math.sqrt(128.0 / m.d_model)
    if e.name == "E":
        return 0.01 * r
    if e.name.startswith("dec.") and e.name.endswith(_LIVELY_DEC_ATTN):
        return 0.4 * r
    if e.name.endswith((".rel_k", ".rel_v")):
        return 0.5
    return std


def make_weights(m: ModelShape, seed: int = 0, eos_boost: float | None = None,
                 std: float = 0.02, lively: bool = False, plain_stack: bool = False) -> np.ndarray:
    """Draw the fp32 weight blob in canonical order.

    Every entry is N(0, std) drawn in fp64; LayerNorm gains get +1 and DLCL row l
    gets +1/l (uniform averaging plus noise).

    Under N(0, 0.02) the tied projection makes a random decoder repeat one token
    forever and EOS practically never wins, which is fine for throughput but
    exercises little of the search.  ``lively=True`` (tests only) draws E with a
    smaller std and the decoder's attention matrices with a larger one, so the
    emitted tokens depend on the source and the step, and boosts the EOS row of E
    (default x5) so hypotheses finish at varied steps.  ``eos_boost`` scales the EOS
    row of E explicitly.  ``plain_stack=True`` makes every DLCL row one-hot on its last
    entry (W[l, l-1] = 1), the weights of a model without layer combination; it is run
    with the history LayerNorm off.
    """
    rng = np.random.default_rng(seed)
    lay = weight_layout(m)
    blob = np.empty(sum(e.size for e in lay), dtype=np.float32)
    off = 0
    for e in lay:
        s = _lively_std(e, m, std) if lively else std
        x = rng.normal(0.0, s, e.size)
        if e.init == "gamma":
            x += 1.0
        elif e.init == "dlcl":
            if plain_stack:
                x = np.zeros(e.size)
                x[-1] = 1.0
            else:
                x += 1.0 / e.dlcl_row
        blob[off:off + e.size] = x
        off += e.size
    if lively and eos_boost is None:
        eos_boost = 5.0
    if eos_boost is not None:
        d = m.d_model
        blob[EOS_ID * d:(EOS_ID + 1) * d] *= np.float32(eos_boost)
    return blob


def unpack(m: ModelShape, blob: np.ndarray) -> dict:
    """Named views into a blob (no copy)."""
    out = {}
    off = 0
    for e in weight_layout(m):
        out[e.name] = blob[off:off + e.size].reshape(e.shape)
        off += e.size
    assert off == blob.size, (off, blob.size)
    return out


def pack(m: ModelShape, named: dict) -> np.ndarray:
    """Inverse of :func:`unpack` (used by tests that build special weights)."""
    parts = [np.asarray(named[e.name], dtype=np.float32).reshape(-1) for e in weight_layout(m)]
    return np.concatenate(parts)


# --------------------------------------------------------------------------
# Token batches
# --------------------------------------------------------------------------
def zipf_cdf(n_ranks: int, s: float) -> np.ndarray:
    p = np.arange(1, n_ranks + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(p)
    return c / c[-1]


def make_sentences(data: DataSetup, vocab: int, seed: int = 1, n_sent: int | None = None):
    """Source sentences in CSR form: (ids int32 [sum len], offsets int64 [n+1]).

    Lengths are drawn first (uniform, or clip(rint(exp(N(ln(mean) - 0.125, 0.5))), 1, max)),
    then the IDs sentence by sentence (uniform on [4, V), or a finite Zipf(s) over ranks
    1..V-4 sampled by inverse CDF with ID = 3 + rank).
    """
    n = data.n_sent if n_sent is None else n_sent
    rng = np.random.default_rng(seed)
    if data.length_kind == "uniform":
        lens = rng.integers(int(data.length_a), int(data.length_b) + 1, size=n)
    elif data.length_kind == "lognormal":
        mu = math.log(data.length_a) - 0.125
        lens = np.clip(np.rint(np.exp(rng.normal(mu, 0.5, size=n))), 1, data.length_b)
    else:
        raise ValueError(data.length_kind)
    lens = lens.astype(np.int64)
    offs = np.zeros(n + 1, dtype=np.int64)
    offs[1:] = np.cumsum(lens)
    ids = np.empty(int(offs[-1]), dtype=np.int32)
    cdf = zipf_cdf(vocab - FIRST_WORD_ID, data.zipf_s) if data.id_kind == "zipf" else None
    for i in range(n):
        k = int(lens[i])
        if data.id_kind == "uniform":
            ids[offs[i]:offs[i + 1]] = rng.integers(FIRST_WORD_ID, vocab, size=k)
        elif data.id_kind == "zipf":
            u = rng.random(k)
            r = np.searchsorted(cdf, u, side="right") + 1
            ids[offs[i]:offs[i + 1]] = np.minimum(r, vocab - FIRST_WORD_ID) + (FIRST_WORD_ID - 1)
        else:
            raise ValueError(data.id_kind)
    return ids, offs


def sentence_list(ids: np.ndarray, offs: np.ndarray) -> list:
    return [ids[offs[i]:offs[i + 1]] for i in range(len(offs) - 1)]


def max_target_len(search: SearchSetup, src_len: int) -> int:
    """Per-sentence target cap: floor(a * S_i) + b tokens, EOS included, lowered to
    max_len_cap when that is positive."""
    n = int(math.floor(search.max_len_a * src_len)) + int(search.max_len_b)
    cap = int(getattr(search, "max_len_cap", 0))
    return min(n, cap) if cap > 0 else n


def stratified_subset(offs: np.ndarray, k: int) -> np.ndarray:
    """Indices of every (n/k)-th sentence of the length-sorted order (longest first)."""
    lens = np.diff(offs)
    n = len(lens)
    order = sorted(range(n), key=lambda i: (-int(lens[i]), i))
    if k >= n:
        return np.array(order, dtype=np.int64)
    step = n / k
    return np.array([order[int(j * step)] for j in range(k)], dtype=np.int64)


def small_model(d_model=64, n_heads=4, d_ffn=None, n_enc=3, n_dec=2, vocab=97) -> ModelShape:
    """Shapes for fast tests (several GEMM tiles, a ragged vocab)."""
    return ModelShape(d_model, n_heads, d_ffn or 4 * d_model, n_enc, n_dec, vocab)


def member_weights(w: Workload, **kw) -> list:
    """Weight blobs of an ensemble workload's members, in member order."""
    return [make_weights(mb.model, seed=mb.weights_seed, plain_stack=not mb.dlcl, **kw) for mb in w.members]


def with_search(w: Workload, **kw) -> Workload:
    return replace(w, search=replace(w.search, **kw))
