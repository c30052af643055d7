"""Pins for the oracle model (encoder with DLCL, cached decoder).

* One-hot DLCL rows reduce Eq. 2 to a plain pre-norm stack; that stack is checked
  against torch's own Transformer layers (norm_first) in fp64, a library routine
  written independently of the oracle.
* Eq. 2 is linear in each row of W: a general row equals the W-weighted sum of the
  one-hot results.
* Cached incremental decoding equals full-prefix recomputation (Sec. 4.1).
* Parameter counts of the paper's Tables 1-2 pin the architecture (tied E, F = 4d,
  self + cross attention in the decoder).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from oracle.model import FullRecomputeScorer, IncrementalScorer

HERE = os.path.dirname(__file__)
SHAPE = synth.ModelShape(d_model=32, n_heads=4, d_ffn=128, n_enc=3, n_dec=2, vocab=23)


def _blob(shape=SHAPE, seed=5, lively=True):
    return synth.make_weights(shape, seed=seed, lively=lively)


def _set_dlcl(shape, blob, rows):
    """Return a copy of blob whose DLCL rows are replaced: rows[l] = array of l entries."""
    named = {k: v.copy() for k, v in synth.unpack(shape, blob).items()}
    for l, r in rows.items():
        named[f"dlcl.{l}"][:] = r
    return synth.pack(shape, named)


def _onehot_prev(shape):
    """W[l, l-1] = 1 (layer l reads the previous layer's output only)."""
    return {l: np.eye(l)[l - 1] for l in range(1, shape.n_enc + 2)}


def _torch_stack(torch, shape, blob, src, tgt, hist_ln_between):
    """Reference model out of torch.nn Transformer layers (norm_first, ReLU, no dropout)."""
    d, H = shape.d_model, shape.n_heads
    P = {k: torch.tensor(v.astype(np.float64)) for k, v in synth.unpack(shape, blob).items()}

    def ln(prefix):
        m = torch.nn.LayerNorm(d, eps=1e-5)
        m.weight.data, m.bias.data = P[prefix + ".gamma"].clone(), P[prefix + ".beta"].clone()
        return m

    def pe(n):
        return torch.tensor(oracle.positional_encoding(np.arange(n), d))

    y = math.sqrt(d) * P["E"][torch.tensor(np.asarray(src, dtype=np.int64))] + pe(len(src))
    y = y[None]
    for i in range(shape.n_enc):
        lay = torch.nn.TransformerEncoderLayer(d, H, shape.d_ffn, dropout=0.0, batch_first=True, norm_first=True)
        p = f"enc.{i}."
        lay.self_attn.in_proj_weight.data = P[p + "W_qkv"].T.clone()
        lay.self_attn.in_proj_bias.data = P[p + "b_qkv"].clone()
        lay.self_attn.out_proj.weight.data = P[p + "W_o"].T.clone()
        lay.self_attn.out_proj.bias.data = P[p + "b_o"].clone()
        lay.linear1.weight.data, lay.linear1.bias.data = P[p + "W_1"].T.clone(), P[p + "b_1"].clone()
        lay.linear2.weight.data, lay.linear2.bias.data = P[p + "W_2"].T.clone(), P[p + "b_2"].clone()
        lay.norm1.weight.data, lay.norm1.bias.data = P[p + "ln1.gamma"].clone(), P[p + "ln1.beta"].clone()
        lay.norm2.weight.data, lay.norm2.bias.data = P[p + "ln2.gamma"].clone(), P[p + "ln2.beta"].clone()
        lay.train()
        if hist_ln_between:
            y = ln(f"hist_ln.{i}")(y)
        y = lay(y)
    if hist_ln_between:
        y = ln(f"hist_ln.{shape.n_enc}")(y)
    enc = ln("enc_out_ln")(y)

    inp = [synth.BOS_ID] + list(tgt)
    z = math.sqrt(d) * P["E"][torch.tensor(inp)] + pe(len(inp))
    z = z[None]
    causal = torch.nn.Transformer.generate_square_subsequent_mask(len(inp), dtype=torch.float64)
    for j in range(shape.n_dec):
        lay = torch.nn.TransformerDecoderLayer(d, H, shape.d_ffn, dropout=0.0, batch_first=True, norm_first=True)
        p = f"dec.{j}."
        lay.self_attn.in_proj_weight.data = P[p + "W_qkv"].T.clone()
        lay.self_attn.in_proj_bias.data = P[p + "b_qkv"].clone()
        lay.self_attn.out_proj.weight.data = P[p + "W_o"].T.clone()
        lay.self_attn.out_proj.bias.data = P[p + "b_o"].clone()
        lay.multihead_attn.in_proj_weight.data = torch.cat([P[p + "W_q"], P[p + "W_kv"]], 1).T.clone()
        lay.multihead_attn.in_proj_bias.data = torch.cat([P[p + "b_q"], P[p + "b_kv"]]).clone()
        lay.multihead_attn.out_proj.weight.data = P[p + "W_oc"].T.clone()
        lay.multihead_attn.out_proj.bias.data = P[p + "b_oc"].clone()
        lay.linear1.weight.data, lay.linear1.bias.data = P[p + "W_1"].T.clone(), P[p + "b_1"].clone()
        lay.linear2.weight.data, lay.linear2.bias.data = P[p + "W_2"].T.clone(), P[p + "b_2"].clone()
        for n in (1, 2, 3):
            norm = getattr(lay, f"norm{n}")
            norm.weight.data, norm.bias.data = P[p + f"ln{n}.gamma"].clone(), P[p + f"ln{n}.beta"].clone()
        lay.train()
        z = lay(z, enc, tgt_mask=causal)
    logits = ln("dec_out_ln")(z)[0] @ P["E"].T
    return enc[0].detach().numpy(), logits.detach().numpy()


SRC = [5, 9, 17, 4, 22, 8, 13]
TGT = [7, 3, 19, 2, 11]


@pytest.mark.parametrize("hist_norm", [False, True])
def test_onehot_dlcl_matches_torch_prenorm_stack(torch_cpu64, hist_norm):
    blob = _set_dlcl(SHAPE, _blob(), _onehot_prev(SHAPE))
    m = oracle.OracleModel(SHAPE, blob, hist_norm=hist_norm)
    enc = m.encode(SRC)
    logits = m.teacher_forced_logits(SRC, TGT)
    enc_ref, logits_ref = _torch_stack(torch_cpu64, SHAPE, blob, SRC, TGT, hist_ln_between=hist_norm)
    np.testing.assert_allclose(enc, enc_ref, atol=1e-11)
    np.testing.assert_allclose(logits, logits_ref, atol=1e-11)


def test_onehot_identity_history_is_an_exact_copy():
    """With one-hot rows and N = identity the combine is 1*h + 0*others: bitwise the layer chain."""
    blob = _set_dlcl(SHAPE, _blob(), _onehot_prev(SHAPE))
    m = oracle.OracleModel(SHAPE, blob, hist_norm=False)
    y = m.embed(SRC, np.arange(len(SRC)))
    for i in range(SHAPE.n_enc):
        y = m.enc_layer(y, i)
    np.testing.assert_array_equal(m.encode(SRC), m.ln(y, "enc_out_ln"))


def test_dlcl_combination_is_linear_in_each_row():
    """x_l(W) = sum_k W[l,k] x_l(e_k): entries of row l do not feed any history entry."""
    base = _blob()
    L = SHAPE.n_enc
    l = L + 1                                   # the row that forms the encoder output
    w = np.array([0.7, -0.2, 1.3, 0.45])
    rows = {l: w}
    m = oracle.OracleModel(SHAPE, _set_dlcl(SHAPE, base, rows))
    _, hist = m.encode(SRC, return_history=True)
    x_direct = sum(w[k] * hist[k] for k in range(l))
    parts = []
    for k in range(l):
        mk = oracle.OracleModel(SHAPE, _set_dlcl(SHAPE, base, {l: np.eye(l)[k]}))
        _, hk = mk.encode(SRC, return_history=True)
        parts.append(hk[k])
    np.testing.assert_allclose(x_direct, sum(w[k] * parts[k] for k in range(l)), atol=1e-13)
    # and the encoder output is LN_out of that combination
    np.testing.assert_allclose(m.encode(SRC), m.ln(x_direct, "enc_out_ln"), atol=1e-13)


def test_history_entries_do_not_depend_on_later_rows():
    base = _blob()
    m1 = oracle.OracleModel(SHAPE, base)
    m2 = oracle.OracleModel(SHAPE, _set_dlcl(SHAPE, base, {3: np.array([5.0, -1.0, 2.0])}))
    _, h1 = m1.encode(SRC, return_history=True)
    _, h2 = m2.encode(SRC, return_history=True)
    for k in range(3):
        np.testing.assert_array_equal(h1[k], h2[k])
    assert not np.allclose(h1[3], h2[3])


@pytest.mark.parametrize("shape", [SHAPE, synth.ModelShape(48, 3, 96, 2, 3, 31)])
def test_incremental_decoding_equals_full_recompute(shape):
    blob = _blob(shape)
    m = oracle.OracleModel(shape, blob)
    src = [4, 9, 12, 6, 5, 7, 8, 10, 11][: 6]
    tgt = [3, 14, 2, 9, 9, 1, 20, 5]
    inc = m.teacher_forced_logits(src, tgt, incremental=True)
    full = m.teacher_forced_logits(src, tgt, incremental=False)
    np.testing.assert_allclose(inc, full, rtol=0, atol=1e-12)
    # the scorer used by the searches agrees with the full recompute on a beam of prefixes
    inc_sc, full_sc = IncrementalScorer(m, src), FullRecomputeScorer(m, src)
    prefixes = [[]]
    for t in range(4):
        a, la = inc_sc(prefixes)
        b, lb = full_sc(prefixes)
        np.testing.assert_allclose(a, b, atol=1e-12)
        np.testing.assert_allclose(la, lb, atol=1e-12)
        prefixes = [p + [w] for p in prefixes[:2] for w in (3, 5)]
        prefixes = prefixes[:3]
        while len(set(map(len, prefixes))) != 1:
            prefixes.pop()


def test_fp32_oracle_tracks_fp64():
    blob = _blob()
    m64 = oracle.OracleModel(SHAPE, blob)
    m32 = oracle.OracleModel(SHAPE, blob, dtype=np.float32)
    a = m64.teacher_forced_logits(SRC, TGT)
    b = m32.teacher_forced_logits(SRC, TGT)
    assert b.dtype == np.float32
    np.testing.assert_allclose(a, b, atol=1e-4)


def test_param_counts_match_tables():
    with open(os.path.join(HERE, "golden", "param_counts.json")) as f:
        g = json.load(f)
    d, F, V = g["d_model"], g["d_ffn"], g["vocab"]
    for mdl in g["models"]:
        n = oracle.param_count_formula(V, d, F, mdl["n_enc"], mdl["n_dec"])
        shape = synth.ModelShape(d, 8, F, mdl["n_enc"], mdl["n_dec"], V)
        # every parameter of the layout (matrices, biases, LayerNorms, DLCL scalars)
        # rounds to the printed count
        assert round(synth.blob_size(shape) / 1e6) == mdl["params_M"], (mdl, synth.blob_size(shape))
        # the matrices are exactly the formula's, and dominate
        mats = sum(e.size for e in synth.weight_layout(shape) if e.name == "E" or ".W_" in e.name)
        assert mats == n
        assert abs(n / 1e6 - mdl["params_M"]) < 0.7
    # untied embeddings or a decoder without cross attention would not fit the tables
    assert round(oracle.param_count_formula(V, d, F, 35, 6) / 1e6 + 2 * V * d / 1e6) != 152
    fp16 = g["fp16_file"]
    assert abs(fp16["params_M"] * 1e6 * 2 / 2 ** 20 - fp16["MiB"]) < 3


def test_embedding_pad_and_scale():
    blob = _blob(lively=False)
    m = oracle.OracleModel(SHAPE, blob)
    y = m.embed([5], [3])[0]
    E = synth.unpack(SHAPE, blob)["E"].astype(np.float64)
    np.testing.assert_allclose(y - math.sqrt(SHAPE.d_model) * E[5], oracle.positional_encoding([3], 32)[0], atol=1e-14)
