"""P11: a one-layer encoder and decoder with d = 4 and one head, small enough to work
out by hand, against the oracle in fp64.

The weights are chosen so that every step has a closed form a reader can follow on
paper: the query and key projections are zero, so every attention weight is uniform and
each attention output is the plain mean of its value rows; the value and output
projections are identities (plus a bias), the FFN is 0.5 ReLU(LN(x) + b1) + b2, the DLCL
rows are one-hot with the history normalisation switched off (N = identity, Eq. 2 with
the layer norm removed), so the encoder output is LN_out(y_1).  The LayerNorm gains and
biases are not 1 and 0 where a swap or a dropped term would go unnoticed, and every
weight is a dyadic fraction, exact in the fp32 blob.  Everything
below is written out for this case with scalar arithmetic; nothing calls the oracle's
layers.  A wrong operand column (Q, K and V of the fused projection), a missing residual,
a wrong positional phase, the embedding scale, the attention span of the decoder's
self-attention (slots 0..t) or the tied output projection changes the logits far beyond
the 1e-12 bound.
"""
import math

import numpy as np

import oracle
import synth

D, V = 4, 6
SHAPE = synth.ModelShape(D, 1, D, 1, 1, V)
EPS = 1e-5


def _weights():
    z = lambda *s: np.zeros(s)
    eye = np.eye(D)
    E = np.array([[(w + 1) / 8, -w / 16, w * w / 64, (2.5 - w) / 8] for w in range(V)])
    named = {"E": E}
    for k in range(2):
        named[f"hist_ln.{k}.gamma"] = np.ones(D)
        named[f"hist_ln.{k}.beta"] = z(D)
    named["dlcl.1"] = np.array([1.0])
    named["dlcl.2"] = np.array([0.0, 1.0])
    p = "enc.0."
    named.update({
        p + "ln1.gamma": np.array([1.0, 2.0, 1.0, 0.5]), p + "ln1.beta": np.array([0.0, 0.125, -0.125, 0.0]),
        p + "W_qkv": np.hstack([z(D, D), z(D, D), eye]), p + "b_qkv": np.r_[z(D), z(D), [0.0625, 0.0, -0.0625, 0.0]],
        p + "W_o": eye, p + "b_o": np.array([0.015625, 0.0, 0.0, 0.0]),
        p + "ln2.gamma": np.ones(D), p + "ln2.beta": z(D),
        p + "W_1": eye, p + "b_1": np.array([0.0, -0.125, 0.0, 0.125]),
        p + "W_2": 0.5 * eye, p + "b_2": np.array([0.0, 0.0, 0.03125, 0.0]),
    })
    named["enc_out_ln.gamma"] = np.array([1.0, 1.0, 2.0, 1.0])
    named["enc_out_ln.beta"] = np.array([0.0, 0.0, 0.0, 0.25])
    p = "dec.0."
    named.update({
        p + "ln1.gamma": np.ones(D), p + "ln1.beta": z(D),
        p + "W_qkv": np.hstack([z(D, D), z(D, D), eye]), p + "b_qkv": z(3 * D),
        p + "W_o": eye, p + "b_o": z(D),
        p + "ln2.gamma": np.ones(D), p + "ln2.beta": z(D),
        p + "W_q": z(D, D), p + "b_q": z(D),
        p + "W_kv": np.hstack([z(D, D), eye]), p + "b_kv": z(2 * D),
        p + "W_oc": eye, p + "b_oc": np.array([0.0, 0.046875, 0.0, 0.0]),
        p + "ln3.gamma": np.ones(D), p + "ln3.beta": z(D),
        p + "W_1": eye, p + "b_1": z(D),
        p + "W_2": 0.5 * eye, p + "b_2": z(D),
    })
    named["dec_out_ln.gamma"] = np.ones(D)
    named["dec_out_ln.beta"] = z(D)
    return E, named


# --- the example, worked with scalars -------------------------------------------------
def _ln(x, g=(1, 1, 1, 1), b=(0, 0, 0, 0)):
    mu = sum(x) / 4
    var = sum((xi - mu) ** 2 for xi in x) / 4
    r = 1 / math.sqrt(var + EPS)
    return [(x[i] - mu) * r * g[i] + b[i] for i in range(4)]


def _pe(p):
    # d = 4: frequencies 1 and 1/10000^(2/4) = 1/100, interleaved sin / cos
    return [math.sin(p), math.cos(p), math.sin(p / 100), math.cos(p / 100)]


def _add(*vs):
    return [sum(v[i] for v in vs) for i in range(4)]


def _mean(rows):
    return [sum(r[i] for r in rows) / len(rows) for i in range(4)]


def _by_hand(E, src, tgt):
    emb = lambda w, p: _add([2 * E[w][i] for i in range(4)], _pe(p))   # sqrt(d) = 2
    # encoder: x_1 = y_0 (one-hot row, N = identity)
    x = [emb(w, i) for i, w in enumerate(src)]
    u = [_ln(xi, (1, 2, 1, 0.5), (0, 0.125, -0.125, 0)) for xi in x]
    att = _mean([_add(ui, [0.0625, 0, -0.0625, 0]) for ui in u])            # uniform weights, V = I + b_v
    a = [_add(xi, att, [0.015625, 0, 0, 0]) for xi in x]                    # W_o = I, b_o
    y = [_add(ai, [0.5 * max(v, 0.0) for v in _add(_ln(ai), [0, -0.125, 0, 0.125])], [0, 0, 0.03125, 0]) for ai in a]
    enc = [_ln(yi, (1, 1, 2, 1), (0, 0, 0, 0.25)) for yi in y]           # LN_out(h_1), h_1 = y_1
    cross = _mean(enc)                                                  # W_q = 0: uniform over the source
    rows = []
    prefix = [synth.BOS_ID] + list(tgt)
    for t in range(len(tgt) + 1):
        zs = [emb(prefix[s], s) for s in range(t + 1)]
        z1 = _add(zs[t], _mean([_ln(zz) for zz in zs]))                 # self-attention over slots 0..t
        z2 = _add(z1, cross, [0, 0.046875, 0, 0])                           # W_oc = I, b_oc
        z3 = _add(z2, [0.5 * max(v, 0.0) for v in _ln(z2)])
        h = _ln(z3)
        rows.append([sum(h[i] * E[w][i] for i in range(4)) for w in range(V)])   # tied projection
    return np.array(rows)


def test_handworked_one_layer_example():
    E, named = _weights()
    blob = synth.pack(SHAPE, named)
    om = oracle.OracleModel(SHAPE, blob, np.float64, hist_norm=False)
    src, tgt = [4, 5, 3], [4, 2]
    want = _by_hand(E.tolist(), src, tgt)
    got = om.teacher_forced_logits(src, tgt)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    # the example is not degenerate: the source and the step both move the logits
    other = _by_hand(E.tolist(), [5, 4], tgt)
    assert np.abs(other - want).max() > 1e-3
    assert np.abs(want[1] - want[0]).max() > 1e-3
