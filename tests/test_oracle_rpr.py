"""Pins of the oracle's relative position representations (encoder self-attention; the
teachers' RPR of Sec. 3.1, with a maximum relative length of 8).

Each check fixes the result from the mathematics, not from the oracle's own formula:
zero tables reduce to plain attention; a constant key row shifts every score of a query
equally (softmax is unchanged); a constant value row adds itself to every output (the
weights sum to 1); a large key row at offset +1 makes every query attend to its next
token (the sign of j - i); a large key row at the +k edge spreads the attention evenly
over every key at distance >= k (the clip); a two-key case gives the closed-form
sigmoid weight with the 1/sqrt(dh) scale.
"""
import math

import numpy as np
import pytest

import synth
from oracle import model as M


def _qkv(t, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((t, d)), rng.standard_normal((t, d)), rng.standard_normal((t, d)))


@pytest.mark.parametrize("rel_k", [1, 3, 8])
def test_zero_tables_are_plain_attention(rel_k):
    q, k, v = _qkv(11, 16, 1)
    z = np.zeros((2 * rel_k + 1, 8))
    np.testing.assert_allclose(M.attention(q, k, v, 2, rel=(z, z, rel_k)), M.attention(q, k, v, 2), atol=1e-13)


def test_constant_key_row_changes_nothing_and_constant_value_row_adds_itself():
    q, k, v = _qkv(9, 12, 2)
    rel_k, dh = 3, 4
    a = np.random.default_rng(3).standard_normal(dh)
    c = np.random.default_rng(4).standard_normal(dh)
    tk = np.tile(a, (2 * rel_k + 1, 1))
    tv = np.tile(c, (2 * rel_k + 1, 1))
    plain = M.attention(q, k, v, 3)
    np.testing.assert_allclose(M.attention(q, k, v, 3, rel=(tk, np.zeros_like(tv), rel_k)), plain, atol=1e-12)
    np.testing.assert_allclose(M.attention(q, k, v, 3, rel=(np.zeros_like(tk), tv, rel_k)), plain + np.tile(c, 3),
                               atol=1e-12)


def test_offset_plus_one_attends_to_the_next_token():
    t, dh, rel_k = 7, 4, 2
    q = np.ones((t, dh))
    k = np.zeros((t, dh))
    v = np.arange(t, dtype=np.float64)[:, None] * np.ones((1, dh))
    tk = np.zeros((2 * rel_k + 1, dh))
    tk[rel_k + 1] = 200.0           # offset j - i = +1
    out = M.attention(q, k, v, 1, rel=(tk, np.zeros_like(tk), rel_k))
    np.testing.assert_allclose(out[:-1, 0], np.arange(1, t), atol=1e-9)   # query i -> value of token i+1
    # the last token has no successor: it averages its keys evenly
    np.testing.assert_allclose(out[-1, 0], np.mean(np.arange(t)), atol=1e-9)


def test_edge_row_covers_every_distance_beyond_the_clip():
    t, dh, rel_k = 12, 4, 3
    q = np.ones((t, dh))
    k = np.zeros((t, dh))
    v = np.arange(t, dtype=np.float64)[:, None] * np.ones((1, dh))
    tk = np.zeros((2 * rel_k + 1, dh))
    tk[2 * rel_k] = 200.0           # every offset >= +rel_k
    out = M.attention(q, k, v, 1, rel=(tk, np.zeros_like(tk), rel_k))
    for i in range(t - rel_k):
        np.testing.assert_allclose(out[i, 0], np.mean(np.arange(i + rel_k, t)), atol=1e-9)


def test_two_keys_closed_form_with_scale():
    dh, rel_k = 16, 1
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, dh))
    k = np.zeros((2, dh))
    v = rng.standard_normal((2, dh))
    tk = np.zeros((3, dh))
    a = rng.standard_normal(dh)
    tk[rel_k + 1] = a               # key 1 is at offset +1 from query 0; key 0 at offset 0
    out = M.attention(q, k, v, 1, rel=(tk, np.zeros_like(tk), rel_k))
    p1 = 1.0 / (1.0 + math.exp(-(q[0] @ a) / math.sqrt(dh)))
    np.testing.assert_allclose(out[0], (1 - p1) * v[0] + p1 * v[1], atol=1e-12)


def test_layout_and_model_with_relative_positions():
    shape = synth.ModelShape(64, 2, 128, 2, 1, 50, rel_k=4)
    names = [e.name for e in synth.weight_layout(shape)]
    assert "enc.0.rel_k" in names and "enc.1.rel_v" in names
    assert synth.blob_size(shape) == synth.blob_size(synth.ModelShape(64, 2, 128, 2, 1, 50)) + 2 * 2 * 9 * 32
    blob = synth.make_weights(shape, seed=1, lively=True)
    om = M.OracleModel(shape, blob)
    src = [5, 9, 13, 7, 21, 4]
    enc = om.encode(src)
    assert enc.shape == (6, 64) and np.isfinite(enc).all()
    # zeroing the tables gives the model without relative positions
    named = synth.unpack(shape, blob.copy())
    named_blob = synth.pack(shape, {n: (np.zeros_like(x) if n.endswith(("rel_k", "rel_v")) else x)
                                    for n, x in named.items()})
    plain_shape = synth.ModelShape(64, 2, 128, 2, 1, 50)
    plain_blob = synth.pack(plain_shape, {n: x for n, x in named.items() if not n.endswith(("rel_k", "rel_v"))})
    np.testing.assert_allclose(M.OracleModel(shape, named_blob).encode(src),
                               M.OracleModel(plain_shape, plain_blob).encode(src), atol=1e-12)
