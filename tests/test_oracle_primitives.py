"""Pins for the oracle's primitives: closed forms, invariants and library routines.

LayerNorm, softmax and attention are checked against torch CPU fp64 (an independent
implementation), and against special cases whose value is known without computing
the primitive (constant rows, zero queries, a single key).
"""
import math

import numpy as np
import pytest

import oracle

RNG = np.random.default_rng(1234)


def test_layer_norm_constant_row_gives_beta():
    x = np.full((3, 16), 7.25)
    g, b = RNG.normal(size=16), RNG.normal(size=16)
    np.testing.assert_array_equal(oracle.layer_norm(x, g, b), np.broadcast_to(b, (3, 16)))


def test_layer_norm_matches_torch(torch_cpu64):
    torch = torch_cpu64
    x = RNG.normal(size=(5, 64)) * 3 + 1
    g, b = RNG.normal(size=64), RNG.normal(size=64)
    ref = torch.nn.functional.layer_norm(torch.tensor(x), (64,), torch.tensor(g), torch.tensor(b), eps=1e-5)
    np.testing.assert_allclose(oracle.layer_norm(x, g, b, 1e-5), ref.numpy(), rtol=0, atol=1e-12)


def test_layer_norm_output_moments():
    x = RNG.normal(size=(4, 128)) * 5 - 2
    y = oracle.layer_norm(x, np.ones(128), np.zeros(128), eps=0.0)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(-1), 1, atol=1e-12)


def test_softmax_rows_sum_to_one_and_lse():
    x = RNG.normal(size=(7, 1000)) * 4
    p = oracle.softmax(x)
    np.testing.assert_allclose(p.sum(-1), 1, atol=1e-12)
    logp = x - oracle.logsumexp(x)[:, None]
    np.testing.assert_allclose(oracle.logsumexp(logp), 0, atol=1e-12)


def test_softmax_and_lse_match_torch(torch_cpu64):
    torch = torch_cpu64
    x = RNG.normal(size=(3, 500)) * 10
    np.testing.assert_allclose(oracle.softmax(x), torch.softmax(torch.tensor(x), -1).numpy(), atol=1e-14)
    np.testing.assert_allclose(oracle.logsumexp(x), torch.logsumexp(torch.tensor(x), -1).numpy(), atol=1e-12)


def test_logsumexp_large_values_stable():
    x = np.array([[1000.0, 1000.0], [-1000.0, -1000.0]])
    np.testing.assert_allclose(oracle.logsumexp(x), [1000 + math.log(2), -1000 + math.log(2)], atol=1e-12)


def test_attention_zero_query_gives_mean_of_values():
    d, H, tk = 32, 4, 9
    q = np.zeros((2, d))
    k, v = RNG.normal(size=(tk, d)), RNG.normal(size=(tk, d))
    out = oracle.attention(q, k, v, H)
    np.testing.assert_allclose(out, np.broadcast_to(v.mean(0), (2, d)), atol=1e-14)


def test_attention_single_key_gives_value():
    d, H = 32, 4
    q, k, v = RNG.normal(size=(3, d)), RNG.normal(size=(1, d)), RNG.normal(size=(1, d))
    np.testing.assert_allclose(oracle.attention(q, k, v, H), np.broadcast_to(v, (3, d)), atol=1e-14)


def test_attention_masked_keys_are_inert():
    d, H = 32, 2
    q, k, v = RNG.normal(size=(4, d)), RNG.normal(size=(6, d)), RNG.normal(size=(6, d))
    allowed = np.zeros((4, 6), dtype=bool)
    allowed[:, :4] = True
    k2, v2 = k.copy(), v.copy()
    k2[4:], v2[4:] = 1e3, -1e3
    a = oracle.attention(q, k, v, H, allowed)
    b = oracle.attention(q, k2, v2, H, allowed)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_allclose(a, oracle.attention(q, k[:4], v[:4], H), atol=1e-14)


def test_attention_matches_torch_sdpa(torch_cpu64):
    torch = torch_cpu64
    d, H, tq, tk = 64, 8, 5, 11
    dh = d // H
    q, k, v = RNG.normal(size=(tq, d)), RNG.normal(size=(tk, d)), RNG.normal(size=(tk, d))
    allowed = RNG.random((tq, tk)) < 0.7
    allowed[:, 0] = True

    def heads(x):
        return torch.tensor(x).reshape(x.shape[0], H, dh).transpose(0, 1)

    ref = torch.nn.functional.scaled_dot_product_attention(
        heads(q), heads(k), heads(v), attn_mask=torch.tensor(allowed)[None])
    ref = ref.transpose(0, 1).reshape(tq, d).numpy()
    np.testing.assert_allclose(oracle.attention(q, k, v, H, allowed), ref, atol=1e-12)


def test_positional_encoding_position_zero():
    pe = oracle.positional_encoding([0], 16)[0]
    np.testing.assert_array_equal(pe, np.tile([0.0, 1.0], 8))


def test_positional_encoding_pairs_on_unit_circle_and_rotate():
    d = 64
    pe = oracle.positional_encoding(np.arange(50), d)
    np.testing.assert_allclose(pe[:, 0::2] ** 2 + pe[:, 1::2] ** 2, 1.0, atol=1e-14)
    # the first pair has frequency 1: position p holds (sin p, cos p)
    np.testing.assert_allclose(pe[:, 0], np.sin(np.arange(50)), atol=1e-14)
    # the last pair has the lowest frequency, 10000^(-(d-2)/d): it moves by that angle per step
    w = 10000.0 ** (-(d - 2) / d)
    ang = np.arctan2(pe[:, d - 2], pe[:, d - 1])
    np.testing.assert_allclose(np.diff(ang), w, atol=1e-12)


@pytest.mark.parametrize("precision", ["f16", "bf16"])
def test_round_weights_touches_only_matrices(precision):
    import synth
    shape = synth.small_model(d_model=32, n_heads=2, n_enc=1, n_dec=1, vocab=11)
    blob = synth.make_weights(shape)
    r = oracle.round_weights(blob, shape, precision)
    off = 0
    for e in synth.weight_layout(shape):
        a, b = blob[off:off + e.size], r[off:off + e.size]
        if e.name == "E" or ".W_" in e.name:
            assert not np.array_equal(a, b)
            if precision == "f16":
                np.testing.assert_array_equal(b, a.astype(np.float16).astype(np.float32))
        else:
            np.testing.assert_array_equal(a, b)
        off += e.size


def test_bf16_rounding_is_nearest_even():
    import synth
    shape = synth.ModelShape(d_model=4, n_heads=1, d_ffn=4, n_enc=0, n_dec=0, vocab=2)
    # E holds 8 values; ties go to the even mantissa, others to nearest
    vals = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20,
                     -(1 + 2 ** -8), 3.0, 1 - 2 ** -9, 65504.0], dtype=np.float32)
    expect = np.array([1.0, 1.0, 1 + 2 ** -6, 1 + 2 ** -7, -1.0, 3.0, 1.0, 65536.0], dtype=np.float32)
    blob = synth.make_weights(shape)
    blob[:8] = vals
    r = oracle.round_weights(blob, shape, "bf16")
    np.testing.assert_array_equal(r[:8], expect)
