"""Pins for the oracle's FP8 weight quantization (lower-precision weights, Sec. 6).

* Library routine: e4m3_round equals torch's float8_e4m3fn cast (round to nearest even)
  on values across the whole range, subnormals and exact ties included, and every
  finite E4M3 value round-trips.
* Hand-worked cases: ties to even in the normal and subnormal ranges, the step of each
  binade, saturation at 448, signed zero.
* Per-column scaling: each column's largest magnitude maps to exactly 448, the error of
  a normal-range element is at most 1/16 of it, a zero column stays zero.
* round_weights("f8") changes exactly the projection matrices (and E to fp16), and the
  biases of the decoder projections that take a pre-norm LayerNorm's output.
* Those folded projections (reading: their FP8 weights quantize diag(gamma) W): the
  weights round_weights returns give LN(u; gamma, beta) W' + b' equal to
  LN0(u) Q + b + beta W, with Q the per-column E4M3 quantization of diag(gamma) W formed by
  torch's float8_e4m3fn cast and LN0 torch's layer_norm without gain or bias; a row with
  zero gain included.
"""
import math

import numpy as np
import pytest

import oracle
import synth


def torch_e4m3(x):
    import torch
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_matches_torch_float8_e4m3fn():
    rng = np.random.default_rng(0)
    # magnitudes from deep subnormal to the top binade, both signs
    x = np.ldexp(rng.uniform(1.0, 2.0, 20000), rng.integers(-14, 9, 20000)) * rng.choice([-1.0, 1.0], 20000)
    x = x[np.abs(x) < 448.0].astype(np.float32)
    # exact midpoints between neighbouring E4M3 values (the ties)
    import torch
    grid = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    grid = np.unique(grid[np.isfinite(grid)])
    mids = ((grid[1:] + grid[:-1]) / 2).astype(np.float32)
    for v in (x, mids, grid.astype(np.float32)):
        np.testing.assert_array_equal(oracle.e4m3_round(v), torch_e4m3(v))
    assert len(grid) == 253   # 126 positive, 126 negative and one zero (-0 == 0 in unique)


@pytest.mark.parametrize("x,want", [
    (1.0625, 1.0), (1.1875, 1.25), (232.0, 224.0), (240.0, 240.0), (448.0, 448.0), (449.0, 448.0),
    (470.0, 448.0), (1e6, 448.0), (-3.3, -3.25), (2.0 ** -9, 2.0 ** -9), (1.5 * 2.0 ** -9, 2.0 ** -8),
    (2.5 * 2.0 ** -9, 2.0 * 2.0 ** -9), (0.4 * 2.0 ** -9, 0.0), (0.5 * 2.0 ** -9, 0.0), (2.0 ** -6, 2.0 ** -6),
    (0.0, 0.0),
])
def test_hand_worked_cases(x, want):
    assert oracle.e4m3_round(np.float32(x)) == want


def test_signed_zero_and_binade_steps():
    assert math.copysign(1.0, float(oracle.e4m3_round(np.float32(-0.0)))) == -1.0
    for e in range(-6, 9):   # normal binades: 8 values each, step 2^(e-3); the top one stops at 448
        lo, n = 2.0 ** e, 8 if e < 8 else 7
        vals = oracle.e4m3_round(np.float32(lo) + np.arange(n, dtype=np.float32) * np.float32(2.0 ** (e - 3)))
        np.testing.assert_array_equal(vals, lo + np.arange(n) * 2.0 ** (e - 3))


def test_per_column_scaling():
    rng = np.random.default_rng(1)
    w = rng.normal(0, 0.02, size=(64, 48)).astype(np.float32)
    w[:, 5] = 0.0
    w[3, 7] = 5.0                                 # one column with an outlier
    q, sc = oracle.quantize_fp8_columns(w)
    assert q.dtype == np.float64 and sc.dtype == np.float32
    np.testing.assert_array_equal(np.abs(q).max(axis=0)[np.arange(48) != 5], 448.0)
    assert sc[5] == 1.0 and not q[:, 5].any()
    np.testing.assert_array_equal(sc, np.where(np.abs(w).max(0) > 0, np.abs(w).max(0) / np.float32(448), 1))
    deq = q * sc.astype(np.float64)
    normal = np.abs(w) >= sc[None, :] * 2.0 ** -6
    assert np.all(np.abs(deq - w)[normal] <= np.abs(w)[normal] / 16)
    assert np.all(np.abs(deq - w)[~normal] <= (sc[None, :] * 2.0 ** -10 + 0 * w)[~normal])
    # every quantized value is an E4M3 value
    np.testing.assert_array_equal(oracle.e4m3_round(q.astype(np.float32)), q)


def test_round_weights_f8_changes_exactly_the_matrices():
    shape = synth.ModelShape(64, 2, 256, 2, 1, 50, rel_k=2)
    blob = synth.make_weights(shape, seed=3)
    r = oracle.round_weights(blob, shape, "f8")
    assert r.dtype == np.float64
    off = 0
    for e in synth.weight_layout(shape):
        a, b = blob[off:off + e.size].astype(np.float64), r[off:off + e.size]
        folded_bias = e.name.startswith("dec.") and e.name.endswith((".b_qkv", ".b_q", ".b_1"))
        if e.name == "E":
            np.testing.assert_array_equal(b, blob[off:off + e.size].astype(np.float16))
        elif ".W_" in e.name:
            assert not np.array_equal(a, b)
            assert np.abs(a - b).max() <= np.abs(a).max() / 8   # gain-scaled ones: 1/16 of max|gamma W| / min gamma
        elif folded_bias:
            assert not np.array_equal(a, b)
        else:
            np.testing.assert_array_equal(a, b)
        off += e.size


def _torch_fp8_columns(w32):
    """Per-column E4M3 quantization by torch: scale = max |column| / 448 (fp32), codes by
    the float8_e4m3fn cast of w / scale (fp32); returns the dequantized fp64 matrix."""
    import torch
    w = torch.from_numpy(w32)
    amax = w.abs().amax(dim=0)
    scale = torch.where(amax > 0, amax / torch.tensor(448.0, dtype=torch.float32), torch.tensor(1.0))
    q = (w / scale[None, :]).to(torch.float8_e4m3fn).to(torch.float64)
    return (q * scale.to(torch.float64)[None, :]).numpy()


@pytest.mark.parametrize("ln,w,b", [("ln1", "W_qkv", "b_qkv"), ("ln2", "W_q", "b_q"), ("ln3", "W_1", "b_1")])
def test_fp8_decoder_projection_folds_the_layernorm_gain(torch_cpu64, ln, w, b):
    torch = torch_cpu64
    shape = synth.ModelShape(64, 2, 256, 1, 2, 50)
    blob = synth.make_weights(shape, seed=5)
    named = synth.unpack(shape, blob.copy())
    p = "dec.1."
    named[p + ln + ".gamma"][:] = 1.0 + 0.5 * np.random.default_rng(6).standard_normal(shape.d_model)
    named[p + ln + ".gamma"][7] = 0.0                       # a row whose LayerNorm output is the constant beta
    named[p + ln + ".beta"][:] = 0.3 * np.random.default_rng(7).standard_normal(shape.d_model)
    blob = synth.pack(shape, named)
    named = synth.unpack(shape, blob)
    r = synth.unpack(shape, oracle.round_weights(blob, shape, "f8"))
    gamma, beta = named[p + ln + ".gamma"], named[p + ln + ".beta"]
    W, bias = named[p + w], named[p + b]
    Q = _torch_fp8_columns((gamma[:, None] * W).astype(np.float32))
    u = torch.from_numpy(np.random.default_rng(8).normal(0.4, 1.3, size=(9, shape.d_model)))
    ln0 = torch.nn.functional.layer_norm(u, (shape.d_model,), eps=1e-5).numpy()
    want = ln0 @ Q + bias.astype(np.float64) + beta.astype(np.float64) @ W.astype(np.float64)
    got = oracle.layer_norm(u.numpy(), gamma.astype(np.float64), beta.astype(np.float64)) @ r[p + w] + r[p + b]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    assert not r[p + w][7].any()
    # and it is not the unfolded quantization: Q / gamma differs from fp8(W)
    plain = _torch_fp8_columns(W.astype(np.float32))
    assert np.abs(r[p + w] - plain).max() > 1e-4


def _torch_decoder_fp8_kv(torch, shape, blob, enc, tgt):
    """Reference decoder in torch (fp64) whose self-attention keys and values go through
    torch's float8_e4m3fn cast before scaled_dot_product_attention (causal): the FP8 cache."""
    F = torch.nn.functional
    d, H = shape.d_model, shape.n_heads
    dh = d // H
    P = {k: torch.tensor(v.astype(np.float64)) for k, v in synth.unpack(shape, blob).items()}
    enc = torch.tensor(enc)

    def ln(x, p):
        return F.layer_norm(x, (d,), P[p + ".gamma"], P[p + ".beta"], eps=1e-5)

    def heads(x):
        return x.reshape(x.shape[0], H, dh).transpose(0, 1)

    inp = torch.tensor([synth.BOS_ID] + list(tgt))
    n = len(inp)
    z = math.sqrt(d) * P["E"][inp] + torch.tensor(oracle.positional_encoding(np.arange(n), d))
    for j in range(shape.n_dec):
        p = f"dec.{j}."
        qkv = ln(z, p + "ln1") @ P[p + "W_qkv"] + P[p + "b_qkv"]
        q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
        k8 = k.float().to(torch.float8_e4m3fn).to(torch.float64)
        v8 = v.float().to(torch.float8_e4m3fn).to(torch.float64)
        att = F.scaled_dot_product_attention(heads(q), heads(k8), heads(v8), is_causal=True)
        z = z + att.transpose(0, 1).reshape(n, d) @ P[p + "W_o"] + P[p + "b_o"]
        qc = ln(z, p + "ln2") @ P[p + "W_q"] + P[p + "b_q"]
        kv = enc @ P[p + "W_kv"] + P[p + "b_kv"]
        att = F.scaled_dot_product_attention(heads(qc), heads(kv[:, :d]), heads(kv[:, d:]))
        z = z + att.transpose(0, 1).reshape(n, d) @ P[p + "W_oc"] + P[p + "b_oc"]
        f = torch.relu(ln(z, p + "ln3") @ P[p + "W_1"] + P[p + "b_1"])
        z = z + f @ P[p + "W_2"] + P[p + "b_2"]
    return (ln(z, "dec_out_ln") @ P["E"].T).numpy()


def test_fp8_kv_cache_matches_torch_float8_decoder(torch_cpu64):
    """The oracle's FP8 key/value cache against torch's float8 cast and attention, on a
    model with large self-attention keys and values (lively weights) so that the rounding
    matters; incremental decoding equals full recomputation with the cache quantized; and
    the quantization moves the logits."""
    torch = torch_cpu64
    shape = synth.ModelShape(32, 4, 128, 2, 2, 23)
    blob = synth.make_weights(shape, seed=12, lively=True)
    src, tgt = [5, 9, 17, 4, 22, 8], [7, 3, 19, 2, 11, 6]
    om = oracle.OracleModel(shape, blob, np.float64, kv_fp8=True)
    want = _torch_decoder_fp8_kv(torch, shape, blob, om.encode(src), tgt)
    inc = om.teacher_forced_logits(src, tgt)
    full = om.teacher_forced_logits(src, tgt, incremental=False)
    np.testing.assert_allclose(inc, want, rtol=0, atol=1e-10)
    np.testing.assert_allclose(inc, full, rtol=0, atol=1e-12)
    plain = oracle.OracleModel(shape, blob, np.float64).teacher_forced_logits(src, tgt)
    assert np.abs(plain - inc).max() > 1e-3
    assert oracle.OracleModel(shape, blob, np.float64, precision="f8").kv_fp8
    weights_only = oracle.OracleModel(shape, blob, np.float64, precision="f8w")
    assert not weights_only.kv_fp8
    np.testing.assert_array_equal(oracle.round_weights(blob, shape, "f8w"), oracle.round_weights(blob, shape, "f8"))
