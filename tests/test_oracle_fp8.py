"""Pins for the oracle's FP8 weight quantization (lower-precision weights, Sec. 6).

* Library routine: e4m3_round equals torch's float8_e4m3fn cast (round to nearest even)
  on values across the whole range, subnormals and exact ties included, and every
  finite E4M3 value round-trips.
* Hand-worked cases: ties to even in the normal and subnormal ranges, the step of each
  binade, saturation at 448, signed zero.
* Per-column scaling: each column's largest magnitude maps to exactly 448, the error of
  a normal-range element is at most 1/16 of it, a zero column stays zero.
* round_weights("f8") changes exactly the projection matrices (and E to fp16).
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
        if e.name == "E":
            np.testing.assert_array_equal(b, blob[off:off + e.size].astype(np.float16))
        elif ".W_" in e.name:
            assert not np.array_equal(a, b)
            assert np.abs(a - b).max() <= np.abs(a).max() / 16
        else:
            np.testing.assert_array_equal(a, b)
        off += e.size
