"""GPU: the beam step's selection (top-k logits in (value desc, index asc) order plus the
row's log-sum-exp) against NumPy, through nt_op_select (a scan of the whole row) and
nt_op_select_tiled (from per-128-column-tile records, reading back only the tiles that
can hold one of the k largest).

Covers the register-resident kernel (V % 4 == 0, V <= 32768) and the streaming kernel
(other V), heavy ties (values drawn from a few integers, equal rows -- many tiles then
share the k-th largest maximum), a row whose maximum is its last logit, -inf logits
(never selected; whole tiles of -inf), V below one tile and not a multiple of it, and k
up to 32.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

INT_MAX = np.iinfo(np.int32).max


def _expected(x, k):
    vals, idxs = [], []
    for row in x:
        finite = np.flatnonzero(row > -np.inf)
        order = finite[np.lexsort((finite, -row[finite].astype(np.float64)))][:k]
        v = np.full(k, -np.inf, dtype=np.float32)
        i = np.full(k, INT_MAX, dtype=np.int64)
        v[: len(order)] = row[order]
        i[: len(order)] = order
        vals.append(v)
        idxs.append(i)
    with np.errstate(divide="ignore"):
        lse = np.array([np.logaddexp.reduce(r.astype(np.float64)) for r in x])
    return np.array(vals), np.array(idxs), lse


def _run(x, k, entry="nt_op_select"):
    import torch
    from paper_2109_08008_amd import nt
    rows, V = x.shape
    dx = torch.from_numpy(x).cuda()
    tv = torch.empty(rows, k, dtype=torch.float32, device="cuda")
    ti = torch.empty(rows, k, dtype=torch.int32, device="cuda")
    ls = torch.empty(rows, dtype=torch.float32, device="cuda")
    getattr(nt, entry)(dx.data_ptr(), rows, V, k, tv.data_ptr(), ti.data_ptr(), ls.data_ptr())
    torch.cuda.synchronize()
    return tv.cpu().numpy(), ti.cpu().numpy().astype(np.int64), ls.cpu().numpy()


def _logits(V, rows, kind, seed):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        x = rng.standard_normal((rows, V)).astype(np.float32) * 4
    elif kind == "ties":
        x = rng.integers(0, 4, size=(rows, V)).astype(np.float32)
    else:   # structured rows: all equal, max at the end, a few finite among -inf, huge magnitudes
        x = rng.standard_normal((rows, V)).astype(np.float32)
        x[0] = 1.5
        x[1, -1] = 50.0
        x[2] = -np.inf
        x[2, rng.choice(V, size=min(V, 3), replace=False)] = [1.0, 2.0, 2.0][: min(V, 3)]
        x[3] *= 1e4
    return x


@pytest.mark.parametrize("entry", ["nt_op_select", "nt_op_select_tiled"])
@pytest.mark.parametrize("V", [7, 101, 1000, 4096, 32000, 40000])
@pytest.mark.parametrize("kind", ["normal", "ties", "rows"])
def test_select_matches_numpy(V, kind, entry):
    rows = 12
    x = _logits(V, rows, kind, seed=V + len(kind))
    for k in (1, 4, 8) + ((16, 32) if V >= 32 else ()):
        if k > V:
            continue
        tv, ti, ls = _run(x, k, entry)
        ev, ei, el = _expected(x, k)
        np.testing.assert_array_equal(ti, ei, err_msg=f"k={k}")
        np.testing.assert_array_equal(tv, ev, err_msg=f"k={k}")
        fin = np.isfinite(el)
        np.testing.assert_allclose(ls[fin], el[fin], rtol=2e-6, atol=2e-5)
        assert np.array_equal(np.isfinite(ls), fin)
