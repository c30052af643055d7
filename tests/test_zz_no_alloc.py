"""GPU: the allocation-free tiled selection (nt_op_select_tiled_noalloc), through the C ABI,
against the allocating entry point (nt_op_select_tiled) that runs the same kernels: two
calls in a row, the second with a smaller input, give identical indices, values and
log-sum-exps; an input beyond the static records array is refused before any launch."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _logits(rows, V, seed):
    import torch
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(rows, V, generator=g) * 3.0
    x[:, 5] = x[:, 7]                      # ties across tiles: the lower index comes first
    x[: rows // 3, 200:300] = float("-inf")
    x[:, V - 1] = x[:, 0]
    return x.cuda()


def _select(fn, x, k):
    import torch
    rows, V = x.shape
    topv = torch.full((rows, k), float("nan"), device="cuda")
    topi = torch.full((rows, k), -7, dtype=torch.int32, device="cuda")
    lse = torch.full((rows,), float("nan"), device="cuda")
    fn(x.data_ptr(), rows, V, k, topv.data_ptr(), topi.data_ptr(), lse.data_ptr())
    torch.cuda.synchronize()
    return topv.cpu(), topi.cpu(), lse.cpu()


def test_noalloc_selection_matches_the_allocating_entry_point():
    import torch
    from paper_2109_08008_amd import nt
    for rows, V, k, seed in [(3000, 32000, 8, 1), (37, 1000, 4, 2)]:   # second call: a smaller input
        x = _logits(rows, V, seed)
        want = _select(nt.nt_op_select_tiled, x, k)
        got = _select(nt.nt_op_select_tiled_noalloc, x, k)
        for a, b in zip(want, got):
            assert torch.equal(a, b)
        # and the selection itself, against torch on the host
        ref_v, _ = torch.topk(x.cpu().double(), k, dim=1)
        np.testing.assert_array_equal(got[0].double().numpy(), ref_v.numpy())
        np.testing.assert_allclose(got[2].double().numpy(), torch.logsumexp(x.cpu().double(), 1).numpy(), atol=1e-4)
    n_tiles = (32000 + 127) // 128
    too_many = nt.NT_SELECT_NOALLOC_MAX_RECORDS // n_tiles + 1
    x = torch.zeros(1, 32000, device="cuda")
    with pytest.raises(nt.NTError) as err:
        nt.nt_op_select_tiled_noalloc(x.data_ptr(), too_many, 32000, 8, x.data_ptr(), x.data_ptr(), x.data_ptr())
    assert err.value.status == nt.NT_E_UNSUPPORTED, err.value
