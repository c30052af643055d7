"""GPU: the MFMA GEMM (nt_op_gemm) against a plain fp64 matrix product.

Covers every tile shape, every dtype, the bias / ReLU / residual / fp32-output
epilogues, ragged M and N and K spanning several pipeline stages.  The same rows
computed with either tile shape, or as part of a larger M, are bitwise identical
(each output is reduced over K in one fixed order).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TORCH_DT = {"f32": "float32", "f16": "float16", "bf16": "bfloat16"}
ULP = {"f32": 2.0 ** -23, "f16": 2.0 ** -10, "bf16": 2.0 ** -7}


def _setup(dtype, M, N, K, seed):
    import torch
    g = torch.Generator().manual_seed(seed)
    tdt = getattr(torch, TORCH_DT[dtype])
    A = torch.randn(M, K, generator=g).to(tdt)
    Bt = torch.randn(N, K, generator=g).to(tdt)
    bias = torch.randn(N, generator=g, dtype=torch.float32)
    R = torch.randn(M, N, generator=g).to(tdt)
    return A, Bt, bias, R


def _run(dtype, A, Bt, bias=None, resid=None, relu=False, out_f32=False, tile=0, bscale=None):
    import torch
    from paper_2109_08008_amd import nt
    M, K = A.shape
    N = Bt.shape[0]
    dA, dB = A.cuda(), Bt.cuda()
    dbias = bias.cuda() if bias is not None else None
    dres = resid.cuda() if resid is not None else None
    dsc = bscale.cuda() if bscale is not None else None
    out = torch.full((M, N), float("nan"), dtype=torch.float32 if out_f32 else A.dtype, device="cuda")
    nt.nt_op_gemm(dtype, dA.data_ptr(), K, dB.data_ptr(), M, N, K, dbias.data_ptr() if dbias is not None else 0,
                  dres.data_ptr() if dres is not None else 0, out.data_ptr(), N, out_f32, relu, tile,
                  dsc.data_ptr() if dsc is not None else None)
    torch.cuda.synchronize()
    return out.cpu()


def _fp8_weights(N, K, seed):
    """Random weights quantized by the library's own FP8 quantizer: (codes [N][K] uint8,
    scales [N] fp32, the dequantized weights [N][K] fp64)."""
    import torch
    from paper_2109_08008_amd import nt
    w = np.random.default_rng(seed).normal(0.0, 1.0, size=(K, N)).astype(np.float32)   # [in][out]
    q, sc = nt.nt_quantize_fp8(w)
    qt = torch.from_numpy(q)
    deq = qt.view(torch.float8_e4m3fn).double() * torch.from_numpy(sc).double()[:, None]
    return qt, torch.from_numpy(sc), deq


@pytest.mark.parametrize("tile", [1, 2, 3, 4])
@pytest.mark.parametrize("M,N,K", [(1, 8, 64), (37, 100, 512), (200, 520, 128), (300, 1000, 2048), (129, 136, 576)])
def test_fp8_weight_gemm_matches_fp64(tile, M, N, K):
    """fp16 activations times FP8 E4M3 weights with column scales: the product of the
    activations with the dequantized weights, to the fp16 GEMM's bound."""
    import torch
    A, _, bias, R = _setup("f16", M, N, K, seed=M * 5 + N + K)
    q, sc, deq = _fp8_weights(N, K, seed=M + N * 3 + K)
    ref = A.double() @ deq.T
    for mode in ("plain", "bias", "relu", "resid", "f32out"):
        kw = {}
        want = ref.clone()
        if mode in ("bias", "relu", "resid"):
            kw["bias"] = bias
            want = want + bias.double()
        if mode == "relu":
            kw["relu"] = True
            want = want.clamp_min(0)
        if mode == "resid":
            kw["resid"] = R
            want = want + R.double()
        if mode == "f32out":
            kw["out_f32"] = True
        got = _run("f16", A, q, tile=tile, bscale=sc, **kw)
        assert not torch.isnan(got).any(), mode
        ulp = ULP["f32"] if mode == "f32out" else ULP["f16"]
        tol = want.abs().max().item() * ulp + 8 * 2.0 ** -24 * K * np.sqrt(K)
        err = (got.double() - want).abs().max().item()
        assert err <= tol, (mode, err, tol)


def test_fp8_weight_gemm_rows_do_not_depend_on_tile_or_batch():
    A, _, bias, _ = _setup("f16", 700, 384, 1024, seed=5)
    q, sc, _ = _fp8_weights(384, 1024, seed=6)
    full = _run("f16", A, q, bias=bias, tile=2, bscale=sc)
    for tile in (1, 3, 4):
        assert torch_equal(_run("f16", A, q, bias=bias, tile=tile, bscale=sc), full)
    assert torch_equal(_run("f16", A[:123], q, bias=bias, tile=1, bscale=sc), full[:123])


def test_fp8_weights_need_fp16():
    import torch
    from paper_2109_08008_amd import nt
    A, Bt, _, _ = _setup("bf16", 16, 64, 64, seed=1)
    sc = torch.ones(64).cuda()
    with pytest.raises(nt.NTError) as e:
        _run("bf16", A, Bt, bscale=sc)
    assert e.value.status == nt.NT_E_UNSUPPORTED


@pytest.mark.parametrize("tile", [1, 2, 3, 4])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("M,N,K", [(1, 8, 64), (37, 100, 512), (200, 520, 128), (300, 1000, 2048), (129, 136, 576)])
def test_gemm_matches_fp64(dtype, tile, M, N, K):
    import torch
    A, Bt, bias, R = _setup(dtype, M, N, K, seed=M * 7 + N + K)
    ref = A.double() @ Bt.double().T
    for mode in ("plain", "bias", "relu", "resid", "f32out"):
        kw = {}
        want = ref.clone()
        if mode in ("bias", "relu", "resid"):
            kw["bias"] = bias
            want = want + bias.double()
        if mode == "relu":
            kw["relu"] = True
            want = want.clamp_min(0)
        if mode == "resid":
            kw["resid"] = R
            want = want + R.double()
        if mode == "f32out":
            kw["out_f32"] = True
        got = _run(dtype, A, Bt, tile=tile, **kw)
        assert not torch.isnan(got).any(), mode
        ulp = ULP["f32"] if mode == "f32out" else ULP[dtype]
        # output rounding + fp32 accumulation over K terms of size ~1 (a tiling or indexing
        # mistake moves results by O(1) or more)
        tol = want.abs().max().item() * ulp + 8 * 2.0 ** -24 * K * np.sqrt(K)
        err = (got.double() - want).abs().max().item()
        assert err <= tol, (mode, err, tol)


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_gemm_rows_do_not_depend_on_tile_or_batch(dtype):
    A, Bt, bias, _ = _setup(dtype, 700, 384, 1024, seed=3)
    full64 = _run(dtype, A, Bt, bias=bias, tile=1)
    full128 = _run(dtype, A, Bt, bias=bias, tile=2)
    assert torch_equal(full64, full128)
    assert torch_equal(_run(dtype, A, Bt, bias=bias, tile=3), full128)
    assert torch_equal(_run(dtype, A, Bt, bias=bias, tile=4), full128)
    part = _run(dtype, A[100:133].contiguous(), Bt, bias=bias, tile=1)
    assert torch_equal(part, full128[100:133])
    one = _run(dtype, A[5:6].contiguous(), Bt, bias=bias, tile=0)
    assert torch_equal(one, full64[5:6])


def torch_equal(a, b):
    import torch
    return bool(torch.equal(a, b))
