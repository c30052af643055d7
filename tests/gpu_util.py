"""Helpers shared by the GPU parity tests: device setup through the C ABI binding and
the oracle-side references.  Imported only by tests marked ``gpu``."""
from __future__ import annotations

import numpy as np

import oracle
import synth
from oracle.model import IncrementalScorer

EOS = synth.EOS_ID


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def new_model(shape, blob, dtype, hist_norm=True):
    from paper_2109_08008_amd import nt
    torch_cuda()
    return nt.Model(shape, blob, dtype, hist_norm)


def pad_batch(srcs):
    B, S = len(srcs), max(len(s) for s in srcs)
    arr = np.zeros((B, S), dtype=np.int32)
    for i, s in enumerate(srcs):
        arr[i, :len(s)] = s
    return arr, np.array([len(s) for s in srcs], dtype=np.int32)


def gpu_encode(model, srcs, search):
    """nt_encode on a padded batch; returns (state, torch tensors kept alive)."""
    from paper_2109_08008_amd import nt
    torch = torch_cuda()
    arr, lens = pad_batch(srcs)
    B, S = arr.shape
    sc = nt.search_cfg(search)
    ws_bytes = nt.nt_workspace_size(model.handle, sc, B, S)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    d_src = torch.from_numpy(arr).cuda()
    d_len = torch.from_numpy(lens).cuda()
    st = nt.nt_encode(model.handle, d_src.data_ptr(), d_len.data_ptr(), lens, B, S, sc, ws.data_ptr(), ws_bytes)
    return st, (ws, d_src, d_len)


def gpu_teacher_forced(model, srcs, tgts, V):
    """Teacher-forced decoder logits for every sentence: list of [len(tgt)+1, V] arrays.

    Step t feeds tgt[t] (EOS after the target), so row t holds the logits that predict
    position t; the search then follows the forced tokens until EOS."""
    from paper_2109_08008_amd import nt
    torch = torch_cuda()
    T = max(len(t) for t in tgts) + 1
    search = synth.SearchSetup(beam=1, max_len_a=0.0, max_len_b=T, token_budget=0, prune=1)
    st, keep = gpu_encode(model, srcs, search)
    B = len(srcs)
    logits = torch.full((B, V), float("nan"), dtype=torch.float32, device="cuda")
    out = [np.zeros((len(t) + 1, V), dtype=np.float32) for t in tgts]
    try:
        for t in range(T):
            forced = np.array([tg[t] if t < len(tg) else EOS for tg in tgts], dtype=np.int32)
            d_forced = torch.from_numpy(forced).cuda()
            logits.fill_(float("nan"))
            alive = nt.nt_decode_step(st, d_forced.data_ptr(), logits.data_ptr())
            host = logits.cpu().numpy()
            for b, tg in enumerate(tgts):
                if t <= len(tg):
                    out[b][t] = host[b]
            if alive == 0:
                break
        toks, scores, logp = nt.nt_dec_state_read(st)
    finally:
        nt.nt_free_state(st)
    for b, tg in enumerate(tgts):
        assert list(toks[b]) == list(tg), (b, list(toks[b]), list(tg))
    return out, scores, logp


def oracle_model(shape, blob, precision, hist_norm=True):
    return oracle.OracleModel(shape, blob, np.float64, precision=precision, hist_norm=hist_norm)


def compare_greedy_ids(om, src, gpu_tokens, max_tgt, tau=1e-4):
    """Token-ID identity with the near-tie protocol: at a divergence, the oracle's fp64 logit
    gap between its token and the GPU's must be <= tau; the oracle then continues from the
    GPU's prefix.  Returns the number of near-ties (raises on a real mismatch)."""
    sc = IncrementalScorer(om, src)
    prefix: list = []
    ties = 0
    gpu = list(int(x) for x in gpu_tokens)
    for t in range(max_tgt):
        logits, _ = sc([prefix])
        row = logits[0]
        w = int(np.argmax(row))
        g = gpu[t] if t < len(gpu) else EOS
        if w != g:
            gap = float(row[w] - row[g])
            assert gap <= tau, f"step {t}: oracle {w} vs GPU {g}, fp64 logit gap {gap:.3g}"
            ties += 1
        if g == EOS:
            assert t == len(gpu)
            return ties
        prefix = prefix + [g]
    assert len(gpu) == max_tgt
    return ties
