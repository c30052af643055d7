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


# ---- the oracle over host processes -----------------------------------------------------
# The parity tests at full model shape run the fp64 oracle on tens of sentences.  Each
# sentence is independent (the oracle decodes one sentence at a time), so they are
# spread over forked host processes, one BLAS thread each, the way the paper splits CPU
# decoding by lines (Sec. 4.3).  The children inherit POOL (the oracle model, the
# sentences and the GPU's results, gathered before the fork) and use only NumPy.
POOL: dict = {}


def _pool_call(arg):
    from threadpoolctl import threadpool_limits
    fn, item = arg
    with threadpool_limits(limits=1):
        return fn(item)


def oracle_map(fn, items, procs=None):
    """[fn(x) for x in items] over min(16, cores) forked processes (fn at module level,
    reading its inputs from POOL).  Items are handed out one at a time in the given
    order, so the longest sentences should come first."""
    import multiprocessing as mp
    import os
    items = list(items)
    if not items:
        return []
    import time
    P = min(procs or 16, os.cpu_count() or 1, len(items))
    out = []
    t0 = last = time.time()
    with mp.get_context("fork").Pool(P) as pool:
        for r in pool.imap(_pool_call, [(fn, x) for x in items], chunksize=1):
            out.append(r)
            if time.time() - last > 20:
                last = time.time()
                print(f"  oracle: {len(out)}/{len(items)} sentences after {last - t0:.0f} s", flush=True)
    return out


def greedy_follow(om, src, gpu_tokens, max_tgt, tau=1e-4):
    """compare_greedy_ids that also returns the oracle's fp64 logits along the GPU's
    tokens: (near-ties, [len+1 or max_tgt, V] rows; row t predicts token t)."""
    sc = IncrementalScorer(om, src)
    prefix: list = []
    ties = 0
    rows = []
    gpu = list(int(x) for x in gpu_tokens)
    for t in range(max_tgt):
        logits, _ = sc([prefix])
        row = logits[0]
        rows.append(row)
        w = int(np.argmax(row))
        g = gpu[t] if t < len(gpu) else EOS
        if w != g:
            gap = float(row[w] - row[g])
            assert gap <= tau, f"step {t}: oracle {w} vs GPU {g}, fp64 logit gap {gap:.3g}"
            ties += 1
        if g == EOS:
            assert t == len(gpu)
            return ties, np.stack(rows)
        prefix = prefix + [g]
    assert len(gpu) == max_tgt
    return ties, np.stack(rows)


class BeamFollower:
    """on_step observer for oracle.beam_search that follows one hypothesis (the GPU's
    output tokens).  It keeps the oracle's logits of every prefix of that hypothesis
    while the prefix is live in the oracle's beam, and notes the first step at which the
    hypothesis leaves the beam, with the oracle's fp64 gap there: between the candidate
    kept at the boundary (the K-th live one, or the 2K-th walked one for an EOS
    candidate) and the hypothesis's own candidate."""

    def __init__(self, tokens, K, eos=EOS):
        self.g = [int(x) for x in tokens]
        self.K = K
        self.eos = eos
        self.rows: dict = {}
        self.left = None
        self.gap = None

    def __call__(self, t, live, logits, cand, order):
        if self.left is not None or t > len(self.g):
            return
        pre = self.g[:t]
        h = next((i for i, toks in enumerate(live) if list(toks) == pre), None)
        if h is None:
            self.left, self.gap = t, float("inf")
            return
        self.rows[t] = np.array(logits[h])
        V = logits.shape[1]
        w = self.g[t] if t < len(self.g) else self.eos
        idx = h * V + w
        walked = [int(i) for i in order[:min(2 * self.K, cand.size)]]
        if w == self.eos:
            if idx not in walked:
                self.left, self.gap = t, float(cand[walked[-1]] - cand[idx])
        else:
            kept = [i for i in walked if i % V != self.eos][:self.K]
            if idx not in kept:
                self.left, self.gap = t, float(cand[kept[-1]] - cand[idx])


def hypothesis_score(rows, tokens, n_steps, alpha, eos_emitted):
    """Normalised score of a hypothesis from the logits rows along it (row t predicts
    token t): the sum of its log-probs (EOS included when emitted) over lp(n)."""
    lp = [float(rows[t][w] - oracle.logsumexp(rows[t])) for t, w in enumerate(tokens)]
    raw = sum(lp) + (float(rows[len(tokens)][EOS] - oracle.logsumexp(rows[len(tokens)])) if eos_emitted else 0.0)
    return raw / oracle.length_penalty(n_steps, alpha), lp
