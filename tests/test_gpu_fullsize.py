"""GPU parity at the benchmark workloads' full sizes.

* Sampled outputs in the benchmark's own configuration: every workload's full sentence
  set, with the benchmark's weights, translated by nt_translate exactly as bench.py
  times it (four batches in flight, graph replay, the workload's token budget and
  search).  For a length-stratified sample of sentences the oracle (fp64 on the
  GPU's rounded weights) is teacher-forced on the GPU's output: every per-token
  log-prob must agree within the fp16 bound (1e-2), and the reported score must be the
  length-normalised sum of those log-probs.  Properties that hold at any size are
  checked on every sentence: the output respects the length limit, never contains
  EOS (generation is not masked otherwise), and the score is finite.
* fp32 at full model shapes: a stratified subset translated greedily and with beam 4
  gives the oracle's token IDs (near-tie protocol for greedy).
"""
import numpy as np
import pytest

import oracle
import synth
from oracle.ensemble import combine
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

FULL = ["base-6-6", "deep-shallow-greedy", "deep-shallow-beam", "wide-30-6", "base-6-6-rpr", "teacher-ensemble",
        "base-6-6-fp8", "wide-30-6-fp8"]
N_SAMPLE = {"teacher-ensemble": 3, "wide-30-6": 4}


def _gpu_model(w, blobs):
    from paper_2109_08008_amd import nt
    if w.members:
        return nt.Ensemble([G.new_model(mb.model, b, w.dtype, hist_norm=mb.dlcl) for mb, b in zip(w.members, blobs)],
                           w.ensemble_rule)
    return G.new_model(w.model, blobs[0], w.dtype)


def _oracle_logp(w, oms, src, toks):
    """[len(toks)+1, V] per-token scores of the oracle teacher-forced on toks."""
    lps = []
    for om in oms:
        lg = om.teacher_forced_logits(src, list(toks))
        lps.append(lg - oracle.logsumexp(lg)[:, None])
    return combine(lps, w.ensemble_rule) if w.members else lps[0]


@pytest.mark.parametrize("name", FULL)
def test_full_workload_sampled_against_oracle(name):
    from paper_2109_08008_amd import nt
    w = synth.WORKLOADS[name]
    blobs = synth.member_weights(w) if w.members else [synth.make_weights(w.model, seed=w.weights_seed)]
    ids, offs = synth.make_sentences(w.data, w.model.vocab, seed=w.data_seed)
    srcs = synth.sentence_list(ids, offs)
    nt.nt_set_streams(4)
    nt.nt_set_graphs(True)
    model = _gpu_model(w, blobs)
    toks, scores, logp = model.translate(ids, offs, w.search)
    # properties of every output
    for s, tk, sc in zip(srcs, toks, scores):
        assert len(tk) <= synth.max_target_len(w.search, len(s))
        assert not (np.asarray(tk) == synth.EOS_ID).any()   # EOS ends a hypothesis; any other ID may be emitted
        assert np.isfinite(sc)
    # sampled sentences against the oracle
    if w.members:
        oms = [G.oracle_model(mb.model, b, w.dtype, hist_norm=mb.dlcl) for mb, b in zip(w.members, blobs)]
    else:
        oms = [G.oracle_model(w.model, blobs[0], w.dtype)]
    worst = 0.0
    for i in synth.stratified_subset(offs, N_SAMPLE.get(name, 6)):
        s, tk = srcs[i], toks[i]
        ref = _oracle_logp(w, oms, s, tk)
        want = np.array([ref[t, tk[t]] for t in range(len(tk))])
        worst = max(worst, float(np.abs(np.asarray(logp[i]) - want).max(initial=0)))
        n = len(tk)
        eos_emitted = n < synth.max_target_len(w.search, len(s))
        raw = float(np.sum(logp[i], dtype=np.float64)) + (ref[n, synth.EOS_ID] if eos_emitted else 0.0)
        norm = oracle.length_penalty(n + (1 if eos_emitted else 0), w.search.len_penalty) if w.search.beam > 1 else 1.0
        assert abs(scores[i] - raw / norm) <= 2e-2 * max(1.0, n / 10), (i, scores[i], raw / norm)
    print(f"{name}: {len(srcs)} sentences, sampled per-token max abs err {worst:.3g}")
    assert worst <= 1e-2
    model.close()


@pytest.mark.parametrize("name,beam", [("base-6-6", 1), ("base-6-6", 4), ("deep-shallow-greedy", 1)])
def test_fp32_full_shape_token_ids(name, beam):
    w = synth.WORKLOADS[name]
    blob = synth.make_weights(w.model, seed=w.weights_seed, lively=True)
    ids, offs = synth.make_sentences(w.data, w.model.vocab, seed=w.data_seed)
    sub = synth.stratified_subset(offs, 16)
    srcs = [synth.sentence_list(ids, offs)[i] for i in sub]
    sub_ids = np.concatenate([np.asarray(s, dtype=np.int32) for s in srcs])
    sub_offs = np.concatenate([[0], np.cumsum([len(s) for s in srcs])]).astype(np.int64)
    search = synth.replace(w.search, beam=beam)
    model = G.new_model(w.model, blob, "f32")
    toks, scores, _ = model.translate(sub_ids, sub_offs, search)
    om = G.oracle_model(w.model, blob, "f32")
    ties = 0
    checked = [0, len(srcs) // 2] if beam > 1 else range(0, len(srcs), 3)
    for k in checked:
        s, tk = srcs[k], toks[k]
        mt = synth.max_target_len(search, len(s))
        if beam == 1:
            ties += G.compare_greedy_ids(om, s, tk, mt)
        else:
            ref = oracle.translate(om, s, search)
            assert list(tk) == list(ref.tokens), k
            assert abs(scores[k] - ref.score) <= 1e-3
    print(f"{name} beam {beam}: near-ties {ties}, lengths {[len(t) for t in toks]}")
    assert ties <= 1
    model.close()
