"""GPU parity of ensemble decoding (the teacher ensemble of Sec. 2.2) against the oracle.

Members differ in width, heads, depth, FFN size, DLCL (on, or a plain pre-norm stack) and
relative positions, as the paper's teachers do.  Tolerances are those of one model:
fp32 combined scores <= 1e-3 max abs under teacher forcing and identical token IDs;
fp16 scores <= 5e-2 and per-token scores of the returned hypothesis <= 1e-2.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle.ensemble import LOG_MEAN_P, MEAN_LOGP, combine, translate_ensemble
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

V = 203
MEMBERS = [  # (shape, seed, dlcl)
    (synth.ModelShape(128, 4, 512, 3, 2, V), 41, True),
    (synth.ModelShape(128, 2, 256, 2, 1, V), 42, False),
    (synth.ModelShape(64, 2, 256, 2, 2, V, rel_k=4), 43, True),
]
SCORE_TOL = {"f32": 1e-3, "f16": 5e-2}
LOGP_TOL = {"f32": 1e-3, "f16": 1e-2}   # per-token combined score of the returned hypothesis


def _blobs():
    return [synth.make_weights(sh, seed=sd, lively=True, eos_boost=4.0, plain_stack=not dl)
            for sh, sd, dl in MEMBERS]


def _gpu_ensemble(dtype, rule, blobs=None, members=MEMBERS):
    from paper_2109_08008_amd import nt
    blobs = blobs or _blobs()
    models = [G.new_model(sh, b, dtype, hist_norm=dl) for (sh, _, dl), b in zip(members, blobs)]
    return nt.Ensemble(models, rule)


def _oracle_members(dtype, blobs=None, members=MEMBERS):
    blobs = blobs or _blobs()
    return [G.oracle_model(sh, b, dtype, hist_norm=dl) for (sh, _, dl), b in zip(members, blobs)]


def _sentences(n, lo, hi, seed):
    ids, offs = synth.make_sentences(synth.DataSetup(n, "uniform", lo, hi, "uniform"), V, seed=seed)
    return synth.sentence_list(ids, offs), ids, offs


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("rule", [MEAN_LOGP, LOG_MEAN_P])
def test_teacher_forced_combined_scores(dtype, rule):
    srcs, _, _ = _sentences(7, 1, 26, seed=8)
    rng = np.random.default_rng(9)
    tgts = [list(rng.integers(3, V, size=int(rng.integers(0, 10)))) for _ in srcs]
    ens = _gpu_ensemble(dtype, rule)
    got, scores, logp = G.gpu_teacher_forced(ens, srcs, tgts, V)
    oms = _oracle_members(dtype)
    err = 0.0
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        lps = []
        for om in oms:
            lg = om.teacher_forced_logits(s, tg)
            lps.append(lg - oracle.logsumexp(lg)[:, None])
        ref = combine(lps, rule)
        err = max(err, float(np.abs(got[b] - ref).max()))
        # the recorded per-token values and the score are sums of combined scores
        want = [ref[t, tg[t]] for t in range(len(tg))]
        assert np.abs(np.asarray(logp[b]) - want).max(initial=0) <= LOGP_TOL[dtype]
        assert abs(scores[b] - (sum(want) + ref[len(tg), synth.EOS_ID])) <= LOGP_TOL[dtype] * (len(tg) + 1)
    print(f"rule {rule} {dtype}: combined scores max abs err {err:.3g}")
    assert err <= SCORE_TOL[dtype]


@pytest.mark.parametrize("rule", [MEAN_LOGP, LOG_MEAN_P])
@pytest.mark.parametrize("beam,alpha", [(1, 0.0), (4, 0.0), (4, 0.6)])
def test_fp32_token_ids(rule, beam, alpha):
    srcs, ids, offs = _sentences(10, 2, 18, seed=10)
    search = synth.SearchSetup(beam=beam, len_penalty=alpha, max_len_a=1.0, max_len_b=6)
    ens = _gpu_ensemble("f32", rule)
    toks, scores, logp = ens.translate(ids, offs, search)
    oms = _oracle_members("f32")
    for s, tk, sc, lp in zip(srcs, toks, scores, logp):
        ref = translate_ensemble(oms, s, search, rule)
        assert list(tk) == list(ref.tokens)
        assert abs(sc - ref.score) <= 1e-3
        np.testing.assert_allclose(lp, ref.tok_logp, atol=1e-3)
    lens = [len(t) for t in toks]
    print("lengths:", lens)
    assert min(lens) < max(synth.max_target_len(search, len(s)) for s in srcs)   # something finished early


def test_fp16_returned_hypothesis_scores():
    rule = MEAN_LOGP
    srcs, ids, offs = _sentences(12, 2, 24, seed=11)
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.5, max_len_b=5)
    ens = _gpu_ensemble("f16", rule)
    toks, scores, logp = ens.translate(ids, offs, search)
    oms = _oracle_members("f16")
    worst = 0.0
    for s, tk, lp in zip(srcs, toks, logp):
        lps = []
        for om in oms:
            lg = om.teacher_forced_logits(s, list(tk))
            lps.append(lg - oracle.logsumexp(lg)[:, None])
        ref = combine(lps, rule)
        want = np.array([ref[t, tk[t]] for t in range(len(tk))])
        worst = max(worst, float(np.abs(np.asarray(lp) - want).max(initial=0)))
    print(f"fp16 per-token combined score max abs err {worst:.3g}")
    assert worst <= 1e-2


def test_one_member_is_the_model():
    from paper_2109_08008_amd import nt
    sh, sd, dl = MEMBERS[0]
    blob = synth.make_weights(sh, seed=sd, lively=True, eos_boost=4.0)
    model = G.new_model(sh, blob, "f32")
    srcs, ids, offs = _sentences(9, 2, 20, seed=12)
    for beam in (1, 4):
        search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.0, max_len_b=6)
        ref_t, ref_s, ref_lp = model.translate(ids, offs, search)
        for rule in (MEAN_LOGP, LOG_MEAN_P):
            ens = nt.Ensemble([model], rule)
            t, s, lp = ens.translate(ids, offs, search)
            for a, b in zip(ref_t, t):
                np.testing.assert_array_equal(a, b)
            np.testing.assert_allclose(s, ref_s, atol=1e-5)
            for a, b in zip(ref_lp, lp):
                np.testing.assert_allclose(a, b, atol=1e-5)
            ens.close()


@pytest.mark.parametrize("beam", [1, 4])
def test_scheduling_does_not_change_results(beam):
    """Batching, pruning, concurrent batches and graph replay leave the ensemble's output
    bitwise unchanged, as they do for one model."""
    from paper_2109_08008_amd import nt
    srcs, ids, offs = _sentences(20, 1, 26, seed=13)
    ens = _gpu_ensemble("f16", LOG_MEAN_P)
    base = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=8192, prune=1)
    ref = ens.translate(ids, offs, base)
    variants = [(dict(prune=0), 4, True), (dict(token_budget=64), 4, True), (dict(token_budget=96), 1, True),
                (dict(token_budget=96), 3, False)]
    try:
        for kw, streams, graphs in variants:
            nt.nt_set_streams(streams)
            nt.nt_set_graphs(graphs)
            t, s, lp = ens.translate(ids, offs, synth.replace(base, **kw))
            for a, b in zip(ref[0], t):
                np.testing.assert_array_equal(a, b)
            np.testing.assert_array_equal(ref[1], s)
            for a, b in zip(ref[2], lp):
                np.testing.assert_array_equal(a, b)
    finally:
        nt.nt_set_streams(4)
        nt.nt_set_graphs(True)


def test_invalid_ensembles_are_rejected():
    from paper_2109_08008_amd import nt
    blobs = _blobs()
    a = G.new_model(MEMBERS[0][0], blobs[0], "f32")
    b16 = G.new_model(MEMBERS[1][0], blobs[1], "f16", hist_norm=False)
    other_v = synth.ModelShape(64, 2, 256, 1, 1, V + 1)
    c = G.new_model(other_v, synth.make_weights(other_v, seed=1), "f32")
    ens = nt.Ensemble([a], MEAN_LOGP)
    cases = [([a, b16], MEAN_LOGP), ([a, c], MEAN_LOGP), ([a, ens], MEAN_LOGP), ([a], 2), ([], MEAN_LOGP),
             ([a] * 9, MEAN_LOGP)]
    for members, rule in cases:
        with pytest.raises(nt.NTError) as e:
            nt.nt_ensemble([m.handle for m in members], rule)
        assert e.value.status == nt.NT_E_INVALID, (len(members), rule)
