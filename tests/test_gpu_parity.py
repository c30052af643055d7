"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Tolerances: fp32 logits <= 1e-3 max abs, per-token log-probs <= 1e-3 and identical token
IDs (near-tie protocol); fp16 teacher-forced logits <= 5e-2 max abs and per-token
log-probs <= 1e-2; bf16 (8 mantissa bits against fp16's 11, so 8x the rounding error)
logits <= 0.4 and per-token log-probs <= 8e-2.  A score (a sum of per-token log-probs)
is held to the per-token bound times the number of its terms.  The oracle always runs in
fp64 on the weights as the GPU stores them (matrices rounded to the 16-bit type).
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

LOGIT_TOL = {"f32": 1e-3, "f16": 5e-2, "bf16": 0.4}
LOGP_TOL = {"f32": 1e-3, "f16": 1e-2, "bf16": 8e-2}
ENC_TOL = {"f32": 1e-4, "f16": 3e-2, "bf16": 0.25}

SHAPES = {
    "d64": synth.ModelShape(64, 2, 256, 2, 1, 101),
    "d128": synth.ModelShape(128, 4, 512, 3, 2, 203),
    "d256": synth.ModelShape(256, 4, 1024, 2, 1, 517),
}


def _sentences(n, lo, hi, V, seed):
    ids, offs = synth.make_sentences(synth.DataSetup(n, "uniform", lo, hi, "uniform"), V, seed=seed)
    return synth.sentence_list(ids, offs), ids, offs


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("name", list(SHAPES))
def test_encoder_output(name, dtype):
    shape = SHAPES[name]
    blob = synth.make_weights(shape, seed=11, lively=True)
    srcs, _, _ = _sentences(12, 1, 23, shape.vocab, seed=3)
    model = G.new_model(shape, blob, dtype)
    st, keep = G.gpu_encode(model, srcs, synth.SearchSetup(beam=1, max_len_b=4))
    from paper_2109_08008_amd import nt
    try:
        enc = nt.nt_dec_state_encoder_out(st, shape.d_model)
    finally:
        nt.nt_free_state(st)
    om = G.oracle_model(shape, blob, dtype)
    err = 0.0
    for b, s in enumerate(srcs):
        ref = om.encode(s)
        err = max(err, float(np.abs(enc[b, :len(s)] - ref).max()))
    print(f"{name} {dtype}: encoder max abs err {err:.3g}")
    assert err <= ENC_TOL[dtype]


# Deep encoders (Sec. 3.1): at these depths the layer-input combination runs blocked, each
# block start also summing the older history entries for the next few rows (up to two
# rows at d <= 512, up to four at d = 1024).
DEEP = {
    "d64-L13": synth.ModelShape(64, 2, 256, 13, 1, 101),
    "d128-L18": synth.ModelShape(128, 4, 512, 18, 1, 203),
    "d1024-L14": synth.ModelShape(1024, 8, 1024, 14, 1, 101),
}


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("name", list(DEEP))
def test_deep_encoder_output_and_logits(name, dtype):
    from paper_2109_08008_amd import nt
    shape = DEEP[name]
    blob = synth.make_weights(shape, seed=13, lively=True)
    srcs, _, _ = _sentences(10, 1, 29, shape.vocab, seed=6)
    model = G.new_model(shape, blob, dtype)
    st, keep = G.gpu_encode(model, srcs, synth.SearchSetup(beam=1, max_len_b=4))
    try:
        enc = nt.nt_dec_state_encoder_out(st, shape.d_model)
    finally:
        nt.nt_free_state(st)
    om = G.oracle_model(shape, blob, dtype)
    enc_err = max(float(np.abs(enc[b, :len(s)] - om.encode(s)).max()) for b, s in enumerate(srcs))
    rng = np.random.default_rng(7)
    tgts = [list(rng.integers(3, shape.vocab, size=int(rng.integers(0, 9)))) for _ in srcs]
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    log_err = max(float(np.abs(got[b] - om.teacher_forced_logits(s, tg)).max())
                  for b, (s, tg) in enumerate(zip(srcs, tgts)))
    print(f"{name} {dtype}: encoder max abs err {enc_err:.3g}, logits {log_err:.3g}")
    assert enc_err <= ENC_TOL[dtype]
    assert log_err <= LOGIT_TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("name", list(SHAPES))
def test_teacher_forced_logits(name, dtype):
    shape = SHAPES[name]
    blob = synth.make_weights(shape, seed=12, lively=True)
    srcs, _, _ = _sentences(9, 1, 30, shape.vocab, seed=4)
    rng = np.random.default_rng(5)
    tgts = [list(rng.integers(3, shape.vocab, size=int(rng.integers(0, 12)))) for _ in srcs]
    model = G.new_model(shape, blob, dtype)
    got, scores, logp = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, dtype)
    err = 0.0
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        ref = om.teacher_forced_logits(s, tg)
        err = max(err, float(np.abs(got[b] - ref).max()))
        # the recorded per-token log-probs are the forced tokens' log_softmax values
        ref_lp = ref - np.log(np.exp(ref - ref.max(1, keepdims=True)).sum(1, keepdims=True)) - ref.max(1, keepdims=True)
        want = [ref_lp[t, tg[t]] for t in range(len(tg))]
        assert np.abs(np.asarray(logp[b]) - want).max(initial=0) <= LOGP_TOL[dtype]
        full = sum(want) + ref_lp[len(tg), synth.EOS_ID]
        assert abs(scores[b] - full) <= LOGP_TOL[dtype] * (len(tg) + 1)
    print(f"{name} {dtype}: teacher-forced logits max abs err {err:.3g}")
    assert err <= LOGIT_TOL[dtype]


def test_tiny_greedy_fp32_token_ids():
    w = synth.WORKLOADS["tiny"]
    blob = synth.make_weights(w.model, lively=True)
    ids, offs = synth.make_sentences(w.data, w.model.vocab)
    srcs = synth.sentence_list(ids, offs)
    model = G.new_model(w.model, blob, "f32")
    toks, scores, _ = model.translate(ids, offs, w.search)
    om = G.oracle_model(w.model, blob, "f32")
    import oracle
    ties = 0
    for s, tk, sc in zip(srcs, toks, scores):
        ties += G.compare_greedy_ids(om, s, tk, 24)
        ref = oracle.translate(om, s, w.search)
        if list(ref.tokens) == list(tk):
            assert abs(ref.score - sc) <= 1e-3
    print("near-ties:", ties, "lengths:", [len(t) for t in toks])
    assert ties <= 1


@pytest.mark.parametrize("beam,alpha,early", [(4, 0.0, 1), (4, 0.6, 1), (4, 0.6, 0), (2, 0.0, 1), (2, 0.6, 1),
                                              (3, 0.6, 1), (5, 0.0, 1), (6, 0.6, 0), (7, 0.6, 1), (12, 0.6, 1),
                                              (8, 0.0, 1), (8, 0.6, 1), (16, 0.0, 1), (16, 0.6, 1), (16, 0.6, 0)])
def test_beam_fp32_token_ids(beam, alpha, early):
    """Beam widths 2 to 16 (the widest the library accepts; 2K = 32 candidates a row).  The
    EOS row's boost is set so that hypotheses end at varied steps: some at once, some in
    between, some at the length limit (a wider beam keeps an early EOS more easily, so
    K = 16 gets a smaller boost)."""
    import oracle
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=21, lively=True, eos_boost=1.0 if beam > 8 else 1.2)
    srcs, ids, offs = _sentences(10, 2, 20, shape.vocab, seed=6)
    search = synth.SearchSetup(beam=beam, len_penalty=alpha, max_len_a=1.0, max_len_b=6, early_stop=early)
    model = G.new_model(shape, blob, "f32")
    toks, scores, logp = model.translate(ids, offs, search)
    om = G.oracle_model(shape, blob, "f32")
    for s, tk, sc, lp in zip(srcs, toks, scores, logp):
        ref = oracle.translate(om, s, search)
        assert list(tk) == list(ref.tokens)
        assert abs(sc - ref.score) <= 1e-3
        np.testing.assert_allclose(lp, ref.tok_logp, atol=1e-3)
    lens = [len(t) for t in toks]
    limits = [synth.max_target_len(search, len(s)) for s in srcs]
    print("lengths:", lens, "limits:", limits)
    assert sum(n > 0 for n in lens) >= 3 and any(0 < n < m for n, m in zip(lens, limits)), "degenerate search"


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("beam", [1, 4])
def test_batching_and_pruning_do_not_change_results(dtype, beam):
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=31, lively=True, eos_boost=4.0)
    srcs, ids, offs = _sentences(24, 1, 30, shape.vocab, seed=7)
    model = G.new_model(shape, blob, dtype)
    base = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=8192, prune=1)
    ref_t, ref_s, ref_lp = model.translate(ids, offs, base)
    assert any(len(t) < synth.max_target_len(base, len(s)) for t, s in zip(ref_t, srcs)), "nothing finished early"
    for kw in [dict(prune=0), dict(token_budget=64), dict(token_budget=0, max_batch_sents=1),
               dict(token_budget=16384, max_batch_sents=5)]:
        t, s, lp = model.translate(ids, offs, synth.replace(base, **kw))
        for a, b in zip(ref_t, t):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(ref_s, s)
        for a, b in zip(ref_lp, lp):
            np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("beam,prune", [(1, 1), (1, 0), (4, 1), (4, 0)])
def test_concurrency_and_graph_replay_do_not_change_results(beam, prune):
    """Batches decoded one or several at a time, steps replayed as one captured decoder
    step per batch (the default) or launched kernel by kernel, with or without every
    third step issued directly for event timing: the results are bitwise the same."""
    from paper_2109_08008_amd import nt
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=33, lively=True, eos_boost=4.0)
    srcs, ids, offs = _sentences(40, 1, 30, shape.vocab, seed=17)
    model = G.new_model(shape, blob, "f16")
    search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=256, prune=prune)
    ref_t, ref_s, ref_lp = model.translate(ids, offs, search)
    assert any(len(t) < synth.max_target_len(search, len(s)) for t, s in zip(ref_t, srcs)), "nothing finished early"
    runs = []
    try:
        nt.nt_set_graphs(False)
        for streams in (1, 2):
            nt.nt_set_streams(streams)
            runs.append(model.translate(ids, offs, search))
        nt.nt_set_graphs(True)
        nt.nt_set_streams(1)
        runs.append(model.translate(ids, offs, search))
        nt.nt_set_streams(3)
        nt.nt_prof_reset()
        nt.nt_prof_config((1 << len(nt.KERNEL_CLASSES)) - 1, 3)
        runs.append(model.translate(ids, offs, search))
        timed = nt.nt_prof_get(nt.KERNEL_CLASSES.index("gemm_vocab"))
    finally:
        nt.nt_set_graphs(True)
        nt.nt_set_streams(4)
        nt.nt_prof_enable(0)
        nt.nt_prof_reset()
    assert timed["launches"] > 0
    for t, s, lp in runs:
        for a, b in zip(ref_t, t):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(ref_s, s)
        for a, b in zip(ref_lp, lp):
            np.testing.assert_array_equal(a, b)


def test_fp16_translation_logprobs_within_tolerance():
    shape = SHAPES["d256"]
    blob = synth.make_weights(shape, seed=41, lively=True, eos_boost=4.0)
    srcs, ids, offs = _sentences(10, 3, 25, shape.vocab, seed=8)
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.5, max_len_b=5)
    model = G.new_model(shape, blob, "f16")
    toks, scores, logp = model.translate(ids, offs, search)
    om = G.oracle_model(shape, blob, "f16")
    worst = 0.0
    for s, tk, lp in zip(srcs, toks, logp):
        ref = om.teacher_forced_logits(s, list(tk))
        lse = np.log(np.exp(ref - ref.max(1, keepdims=True)).sum(1)) + ref.max(1)
        want = np.array([ref[t, tk[t]] - lse[t] for t in range(len(tk))])
        if len(tk):
            worst = max(worst, float(np.abs(lp - want).max()))
    print("fp16 per-token log-prob max abs err", worst)
    assert worst <= 1e-2


def test_long_and_single_token_sentences():
    """Attention over several 64-key chunks (S = 150) next to one-token sentences."""
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=51, lively=True)
    rng = np.random.default_rng(9)
    srcs = [list(rng.integers(4, shape.vocab, size=n)) for n in (150, 1, 77, 1, 64, 65)]
    tgts = [list(rng.integers(3, shape.vocab, size=4)) for _ in srcs]
    model = G.new_model(shape, blob, "f32")
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, "f32")
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        np.testing.assert_allclose(got[b], om.teacher_forced_logits(s, tg), atol=1e-3)
