"""GPU parity of the FP8 models against the oracle run on the same quantized weights
(fp64 arithmetic): "f8w" (fp16 activations, E4M3 projection weights with column scales)
and "f8" (the same, with an E4M3 self-attention key/value cache).

The weight quantization itself is pinned on the CPU (the library's quantizer equals the
oracle's bit for bit), so the FP8-weight tests measure arithmetic error only and take
the fp16 bounds: encoder output <= 3e-2, teacher-forced logits <= 5e-2, per-token
log-probs of a returned beam hypothesis <= 1e-2.  A check that the FP8 model really
differs from the fp16 one guards against the weights silently staying in fp16.

The cache rounds every key and value to E4M3 on both sides, but from values that already
differ by fp16 rounding: where one lies next to a midpoint between two E4M3 values the
two sides can round it apart, by one E4M3 step (1/16 to 1/8 of its magnitude).  Such a
step moves the logits by more than fp16 rounding does.  If a fraction p of the cached
values round apart, the two sides differ by one step there, while the cache's own effect
(the oracle with against without it) is the rounding error of every value, about a
quarter step on average: the difference is near sqrt(12 p) of the cache's effect.  The
tests allow half of it (p up to 2%; fp16 rounding of the projection's inputs gives p
near 1%), at most 0.1 on the logits, and twice the fp16 bound (2e-2) on the per-token
log-probs of a returned hypothesis.
"""
import numpy as np
import pytest

import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPES = {
    "d64": synth.ModelShape(64, 2, 256, 2, 1, 101),
    "d128": synth.ModelShape(128, 4, 512, 3, 2, 203),
    "d256-rpr": synth.ModelShape(256, 4, 1024, 2, 1, 517, rel_k=4),
}


def _sentences(n, lo, hi, V, seed):
    ids, offs = synth.make_sentences(synth.DataSetup(n, "uniform", lo, hi, "uniform"), V, seed=seed)
    return synth.sentence_list(ids, offs), ids, offs


@pytest.mark.parametrize("name", list(SHAPES))
def test_encoder_output_and_teacher_forced_logits(name):
    from paper_2109_08008_amd import nt
    shape = SHAPES[name]
    blob = synth.make_weights(shape, seed=61, lively=True)
    srcs, _, _ = _sentences(9, 1, 30, shape.vocab, seed=62)
    rng = np.random.default_rng(63)
    tgts = [list(rng.integers(3, shape.vocab, size=int(rng.integers(0, 12)))) for _ in srcs]
    model = G.new_model(shape, blob, "f8w")
    st, keep = G.gpu_encode(model, srcs, synth.SearchSetup(beam=1, max_len_b=4))
    try:
        enc = nt.nt_dec_state_encoder_out(st, shape.d_model)
    finally:
        nt.nt_free_state(st)
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, "f8w")
    enc_err = max(float(np.abs(enc[b, :len(s)] - om.encode(s)).max()) for b, s in enumerate(srcs))
    log_err = max(float(np.abs(got[b] - om.teacher_forced_logits(s, tg)).max())
                  for b, (s, tg) in enumerate(zip(srcs, tgts)))
    # the same model in fp16: the FP8 weights must move the logits well past that noise
    ref16 = G.new_model(shape, blob, "f16")
    got16, _, _ = G.gpu_teacher_forced(ref16, srcs, tgts, shape.vocab)
    moved = max(float(np.abs(a - b).max()) for a, b in zip(got, got16))
    print(f"{name}: encoder err {enc_err:.3g}, logits err {log_err:.3g}, fp8 vs fp16 {moved:.3g}")
    assert enc_err <= 3e-2
    assert log_err <= 5e-2
    assert moved > 4 * log_err


def test_beam_translation_per_token_logprobs():
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=64, lively=True, eos_boost=4.0)
    srcs, ids, offs = _sentences(12, 2, 24, shape.vocab, seed=65)
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.5, max_len_b=5)
    model = G.new_model(shape, blob, "f8w")
    toks, scores, logp = model.translate(ids, offs, search)
    om = G.oracle_model(shape, blob, "f8w")
    worst = 0.0
    for s, tk, lp in zip(srcs, toks, logp):
        ref = om.teacher_forced_logits(s, list(tk))
        lse = np.log(np.exp(ref - ref.max(1, keepdims=True)).sum(1)) + ref.max(1)
        want = np.array([ref[t, tk[t]] - lse[t] for t in range(len(tk))])
        worst = max(worst, float(np.abs(np.asarray(lp) - want).max(initial=0)))
    print("fp8 per-token log-prob max abs err", worst, "lengths", [len(t) for t in toks])
    assert worst <= 1e-2


@pytest.mark.parametrize("beam", [1, 4])
def test_batching_and_pruning_do_not_change_results(beam):
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=66, lively=True, eos_boost=4.0)
    _, ids, offs = _sentences(24, 1, 30, shape.vocab, seed=67)
    model = G.new_model(shape, blob, "f8w")
    base = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=8192, prune=1)
    ref = model.translate(ids, offs, base)
    for kw in [dict(prune=0), dict(token_budget=64), dict(token_budget=0, max_batch_sents=1)]:
        t, s, lp = model.translate(ids, offs, synth.replace(base, **kw))
        for a, b in zip(ref[0], t):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(ref[1], s)


@pytest.mark.parametrize("name", list(SHAPES))
def test_fp8_cache_teacher_forced_logits(name):
    shape = SHAPES[name]
    blob = synth.make_weights(shape, seed=81, lively=True)
    srcs, _, _ = _sentences(9, 1, 30, shape.vocab, seed=82)
    rng = np.random.default_rng(83)
    tgts = [list(rng.integers(3, shape.vocab, size=int(rng.integers(4, 16)))) for _ in srcs]
    got, _, _ = G.gpu_teacher_forced(G.new_model(shape, blob, "f8"), srcs, tgts, shape.vocab)
    om = G.oracle_model(shape, blob, "f8")
    ow = G.oracle_model(shape, blob, "f8w")
    assert om.kv_fp8 and not ow.kv_fp8
    err = cache_effect = 0.0
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        want = om.teacher_forced_logits(s, tg)
        err = max(err, float(np.abs(got[b] - want).max()))
        cache_effect = max(cache_effect, float(np.abs(ow.teacher_forced_logits(s, tg) - want).max()))
    print(f"{name}: FP8 cache logits err {err:.3g}, oracle with vs without the FP8 cache {cache_effect:.3g}")
    assert err <= 0.1
    assert err < 0.5 * cache_effect


def test_fp8_cache_beam_translation_per_token_logprobs():
    shape = SHAPES["d128"]
    blob = synth.make_weights(shape, seed=84, lively=True, eos_boost=4.0)
    srcs, ids, offs = _sentences(12, 2, 24, shape.vocab, seed=85)
    search = synth.SearchSetup(beam=4, len_penalty=0.6, max_len_a=1.5, max_len_b=5)
    toks, scores, logp = G.new_model(shape, blob, "f8").translate(ids, offs, search)
    om = G.oracle_model(shape, blob, "f8")
    ow = G.oracle_model(shape, blob, "f8w")

    def token_logp(model, s, tk):
        ref = model.teacher_forced_logits(s, list(tk))
        lse = np.log(np.exp(ref - ref.max(1, keepdims=True)).sum(1)) + ref.max(1)
        return np.array([ref[t, tk[t]] - lse[t] for t in range(len(tk))])

    worst = cache_effect = 0.0
    for s, tk, lp in zip(srcs, toks, logp):
        want = token_logp(om, s, tk)
        worst = max(worst, float(np.abs(np.asarray(lp) - want).max(initial=0)))
        cache_effect = max(cache_effect, float(np.abs(token_logp(ow, s, tk) - want).max(initial=0)))
    print("FP8 cache per-token log-prob max abs err", worst, "oracle with vs without the FP8 cache", cache_effect,
          "lengths", [len(t) for t in toks])
    assert sum(len(t) for t in toks) > len(toks)
    # the derived bound of the FP8 cache (values one E4M3 step apart for up to 2% of the
    # cache: half the cache's own effect), as for the logits, and never above 5e-2
    assert worst <= min(5e-2, 0.5 * cache_effect)


@pytest.mark.parametrize("beam", [1, 4])
def test_fp8_cache_batching_and_pruning_do_not_change_results(beam):
    shape = SHAPES["d256-rpr"]
    blob = synth.make_weights(shape, seed=86, lively=True, eos_boost=4.0)
    _, ids, offs = _sentences(24, 1, 30, shape.vocab, seed=87)
    model = G.new_model(shape, blob, "f8")
    base = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=1.5, max_len_b=5, token_budget=8192, prune=1)
    ref = model.translate(ids, offs, base)
    for kw in [dict(prune=0), dict(token_budget=64), dict(token_budget=0, max_batch_sents=1)]:
        t, s, lp = model.translate(ids, offs, synth.replace(base, **kw))
        for a, b in zip(ref[0], t):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(ref[1], s)
