"""GPU edge cases of nt_translate: input it must reject (an empty sentence, a source past
the position table, a token ID outside the vocabulary, a target limit past the position
table), a model that keeps working after a rejected call, the longest source the
position table allows, and one-step target limits.  Parity is against the oracle in
fp32 (token IDs under the near-tie protocol, teacher-forced logits within 1e-3)."""
import numpy as np
import pytest

import oracle
import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

SHAPE = synth.ModelShape(64, 2, 256, 2, 1, 101)


def _csr(sents):
    ids = np.concatenate([np.asarray(s, dtype=np.int32) for s in sents])
    offs = np.concatenate([[0], np.cumsum([len(s) for s in sents])]).astype(np.int64)
    return ids, offs


def test_invalid_inputs_are_rejected_and_the_model_stays_usable():
    from paper_2109_08008_amd import nt
    blob = synth.make_weights(SHAPE, seed=71, lively=True)
    model = G.new_model(SHAPE, blob, "f32")
    search = synth.SearchSetup(beam=1, max_len_a=1.0, max_len_b=4)
    P = synth.MAX_POSITIONS
    cases = {
        "empty sentence": ([[5, 6], [], [7]], search),
        "source past the position table": ([[5] * (P + 1)], search),
        "token id = vocab": ([[5, SHAPE.vocab, 7]], search),
        "negative token id": ([[5, -1]], search),
        "target limit past the position table": ([[5] * 600], synth.replace(search, max_len_a=2.0, max_len_b=0)),
    }
    for name, (sents, s) in cases.items():
        ids, offs = _csr(sents)
        with pytest.raises(nt.NTError) as err:
            model.translate(ids, offs, s)
        assert err.value.status == nt.NT_E_INVALID, (name, err.value)
    srcs = [[5, 6, 7, 8], [9], [10, 11, 12]]
    ids, offs = _csr(srcs)
    toks, scores, _ = model.translate(ids, offs, search)
    om = G.oracle_model(SHAPE, blob, "f32")
    ties = sum(G.compare_greedy_ids(om, s, tk, synth.max_target_len(search, len(s))) for s, tk in zip(srcs, toks))
    assert ties <= 1
    model.close()


def test_longest_source_the_position_table_allows():
    blob = synth.make_weights(SHAPE, seed=72, lively=True)
    rng = np.random.default_rng(73)
    P = synth.MAX_POSITIONS
    srcs = [list(rng.integers(3, SHAPE.vocab, size=P)), [4], list(rng.integers(3, SHAPE.vocab, size=P - 1))]
    tgts = [list(rng.integers(3, SHAPE.vocab, size=3)) for _ in srcs]
    model = G.new_model(SHAPE, blob, "f32")
    got, _, _ = G.gpu_teacher_forced(model, srcs, tgts, SHAPE.vocab)
    om = G.oracle_model(SHAPE, blob, "f32")
    for b, (s, tg) in enumerate(zip(srcs, tgts)):
        np.testing.assert_allclose(got[b], om.teacher_forced_logits(s, tg), atol=1e-3)
    # and translated with greedy search
    search = synth.SearchSetup(beam=1, max_len_a=0.0, max_len_b=6)
    ids, offs = _csr(srcs)
    toks, _, _ = model.translate(ids, offs, search)
    ties = sum(G.compare_greedy_ids(om, s, tk, 6) for s, tk in zip(srcs, toks))
    assert ties <= 1
    model.close()


@pytest.mark.parametrize("beam", [1, 4])
def test_one_step_target_limit(beam):
    """max target length 1: every hypothesis ends after one step (EOS or the limit)."""
    blob = synth.make_weights(SHAPE, seed=74, lively=True)
    srcs = [[5, 6, 7], [8], [9, 10]]
    ids, offs = _csr(srcs)
    search = synth.SearchSetup(beam=beam, len_penalty=0.6, max_len_a=0.0, max_len_b=1)
    model = G.new_model(SHAPE, blob, "f32")
    toks, scores, _ = model.translate(ids, offs, search)
    om = G.oracle_model(SHAPE, blob, "f32")
    for s, tk, sc in zip(srcs, toks, scores):
        assert len(tk) <= 1
        if beam > 1:
            ref = oracle.translate(om, s, search)
            assert list(tk) == list(ref.tokens)
            assert abs(sc - ref.score) <= 1e-3
        else:
            assert G.compare_greedy_ids(om, s, tk, 1) <= 1
    model.close()
