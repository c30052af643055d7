"""Pins for the oracle's ensemble decoding (the teacher ensemble of Sec. 2.2).

* Closed forms: two hand-written member distributions, given as logits shifted by
  arbitrary per-member constants, combine to values worked out by hand for both rules;
  the ensemble's choice there differs from both members' choices.
* Special cases: one member is that model; M copies of one model are that model.
* Invariants: the log of the mean probability is normalised; the mean of the
  log-probabilities is at most it (Jensen) and sums to at most one probability (AM-GM);
  member order does not matter.
* Brute force: over a vocabulary of 6 and 4 target tokens, a beam wide enough to keep
  every prefix returns the best sequence under the combined scores, found exhaustively.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from oracle.ensemble import LOG_MEAN_P, MEAN_LOGP, EnsembleScorer, combine, translate_ensemble
from oracle.model import IncrementalScorer
from tests.test_oracle_search import TINY_V, Memo


def shifted_logits(probs, shift):
    return np.log(np.asarray(probs, dtype=np.float64)) + shift


class Fixed:
    """A scorer returning one fixed logits row for every prefix."""

    def __init__(self, row):
        self.row = np.asarray(row, dtype=np.float64)

    def __call__(self, prefixes):
        logits = np.tile(self.row, (len(prefixes), 1))
        return logits, oracle.logsumexp(logits)


def test_combine_closed_form():
    # ids 0..2 (PAD, BOS, EOS) get a small equal share; words 3..5 carry the example
    pa = [0.02, 0.02, 0.02, 0.46, 0.08, 0.40]
    pb = [0.02, 0.02, 0.02, 0.08, 0.46, 0.40]
    # logits up to a per-member constant: the combination must remove each member's own
    # normaliser before mixing
    members = lambda: [Fixed(shifted_logits(pa, 5.0)), Fixed(shifted_logits(pb, -3.0))]
    s0, z0 = EnsembleScorer(members(), MEAN_LOGP)([[]])
    s1, z1 = EnsembleScorer(members(), LOG_MEAN_P)([[]])
    assert np.all(z0 == 0) and np.all(z1 == 0)
    # mean of logs: log 0.02 for ids 0..2, log sqrt(0.46 * 0.08) for words 3 and 4, log 0.4
    g = 0.5 * math.log(0.0368)
    want0 = [math.log(0.02)] * 3 + [g, g, math.log(0.4)]
    # log of the mean: log 0.02, log 0.27 twice, log 0.4
    want1 = [math.log(0.02)] * 3 + [math.log(0.27), math.log(0.27), math.log(0.4)]
    np.testing.assert_allclose(s0[0], want0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(s1[0], want1, rtol=0, atol=1e-14)
    # each member alone picks its own favourite; the ensemble picks the shared second choice
    assert np.argmax(pa) == 3 and np.argmax(pb) == 4
    assert np.argmax(s0[0]) == 5 and np.argmax(s1[0]) == 5
    # greedy over the ensemble takes that word with that score
    h = oracle.greedy_search(EnsembleScorer(members(), LOG_MEAN_P), 1)
    assert h.tokens == [5] and h.score == pytest.approx(math.log(0.4), abs=1e-14)


@pytest.mark.parametrize("mode", [MEAN_LOGP, LOG_MEAN_P])
def test_single_member_is_the_model(mode):
    rng = np.random.default_rng(3)
    lp = rng.normal(size=(5, 11))
    lp = lp - oracle.logsumexp(lp)[:, None]
    np.testing.assert_array_equal(combine([lp], mode), lp)
    blob = synth.make_weights(TINY_V, seed=4, std=0.5)
    m = oracle.OracleModel(TINY_V, blob)
    src = [4, 5, 3, 4, 5]
    for search in (synth.SearchSetup(beam=1, max_len_a=0.0, max_len_b=6),
                   synth.SearchSetup(beam=3, len_penalty=0.6, max_len_a=0.0, max_len_b=6)):
        one = oracle.translate(m, src, search)
        ens = translate_ensemble([m], src, search, mode)
        assert ens.tokens == one.tokens
        assert ens.score == pytest.approx(one.score, abs=1e-12)
        np.testing.assert_allclose(ens.tok_logp, one.tok_logp, rtol=0, atol=1e-12)


@pytest.mark.parametrize("mode", [MEAN_LOGP, LOG_MEAN_P])
def test_copies_of_one_model_are_that_model(mode):
    blob = synth.make_weights(TINY_V, seed=5, std=0.5)
    m = oracle.OracleModel(TINY_V, blob)
    src = [5, 4, 4, 3]
    search = synth.SearchSetup(beam=4, len_penalty=0.0, max_len_a=0.0, max_len_b=5)
    one = oracle.translate(m, src, search)
    ens = translate_ensemble([m, m, m], src, search, mode)
    assert ens.tokens == one.tokens
    assert ens.score == pytest.approx(one.score, abs=1e-12)


def test_normalisation_jensen_and_member_order():
    rng = np.random.default_rng(7)
    members = []
    for _ in range(4):
        x = rng.normal(scale=2.0, size=(6, 50))
        members.append(x - oracle.logsumexp(x)[:, None])
    s0 = combine(members, MEAN_LOGP)
    s1 = combine(members, LOG_MEAN_P)
    np.testing.assert_allclose(oracle.logsumexp(s1), 0.0, atol=1e-12)
    assert np.all(oracle.logsumexp(s0) <= 1e-12)
    assert np.all(s0 <= s1 + 1e-12)
    assert np.all(s1 - s0 > 1e-3)          # members disagree, so the bound is strict here
    perm = [members[i] for i in (2, 0, 3, 1)]
    np.testing.assert_allclose(combine(perm, MEAN_LOGP), s0, rtol=0, atol=1e-12)
    np.testing.assert_allclose(combine(perm, LOG_MEAN_P), s1, rtol=0, atol=1e-12)
    with pytest.raises(ValueError):
        combine(members, 2)


@pytest.mark.parametrize("mode", [MEAN_LOGP, LOG_MEAN_P])
@pytest.mark.parametrize("alpha", [0.0, 0.6])
def test_wide_ensemble_beam_equals_brute_force(mode, alpha):
    src = [4, 5, 3, 4]
    members = [oracle.OracleModel(TINY_V, synth.make_weights(TINY_V, seed=s, std=0.5)) for s in (0, 1)]
    sc = EnsembleScorer([Memo(m, src) for m in members], mode)
    best = oracle.brute_force_best(sc, 6, 4, alpha)
    got = oracle.beam_search(sc, 125, 4, alpha, early_stop=False)
    assert got.tokens == best.tokens
    assert got.score == pytest.approx(best.score, abs=1e-12)
    # the incremental members give the same search result as full recompute
    inc = EnsembleScorer([IncrementalScorer(m, src) for m in members], mode)
    assert oracle.beam_search(inc, 125, 4, alpha, early_stop=False).tokens == best.tokens


def test_teacher_ensemble_members_match_table_1():
    """The teacher-ensemble workload's members have the sizes Table 1 prints: 152M for a
    35-6 teacher, 168M for a 40-6 one and 640M for the ensemble of the four (every
    parameter of the blob: matrices, biases, LayerNorms, DLCL weights, relative-position
    tables)."""
    w = synth.WORKLOADS["teacher-ensemble"]
    counts = [synth.blob_size(m.model) for m in w.members]
    assert [round(c / 1e6) for c in counts] == [152, 152, 168, 168]
    assert round(sum(counts) / 1e6) == 640
    assert sorted(m.dlcl for m in w.members) == [False, False, True, True]
    assert all(m.model.rel_k == 8 and m.model.n_dec == 6 and m.model.n_heads == 8 for m in w.members)
