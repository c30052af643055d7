"""Pins for the oracle's greedy and beam search.

* Brute force: with a vocabulary of 6 and at most 4 target tokens, a beam wide enough
  to keep every prefix returns the best of all sequences (enumerated exhaustively).
* Beam K=1 (alpha=0) has a closed form in terms of the greedy trajectory.
* With alpha=0 the paper's early-stop rule (Sec. 4.1) returns the same hypothesis as
  running to the length limit, since log-probs only lower a score.
* Greedy's argmax over logits equals the argmax over log-probs (Sec. 4.4).
* A hand-worked table scorer fixes the walk order, EOS handling and stop rule.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from oracle.model import IncrementalScorer

EOS = synth.EOS_ID


class Memo:
    """Cache a scorer's result per prefix (the brute force asks for each prefix many times)."""

    def __init__(self, model, src):
        self.m, self.cross = model, model.cross_kv(model.encode(src))
        self.memo = {}

    def __call__(self, prefixes):
        out_l, out_s = [], []
        for p in prefixes:
            key = tuple(p)
            if key not in self.memo:
                logits = self.m.decode_full(self.cross, list(p))[-1]
                self.memo[key] = (logits, oracle.logsumexp(logits))
            out_l.append(self.memo[key][0])
            out_s.append(self.memo[key][1])
        return np.stack(out_l), np.array(out_s)


class TableScorer:
    """Scorer defined by a dict prefix -> logits; prefixes not in the table get a uniform row."""

    def __init__(self, table, V):
        self.table, self.V = table, V

    def __call__(self, prefixes):
        rows = [np.asarray(self.table.get(tuple(p), np.zeros(self.V)), dtype=np.float64) for p in prefixes]
        logits = np.stack(rows)
        return logits, oracle.logsumexp(logits)


def logp_row(V, spec):
    """Exact log-probabilities: the words in spec get their given log p, the rest share
    the remaining mass equally."""
    rest = [w for w in range(V) if w not in spec]
    mass = 1.0 - sum(math.exp(v) for v in spec.values())
    assert mass > 0
    row = np.full(V, math.log(mass / len(rest)))
    for w, v in spec.items():
        row[w] = v
    return row


TINY_V = synth.ModelShape(d_model=8, n_heads=2, d_ffn=16, n_enc=2, n_dec=1, vocab=6)


@pytest.mark.parametrize("alpha", [0.0, 0.6])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_wide_beam_equals_brute_force(alpha, seed):
    blob = synth.make_weights(TINY_V, seed=seed, std=0.5)
    m = oracle.OracleModel(TINY_V, blob)
    sc = Memo(m, [4, 5, 3, 4])
    best = oracle.brute_force_best(sc, 6, 4, alpha)
    got = oracle.beam_search(sc, 125, 4, alpha, early_stop=False)
    assert got.tokens == best.tokens
    assert (got.eos_logp is None) == (best.eos_logp is None)
    assert got.score == pytest.approx(best.score, abs=1e-12)
    # a wider beam changes nothing
    assert oracle.beam_search(sc, 200, 4, alpha, early_stop=False).tokens == best.tokens


def _beam1_closed_form(sc, max_tgt):
    """Best of {greedy prefix[:s] + EOS when EOS ranked in the top 2 at step s} U {greedy}."""
    prefix, total, best = [], 0.0, None
    for t in range(max_tgt):
        logits, lse = sc([prefix])
        logp = logits[0] - lse[0]
        order = np.lexsort((np.arange(logp.size), -logp))
        w = int(order[0])
        if w != EOS and int(order[1]) == EOS:
            cand = (total + logp[EOS], list(prefix))
            if best is None or cand[0] > best[0]:
                best = cand
        total += logp[w]
        if w == EOS:
            cand = (total, list(prefix))
            return cand if best is None or cand[0] > best[0] else best
        prefix.append(w)
    cand = (total, list(prefix))
    return cand if best is None or cand[0] > best[0] else best


@pytest.mark.parametrize("seed", range(6))
def test_beam_one_closed_form_from_greedy(seed):
    shape = synth.ModelShape(16, 2, 32, 2, 1, 9)
    blob = synth.make_weights(shape, seed=seed, lively=True, eos_boost=2.0 + seed)
    m = oracle.OracleModel(shape, blob)
    src = [4, 7, 8, 5, 6]
    sc = IncrementalScorer(m, src)
    g = oracle.greedy_search(IncrementalScorer(m, src), 12)
    b = oracle.beam_search(IncrementalScorer(m, src), 1, 12, 0.0, early_stop=True)
    b_full = oracle.beam_search(IncrementalScorer(m, src), 1, 12, 0.0, early_stop=False)
    score, toks = _beam1_closed_form(sc, 12)
    assert b.tokens == toks and b_full.tokens == toks
    assert b.score == pytest.approx(score, abs=1e-12)
    assert b.score >= g.score - 1e-12


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("K", [2, 4])
def test_early_stop_is_exact_without_length_penalty(seed, K):
    shape = synth.ModelShape(16, 2, 32, 2, 1, 13)
    blob = synth.make_weights(shape, seed=seed, lively=True, eos_boost=3.0)
    m = oracle.OracleModel(shape, blob)
    src = [4, 9, 10, 12, 5, 5]
    a = oracle.beam_search(IncrementalScorer(m, src), K, 15, 0.0, early_stop=True)
    b = oracle.beam_search(IncrementalScorer(m, src), K, 15, 0.0, early_stop=False)
    assert a.tokens == b.tokens
    assert a.score == pytest.approx(b.score, abs=1e-12)


def test_greedy_argmax_logits_equals_argmax_logprobs():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(50, 1000)) * 3
    logp = x - oracle.logsumexp(x)[:, None]
    np.testing.assert_array_equal(np.argmax(x, -1), np.argmax(logp, -1))


def test_greedy_ties_go_to_lowest_id():
    V = 6
    tab = {(): [0, 0, -9, 1, 1, 1], (3,): [0, 0, 5, 0, 0, 0]}
    h = oracle.greedy_search(TableScorer(tab, V), 5)
    assert h.tokens == [3]
    lse0 = math.log(2 + math.exp(-9) + 3 * math.e)
    assert h.tok_logp[0] == pytest.approx(1 - lse0)


def test_hand_worked_beam_example():
    """V = 4 (PAD, BOS, EOS, w=3), K = 2; log p(PAD) = log p(BOS) share the rest.

    Step 0 from []: log p(EOS) = -1.0, log p(3) = -0.5, log p(PAD) = log p(BOS) = -4.36.
      Walk: [3] -0.5 (live), EOS -1.0 (finished, score -1.0), [0] -4.36 (live).
      Stop test: -1.0 >= -0.5?  No.
    Step 1 from [3]: log p(EOS) = -0.2 -> finished -0.7 (better); [3,3] -2.5 live, [3,0] live.
      Stop test: -0.7 >= -2.5 -> stop.  Result: tokens [3], score -0.7.
    """
    tab = {(): logp_row(4, {EOS: -1.0, 3: -0.5}), (3,): logp_row(4, {EOS: -0.2, 3: -2.0})}
    h = oracle.beam_search(TableScorer(tab, 4), 2, 10, 0.0, early_stop=True)
    assert h.tokens == [3]
    assert h.score == pytest.approx(-0.7, abs=1e-12)
    assert h.tok_logp == pytest.approx([-0.5], abs=1e-12)
    assert h.eos_logp == pytest.approx(-0.2, abs=1e-12)
    # the length-limited run with alpha = 1: scores are divided by (5+n)/6
    h = oracle.beam_search(TableScorer(tab, 4), 2, 2, 1.0, early_stop=False)
    assert h.tokens == [3]
    assert h.score == pytest.approx(-0.7 / (7 / 6), abs=1e-12)


def test_length_limit_finalises_live_hypotheses():
    # EOS is never likely: the beam runs to max_tgt and returns the best live hypothesis
    V = 5
    tab = {}
    for n in range(4):
        import itertools
        for p in itertools.product([0, 1, 3, 4], repeat=n):
            tab[p] = [-3.0, -2.0, -20.0, -1.0 - 0.1 * n, -1.5]
    h = oracle.beam_search(TableScorer(tab, V), 3, 3, 0.0)
    assert h.tokens == [3, 3, 3]
    assert h.eos_logp is None
    g = oracle.greedy_search(TableScorer(tab, V), 3)
    assert g.tokens == [3, 3, 3]
    lse = oracle.logsumexp(np.array(tab[()]))
    assert g.tok_logp[0] == pytest.approx(-1.0 - lse)


def test_alpha_changes_ranking_of_finished_lengths():
    # Finished candidates: [] + EOS with raw -1.2 (n=1) and [3] + EOS with raw -1.35 (n=2).
    # alpha = 0 prefers the short one; alpha = 2 divides by ((5+n)/6)^2 and prefers the long one.
    tab = {(): logp_row(5, {EOS: -1.2, 3: -0.4}), (3,): logp_row(5, {EOS: -0.95})}
    a0 = oracle.beam_search(TableScorer(tab, 5), 2, 3, 0.0, early_stop=False)
    a2 = oracle.beam_search(TableScorer(tab, 5), 2, 3, 2.0, early_stop=False)
    assert a0.tokens == [] and a0.score == pytest.approx(-1.2, abs=1e-12)
    assert a2.tokens == [3] and a2.score == pytest.approx(-1.35 / (7 / 6) ** 2, abs=1e-12)
