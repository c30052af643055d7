"""Oracle ensemble decoding: several models score every step together.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The teacher ensemble of Sec. 2.2 (Table 1: four deep teachers, 35 or 40 encoder layers,
with and without DLCL, six decoder layers, beam 4) decodes with all members at once:
at every step each member scores the next token given the shared prefix, and the search
ranks words by a combination of the members' distributions.  The paper names the
ensemble but not its combination rule, so both common readings are provided:

* ``MEAN_LOGP`` (0): s(w) = (1/M) * sum_m log p_m(w), the average of the members'
  log-probabilities (a normalised geometric mean of the probabilities up to a
  per-step constant; s itself is not renormalised);
* ``LOG_MEAN_P`` (1): s(w) = log((1/M) * sum_m p_m(w)), the log of the average
  probability (normalised by construction).

s(w) is the per-token score the search adds to a hypothesis, in the place of one
model's log p(w): greedy takes its argmax, beam search ranks score + s(w) and applies
the length penalty and the stop rule to the sums exactly as for one model.  Each member
keeps its own encoder output and key/value caches; only the prefix is shared.
"""
from __future__ import annotations

import math

import numpy as np

import synth

from .model import IncrementalScorer, OracleModel, logsumexp
from .search import Hypothesis, beam_search, greedy_search

MEAN_LOGP, LOG_MEAN_P = 0, 1


def combine(member_logp, mode: int) -> np.ndarray:
    """Combined per-token scores from a list of M member log-probability arrays of one
    shape ([n, V]), by the rule ``mode``."""
    lp = np.stack([np.asarray(x) for x in member_logp])      # [M, n, V]
    M = lp.shape[0]
    if mode == MEAN_LOGP:
        return lp.sum(axis=0) / M
    if mode == LOG_MEAN_P:
        return logsumexp(lp, axis=0) - math.log(M)
    raise ValueError(f"unknown ensemble combination {mode}")


class EnsembleScorer:
    """Scorer interface of the search (prefixes -> (scores [n, V], lse [n])) over M member
    scorers.  The combined scores are already per-token scores, so the returned lse is 0
    and the search adds them as they are."""

    def __init__(self, scorers, mode: int):
        if not scorers:
            raise ValueError("an ensemble needs at least one member")
        self.scorers = list(scorers)
        self.mode = mode

    def __call__(self, prefixes):
        lps = []
        for sc in self.scorers:
            logits, lse = sc(prefixes)
            lps.append(logits - lse[:, None])
        s = combine(lps, self.mode)
        return s, np.zeros(s.shape[0], dtype=s.dtype)


def translate_ensemble(models: list[OracleModel], src, search: synth.SearchSetup, mode: int) -> Hypothesis:
    """Translate one sentence with every member scoring each step (same search as one
    model, over the combined scores)."""
    max_tgt = synth.max_target_len(search, len(src))
    sc = EnsembleScorer([IncrementalScorer(m, src) for m in models], mode)
    if search.beam <= 1:
        return greedy_search(sc, max_tgt)
    return beam_search(sc, search.beam, max_tgt, search.len_penalty, bool(search.early_stop))
