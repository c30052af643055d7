"""Oracle search: greedy and beam search over any next-token scorer.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A scorer maps a list of target prefixes (all of one length t, BOS excluded) to
(logits [n, V], logsumexp [n]); log p = logits - lse.

Greedy (Sec. 4.4, used by every submission): take the argmax of the logits
(lowest ID on ties; the argmax needs no log_softmax, Sec. 4.4 profile notes), stop
at EOS or after max_tgt generated tokens (EOS counted).

Beam search with the paper's faster stop rule (Sec. 4.1: stop once a candidate has
produced EOS and no live candidate scores higher).  Readings of what the paper leaves
open:

* Candidates c = score_h + log p_h(w) over every live h and word w, ordered by
  (c descending, rank_h * V + w ascending); the first 2K are walked in order.
* An EOS candidate becomes a finished hypothesis with score c / lp(n), where n counts
  the generated tokens including EOS and lp(n) = ((5 + n) / 6) ** alpha (GNMT form;
  alpha comes from the workload, not the paper).  Only the best finished hypothesis is
  kept; on equal scores the earlier one stays.
* The first K non-EOS candidates become the next live set, in walk order.
* Stop rule: a finished hypothesis exists and its score >= max over live of
  c / lp(n_live).  Otherwise stop at max_tgt, where live hypotheses are finalised with
  c / lp(max_tgt) after that step's EOS candidates.  early_stop=False runs to max_tgt.
* Output tokens exclude BOS and EOS; the score includes the EOS log-prob.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field

import numpy as np

import synth


@dataclass
class Hypothesis:
    tokens: list                       # generated tokens, EOS excluded
    score: float                       # normalised score (raw sum of log-probs for greedy)
    tok_logp: list = field(default_factory=list)   # log p of each output token
    eos_logp: float | None = None      # log p of the final EOS, if emitted
    raw: float = 0.0                   # un-normalised sum of log-probs incl. EOS


def length_penalty(n, alpha):
    return ((5.0 + n) / 6.0) ** alpha


def greedy_search(scorer, max_tgt, eos=synth.EOS_ID) -> Hypothesis:
    prefix: list = []
    lps: list = []
    total = 0.0
    for t in range(max_tgt):
        logits, lse = scorer([prefix])
        w = int(np.argmax(logits[0]))          # first maximum = lowest ID
        lp = float(logits[0, w] - lse[0])
        total += lp
        if w == eos:
            return Hypothesis(prefix, total, lps, lp, total)
        prefix = prefix + [w]
        lps = lps + [lp]
    return Hypothesis(prefix, total, lps, None, total)


def beam_search(scorer, K, max_tgt, alpha=0.0, early_stop=True, eos=synth.EOS_ID, on_step=None) -> Hypothesis:
    """``on_step`` (optional, for diagnostics) is called at every step, before the
    candidates are walked, as on_step(t, live_tokens, logits, cand, order): the live
    prefixes, their logits [n, V], the candidate scores c (flattened h*V + w) and the
    candidate order; it changes nothing."""
    live = [([], 0.0, [])]                      # (tokens, raw score, per-token logp)
    best: Hypothesis | None = None

    def offer(h: Hypothesis):
        nonlocal best
        if best is None or h.score > best.score:
            best = h

    for t in range(max_tgt):
        n = t + 1
        logits, lse = scorer([h[0] for h in live])
        logp = logits - lse[:, None]
        V = logp.shape[1]
        cand = (np.array([h[1] for h in live], dtype=logp.dtype)[:, None] + logp).reshape(-1)
        order = np.lexsort((np.arange(cand.size), -cand))
        if on_step is not None:
            on_step(t, [h[0] for h in live], logits, cand, order)
        new_live = []
        for idx in order[:min(2 * K, cand.size)]:
            h, w = divmod(int(idx), V)
            c = float(cand[idx])
            toks, _, lps = live[h]
            if w == eos:
                offer(Hypothesis(list(toks), c / length_penalty(n, alpha), list(lps),
                                 float(logp[h, w]), c))
            elif len(new_live) < K:
                new_live.append((toks + [w], c, lps + [float(logp[h, w])]))
        live = new_live
        if n == max_tgt:
            for toks, c, lps in live:
                offer(Hypothesis(list(toks), c / length_penalty(n, alpha), list(lps), None, c))
            break
        if not live:
            break
        if early_stop and best is not None:
            if best.score >= max(h[1] for h in live) / length_penalty(n, alpha):
                break
    return best


def translate(model, src, search: synth.SearchSetup, on_step=None) -> Hypothesis:
    """Translate one sentence with the workload's search setup (``on_step``: see
    beam_search; beam only)."""
    from .model import IncrementalScorer
    max_tgt = synth.max_target_len(search, len(src))
    sc = IncrementalScorer(model, src)
    if search.beam <= 1:
        return greedy_search(sc, max_tgt)
    return beam_search(sc, search.beam, max_tgt, search.len_penalty, bool(search.early_stop), on_step=on_step)


def brute_force_best(scorer, V, max_tgt, alpha=0.0, eos=synth.EOS_ID) -> Hypothesis:
    """Exhaustive search: every sequence that ends in EOS within max_tgt tokens or runs to
    max_tgt without EOS; returns the one with the highest c / lp(n) (earliest on ties,
    enumerating shorter sequences first).  For tiny vocabularies only."""
    words = [w for w in range(V) if w != eos]
    best: Hypothesis | None = None
    for n in range(1, max_tgt + 1):
        for body in itertools.product(words, repeat=n - 1):
            for last in ([eos] + words if n == max_tgt else [eos]):
                seq = list(body) + [last]
                total = 0.0
                lps = []
                for t in range(n):
                    logits, lse = scorer([seq[:t]])
                    lps.append(float(logits[0, seq[t]] - lse[0]))
                    total += lps[-1]
                s = total / length_penalty(n, alpha)
                if best is None or s > best.score:
                    if last == eos:
                        best = Hypothesis(list(body), s, lps[:-1], lps[-1], total)
                    else:
                        best = Hypothesis(seq, s, lps, None, total)
    return best
