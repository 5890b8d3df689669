"""Exhaustive enumeration of CTC alignments for tiny inputs (a pin for the oracle).

Every alignment a in C^T over a small class subset C is scored as
sum_t D[t, a_t], collapsed (merge repeats, drop blanks) and grouped by the
collapsed symbol sequence; alignments with symbols outside the lexicon are
discarded.  A complete hypothesis (empty, or ending in the separator) then
scores LSE over its alignments (or the best alignment alone, for the max
recombination), plus the token / word bonuses, plus the best word-level
reading over its homophones.  No beam, no pruning, no prefix
search: the definition of the search target written out.
"""

from __future__ import annotations

import itertools
import math
from typing import Callable, Dict, List, Sequence, Tuple

import numpy as np

BLANK, SEP = 0, 40


def collapse(a: Sequence[int]) -> Tuple[int, ...]:
    out = []
    prev = None
    for s in a:
        if s != prev and s != BLANK:
            out.append(int(s))
        prev = s
    return tuple(out)


def alignment_lse(D: np.ndarray, classes: Sequence[int], reduce: str = "lse") -> Dict[Tuple[int, ...], float]:
    """log-sum-exp (reduce="lse") or maximum (reduce="max") over alignments of D
    (float64 [T, 41]) per collapsed sequence."""
    T = D.shape[0]
    C = np.asarray(classes)
    grid = np.array(list(itertools.product(range(len(C)), repeat=T)), dtype=np.int64)
    A = C[grid]
    scores = D[np.arange(T)[None, :], A].sum(axis=1)
    acc: Dict[Tuple[int, ...], float] = {}
    for row, sc in zip(A, scores):
        y = collapse(row)
        prev = acc.get(y, -math.inf)
        acc[y] = float(np.logaddexp(prev, sc)) if reduce == "lse" else float(max(prev, sc))
    return acc


def segments(y: Tuple[int, ...]):
    """Split y into words; returns (complete words, trailing partial word)."""
    words, cur = [], []
    for s in y:
        if s == SEP:
            words.append(tuple(cur))
            cur = []
        else:
            cur.append(s)
    return words, tuple(cur)


def complete_hypotheses(D: np.ndarray, classes: Sequence[int], lex_words: List[Tuple[int, ...]],
                        beta: float, gamma: float,
                        reading_score: Callable[[List[int]], float], reduce: str = "lse",
                        entry_word: Sequence[int] = None):
    """{y: (total, best reading)} over every lexicon-valid complete hypothesis.

    ``lex_words[e]`` spells word ``entry_word[e]`` (default: word e)."""
    homs: Dict[Tuple[int, ...], List[int]] = {}
    for e, ph in enumerate(lex_words):
        w = e if entry_word is None else int(entry_word[e])
        lst = homs.setdefault(tuple(ph), [])
        if w not in lst:
            lst.append(w)
    for k in homs:
        homs[k].sort()
    out = {}
    for y, lse in alignment_lse(D, classes, reduce).items():
        words, partial = segments(y)
        if partial:
            continue
        if any(len(w) == 0 or w not in homs for w in words):
            continue
        n_ph = sum(len(w) for w in words)
        best, best_r = -math.inf, None
        for reading in itertools.product(*[homs[w] for w in words]):
            s = reading_score(list(reading))
            if s > best:
                best, best_r = s, list(reading)
        out[y] = (lse + beta * n_ph + gamma * len(words) + best, best_r, lse)
    return out
