"""Parity protocol between ranked decoder outputs and the oracle's (no GPU).

An utterance's output is its ranked list of (word sequence, fp32 total).  It
matches the oracle's when every rank holds the same word sequence and the
scores agree within SCORE_TOL.  A near-tie is an utterance whose oracle
ranking has two adjacent totals less than NEAR_TIE apart, or whose last frame
kept its K-th candidate less than NEAR_TIE above the (K+1)-th: near-ties are
counted and reported.  A differing output is excused only

* at a near-tie, if every rank above the first near-tied pair matches
  ("near_tie_excused"), or
* when some decision inside the search (top-K, theta, top-o, lambda, top-F)
  was taken at a margin below EXCUSE_TOL, where rounding may flip it
  ("tie_divergent": both sides compute in fp64, so the window is tiny).

Anything else is a mismatch.  Word sequences are compared through a 64-bit
hash so that stored oracle results stay small.
"""

from __future__ import annotations

import hashlib
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

SCORE_TOL = 1e-4     # fp32 hypothesis scores, absolute
NEAR_TIE = 1e-4      # adjacent totals / the last frame's K-th vs (K+1)-th below this: a near-tie
EXCUSE_TOL = 1e-9    # a decision margin below this may flip under fp64 rounding
SEARCH_MARGINS = ("topk", "theta", "homophone", "lambda", "fusion")


def word_hash(words: Sequence[int]) -> int:
    """64-bit hash of a word-id sequence."""
    a = np.ascontiguousarray(np.asarray(list(words), dtype=np.int32))
    return int.from_bytes(hashlib.blake2b(a.tobytes(), digest_size=8).digest(), "little")


@dataclass
class Expected:
    """The oracle's ranked output for one utterance."""

    hashes: np.ndarray            # uint64 [n], word_hash of each rank's words
    total: np.ndarray             # float64 [n]
    margins: Dict[str, float]
    words: Optional[List[List[int]]] = None

    @classmethod
    def from_oracle(cls, res, K: int) -> "Expected":
        ws = [[int(x) for x in w] for w in res.words[:K]]
        return cls(np.array([word_hash(w) for w in ws], dtype=np.uint64), np.asarray(res.total[:K], np.float64),
                   dict(res.margins), ws)


def near_tie_ranks(exp: Expected) -> List[int]:
    """Ranks r whose total is less than NEAR_TIE above rank r+1's (the last rank
    when the last frame's K-th candidate was that close to the (K+1)-th)."""
    t = exp.total
    r = [i for i in range(len(t) - 1) if t[i] - t[i + 1] < NEAR_TIE]
    if exp.margins.get("last_topk", np.inf) < NEAR_TIE and len(t):
        r.append(len(t) - 1)
    return r


@dataclass
class Parity:
    utterances: int = 0
    exact: int = 0
    near_tie: int = 0           # utterances with a near-tie (reported, whatever the outcome)
    near_tie_excused: int = 0   # differ below the first near-tied pair, match above it
    tie_divergent: int = 0      # differ after a search decision taken at a margin < EXCUSE_TOL
    mismatch: List[str] = field(default_factory=list)
    empty: int = 0              # utterances whose oracle output is empty
    n_hyps: int = 0             # hypotheses compared and matched
    max_score_err: float = 0.0

    def add(self, b: int, gw: List[List[int]], gs: np.ndarray, exp: Expected) -> str:
        """Classifies utterance b: gw / gs are the decoder's ranked words and fp32 scores."""
        self.utterances += 1
        n_o, n_g = len(exp.total), len(gw)
        self.empty += n_o == 0
        ties = near_tie_ranks(exp)
        self.near_tie += bool(ties)
        k = 0
        while k < min(n_g, n_o) and word_hash(gw[k]) == int(exp.hashes[k]) and \
                abs(float(gs[k]) - float(exp.total[k])) <= SCORE_TOL:
            self.max_score_err = max(self.max_score_err, abs(float(gs[k]) - float(exp.total[k])))
            k += 1
        if k == n_g == n_o:
            self.exact += 1
            self.n_hyps += n_o
            return "exact"
        if ties and k >= min(ties):
            self.near_tie_excused += 1
            self.n_hyps += k
            return "near_tie_excused"
        if min(exp.margins.get(m, np.inf) for m in SEARCH_MARGINS) < EXCUSE_TOL:
            self.tie_divergent += 1
            return "tie_divergent"
        ow = exp.words
        self.mismatch.append(
            f"utt {b}: first difference at rank {k}: decoder "
            f"{(gw[k], float(gs[k])) if k < n_g else None} oracle "
            f"{((ow[k] if ow else hex(int(exp.hashes[k]))), float(exp.total[k])) if k < n_o else None}; "
            f"n decoder={n_g} oracle={n_o}; margins={exp.margins}")
        return "mismatch"

    def counts(self) -> dict:
        return dict(utterances=self.utterances, exact=self.exact, near_tie=self.near_tie,
                    near_tie_excused=self.near_tie_excused, tie_divergent=self.tie_divergent,
                    mismatch=len(self.mismatch), empty=self.empty, hyps_compared=self.n_hyps,
                    max_abs_score_err=self.max_score_err)

    def report(self, name: str) -> str:
        c = self.counts()
        return (f"[parity] {name}: utts={c['utterances']} exact={c['exact']} near_tie={c['near_tie']} "
                f"excused={c['near_tie_excused']} tie_divergent={c['tie_divergent']} mismatch={c['mismatch']} "
                f"empty={c['empty']} hyps={c['hyps_compared']} max|dscore|={c['max_abs_score_err']:.2e}")
