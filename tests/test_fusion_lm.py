"""The external fusion scorer's stand-in LLM and the caller's request scoring
(no GPU): the model is a proper causal distribution over words, scores do not
depend on batching or padding, and each distinct request is scored once."""

import numpy as np
import pytest
import torch

from workloads.fusion_lm import CausalWordLM, RoundTripStats, score_requests

V, BOS = 37, 36


@pytest.fixture(scope="module")
def lm():
    return CausalWordLM(V, BOS, d_model=32, n_layers=2, n_heads=4, max_len=64, seed=7)


def one(lm, ws):
    t = torch.tensor([ws or [0]], dtype=torch.int32)
    return float(lm.score(t, torch.tensor([len(ws)]))[0])


def test_next_word_distribution_sums_to_one(lm):
    """For any context, sum_w p(w | <s> ctx) = 1: the increments of the full
    score over every next word log-sum-exp to 0."""
    rng = np.random.default_rng(0)
    for n in (0, 1, 4):
        ctx = [int(x) for x in rng.integers(0, V, n)]
        rows = torch.tensor([ctx + [w] for w in range(V)], dtype=torch.int32)
        s = lm.score(rows, torch.full((V,), n + 1)).double()
        inc = s - one(lm, ctx)
        assert abs(float(torch.logsumexp(inc, 0))) < 1e-5
        assert float(inc.max()) < 0.0


def test_empty_sequence_scores_zero(lm):
    assert one(lm, []) == 0.0


def test_scores_independent_of_batch_and_padding(lm):
    """A sequence's score is the same alone, in a batch with longer sequences
    (padded), and whatever the pad values; a longer score is the chain-rule
    continuation of its prefix (causality)."""
    rng = np.random.default_rng(1)
    seqs = [[int(x) for x in rng.integers(0, V, n)] for n in (1, 3, 7, 2, 5)]
    L = max(map(len, seqs))
    for pad in (0, 5, -1):
        rows = torch.full((len(seqs), L), pad, dtype=torch.int32)
        for i, s in enumerate(seqs):
            rows[i, :len(s)] = torch.tensor(s)
        got = lm.score(rows, torch.tensor([len(s) for s in seqs]))
        for i, s in enumerate(seqs):
            assert abs(float(got[i]) - one(lm, s)) < 1e-4
    s = seqs[2]
    full = torch.tensor([s], dtype=torch.int32)
    prefix_scores = [one(lm, s[:k]) for k in range(len(s) + 1)]
    assert all(b < a for a, b in zip(prefix_scores, prefix_scores[1:]))
    assert abs(float(lm.score(full, torch.tensor([len(s)]))[0]) - prefix_scores[-1]) < 1e-5


def test_score_requests_dedups_and_fills(lm):
    """Request layout [B][K][o][W] with counts (-1 = not asked): every asked
    sub-beam gets its sequence's score, distinct sequences are scored once,
    the rest get 0."""
    B, K, O, W = 2, 3, 2, 6
    words = torch.full((B, K, O, W), 99, dtype=torch.int32)
    nw = torch.full((B, K, O), -1, dtype=torch.int32)
    seqs = {(0, 0, 0): [1, 2, 3], (0, 0, 1): [1, 2], (0, 1, 0): [1, 2, 3], (1, 2, 1): [],
            (1, 0, 0): [4], (1, 1, 0): [1, 2]}
    for (b, k, j), s in seqs.items():
        words[b, k, j, :len(s)] = torch.tensor(s or [0])[:len(s)]
        nw[b, k, j] = len(s)
    seen = []

    def scorer(rows, lens):
        seen.extend(tuple(int(x) for x in r[:n]) for r, n in zip(rows, lens))
        return lm.score(rows, lens)

    st = RoundTripStats()
    out = score_requests(words, nw, scorer, batch=2, stats=st)
    assert out.shape == (B, K, O) and out.dtype == torch.float32
    for b in range(B):
        for k in range(K):
            for j in range(O):
                if (b, k, j) in seqs:
                    assert abs(float(out[b, k, j]) - one(lm, seqs[(b, k, j)])) < 1e-4
                else:
                    assert float(out[b, k, j]) == 0.0
    assert sorted(seen) == sorted(set(map(tuple, seqs.values())))
    assert st.requested == len(seqs) and st.scored == 4 and st.batches == 2
