"""Pins of the oracle's pruning decisions, worked by hand (no GPU).

The brute-force pins run without pruning; these tiny cases make each pruning
decision of the search bind and fix its outcome by hand arithmetic:

* Alg. 1's top-K selection and its theta cut (best - theta, taken over the
  totals of the current frame, word-level score included, an entry exactly
  at the cut kept), and the order of Alg. 1 that applies the n-gram after
  them;
* the tie-break of equal totals by the 64-bit prefix key, whose values come
  from a SplitMix64 checked here against its published outputs;
* the fusion target set of Sec. 3.4.2 / App. E.4: the top F hypotheses (not
  sub-beams) at a fusion frame, every hypothesis at the end;
* the top-o and lambda cut of Sec. 3.4.1 / App. E.3 (lambda measured from the
  best surviving candidate, not from the parent), and the order (score desc,
  parent sub-beam asc, word id asc) among equal candidates.

Inputs are log-probability rows with -inf outside a few classes, alpha = 1 and
binary-fraction bonuses, so every path score below is exact in fp64; the
n-gram and fusion terms are written out from their definitions.
"""

import math

import numpy as np
import pytest

import oracle
from tests.tinylm import lexicon_from, lm_from_entries
from workloads import DecodeParams

LN10 = math.log(10.0)
NEG = -np.inf
M64 = 2**64 - 1


def splitmix64(x: int) -> int:
    """SplitMix64 output for state x (Steele, Lea & Flood, OOPSLA 2014)."""
    z = (x + 0x9E3779B97F4A7C15) & M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def test_splitmix64_here_matches_published_outputs():
    # the first outputs of SplitMix64 seeded with 0 (states 0, golden, 2*golden)
    assert splitmix64(0) == 0xE220A8397B1DCDAF
    assert splitmix64(0x9E3779B97F4A7C15) == 0x6E789E6AA1B965F4
    assert splitmix64((2 * 0x9E3779B97F4A7C15) & M64) == 0x06C45D188009454F


def frames(*rows):
    """float32 [T][41] rows: -inf except the given {class: log-prob}."""
    out = np.full((len(rows), 41), NEG, np.float64)
    for t, r in enumerate(rows):
        for v, x in r.items():
            out[t, v] = x
    return out.astype(np.float32)


def unigram_lm(n_words, uni, bos_bo=0.0):
    """LM with unigrams only: uni[w] = (log10 p, backoff); <s>, </s>, <unk> appended."""
    W = n_words
    ent = [((w,), p, b) for w, (p, b) in enumerate(uni)]
    ent += [((W,), -99.0, bos_bo), ((W + 1,), -1.0, 0.0), ((W + 2,), -3.0, 0.0)]
    return lm_from_entries(W, [ent, [], [], []])


# alpha = 1 and binary-fraction bonuses: path scores are exact in fp64
BASE = DecodeParams(alpha=1.0, beta=0.5, gamma=0.25, omega=0.0, phi=1.2, theta=1e30, lam=1e30,
                    fusion_interval=0, fusion_top_f=0)


def run(orc, lg, finalize=0, **kw):
    kw.setdefault("beam", 64)
    return orc.decode(lg, oracle.params_from(BASE, finalize=finalize, **kw), max_subs=8)


def labels(res):
    return [tuple(int(s) for s in y) for y in res.labels]


# ------------------------------------------------------------------ top-K and theta

@pytest.fixture(scope="module")
def four_words():
    lex = lexicon_from([(1,), (2,), (3,), (4,)])
    return oracle.Oracle(lex, unigram_lm(4, [(-1.0, 0.0)] * 4))


# One frame from the empty prefix (a_b = 0):
#   ()   blank-stay   0 + D[0]                     = -1.0
#   (1)  extension    0 + D[1] + beta = -0.5 + 0.5 =  0.0
#   (2)               -1.5 + 0.5                   = -1.0
#   (3)               -2.5 + 0.5                   = -2.0
#   (4)               -3.0 + 0.5                   = -2.5
# () and (2) tie exactly at -1.0; key(()) = 0 < key((2)) = splitmix64(2), so ()
# ranks first.
ONE_FRAME = frames({0: -1.0, 1: -0.5, 2: -1.5, 3: -2.5, 4: -3.0})


@pytest.mark.parametrize("K,theta,expect", [
    (2, 30.0, [((1,), 0.0), ((), -1.0)]),                 # K binds: (2) loses the tie on the key
    (3, 30.0, [((1,), 0.0), ((), -1.0), ((2,), -1.0)]),
    (3, 1.0, [((1,), 0.0), ((), -1.0), ((2,), -1.0)]),    # cut = 0 - 1.0: entries at the cut stay
    (3, 0.75, [((1,), 0.0)]),                             # cut = -0.75 drops both -1.0 entries
    (5, 1.75, [((1,), 0.0), ((), -1.0), ((2,), -1.0)]),   # theta binds below K: -2.0, -2.5 < -1.75
    (5, 30.0, [((1,), 0.0), ((), -1.0), ((2,), -1.0), ((3,), -2.0), ((4,), -2.5)]),
])
def test_top_k_and_theta_cut(four_words, K, theta, expect):
    res = run(four_words, ONE_FRAME, beam=K, theta=theta)
    assert labels(res) == [y for y, _ in expect]
    assert res.total.tolist() == [t for _, t in expect]
    assert 0 < splitmix64(2)  # key(()) = 0 is below every other key


def test_top_k_margin_reports_the_boundary(four_words):
    # K = 2: the 2nd and 3rd candidates tie (margin 0); K = 3: -1.0 - (-2.0) = 1.0
    assert run(four_words, ONE_FRAME, beam=2).margins["topk"] == 0.0
    assert run(four_words, ONE_FRAME, beam=3).margins["topk"] == 1.0


def test_exact_total_tie_broken_by_prefix_key(four_words):
    # (1) = (3) = -0.75 + 0.5 = -0.25 exactly, (2) = -1.0 + 0.5 = -0.5, () = -4.
    # key((1)) = splitmix64(1) = 0x910A2DEC89025CC1 > key((3)) = splitmix64(3)
    # = 0x1D0B14E4DB018FED, so (3) ranks before (1) although 3 > 1.
    assert splitmix64(1) == 0x910A2DEC89025CC1 and splitmix64(3) == 0x1D0B14E4DB018FED
    lg = frames({0: -4.0, 1: -0.75, 2: -1.0, 3: -0.75})
    assert labels(run(four_words, lg, beam=1)) == [(3,)]
    res = run(four_words, lg, beam=2)
    assert labels(res) == [(3,), (1,)]
    assert res.total.tolist() == [-0.25, -0.25]
    assert [int(k) for k in res.keys] == [splitmix64(3), splitmix64(1)]


# ------------------------------------------------------------------ theta sees the word-level score

@pytest.fixture(scope="module")
def two_words():
    # w0 = (1), w1 = (2); log10 P(w | <s>) = bo(<s>) + p(w) = p(w): -0.25 and -2.0
    lex = lexicon_from([(1,), (2,)])
    return oracle.Oracle(lex, unigram_lm(2, [(-0.25, 0.0), (-2.0, 0.0)]))


# frame 0: (1) = (2) = -1.0 + 0.5 = -0.5 (blank -inf: the empty prefix dies)
# frame 1: (1 40) = (2 40) = -0.5 - 0.5 + 0.25 = -0.75 (only the separator); both
#          complete a word, and the n-gram (omega = 1) adds after the cut:
#          L0 = ln10 * -0.25 = -0.5756, L1 = ln10 * -2.0 = -4.6052
# frame 2: blank only: acoustic -0.75 - 0.25 = -1.0 for both; totals -1.0 + L;
#          L0 - L1 = 1.75 ln10 = 4.0295, so theta = 4.0 drops (2 40), 4.1 keeps it
THETA_FRAMES = frames({1: -1.0, 2: -1.0}, {40: -0.5}, {0: -0.25})


def test_theta_after_the_word_score_and_before_the_ngram(two_words):
    L0, L1 = LN10 * -0.25, LN10 * -2.0
    # after frame 1 both stay at theta = 4: the cut precedes the n-gram (Alg. 1)
    r2 = run(two_words, THETA_FRAMES[:2], omega=1.0, theta=4.0)
    assert labels(r2) == [(1, 40), (2, 40)]
    np.testing.assert_allclose(r2.total, [-0.75 + L0, -0.75 + L1], rtol=0, atol=1e-12)
    # frame 2 ranks totals with the word-level score: theta = 4.0 cuts (2 40)
    r3 = run(two_words, THETA_FRAMES, omega=1.0, theta=4.0)
    assert labels(r3) == [(1, 40)]
    np.testing.assert_allclose(r3.total, [-1.0 + L0], rtol=0, atol=1e-12)
    r3b = run(two_words, THETA_FRAMES, omega=1.0, theta=4.1)
    assert labels(r3b) == [(1, 40), (2, 40)]
    np.testing.assert_allclose(r3b.total, [-1.0 + L0, -1.0 + L1], rtol=0, atol=1e-12)
    assert r3b.subs[0] == [(pytest.approx(L0, abs=1e-12), [0])]


# ------------------------------------------------------------------ fusion target set

def bg(seed, a, b, lo=-10.0, hi=-0.5):
    """Synthetic bigram fusion score: lo + (hi - lo) * top 16 bits / 2^16."""
    return lo + (hi - lo) * (splitmix64(seed ^ ((a << 32) | b)) >> 48) / 65536.0


def test_fusion_top_f_fuses_hypotheses_not_subbeams():
    # w0 and w1 spell (1); w2 = (2); w3 = (3); omega = 0, so a completed word
    # keeps Lw = 0 and the homophones w0, w1 tie (order by word id: w0, w1).
    lex = lexicon_from([(1,), (1,), (2,), (3,)])
    W, bos = 4, 4
    orc = oracle.Oracle(lex, unigram_lm(W, [(-1.0, 0.0)] * W))
    # seed ^ (<s> << 32 | 1) = 0: Bg(<s>, w1) takes the published splitmix64(0)
    # = 0xE220..., top 16 bits 57888: -10 + 9.5 * 57888 / 65536 = -1.608642578125;
    # Bg(<s>, w0): seed ^ (<s> << 32) = 1, splitmix64(1) >> 48 = 0x910A = 37130:
    # -10 + 9.5 * 37130 / 65536 = -4.6176910400390625
    seed = (bos << 32) | 1
    assert bg(seed, bos, 1) == -1.608642578125 and bg(seed, bos, 0) == -4.6176910400390625
    # frame 0: (1) = 0.0, (2) = -0.5, (3) = -1.0; frame 1: + 0 + gamma 0.25 at the
    # separator: (1 40) = 0.25, (2 40) = -0.25, (3 40) = -0.75, all at the root.
    # Fusion after frame 1 (I = 1) on the top F = 1 hypothesis, (1 40): both
    # of its sub-beams become phi * Bg and re-rank: [w1 1.2 * -1.6086 = -1.9304,
    # w0 1.2 * -4.6177 = -5.5412]; total 0.25 - 1.9304 = -1.6804.
    lg = frames({1: -0.5, 2: -1.0, 3: -1.5}, {40: 0.0})
    f1 = 0.25 + 1.2 * -1.608642578125
    res = run(orc, lg, fusion_interval=1, fusion_top_f=1, fusion_seed=seed)
    assert labels(res) == [(2, 40), (3, 40), (1, 40)]
    assert res.total.tolist() == [-0.25, -0.75, f1]
    assert res.words == [[2], [3], [1]]
    assert res.subs[2] == [(1.2 * -1.608642578125, [1]), (1.2 * -4.6176910400390625, [0])]
    assert res.subs[0] == [(0.0, [2])] and res.subs[1] == [(0.0, [3])]
    assert res.margins["fusion"] == 0.5   # 0.25 - (-0.25): the 1st and 2nd by total
    # F = 2: (2 40) is fused too (seed ^ (<s> << 32 | 2) = 3, splitmix64(3) >> 48 =
    # 0x1D0B = 7435: Bg = -8.92223358154296875); (3 40) is not
    assert bg(seed, bos, 2) == -10.0 + 9.5 * 7435 / 65536
    r2 = run(orc, lg, fusion_interval=1, fusion_top_f=2, fusion_seed=seed)
    assert labels(r2) == [(3, 40), (1, 40), (2, 40)]
    assert r2.total.tolist() == [-0.75, f1, -0.25 + 1.2 * bg(seed, bos, 2)]
    # at the end of the utterance the final fusion covers every hypothesis:
    # (3 40) gets Bg(<s>, w3) (seed ^ ... = 2, splitmix64(2) >> 48 = 0x9758 =
    # 38744: -4.38372802734375)
    assert bg(seed, bos, 3) == -4.38372802734375
    fin = run(orc, lg, finalize=1, fusion_interval=1, fusion_top_f=1, fusion_seed=seed)
    assert labels(fin) == [(1, 40), (3, 40), (2, 40)]
    assert fin.total.tolist() == [f1, -0.75 + 1.2 * -4.38372802734375,
                                  -0.25 + 1.2 * bg(seed, bos, 2)]


def test_fused_subbeams_survive_a_merge_with_an_unfused_parent():
    """Fusion (Sec. 3.4.2) and recombination (App. E.1) over several frames: a
    hypothesis fused at a fusion frame keeps its fused sub-beams when, a frame
    later, the extension of an unfused hypothesis (its parent prefix) merges
    into it: the merged entry takes its word-level state from its own stay,
    not from the extension."""
    lex = lexicon_from([(1,), (2,)])
    W, bos = 2, 2
    orc = oracle.Oracle(lex, unigram_lm(W, [(-1.0, 0.0)] * W))
    # seed ^ (<s> << 32 | w0) = 1: Bg(<s>, w0) from splitmix64(1) >> 48 = 0x910A
    seed = (bos << 32) | 1
    B0 = bg(seed, bos, 0)
    assert B0 == -4.6176910400390625
    # frame 0: (1) = -0.5 + beta 0.5 = 0
    # frame 1: (1 40) = 0 + 0 + gamma 0.25 = 0.25, word w0 (omega = 0: Lw = 0)
    # frame 2: Z = (1 40) by its blank, 0.25 - 1 = -0.75; X = (1 40 2) = 0.25 -
    #          0.5 + 0.5 = 0.25.  Fusion (t = 2, I = 2) on the top F = 1: X
    #          alone, Lw(X) = 1.2 B0; Z keeps Lw = 0.
    # frame 3: X: blank-ending 0.25 - 1 = -0.75; non-blank-ending LSE(its repeat
    #          0.25 - 0.5 = -0.25, Z's extension by 2: -0.75 - 0.5 + 0.5 =
    #          -0.75), with X's own (fused) sub-beam; Z: -0.75 - 1 = -1.75.
    lg = frames({1: -0.5}, {40: 0.0}, {0: -1.0, 2: -0.5}, {0: -1.0, 2: -0.5})

    def lse(a, b):
        return max(a, b) + math.log1p(math.exp(-abs(a - b)))

    ax = lse(-0.75, lse(-0.25, -0.75))
    res = run(orc, lg, fusion_interval=2, fusion_top_f=1, fusion_seed=seed)
    # Z (-1.75) now ranks before X (ax + 1.2 B0 = -4.999); with the extension's
    # sub-beam X would lead at ax = 0.543
    assert labels(res) == [(1, 40), (1, 40, 2)]
    np.testing.assert_allclose(res.total, [-1.75, ax + 1.2 * B0], rtol=0, atol=1e-12)
    assert res.subs[0] == [(0.0, [0])]
    assert res.subs[1] == [(1.2 * B0, [0])]
    # after frame 2: X, which led before the fusion, is the fused one
    r2 = run(orc, lg[:3], fusion_interval=2, fusion_top_f=1, fusion_seed=seed)
    assert labels(r2) == [(1, 40), (1, 40, 2)]
    assert r2.total.tolist() == [-0.75, 0.25 + 1.2 * B0]


# ------------------------------------------------------------------ top-o and lambda

def test_lambda_cut_from_the_best_survivor():
    # three homophones of (1): log10 P(w | <s>) = -1.0, -2.5, -2.875 (unigrams,
    # bo(<s>) = 0); omega = 1: Lw' = ln10 * p = -2.3026, -5.7565, -6.6199.
    # lambda = 4 cuts at -2.3026 - 4 = -6.3026: w2 goes, w1 stays (a cut from
    # the parent's Lw = 0 would be at -4 and take w1 as well).
    lex = lexicon_from([(1,), (1,), (1,)])
    orc = oracle.Oracle(lex, unigram_lm(3, [(-1.0, 0.0), (-2.5, 0.0), (-2.875, 0.0)]))
    lg = frames({1: -0.5}, {40: -0.5})   # (1 40): acoustic -0.5 + 0.5 - 0.5 + 0.25 = -0.25
    Ls = [LN10 * -1.0, LN10 * -2.5, LN10 * -2.875]

    def subs(**kw):
        kw.setdefault("subbeams", 3)
        r = run(orc, lg, omega=1.0, **kw)
        assert labels(r) == [(1, 40)]
        assert abs(r.total[0] - (-0.25 + Ls[0])) <= 1e-12
        return [(round(L, 12), w) for L, w in r.subs[0]]

    exp = [(round(L, 12), [w]) for w, L in enumerate(Ls)]
    assert subs(lam=4.0) == exp[:2]
    assert subs(lam=4.5) == exp                       # cut -6.8026: all three
    assert subs(lam=4.5, subbeams=2) == exp[:2]       # top-o binds first
    assert subs(lam=0.0) == exp[:1]
    r = run(orc, lg, omega=1.0, subbeams=3, lam=4.0)
    assert abs(r.margins["lambda"] - abs(Ls[2] - (Ls[0] - 4.0))) <= 1e-12


def test_equal_candidates_order_by_parent_subbeam_then_word():
    # a0, a1 spell (1); b0, b1 spell (2).  Unigrams a: -1.0 (backoff -0.5), b: -1.5.
    # First word: log10 P(a | <s>) = -1.0 for both -> Lw = -ln10, tied; word id
    # order: sub-beams [a0, a1].
    # Second word: log10 P(b | <s> a) = bo(<s> a) (absent: 0) + bo(a) + p(b) =
    # -0.5 - 1.5 = -2.0 for all four (parent j, b) pairs: Lw = -ln10 - 2 ln10, an
    # exact four-way tie.  Order (score desc, j asc, w asc) keeps, with o = 2,
    # (j=0, b0) and (j=0, b1): readings [a0 b0], [a0 b1]; ordering by word first
    # would give [a0 b0], [a1 b0].
    lex = lexicon_from([(1,), (1,), (2,), (2,)])
    orc = oracle.Oracle(lex, unigram_lm(4, [(-1.0, -0.5), (-1.0, -0.5), (-1.5, 0.0), (-1.5, 0.0)]))
    lg = frames({1: -0.5}, {40: -0.5}, {2: -0.5}, {40: -0.5})
    r = run(orc, lg, omega=1.0, subbeams=2, lam=100.0)
    assert labels(r) == [(1, 40, 2, 40)]
    L = (0.0 + LN10 * -1.0) + LN10 * -2.0
    assert r.subs[0] == [(L, [0, 2]), (L, [0, 3])]
    assert r.margins["homophone"] == 0.0
    # after the first word alone: [a0, a1]
    r1 = run(orc, lg[:2], omega=1.0, subbeams=2, lam=100.0)
    assert r1.subs[0] == [(LN10 * -1.0, [0]), (LN10 * -1.0, [1])]


# ------------------------------------------------------------------ end of the utterance

def test_end_keeps_word_boundaries_else_every_hypothesis(four_words):
    # ONE_FRAME with finalisation: () is the only entry at a word boundary, so
    # it alone is output (total -1.0, no words); (1)..(4) stop inside a word.
    fin = run(four_words, ONE_FRAME, finalize=1, beam=5)
    assert labels(fin) == [()] and fin.total.tolist() == [-1.0] and fin.words == [[]]
    # without a blank the empty prefix dies: no entry ends at a word boundary,
    # so every entry is ranked with its completed words (none yet)
    lg = frames({1: -0.5, 2: -1.5, 3: -2.5, 4: -3.0})
    fin = run(four_words, lg, finalize=1, beam=5)
    assert labels(fin) == [(1,), (2,), (3,), (4,)]
    assert fin.total.tolist() == [0.0, -1.0, -2.0, -2.5] and fin.words == [[], [], [], []]
    # two frames, separator then phoneme: (1 40 2) and (1 40 3) are inside
    # their second word and keep their first, completed word w0
    lg2 = frames({1: -0.5}, {40: -0.5}, {2: -0.5, 3: -1.0})
    fin2 = run(four_words, lg2, finalize=1, beam=5)
    assert labels(fin2) == [(1, 40, 2), (1, 40, 3)] and fin2.words == [[0], [0]]
    # (-0.5 + 0.5) + (-0.5 + 0.25) + (-0.5 + 0.5) = -0.25 and -0.75 (omega = 0)
    assert fin2.total.tolist() == [-0.25, -0.75]
