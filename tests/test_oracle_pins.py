"""Pins of the CPU oracle against facts fixed outside it (no GPU).

* brute force: every CTC alignment of tiny inputs enumerated (the search
  target by definition), with and without the n-gram, with fusion;
* the CTC forward algorithm of ``torch.nn.functional.ctc_loss`` (fp64);
* probability conservation on a complete lexicon;
* hand-computed 4-gram backoff values (tests/golden/ngram_backoff.json);
* the published first outputs of SplitMix64 seeded with 0;
* greedy vs tracked homophones (the example motivating Sec. 3.4.1);
* fusion identity: fusing with the n-gram LM's own score changes nothing.
"""

import ctypes
import math

import numpy as np
import pytest
import torch

import oracle
from tests import brute_force as bf
from tests.tinylm import golden_ngram, lexicon_from, lm_from_entries, peaked_logits, random_small_lm
from workloads import DecodeParams, load_workload

LN10 = math.log(10.0)
BIG = dict(beam=10**7, subbeams=1000, theta=1e30, lam=1e30)

# Phonemes {1,2,3}; homophones (1,2) x2 and (1,) x2; a doubled phoneme (2,2).
TINY_WORDS = [(1,), (2, 2), (1, 2), (1, 2), (3, 1), (2,), (1,)]
TINY_CLASSES = (0, 1, 2, 3, 40)


@pytest.fixture(scope="module")
def tiny():
    lex = lexicon_from(TINY_WORDS)
    lm = random_small_lm(len(TINY_WORDS), 60)
    return lex, lm, oracle.Oracle(lex, lm)


def tiny_logits(T, seed):
    rng = np.random.default_rng(seed)
    raw = rng.standard_normal((T, 41))
    raw[:, list(TINY_CLASSES)] += 2.5
    raw -= raw.max(-1, keepdims=True)
    raw -= np.log(np.exp(raw).sum(-1, keepdims=True))
    return raw.astype(np.float32)


def ngram_reading_score(orc, lm, omega):
    c = omega * LN10

    def score(words):
        s, hist = 0.0, [lm.bos]
        for w in words:
            s = s + c * orc.log10p(hist[-3:], w)
            hist.append(w)
        return s
    return score


def check_against_brute(res, expect, tol=1e-9):
    got = {tuple(int(s) for s in lab): (t, [int(w) for w in ws])
           for lab, t, ws in zip(res.labels, res.total, res.words)}
    assert set(got) == set(expect), (sorted(got), sorted(expect))
    for y, (tot, reading, _) in expect.items():
        assert abs(got[y][0] - tot) <= tol * max(1.0, abs(tot)), (y, got[y][0], tot)
        assert got[y][1] == reading, (y, got[y][1], reading)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("omega", [0.0, 0.5])
def test_brute_force_no_pruning(tiny, seed, omega):
    lex, lm, orc = tiny
    T = 7
    lg = tiny_logits(T, seed)
    p = DecodeParams(omega=omega, fusion_interval=0)
    params = oracle.params_from(p, **BIG)
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                    ngram_reading_score(orc, lm, omega))
    assert len(expect) > 5
    check_against_brute(res, expect)


@pytest.mark.parametrize("seed", range(20))
def test_brute_force_random_lexicons(seed):
    """Random small lexicons over phonemes {1, 2, 3} (one to three phonemes a
    word, so words that are prefixes of others and doubled phonemes occur;
    distinct spellings plus one homophone pair), random bonuses and LM weight:
    without pruning, the oracle's complete hypotheses, totals and readings
    equal the exhaustive enumeration's."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(4, 8))  # (the tiny LM needs five words or more for its 60 n-grams)
    words = []
    while len(words) < n:
        w = tuple(int(x) for x in rng.integers(1, 4, size=int(rng.integers(1, 4))))
        if w not in words:
            words.append(w)
    words.append(words[int(rng.integers(0, n))])
    lex = lexicon_from(words)
    lm = random_small_lm(len(words), 60)
    orc = oracle.Oracle(lex, lm)
    try:
        lg = tiny_logits(6, 50 + seed)
        omega = float(rng.choice([0.0, 0.5, 1.0]))
        p = DecodeParams(omega=omega, beta=float(rng.uniform(0.0, 2.0)), gamma=float(rng.uniform(0.0, 2.0)),
                         fusion_interval=0)
        res = orc.decode(lg, oracle.params_from(p, **BIG))
        D = p.alpha * lg.astype(np.float64)
        expect = bf.complete_hypotheses(D, TINY_CLASSES, words, p.beta, p.gamma,
                                        ngram_reading_score(orc, lm, omega))
        assert len(expect) > 1
        check_against_brute(res, expect)
    finally:
        orc.close()


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("omega", [0.0, 0.5])
def test_brute_force_max_recombination(tiny, seed, omega):
    """merge = max (App. E.1): every complete hypothesis scores its single best
    alignment (Viterbi) plus bonuses plus its best reading."""
    lex, lm, orc = tiny
    T = 7
    lg = tiny_logits(T, seed)
    p = DecodeParams(omega=omega, fusion_interval=0)
    params = oracle.params_from(p, merge_max=1, **BIG)
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                    ngram_reading_score(orc, lm, omega), reduce="max")
    assert len(expect) > 5
    check_against_brute(res, expect)
    # the max never exceeds the sum over alignments
    lse = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                 ngram_reading_score(orc, lm, omega))
    assert all(expect[y][0] <= lse[y][0] + 1e-12 for y in expect)
    assert any(expect[y][0] < lse[y][0] - 1e-3 for y in expect)


@pytest.mark.parametrize("seed", [0, 6])
def test_raw_logits_brute_force(tiny, seed):
    """Raw scores in: each frame is log-softmax-normalised (scipy's log_softmax
    on the same fp32 inputs, in fp64) before the search; a per-frame constant
    shift of the inputs changes nothing."""
    from scipy.special import log_softmax
    lex, lm, orc = tiny
    T = 7
    rng = np.random.default_rng(100 + seed)
    raw = rng.standard_normal((T, 41)) * 2.0
    raw[:, list(TINY_CLASSES)] += 3.0
    raw = raw.astype(np.float32)
    p = DecodeParams(omega=0.5, fusion_interval=0)
    params = oracle.params_from(p, raw_logits=1, **BIG)
    res = orc.decode(raw, params)
    D = p.alpha * log_softmax(raw.astype(np.float64), axis=-1)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                    ngram_reading_score(orc, lm, 0.5))
    check_against_brute(res, expect)
    shifted = (raw + np.arange(T, dtype=np.float32)[:, None] * 8.0).astype(np.float32)
    res2 = orc.decode(shifted, params)
    assert [list(w) for w in res2.words] == [list(w) for w in res.words]
    assert np.allclose(res2.total, res.total, atol=1e-5)


@pytest.mark.parametrize("seed", [3, 4])
def test_brute_force_with_fusion(tiny, seed):
    """Final fusion over all entries: total = acoustic + bonuses + max_reading phi*S_fus."""
    lex, lm, orc = tiny
    T = 7
    lg = tiny_logits(T, seed)
    p = DecodeParams(fusion_interval=2, fusion_top_f=0)
    params = oracle.params_from(p, fusion_seed=12345, **BIG)
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                    lambda ws: p.phi * orc.fusion_score(params, ws))
    check_against_brute(res, expect)
    assert res.stats["fused"] > 0


def test_brute_force_with_caller_scorer(tiny):
    """Fusion scores from a scorer the caller passes in (an arbitrary function of
    the word sequence): the final fusion follows it exactly."""
    lex, lm, orc = tiny
    calls = []

    def scorer(ws):
        calls.append(tuple(ws))
        h = 0
        for w in ws:
            h = (h * 1000003 + w + 1) % 2147483647
        return -0.5 - (h % 977) / 100.0

    T = 7
    lg = tiny_logits(T, 9)
    p = DecodeParams(fusion_interval=3, fusion_top_f=0)
    params = oracle.params_from(p, scorer=scorer, **BIG)
    assert params.fusion_mode == 2
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma, lambda ws: p.phi * scorer(ws))
    check_against_brute(res, expect)
    assert res.stats["fused"] > 0 and calls
    # without a scorer, mode 2 is refused
    with pytest.raises(RuntimeError):
        orc.decode(lg, oracle.params_from(p, fusion_mode=2, **BIG))


def test_brute_force_end_of_sentence_marks(tiny):
    """The final fusion with end-of-sentence marks: every reading's fusion
    score takes its best mark (the first of equals), and the mark follows the
    words of the output."""
    lex, lm, orc = tiny
    T = 7
    lg = tiny_logits(T, 8)
    marks = [lm.eos, lm.unk, 2]
    p = DecodeParams(fusion_interval=3, fusion_top_f=0)
    params = oracle.params_from(p, fusion_seed=99, eos_count=3, eos_ids=(ctypes.c_int32 * 3)(*marks), **BIG)
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)

    def best_mark(ws):
        last = ws[-1] if ws else lm.bos
        vals = [orc.fusion_score(params, [last, m]) - orc.fusion_score(params, [last]) for m in marks]
        k = int(np.argmax(vals))  # first of equals
        return vals[k], marks[k]

    expect = bf.complete_hypotheses(D, TINY_CLASSES, TINY_WORDS, p.beta, p.gamma,
                                    lambda ws: p.phi * (orc.fusion_score(params, ws) + best_mark(ws)[0]))
    expect = {y: (t, r + [best_mark(r)[1]], a) for y, (t, r, a) in expect.items()}
    check_against_brute(res, expect)


@pytest.mark.parametrize("omega,fusion", [(0.5, 0), (0.0, 2)])
def test_brute_force_pronunciation_variants(omega, fusion):
    """Several entries per word (App. I): a word is reachable through each of
    its spellings, and a spelling's homophones are distinct word ids."""
    words = [(1,), (2, 2), (1, 2), (3, 1), (2,)]
    entries = words + [(3,), (1, 2), (2, 1)]      # variants of words 0, 2 (same spelling again) and 4
    entry_word = list(range(len(words))) + [0, 2, 4]
    lex = lexicon_from(entries)
    lex.entry_word = np.array(entry_word, dtype=np.int32)
    lm = random_small_lm(len(words), 40)
    orc = oracle.Oracle(lex, lm)
    T = 7
    lg = tiny_logits(T, 11)
    p = DecodeParams(omega=omega, fusion_interval=fusion, fusion_top_f=0)
    params = oracle.params_from(p, fusion_seed=7, **BIG)
    res = orc.decode(lg, params)
    D = p.alpha * lg.astype(np.float64)
    if fusion:
        score = lambda ws: p.phi * orc.fusion_score(params, ws)
    else:
        score = ngram_reading_score(orc, lm, omega)
    expect = bf.complete_hypotheses(D, TINY_CLASSES, entries, p.beta, p.gamma, score, entry_word=entry_word)
    # word 0 is reachable through its variant spelling (3,), which spells nothing else
    via_variant = False
    for y, (_, r, _) in expect.items():
        ws, _ = bf.segments(y)
        via_variant |= any(w == (3,) and r[i] == 0 for i, w in enumerate(ws))
    assert via_variant
    check_against_brute(res, expect)
    orc.close()


def ctc_forward(lg, alpha, labels):
    """log sum over CTC alignments of alpha*logits, via torch's CTC loss (fp64 CPU)."""
    lp = torch.from_numpy(alpha * lg.astype(np.float64))[:, None, :]
    tgt = torch.tensor([labels], dtype=torch.long) if labels else torch.zeros((1, 0), dtype=torch.long)
    loss = torch.nn.functional.ctc_loss(lp, tgt, torch.tensor([lg.shape[0]]),
                                        torch.tensor([len(labels)]), blank=0, reduction="none",
                                        zero_infinity=False)
    return -float(loss[0])


def bonus(labels, p):
    return sum(p.gamma if s == 40 else p.beta for s in labels)


@pytest.mark.parametrize("seed", [0, 5])
def test_ctc_forward_exact_without_pruning(tiny, seed):
    lex, lm, orc = tiny
    lg = tiny_logits(7, seed)
    p = DecodeParams(fusion_interval=0)
    res = orc.decode(lg, oracle.params_from(p, **BIG))
    assert len(res.labels) > 5
    for lab, ac in zip(res.labels, res.acoustic):
        ref = ctc_forward(lg, p.alpha, [int(s) for s in lab])
        assert abs((ac - bonus(lab, p)) - ref) < 1e-9, (lab, ac, ref)


def test_ctc_forward_upper_bound_under_pruning():
    """With pruning an output keeps a subset of its alignments: acoustic <= CTC forward."""
    d = load_workload("c1")
    p = d.workload.params
    orc = oracle.Oracle(d.lexicon, d.lm)
    for K in (2, 8, 32):
        res = orc.decode(d.logits[0], oracle.params_from(p, beam=K))
        assert len(res.labels) >= 1
        for lab, ac in zip(res.labels, res.acoustic):
            ref = ctc_forward(d.logits[0], p.alpha, [int(s) for s in lab])
            assert ac - bonus(lab, p) <= ref + 1e-9


def test_probability_conservation():
    """alpha=1, no bonuses, no LM, no pruning and every phoneme string a word:
    the beam's acoustic mass stays exactly 1 (log 0) after every frame."""
    T = 8
    words = [w for n in range(1, T + 1) for w in __import__("itertools").product((1, 2), repeat=n)]
    lex = lexicon_from(words)
    lm = random_small_lm(len(words), len(words) + 3 + 30)
    orc = oracle.Oracle(lex, lm)
    rng = np.random.default_rng(7)
    raw = np.full((T, 41), -np.inf)
    raw[:, [0, 1, 2]] = rng.standard_normal((T, 3))
    raw -= np.log(np.exp(raw).sum(-1, keepdims=True))
    p = DecodeParams(alpha=1.0, beta=0.0, gamma=0.0, omega=0.0, fusion_interval=0)
    res = orc.decode(raw.astype(np.float32), oracle.params_from(p, **BIG), frame_lse=True)
    lg32 = raw.astype(np.float32).astype(np.float64)
    # the float32 rounding of the inputs moves the mass by at most a few ulp per frame
    norm = np.cumsum(np.log(np.exp(lg32[:, :3]).sum(-1)))
    np.testing.assert_allclose(res.frame_lse, norm, atol=1e-12)


def test_ngram_backoff_hand_values():
    lm, queries = golden_ngram()
    lex = lexicon_from([(1,), (2,), (3,), (4,)])
    orc = oracle.Oracle(lex, lm)
    for ctx, w, expect, why in queries:
        got = orc.log10p(list(ctx), w)
        assert abs(got - expect) < 1e-6, (ctx, w, got, expect, why)


def test_splitmix64_published_outputs():
    # SplitMix64 seeded with 0: the first three outputs are well known test vectors.
    gold = 0x9E3779B97F4A7C15
    assert oracle.splitmix64(0) == 0xE220A8397B1DCDAF
    assert oracle.splitmix64(gold) == 0x6E789E6AA1B965F4
    assert oracle.splitmix64((2 * gold) & (2**64 - 1)) == 0x06C45D188009454F


def test_fusion_bigram_value_from_published_vector():
    """seed XOR (a<<32|b) == 0 makes the hash the published splitmix64(0) output,
    whose top 16 bits are 0xE220 = 57888: Bg = lo + (hi-lo)*57888/65536."""
    lm, _ = golden_ngram()
    orc = oracle.Oracle(lexicon_from([(1,), (2,), (3,), (4,)]), lm)
    b = 2
    seed = (lm.bos << 32) | b
    p = oracle.params_from(DecodeParams(), fusion_seed=seed)
    assert orc.fusion_score(p, [b]) == -10.0 + 9.5 * 57888 / 65536
    assert orc.fusion_score(p, []) == 0.0


def homophone_case():
    # w0 and w1 are homophones (phoneme 1); w2 is phoneme 2.
    lex = lexicon_from([(1,), (1,), (2,)])
    W = 3
    bos = W
    lm = lm_from_entries(W, [
        [((0,), -1.0, -1.0), ((1,), -0.5, 0.0), ((2,), -2.0, 0.0), ((bos,), -99.0, -0.6),
         ((W + 1,), -1.0, 0.0), ((W + 2,), -3.0, 0.0)],
        [((bos, 0), -0.1, 0.0), ((1, 2), -0.05, 0.0)],
        [],
        [],
    ])
    lg = peaked_logits([1, 0, 40, 0, 2, 0, 40], strong=8.0)
    return lex, lm, lg


def test_greedy_vs_tracked_homophones():
    """'They're happy' (Sec. 3.4.1): the likelier homophone w0 loses once the next
    word is seen.  By hand: P(w0|<s>) = -0.1, P(w1|<s>) = -0.6 + -0.5 = -1.1,
    P(w2|w0) = -1.0 + -2.0 = -3.0, P(w2|w1) = -0.05."""
    lex, lm, lg = homophone_case()
    orc = oracle.Oracle(lex, lm)
    p = DecodeParams(fusion_interval=0)
    c = p.omega * LN10
    greedy = orc.decode(lg, oracle.params_from(p, beam=64, subbeams=1, lam=0.0))
    tracked = orc.decode(lg, oracle.params_from(p, beam=64, subbeams=2))
    ac_ref = ctc_forward(lg, p.alpha, [1, 40, 2, 40]) + 2 * p.beta + 2 * p.gamma
    i = greedy.labels.index([1, 40, 2, 40])
    assert greedy.words[i] == [0, 2]
    assert abs(greedy.total[i] - (ac_ref + c * (-0.1 + -3.0))) < 1e-6
    j = tracked.labels.index([1, 40, 2, 40])
    assert tracked.words[j] == [1, 2]
    assert abs(tracked.total[j] - (ac_ref + c * (-1.1 + -0.05))) < 1e-6


def test_fusion_identity():
    """phi = omega and the n-gram's own ln-scaled sentence score as the fusion score:
    every fusion event is a no-op, so results equal the run without fusion."""
    d = load_workload("t-c1k")
    orc = oracle.Oracle(d.lexicon, d.lm)
    p = d.workload.params
    n_out = 0
    for b in range(4):
        lg = d.logits[b, :d.lengths[b]]
        base = orc.decode(lg, oracle.params_from(p, beam=32, fusion_interval=0))
        fused = orc.decode(lg, oracle.params_from(p, beam=32, fusion_interval=5, fusion_top_f=0,
                                                  phi=p.omega, fusion_mode=1))
        assert fused.stats["fused"] > 0
        assert base.labels == fused.labels and base.words == fused.words
        np.testing.assert_allclose(base.total, fused.total, atol=1e-9)
        n_out += len(base.total)
        # the same through the caller-scorer path, the n-gram score computed here
        own = ngram_reading_score(orc, d.lm, 1.0)
        via = orc.decode(lg, oracle.params_from(p, beam=32, fusion_interval=5, fusion_top_f=0,
                                                phi=p.omega, scorer=own))
        assert via.words == base.words
        np.testing.assert_allclose(via.total, base.total, atol=1e-9)
        other = orc.decode(lg, oracle.params_from(p, beam=32, fusion_interval=5, fusion_top_f=0,
                                                  fusion_seed=d.fusion_seed))
        if len(base.total) and len(other.total):
            assert not np.allclose(other.total[:1], base.total[:1])
    assert n_out > 10


def test_collapse_invariants():
    """Outputs: unique prefixes, lexicon-valid, key = chained splitmix64 of the
    labels, and the best reading spells the labels."""
    d = load_workload("t-c1k")
    orc = oracle.Oracle(d.lexicon, d.lm)
    p = d.workload.params
    homs = {}
    for w in range(d.lexicon.n_words):
        homs.setdefault(tuple(int(x) for x in d.lexicon.word(w)), set()).add(w)
    for b in range(3):
        res = orc.decode(d.logits[b, :d.lengths[b]], oracle.params_from(p, fusion_seed=d.fusion_seed))
        labs = [tuple(l) for l in res.labels]
        assert len(set(labs)) == len(labs)
        assert list(res.total) == sorted(res.total, reverse=True)
        # the outputs all end at a word boundary, or (when no hypothesis did) none does
        complete = [bf.segments(lab)[1] == () for lab in labs]
        assert all(complete) or not any(complete)
        for lab, key, ws in zip(labs, res.keys, res.words):
            assert oracle.prefix_key(lab) == int(key)
            words, partial = bf.segments(lab)
            assert len(words) == len(ws)
            for ph, w in zip(words, ws):
                assert w in homs[ph]
