"""Seeded generators for lexicons, 4-gram backoff LMs and CTC log-probabilities.

Every generator draws from ``numpy.random.default_rng(SeedSequence([...]))``
with a tag that names what is generated, so the same lexicon / LM is produced
for every workload that names it (the 125k-word workloads share one lexicon,
and two of them share the 50M-n-gram LM).  Large artifacts are cached as
``.npy`` files under ``$LB_CACHE_DIR`` (default: ``<tmp>/lb_workloads``).
"""

from __future__ import annotations

import os
import tempfile
import time
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

from .configs import BASE_SEED, BLANK, SEP, N_CLASSES, N_PHONEMES, LexiconSpec, LMSpec, Workload

_TAG_LEXICON = 1
_TAG_LM = 2
_TAG_LOGITS = 3
_TAG_FUSION = 4


def _rng(*tag: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([BASE_SEED, *tag]))


def _cache_dir() -> str:
    d = os.environ.get("LB_CACHE_DIR") or os.path.join(tempfile.gettempdir(), "lb_workloads")
    os.makedirs(d, exist_ok=True)
    return d


def _log(msg: str) -> None:
    if os.environ.get("LB_GEN_VERBOSE"):
        print(f"[workloads] {msg}", flush=True)


# --------------------------------------------------------------------------- lexicon


@dataclass
class Lexicon:
    """Pronunciation dictionary in CSR form.

    Entry e spells ``phonemes[offsets[e] .. offsets[e+1]]`` (values 1..39) and
    stands for word ``entry_word[e]`` (None: word e).  Without variants there
    is one entry per word and ``n_words`` is also the number of words; word ids
    are the LM vocabulary ids of the words.
    """

    n_words: int          # entries
    offsets: np.ndarray   # int32 [n_words + 1]
    phonemes: np.ndarray  # int32 [offsets[-1]]
    entry_word: Optional[np.ndarray] = None  # int32 [n_words]

    def word(self, e: int) -> np.ndarray:
        return self.phonemes[self.offsets[e]:self.offsets[e + 1]]

    def pronunciations(self, w: int) -> List[int]:
        """Entries spelling word w (its default entry w first)."""
        if self.entry_word is None:
            return [w]
        if not hasattr(self, "_prons"):
            prons: dict = {}
            for e, x in enumerate(self.entry_word.tolist()):
                prons.setdefault(x, []).append(e)
            self._prons = prons
        return self._prons.get(w, [w])


def make_lexicon(spec: LexiconSpec) -> Lexicon:
    rng = _rng(_TAG_LEXICON, spec.n_words, spec.max_len)
    lens = rng.integers(1, spec.max_len + 1, size=spec.n_words)
    offsets = np.zeros(spec.n_words + 1, dtype=np.int32)
    np.cumsum(lens, out=offsets[1:])
    phonemes = rng.integers(1, N_PHONEMES + 1, size=int(offsets[-1])).astype(np.int32)
    if spec.variant_frac <= 0:
        return Lexicon(spec.n_words, offsets, phonemes)
    # a second pronunciation for a share of the words: one phoneme substituted,
    # inserted or deleted
    n_var = int(round(spec.variant_frac * spec.n_words))
    base = np.sort(rng.choice(spec.n_words, size=n_var, replace=False))
    extra: List[np.ndarray] = []
    for w in base.tolist():
        ph = phonemes[offsets[w]:offsets[w + 1]].tolist()
        op = int(rng.integers(0, 4))
        k = int(rng.integers(0, len(ph)))
        if op == 2:
            ph.insert(k, int(rng.integers(1, N_PHONEMES + 1)))
        elif op == 3 and len(ph) > 1:
            del ph[k]
        else:
            ph[k] = 1 + (ph[k] - 1 + int(rng.integers(1, N_PHONEMES))) % N_PHONEMES
        extra.append(np.array(ph, dtype=np.int32))
    lens2 = np.array([len(x) for x in extra], dtype=np.int64)
    offsets2 = np.concatenate([offsets, offsets[-1] + np.cumsum(lens2)]).astype(np.int32)
    phonemes2 = np.concatenate([phonemes] + extra).astype(np.int32)
    entry_word = np.concatenate([np.arange(spec.n_words), base]).astype(np.int32)
    return Lexicon(spec.n_words + n_var, offsets2, phonemes2, entry_word)


# --------------------------------------------------------------------------- n-gram LM


@dataclass
class NGramLM:
    """A 4-gram backoff LM in ARPA form, as sorted flat arrays.

    ``ids[n-1]`` is an int32 array ``[count_n, n]`` of word tuples, sorted
    lexicographically and unique; ``logp[n-1]`` the log10 probabilities and
    ``bo[n-1]`` (orders 1..3) the log10 backoff weights, both float32.
    Vocabulary: lexicon words 0..W-1, then ``<s>`` = W, ``</s>`` = W+1,
    ``<unk>`` = W+2.

    ``ctx[n-1]`` (orders 2..4) is the row index of each entry's context in the
    order n-1 arrays and ``key[n-1] = ctx * vocab + word`` (int64, sorted); the
    sentence sampler uses them.
    """

    vocab_size: int
    bos: int
    eos: int
    unk: int
    ids: List[np.ndarray]
    logp: List[np.ndarray]
    bo: List[Optional[np.ndarray]]
    ctx: List[Optional[np.ndarray]]
    key: List[Optional[np.ndarray]]

    @property
    def counts(self) -> List[int]:
        return [int(a.shape[0]) for a in self.ids]

    @property
    def n_words(self) -> int:
        return self.vocab_size - 3


def _draw_unique_keys(count: int, draw, rng: np.random.Generator) -> np.ndarray:
    """Sorted unique keys: draw with ``draw(m)``, drop duplicates, and if more
    than ``count`` distinct keys were drawn, keep a uniformly random subset."""
    kept = np.empty(0, dtype=np.int64)
    while kept.shape[0] < count:
        need = count - kept.shape[0]
        cand = np.unique(draw(int(need * 1.03) + 64))
        if kept.shape[0]:
            pos = np.searchsorted(kept, cand)
            pos[pos >= kept.shape[0]] = 0
            cand = cand[kept[pos] != cand]
        if cand.shape[0] > need:
            drop = rng.choice(cand.shape[0], cand.shape[0] - need, replace=False)
            keep = np.ones(cand.shape[0], dtype=bool)
            keep[drop] = False
            cand = cand[keep]
        kept = np.union1d(kept, cand) if kept.shape[0] else cand
    return kept


def make_lm(spec: LMSpec) -> NGramLM:
    lex = spec.lexicon
    W = lex.n_words
    V = W + 3
    bos, eos, unk = W, W + 1, W + 2
    rng = _rng(_TAG_LM, spec.n_total, W)
    rem = spec.n_total - V
    if rem < 3:
        raise ValueError("n_total must exceed the vocabulary size")
    n2 = int(round(0.40 * rem))
    n3 = int(round(0.35 * rem))
    n4 = rem - n2 - n3

    t0 = time.time()
    ids1 = np.arange(V, dtype=np.int32)[:, None]
    p1 = rng.uniform(-4.0, -0.5, V).astype(np.float32)
    p1[bos] = -99.0
    bo1 = rng.uniform(-1.0, 0.0, V).astype(np.float32)

    # Order 2: context = <s> with probability 1%, else a uniform word.
    def draw2(m):
        ctx = rng.integers(0, W, size=m, dtype=np.int64)
        ctx[rng.random(m) < 0.01] = bos
        w = rng.integers(0, W, size=m, dtype=np.int64)
        return ctx * V + w

    key2 = _draw_unique_keys(n2, draw2, rng)
    ctx2 = key2 // V
    w2 = (key2 % V).astype(np.int32)
    ids2 = np.stack([ctx2.astype(np.int32), w2], axis=1)
    p2 = rng.uniform(-4.0, -0.5, n2).astype(np.float32)
    bo2 = rng.uniform(-1.0, 0.0, n2).astype(np.float32)
    _log(f"{spec.name}: order 2 ({n2}) {time.time() - t0:.1f}s")

    # Orders 3 and 4: context = a uniformly drawn existing entry of order n-1.
    def make_order(n_prev, ids_prev, count):
        def draw(m):
            ctx = rng.integers(0, n_prev, size=m, dtype=np.int64)
            w = rng.integers(0, W, size=m, dtype=np.int64)
            return ctx * V + w
        key = _draw_unique_keys(count, draw, rng)
        ctx = key // V
        w = (key % V).astype(np.int32)
        ids = np.empty((count, ids_prev.shape[1] + 1), dtype=np.int32)
        ids[:, :-1] = ids_prev[ctx]
        ids[:, -1] = w
        return key, ctx, ids

    key3, ctx3, ids3 = make_order(n2, ids2, n3)
    p3 = rng.uniform(-4.0, -0.5, n3).astype(np.float32)
    bo3 = rng.uniform(-1.0, 0.0, n3).astype(np.float32)
    _log(f"{spec.name}: order 3 ({n3}) {time.time() - t0:.1f}s")
    key4, ctx4, ids4 = make_order(n3, ids3, n4)
    p4 = rng.uniform(-4.0, -0.5, n4).astype(np.float32)
    _log(f"{spec.name}: order 4 ({n4}) {time.time() - t0:.1f}s")

    return NGramLM(V, bos, eos, unk,
                   ids=[ids1, ids2, ids3, ids4], logp=[p1, p2, p3, p4],
                   bo=[bo1, bo2, bo3, None],
                   ctx=[None, ctx2, ctx3, ctx4], key=[None, key2, key3, key4])


def _lm_cache_paths(spec: LMSpec):
    d = os.path.join(_cache_dir(), f"{spec.name}-{spec.n_total}-{spec.lexicon.n_words}")
    return d


def load_lm(spec: LMSpec, cache: bool = True) -> NGramLM:
    """``make_lm`` with an on-disk cache for the large LMs."""
    if not cache or spec.n_total < 2_000_000:
        return make_lm(spec)
    d = _lm_cache_paths(spec)
    names = ["ids1", "ids2", "ids3", "ids4", "p1", "p2", "p3", "p4", "bo1", "bo2", "bo3",
             "ctx2", "ctx3", "ctx4", "key2", "key3", "key4"]
    done = os.path.join(d, "DONE")
    if os.path.exists(done):
        a = {n: np.load(os.path.join(d, n + ".npy"), mmap_mode=None) for n in names}
        W = spec.lexicon.n_words
        return NGramLM(W + 3, W, W + 1, W + 2,
                       ids=[a["ids1"], a["ids2"], a["ids3"], a["ids4"]],
                       logp=[a["p1"], a["p2"], a["p3"], a["p4"]],
                       bo=[a["bo1"], a["bo2"], a["bo3"], None],
                       ctx=[None, a["ctx2"], a["ctx3"], a["ctx4"]],
                       key=[None, a["key2"], a["key3"], a["key4"]])
    lm = make_lm(spec)
    os.makedirs(d, exist_ok=True)
    arrs = dict(ids1=lm.ids[0], ids2=lm.ids[1], ids3=lm.ids[2], ids4=lm.ids[3],
                p1=lm.logp[0], p2=lm.logp[1], p3=lm.logp[2], p4=lm.logp[3],
                bo1=lm.bo[0], bo2=lm.bo[1], bo3=lm.bo[2],
                ctx2=lm.ctx[1], ctx3=lm.ctx[2], ctx4=lm.ctx[3],
                key2=lm.key[1], key3=lm.key[2], key4=lm.key[3])
    try:
        for n, arr in arrs.items():
            np.save(os.path.join(d, n + ".npy"), arr)
        open(done, "w").close()
    except OSError:
        pass
    return lm


# --------------------------------------------------------------------------- sentence sampler


class _Sampler:
    """Draws word sequences from the LM: the next word is drawn proportionally
    to 10^log10p among the explicit continuations of the longest context
    (up to 3 words) that has any, falling back to the unigram distribution
    over lexicon words."""

    def __init__(self, lm: NGramLM):
        self.lm = lm
        W = lm.n_words
        p = lm.logp[0][:W].astype(np.float64)
        w = np.power(10.0, p - p.max())
        self.uni_cdf = np.cumsum(w) / w.sum()

    def _range(self, n: int, ctx_row: int):
        c = self.lm.ctx[n - 1]
        lo = int(np.searchsorted(c, ctx_row, "left"))
        hi = int(np.searchsorted(c, ctx_row, "right"))
        return lo, hi

    def _row(self, n: int, ctx_row: int, word: int) -> int:
        """Row of the order-n entry (context row, word), or -1."""
        k = self.lm.key[n - 1]
        q = ctx_row * self.lm.vocab_size + word
        i = int(np.searchsorted(k, q))
        return i if i < k.shape[0] and int(k[i]) == q else -1

    def continuation(self, hist: List[int]):
        """(order n, lo, hi) of the longest context of ``hist`` with continuations."""
        # rows[m-1] = row of the last m history words as an order-m entry (-1 if absent)
        rows = [int(hist[-1])]
        if len(hist) >= 2:
            rows.append(self._row(2, int(hist[-2]), int(hist[-1])))
        if len(hist) >= 3:
            r_prev = self._row(2, int(hist[-3]), int(hist[-2]))
            rows.append(self._row(3, r_prev, int(hist[-1])) if r_prev >= 0 else -1)
        for m in range(len(rows), 0, -1):
            if rows[m - 1] < 0:
                continue
            lo, hi = self._range(m + 1, rows[m - 1])
            if hi > lo:
                return (m + 1, lo, hi)
        return None

    def next_word(self, hist: List[int], rng: np.random.Generator) -> int:
        c = self.continuation(hist)
        if c is None:
            return int(np.searchsorted(self.uni_cdf, rng.random(), "right"))
        n, lo, hi = c
        p = self.lm.logp[n - 1][lo:hi].astype(np.float64)
        w = np.power(10.0, p - p.max())
        cdf = np.cumsum(w) / w.sum()
        j = int(np.searchsorted(cdf, rng.random(), "right"))
        return int(self.lm.ids[n - 1][lo + min(j, hi - lo - 1), -1])

    def sentence(self, n_words: int, rng: np.random.Generator) -> List[int]:
        hist = [self.lm.bos]
        for _ in range(n_words):
            hist.append(self.next_word(hist, rng))
        return hist[1:]


# --------------------------------------------------------------------------- logits


def make_targets(lex: Lexicon, sampler: _Sampler, frames: int, rng: np.random.Generator,
                 fill: bool) -> tuple:
    """Frame-level CTC targets for one utterance.

    Words (3..15 per sentence, drawn from the LM) expand to their phonemes and
    a SEP.  Each symbol is preceded by a blank run of Geom0(0.4) frames (at
    least 1 between identical consecutive symbols) and lasts 1 + Geom0(0.4)
    frames.  Words are appended while they fit; the rest is blank.  With
    ``fill`` (streams) sentences are appended until a word no longer fits.
    Returns (targets int32 [frames], words list).
    """
    tgt = np.zeros(frames, dtype=np.int32)
    pos = 0
    prev = -1
    words_out: List[int] = []
    while True:
        n = int(rng.integers(3, 16))
        words = sampler.sentence(n, rng)
        stop = False
        for w in words:
            prons = lex.pronunciations(w)
            e = prons[int(rng.integers(0, len(prons)))] if len(prons) > 1 else prons[0]
            syms = list(lex.word(e)) + [SEP]
            seg: List[int] = []
            p = prev
            for s in syms:
                nb = int(rng.geometric(0.4)) - 1
                if s == p:
                    nb = max(nb, 1)
                dur = int(rng.geometric(0.4))      # 1 + Geom0(0.4)
                seg.extend([BLANK] * nb)
                seg.extend([int(s)] * dur)
                p = s
            if pos + len(seg) > frames:
                stop = True
                break
            tgt[pos:pos + len(seg)] = seg
            pos += len(seg)
            prev = p
            words_out.append(w)
        if stop or not fill:
            break
    return tgt, words_out


def make_logits(targets: np.ndarray, sigma: float, rng: np.random.Generator) -> np.ndarray:
    """raw = 4*onehot(target) + sigma*N(0,1); log-softmax in float64, stored float32."""
    B, T = targets.shape
    raw = sigma * rng.standard_normal((B, T, N_CLASSES))
    np.put_along_axis(raw, targets[..., None].astype(np.int64),
                      np.take_along_axis(raw, targets[..., None].astype(np.int64), -1) + 4.0, -1)
    m = raw.max(-1, keepdims=True)
    lse = m + np.log(np.exp(raw - m).sum(-1, keepdims=True))
    return (raw - lse).astype(np.float32)


@dataclass
class WorkloadData:
    workload: Workload
    lexicon: Lexicon
    lm: NGramLM
    logits: np.ndarray        # float32 [B, T, 41], log-softmax
    lengths: np.ndarray       # int32 [B]
    targets: np.ndarray       # int32 [B, T]
    words: List[List[int]]    # reference word sequences (not used by the decoder)
    fusion_seed: int          # seed of the synthetic fusion scorer


def load_workload(name_or_wl, batch: Optional[int] = None, cache: bool = True) -> WorkloadData:
    """Build (or load from cache) every input of a workload.

    ``batch`` optionally keeps only the first ``batch`` utterances (the draws of
    utterance b do not depend on the batch size)."""
    from .configs import get_config
    wl = get_config(name_or_wl) if isinstance(name_or_wl, str) else name_or_wl
    t0 = time.time()
    lex = make_lexicon(wl.lexicon)
    lm = load_lm(wl.lm, cache=cache)
    _log(f"{wl.name}: lexicon+lm {time.time() - t0:.1f}s")
    sampler = _Sampler(lm)
    B = wl.batch if batch is None else min(batch, wl.batch)
    T = wl.frames
    targets = np.zeros((B, T), dtype=np.int32)
    words = []
    lengths = np.full(B, T, dtype=np.int32)
    fill = wl.chunk > 0
    for b in range(B):
        r = _rng(_TAG_LOGITS, hash_name(wl.name), b)
        tgt, ws = make_targets(lex, sampler, T, r, fill)
        targets[b] = tgt
        words.append(ws)
        if wl.ragged:
            lengths[b] = int(r.integers(T // 2, T + 1))
    logits = np.empty((B, T, N_CLASSES), dtype=np.float32)
    for b in range(B):
        r = _rng(_TAG_LOGITS, hash_name(wl.name), b, 1)
        logits[b] = make_logits(targets[b:b + 1], wl.sigma, r)[0]
    fseed = int(_rng(_TAG_FUSION, hash_name(wl.name)).integers(0, 2**63 - 1, dtype=np.int64))
    _log(f"{wl.name}: total {time.time() - t0:.1f}s")
    return WorkloadData(wl, lex, lm, logits, lengths, targets, words, fseed)


def hash_name(name: str) -> int:
    """Stable small integer of a workload name (for seed sequences)."""
    h = 0
    for ch in name.encode():
        h = (h * 131 + ch) % (2**31 - 1)
    return h
