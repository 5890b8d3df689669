"""Small hand-made lexicons and LMs for oracle pins and GPU edge cases."""

from __future__ import annotations

import json
import os

import numpy as np

from workloads import Lexicon, NGramLM
from workloads.configs import LexiconSpec, LMSpec
from workloads.gen import make_lm

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def lexicon_from(words) -> Lexicon:
    """Lexicon whose word w has phonemes ``words[w]``."""
    offs = np.zeros(len(words) + 1, np.int32)
    offs[1:] = np.cumsum([len(w) for w in words])
    ph = np.array([p for w in words for p in w], np.int32)
    return Lexicon(len(words), offs, ph)


def lm_from_entries(n_words: int, orders, bos=None) -> NGramLM:
    """orders[n-1] = list of (tuple of ids, log10p, bo) for n = 1..4 (bo ignored for n=4)."""
    V = n_words + 3
    ids, lp, bo = [], [], []
    for n in range(1, 5):
        ent = sorted(orders[n - 1], key=lambda e: tuple(e[0]))
        ids.append(np.array([list(e[0]) for e in ent], np.int32).reshape(len(ent), n))
        lp.append(np.array([e[1] for e in ent], np.float32))
        bo.append(np.array([e[2] if len(e) > 2 else 0.0 for e in ent], np.float32) if n < 4 else None)
    return NGramLM(V, n_words, n_words + 1, n_words + 2, ids=ids, logp=lp, bo=bo,
                   ctx=[None] * 4, key=[None] * 4)


def golden_ngram():
    with open(os.path.join(GOLDEN, "ngram_backoff.json")) as f:
        g = json.load(f)
    voc = g["vocab"]

    def tup(s):
        return tuple(voc[x] for x in s.split())

    orders = [
        [((voc[w],), p, b) for w, p, b in g["unigrams"]],
        [(tup(s), p, b) for s, p, b in g["bigrams"]],
        [(tup(s), p, b) for s, p, b in g["trigrams"]],
        [(tup(s), p) for s, p in g["fourgrams"]],
    ]
    lm = lm_from_entries(g["n_words"], orders)
    queries = [(tup(q["ctx"]) if q["ctx"] else (), voc[q["w"]], q["log10p"], q["why"])
               for q in g["queries"]]
    return lm, queries


def random_small_lm(n_words: int, n_total: int) -> NGramLM:
    """A seeded random 4-gram LM over n_words words (same generator as the workloads)."""
    return make_lm(LMSpec(f"tiny{n_words}", LexiconSpec(f"tiny{n_words}", n_words, 3), n_total))


def peaked_logits(targets, strong=6.0, seed=0, sigma=0.3):
    """Log-softmax frames that favour the given target classes."""
    rng = np.random.default_rng(seed)
    T = len(targets)
    raw = sigma * rng.standard_normal((T, 41))
    raw[np.arange(T), targets] += strong
    raw -= raw.max(-1, keepdims=True)
    raw -= np.log(np.exp(raw).sum(-1, keepdims=True))
    return raw.astype(np.float32)
