"""LightBeam CPU oracle -- TEST INFRASTRUCTURE ONLY.

Python wrapper (ctypes) around ``oracle.cpp``, a plain single-threaded fp64
implementation of the decoding method of LightBeam (arXiv 2603.14002, Alg. 1,
Eq. (1), Eq. (2), App. E).  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the HIP decoder never
does.  ``build()`` compiles ``liboracle.so`` with g++.

Every function of the oracle is pinned by tests that do not re-type it:
brute-force enumeration of CTC alignments, the CTC forward algorithm of
``torch.nn.functional.ctc_loss``, probability conservation, hand-computed
backoff values, a published SplitMix64 output and special cases (fusion
identity, greedy homophones).
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

# minimum decision margins over the decode (the K-th vs (K+1)-th candidate at
# top-K, the distance to the theta cut, the o-th vs (o+1)-th homophone
# candidate, the distance to the lambda cut, the F-th vs (F+1)-th fused
# hypothesis, adjacent output ranks), and the last frame's top-K margin
MARGIN_NAMES = ("topk", "theta", "homophone", "lambda", "fusion", "ranking", "last_topk")


def build(force: bool = True) -> str:
    """Compile liboracle.so (g++, -O2, no FP contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
                               "-fno-fast-math", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


# fusion_mode 2: the caller's scorer, S(words[0..n)) in natural log
SCORER_FN = ctypes.CFUNCTYPE(ctypes.c_double, ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_void_p)


class _Params(ctypes.Structure):
    _fields_ = [("beam", ctypes.c_int32), ("subbeams", ctypes.c_int32),
                ("alpha", ctypes.c_double), ("beta", ctypes.c_double), ("gamma", ctypes.c_double),
                ("omega", ctypes.c_double), ("phi", ctypes.c_double), ("theta", ctypes.c_double),
                ("lam", ctypes.c_double),
                ("fusion_interval", ctypes.c_int32), ("fusion_top_f", ctypes.c_int32),
                ("fusion_mode", ctypes.c_int32), ("finalize", ctypes.c_int32),
                ("merge_max", ctypes.c_int32), ("raw_logits", ctypes.c_int32),
                ("eos_count", ctypes.c_int32), ("eos_ids", ctypes.c_int32 * 3),
                ("fusion_seed", ctypes.c_uint64),
                ("fusion_lo", ctypes.c_double), ("fusion_hi", ctypes.c_double),
                ("scorer", SCORER_FN), ("scorer_ctx", ctypes.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        lib.orc_create.restype = P
        lib.orc_create.argtypes = [ctypes.c_int32, P, P, P, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_int32, P] + [P] * 11
        lib.orc_destroy.argtypes = [P]
        lib.orc_last_error.restype = ctypes.c_char_p
        lib.orc_decode.restype = ctypes.c_int32
        lib.orc_decode.argtypes = [P, ctypes.POINTER(_Params), P, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_int32, ctypes.c_int32] + [P] * 10 + [ctypes.c_int32] + [P] * 4
        lib.orc_log10p.restype = ctypes.c_double
        lib.orc_log10p.argtypes = [P, P, ctypes.c_int32, ctypes.c_int32]
        lib.orc_fusion_score.restype = ctypes.c_double
        lib.orc_fusion_score.argtypes = [P, ctypes.POINTER(_Params), P, ctypes.c_int32]
        lib.orc_splitmix64.restype = ctypes.c_uint64
        lib.orc_splitmix64.argtypes = [ctypes.c_uint64]
        lib.orc_prefix_key.restype = ctypes.c_uint64
        lib.orc_prefix_key.argtypes = [P, ctypes.c_int32]
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


@dataclass
class OracleResult:
    words: List[List[int]]      # best sub-beam word ids, per ranked hypothesis
    total: np.ndarray           # float64 [n]
    acoustic: np.ndarray        # float64 [n]
    labels: List[List[int]]     # collapsed symbol sequences
    keys: np.ndarray            # uint64 [n]
    margins: dict               # min decision margins
    frame_lse: Optional[np.ndarray]
    stats: dict
    subs: Optional[List[List[tuple]]] = None  # per hypothesis: [(Lw, words), ...] best first

    @property
    def min_margin(self) -> float:
        """Smallest margin of any decision taken during the decode."""
        return float(min(v for k, v in self.margins.items() if k != "last_topk"))


def params_from(p, fusion_seed: int = 0, fusion_mode: int = 0, scorer=None, **overrides) -> _Params:
    """orc params from a ``workloads.DecodeParams`` (plus overrides).

    ``scorer``: a Python function of a word-id list returning its fusion score
    (natural log); it selects fusion_mode 2."""
    cb = None
    if scorer is not None:
        fusion_mode = 2
        cb = SCORER_FN(lambda w, n, _ctx: float(scorer([int(w[i]) for i in range(n)])))
    d = dict(beam=p.beam, subbeams=p.subbeams, alpha=p.alpha, beta=p.beta, gamma=p.gamma,
             omega=p.omega, phi=p.phi, theta=p.theta, lam=p.lam,
             fusion_interval=p.fusion_interval, fusion_top_f=p.fusion_top_f,
             fusion_mode=fusion_mode, finalize=1, merge_max=0, raw_logits=0, fusion_seed=fusion_seed,
             fusion_lo=p.fusion_lo, fusion_hi=p.fusion_hi)
    d.update(overrides)
    q = _Params(**d)
    if cb is not None:
        q.scorer = cb
        q._cb = cb  # the callback lives as long as the params
    return q


class Oracle:
    """Holds a lexicon + LM copy inside the C++ oracle.  Thread-safe decode."""

    def __init__(self, lexicon, lm):
        lib = _load()
        self._keep = []
        offs = np.ascontiguousarray(lexicon.offsets, dtype=np.int32)
        phs = np.ascontiguousarray(lexicon.phonemes, dtype=np.int32)
        counts = np.array(lm.counts, dtype=np.int64)
        ids = [np.ascontiguousarray(a, dtype=np.int32) for a in lm.ids]
        lp = [np.ascontiguousarray(a, dtype=np.float32) for a in lm.logp]
        bo = [np.ascontiguousarray(a, dtype=np.float32) for a in lm.bo[:3]]
        ew = getattr(lexicon, "entry_word", None)
        ew = None if ew is None else np.ascontiguousarray(ew, dtype=np.int32)
        self._ew = ew
        self._h = lib.orc_create(int(lexicon.n_words), _ptr(offs), _ptr(phs), _ptr(ew) if ew is not None else None,
                                 int(lm.vocab_size),
                                 int(lm.bos), int(lm.unk), _ptr(counts),
                                 _ptr(ids[0]), _ptr(lp[0]), _ptr(bo[0]),
                                 _ptr(ids[1]), _ptr(lp[1]), _ptr(bo[1]),
                                 _ptr(ids[2]), _ptr(lp[2]), _ptr(bo[2]),
                                 _ptr(ids[3]), _ptr(lp[3]))
        if not self._h:
            raise RuntimeError("oracle create failed: " + lib.orc_last_error().decode())
        self.lib = lib

    def close(self):
        if getattr(self, "_h", None):
            self.lib.orc_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def decode(self, logits: np.ndarray, params: _Params, max_hyps: int = 4096,
               max_words: int = 512, max_labels: int = 2048,
               frame_lse: bool = False, max_subs: int = 0) -> OracleResult:
        """Decodes one utterance.  With max_subs > 0 the result also lists up to
        max_subs sub-beams (word-level score, words) of every hypothesis."""
        lg = np.ascontiguousarray(logits, dtype=np.float32)
        T = int(lg.shape[0])
        assert lg.ndim == 2 and lg.shape[1] == 41
        words = np.empty((max_hyps, max_words), np.int32)
        nwords = np.empty(max_hyps, np.int32)
        tot = np.empty(max_hyps, np.float64)
        ac = np.empty(max_hyps, np.float64)
        labels = np.empty((max_hyps, max_labels), np.int32)
        nlabels = np.empty(max_hyps, np.int32)
        keys = np.empty(max_hyps, np.uint64)
        margins = np.empty(7, np.float64)
        flse = np.empty(max(T, 1), np.float64) if frame_lse else None
        stats = np.empty(4, np.int64)
        S = max(0, int(max_subs))
        nsub = np.zeros(max_hyps, np.int32) if S else None
        subL = np.empty((max_hyps, S), np.float64) if S else None
        subnw = np.empty((max_hyps, S), np.int32) if S else None
        subw = np.empty((max_hyps, S, max_words), np.int32) if S else None
        n = self.lib.orc_decode(self._h, ctypes.byref(params), _ptr(lg), T, max_hyps, max_words,
                                max_labels, _ptr(words), _ptr(nwords), _ptr(tot), _ptr(ac),
                                _ptr(labels), _ptr(nlabels), _ptr(keys), _ptr(margins),
                                _ptr(flse), _ptr(stats), S, _ptr(nsub), _ptr(subL), _ptr(subnw), _ptr(subw))
        if n < 0:
            raise RuntimeError("oracle decode failed: " + self.lib.orc_last_error().decode())
        m = min(n, max_hyps)
        return OracleResult(
            words=[list(words[i, :min(nwords[i], max_words)]) for i in range(m)],
            total=tot[:m].copy(), acoustic=ac[:m].copy(),
            labels=[list(labels[i, :min(nlabels[i], max_labels)]) for i in range(m)],
            keys=keys[:m].copy(),
            margins=dict(zip(MARGIN_NAMES, margins.tolist())),
            frame_lse=None if flse is None else flse[:T].copy(),
            stats=dict(expansions=int(stats[0]), word_events=int(stats[1]),
                       lm_queries=int(stats[2]), fused=int(stats[3])),
            subs=None if not S else [[(float(subL[i, j]), [int(x) for x in subw[i, j, :min(subnw[i, j], max_words)]])
                                      for j in range(nsub[i])] for i in range(m)])

    def log10p(self, ctx, w: int) -> float:
        c = np.ascontiguousarray(list(ctx) or [0], dtype=np.int32)
        return float(self.lib.orc_log10p(self._h, _ptr(c), len(ctx), int(w)))

    def fusion_score(self, params: _Params, words) -> float:
        a = np.ascontiguousarray(list(words) or [0], dtype=np.int32)
        return float(self.lib.orc_fusion_score(self._h, ctypes.byref(params), _ptr(a), len(words)))


def splitmix64(x: int) -> int:
    return int(_load().orc_splitmix64(ctypes.c_uint64(x & (2**64 - 1))))


def prefix_key(y) -> int:
    a = np.ascontiguousarray(list(y) or [0], dtype=np.int32)
    return int(_load().orc_prefix_key(_ptr(a), len(y)))
