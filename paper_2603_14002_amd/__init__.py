"""MI355X (gfx950) LightBeam decoding library: a thin ctypes binding of liblightbeam.so.

The functions below carry the names of the C ABI in ``include/lightbeam.h``
and only marshal arguments: every step of the decode runs in the HIP kernels
of the library.  PyTorch tensors supply device memory and streams.  If the
library has not been built (``python -m paper_2603_14002_amd.build``) the
import of ``lib()`` raises; there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblightbeam.so")

LB_OK, LB_ERR_INVALID_ARG, LB_ERR_STATE, LB_ERR_CAPACITY = 0, 1, 2, 3
LB_ERR_OUT_OF_MEMORY, LB_ERR_HIP, LB_NEED_FUSION = 4, 5, 6
LB_BEGIN, LB_END = 1, 2
LB_FUSION_NONE, LB_FUSION_SYNTH_BIGRAM, LB_FUSION_EXTERNAL = 0, 1, 2
LB_MAX_BEAM, LB_MAX_SUBBEAMS = 256, 4

STATUS_NAMES = {0: "LB_OK", 1: "LB_ERR_INVALID_ARG", 2: "LB_ERR_STATE", 3: "LB_ERR_CAPACITY",
                4: "LB_ERR_OUT_OF_MEMORY", 5: "LB_ERR_HIP", 6: "LB_NEED_FUSION"}

EXPORTED = ("lb_create", "lb_destroy", "lb_decode_batch", "lb_fusion_request", "lb_fusion_scores",
            "lb_get_status", "lb_get_stats", "lb_reset_stats", "lb_set_profiling", "lb_last_error",
            "lb_build_id", "lb_decode_batch_noalloc", "lb_measure_gather")


class LBError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class lb_lexicon_desc(ctypes.Structure):
    _fields_ = [("n_entries", ctypes.c_int32), ("offsets", ctypes.c_void_p), ("phonemes", ctypes.c_void_p),
                ("entry_word", ctypes.c_void_p)]


class lb_ngram_desc(ctypes.Structure):
    _fields_ = [("vocab_size", ctypes.c_int32), ("bos_id", ctypes.c_int32), ("unk_id", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("count", ctypes.c_int64 * 4),
                ("ids", ctypes.c_void_p * 4), ("log10p", ctypes.c_void_p * 4),
                ("backoff", ctypes.c_void_p * 4)]


class lb_params(ctypes.Structure):
    _fields_ = [("beam", ctypes.c_int32), ("subbeams", ctypes.c_int32),
                ("alpha", ctypes.c_double), ("beta", ctypes.c_double), ("gamma", ctypes.c_double),
                ("omega", ctypes.c_double), ("phi", ctypes.c_double), ("theta", ctypes.c_double),
                ("lambda_", ctypes.c_double),
                ("fusion_source", ctypes.c_int32), ("fusion_interval", ctypes.c_int32),
                ("fusion_top_f", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("max_frames", ctypes.c_int32), ("max_words_out", ctypes.c_int32),
                ("fusion_seed", ctypes.c_uint64), ("fusion_lo", ctypes.c_double),
                ("fusion_hi", ctypes.c_double), ("lm_load_factor", ctypes.c_double),
                ("arena_nodes_per_stream", ctypes.c_int64),
                ("merge", ctypes.c_int32), ("input", ctypes.c_int32),
                ("eos_count", ctypes.c_int32), ("eos_ids", ctypes.c_int32 * 3),
                ("heavy_homophones", ctypes.c_int32)]


class lb_stats(ctypes.Structure):
    _fields_ = [("expansions", ctypes.c_int64), ("word_events", ctypes.c_int64),
                ("lm_queries", ctypes.c_int64), ("fused", ctypes.c_int64), ("frames", ctypes.c_int64),
                ("probe_lines", ctypes.c_int64), ("lm_lookups", ctypes.c_int64),
                ("launches", ctypes.c_int64 * 8), ("kernel_ms", ctypes.c_double * 8),
                ("timed", ctypes.c_int64 * 8), ("index_lines", ctypes.c_int64),
                ("phase_cycles", ctypes.c_int64 * 8)]


_lib = None


def lib():
    """The loaded liblightbeam.so.  Raises if it has not been built, or if its
    build id differs from the hash of the sources in this tree (a library built
    from other sources is never used)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2603_14002_amd.build`")
        from .build import source_hash
        L = ctypes.CDLL(LIB_PATH)
        L.lb_build_id.restype = ctypes.c_char_p
        L.lb_build_id.argtypes = []
        have, want = L.lb_build_id().decode(), source_hash()
        if have != want:
            raise ImportError(f"{LIB_PATH} was built from other sources (build id {have[:16]}, sources "
                              f"{want[:16]}): rebuild it with `python -m paper_2603_14002_amd.build`")
        P = ctypes.c_void_p
        L.lb_create.restype = ctypes.c_int32
        L.lb_create.argtypes = [ctypes.POINTER(lb_lexicon_desc), ctypes.POINTER(lb_ngram_desc),
                                ctypes.POINTER(lb_params), ctypes.POINTER(ctypes.c_void_p)]
        L.lb_destroy.restype = None
        L.lb_destroy.argtypes = [P]
        L.lb_decode_batch.restype = ctypes.c_int32
        L.lb_decode_batch.argtypes = [P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint32, P, P, P]
        L.lb_decode_batch_noalloc.restype = ctypes.c_int32
        L.lb_decode_batch_noalloc.argtypes = [P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint32, P, P, P]
        L.lb_measure_gather.restype = ctypes.c_int32
        L.lb_measure_gather.argtypes = [P, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, P, ctypes.c_uint64, P]
        L.lb_fusion_request.restype = ctypes.c_int32
        L.lb_fusion_request.argtypes = [P, P, P, P]
        L.lb_fusion_scores.restype = ctypes.c_int32
        L.lb_fusion_scores.argtypes = [P, P, P]
        L.lb_get_status.restype = ctypes.c_int32
        L.lb_get_status.argtypes = [P, P]
        L.lb_get_stats.restype = ctypes.c_int32
        L.lb_get_stats.argtypes = [P, ctypes.POINTER(lb_stats)]
        L.lb_reset_stats.restype = ctypes.c_int32
        L.lb_reset_stats.argtypes = [P]
        L.lb_set_profiling.restype = ctypes.c_int32
        L.lb_set_profiling.argtypes = [P, ctypes.c_uint32]
        L.lb_last_error.restype = ctypes.c_char_p
        L.lb_last_error.argtypes = []
        _lib = L
    return _lib


def lb_last_error() -> str:
    return lib().lb_last_error().decode()


def lb_build_id() -> str:
    return lib().lb_build_id().decode()


def _check(st: int, allow=(LB_OK,)) -> int:
    if st not in allow:
        raise LBError(st, lb_last_error())
    return st


def _np_ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _dev_ptr(t) -> Optional[int]:
    """Device address of a torch tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------ C-ABI wrappers (same names)


def lb_create(lex: lb_lexicon_desc, lm: lb_ngram_desc, params: lb_params) -> int:
    out = ctypes.c_void_p()
    _check(lib().lb_create(ctypes.byref(lex), ctypes.byref(lm), ctypes.byref(params), ctypes.byref(out)))
    return out.value


def lb_destroy(dec: int) -> None:
    lib().lb_destroy(dec)


def lb_decode_batch(dec: int, logits, lengths, batch: int, frames: int, flags: int, stream,
                    out_hyps, out_scores) -> int:
    return _check(lib().lb_decode_batch(dec, _dev_ptr(logits), _dev_ptr(lengths), batch, frames, flags,
                                        _stream_ptr(stream), _dev_ptr(out_hyps), _dev_ptr(out_scores)),
                  allow=(LB_OK, LB_NEED_FUSION))


def lb_decode_batch_noalloc(dec: int, logits, lengths, batch: int, frames: int, flags: int, stream,
                            out_hyps, out_scores) -> int:
    return _check(lib().lb_decode_batch_noalloc(dec, _dev_ptr(logits), _dev_ptr(lengths), batch, frames, flags,
                                                _stream_ptr(stream), _dev_ptr(out_hyps), _dev_ptr(out_scores)))


def lb_measure_gather(table, table_lines: int, n_lines: int, seed: int, out, out_len: int, stream) -> int:
    return _check(lib().lb_measure_gather(_dev_ptr(table), table_lines, n_lines, seed & (2**64 - 1), _dev_ptr(out),
                                          out_len, _stream_ptr(stream)))


def lb_fusion_request(dec: int, words, n_words, stream) -> int:
    return _check(lib().lb_fusion_request(dec, _dev_ptr(words), _dev_ptr(n_words), _stream_ptr(stream)))


def lb_fusion_scores(dec: int, fusion_logprobs, stream) -> int:
    return _check(lib().lb_fusion_scores(dec, _dev_ptr(fusion_logprobs), _stream_ptr(stream)))


def lb_get_status(dec: int, stream) -> int:
    return lib().lb_get_status(dec, _stream_ptr(stream))


def lb_get_stats(dec: int) -> lb_stats:
    s = lb_stats()
    _check(lib().lb_get_stats(dec, ctypes.byref(s)))
    return s


def lb_reset_stats(dec: int) -> None:
    _check(lib().lb_reset_stats(dec))


# kernel kinds (index of lb_stats.launches / kernel_ms)
KIND_DECODE, KIND_OUTPUT, KIND_FUSE_SELECT, KIND_FUSE_EXPORT, KIND_FUSE_APPLY, KIND_BEGIN = 0, 1, 2, 3, 4, 5
KIND_NAMES = ("decode", "output", "fuse_select", "fuse_export", "fuse_apply", "begin")
LB_MERGE_LOGSUMEXP, LB_MERGE_MAX = 0, 1
LB_INPUT_LOGPROBS, LB_INPUT_LOGITS = 0, 1
LB_PROFILE_ALL, LB_PROFILE_PHASES = 0xFF, 0x100
PHASE_NAMES = ("recombination", "top_k", "new_beam", "ngram_group", "ngram_lookup", "ngram_rank", "fusion_rest",
               "load_writeback_output")


def lb_set_profiling(dec: int, kernel_mask: int) -> None:
    """bit k times kernel kind k with HIP events (0 = off, LB_PROFILE_ALL = all)."""
    _check(lib().lb_set_profiling(dec, int(kernel_mask) & 0xFFFFFFFF))


# ------------------------------------------------------------------ descriptor marshalling


@dataclass
class Descriptors:
    """C descriptors plus the host arrays they point into (kept alive)."""

    lex: lb_lexicon_desc
    lm: lb_ngram_desc
    keep: list


def make_descriptors(lexicon, ngram) -> Descriptors:
    """Descriptors of a lexicon (entries: offsets, phonemes, optional entry ->
    word map) and a 4-gram LM (vocab_size, bos, unk, ids[4], logp[4], bo[3])."""
    keep = []

    def arr(a, dt):
        x = np.ascontiguousarray(a, dtype=dt)
        keep.append(x)
        return x

    offs = arr(lexicon.offsets, np.int32)
    phs = arr(lexicon.phonemes, np.int32)
    ew = getattr(lexicon, "entry_word", None)
    ewp = arr(ew, np.int32).ctypes.data if ew is not None else None
    lex = lb_lexicon_desc(int(lexicon.n_words), offs.ctypes.data, phs.ctypes.data, ewp)
    lm = lb_ngram_desc()
    lm.vocab_size = int(ngram.vocab_size)
    lm.bos_id = int(ngram.bos)
    lm.unk_id = int(ngram.unk)
    for n in range(4):
        ids = arr(ngram.ids[n], np.int32)
        lp = arr(ngram.logp[n], np.float32)
        lm.count[n] = int(ids.shape[0])
        lm.ids[n] = ids.ctypes.data if ids.size else None
        lm.log10p[n] = lp.ctypes.data if lp.size else None
        if n < 3:
            bo = arr(ngram.bo[n], np.float32)
            lm.backoff[n] = bo.ctypes.data if bo.size else None
        else:
            lm.backoff[n] = None
    return Descriptors(lex, lm, keep)


def make_params(p, *, max_batch: int, max_frames: int, fusion_source: Optional[int] = None,
                fusion_seed: int = 0, load_factor: float = 0.0, arena_nodes_per_stream: int = 0,
                **overrides) -> lb_params:
    """lb_params from a ``workloads.DecodeParams``-like object."""
    src = fusion_source
    if src is None:
        src = LB_FUSION_SYNTH_BIGRAM if p.fusion_interval > 0 else LB_FUSION_NONE
    d = dict(beam=p.beam, subbeams=p.subbeams, alpha=p.alpha, beta=p.beta, gamma=p.gamma,
             omega=p.omega, phi=p.phi, theta=p.theta, lambda_=p.lam, fusion_source=src,
             fusion_interval=p.fusion_interval if src != LB_FUSION_NONE else 0,
             fusion_top_f=p.fusion_top_f, max_batch=max_batch, max_frames=max_frames,
             max_words_out=p.max_words_out, fusion_seed=fusion_seed & (2**64 - 1),
             fusion_lo=p.fusion_lo, fusion_hi=p.fusion_hi, lm_load_factor=load_factor,
             arena_nodes_per_stream=arena_nodes_per_stream, merge=LB_MERGE_LOGSUMEXP, input=LB_INPUT_LOGPROBS)
    d.update(overrides)
    return lb_params(**d)


class Decoder:
    """Convenience owner of an lb_decoder handle (argument marshalling only)."""

    def __init__(self, lexicon, ngram, params: lb_params):
        self.desc = make_descriptors(lexicon, ngram)
        self.params = params
        self.handle = lb_create(self.desc.lex, self.desc.lm, params)
        self.desc = None  # the library copied what it keeps

    def close(self):
        if getattr(self, "handle", None):
            lb_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def decode(self, logits, lengths, flags: int = LB_BEGIN | LB_END, stream=None, out_hyps=None,
               out_scores=None):
        """logits: device float32 [B, T, 41]; lengths: device int32 [B].  Returns
        (status, out_hyps int32 [B, K, W], out_scores float32 [B, K])."""
        import torch
        B, T = int(logits.shape[0]), int(logits.shape[1])
        K, W = self.params.beam, self.params.max_words_out
        dev = logits.device
        if out_hyps is None:
            out_hyps = torch.empty((B, K, W), dtype=torch.int32, device=dev)
        if out_scores is None:
            out_scores = torch.empty((B, K), dtype=torch.float32, device=dev)
        st = lb_decode_batch(self.handle, logits, lengths, B, T, flags, stream, out_hyps, out_scores)
        return st, out_hyps, out_scores

    def status(self, stream=None) -> int:
        return lb_get_status(self.handle, stream)

    def stats(self) -> lb_stats:
        return lb_get_stats(self.handle)
