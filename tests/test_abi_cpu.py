"""The C-ABI library loads, exports every symbol the header declares, and rejects
bad arguments on the host before any HIP call (no GPU needed)."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2603_14002_amd as lbm
from tests.tinylm import golden_ngram, lexicon_from
from workloads import DecodeParams

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lightbeam.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:lb_status|void|const char\*)\s+(lb_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    L = lbm.lib()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(lbm.EXPORTED)


def test_struct_sizes_match_header_layout():
    assert ctypes.sizeof(lbm.lb_params) == 160
    assert ctypes.sizeof(lbm.lb_ngram_desc) == 144
    assert ctypes.sizeof(lbm.lb_lexicon_desc) == 32
    assert ctypes.sizeof(lbm.lb_stats) == 320


def _descs():
    lm, _ = golden_ngram()
    lex = lexicon_from([(1,), (2,), (3,), (4,)])
    return lbm.make_descriptors(lex, lm)


def _create(d, params):
    out = ctypes.c_void_p()
    st = lbm.lib().lb_create(ctypes.byref(d.lex), ctypes.byref(d.lm), ctypes.byref(params), ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("field,value", [
    ("beam", 0), ("beam", 257), ("subbeams", 0), ("subbeams", 5), ("max_batch", 0), ("max_frames", 0),
    ("max_words_out", 0), ("fusion_source", 7), ("fusion_top_f", -1), ("theta", -1.0), ("lambda_", float("nan")),
    ("lm_load_factor", 0.95), ("arena_nodes_per_stream", -5), ("merge", 2), ("merge", -1), ("input", 2),
    ("eos_count", 4), ("eos_count", -1),
])
def test_create_rejects_bad_params(field, value):
    d = _descs()
    p = lbm.make_params(DecodeParams(), max_batch=2, max_frames=10)
    setattr(p, field, value)
    st, h = _create(d, p)
    assert st == lbm.LB_ERR_INVALID_ARG and not h
    assert lbm.lb_last_error()


def test_create_rejects_bad_lexicon():
    lm, _ = golden_ngram()
    p = lbm.make_params(DecodeParams(), max_batch=1, max_frames=10)
    for words in ([(1,), ()], [(1,), (40,)], [(0,)]):
        lex = lexicon_from([w if w else () for w in words])
        d = lbm.make_descriptors(lex, lm)
        st, h = _create(d, p)
        assert st == lbm.LB_ERR_INVALID_ARG and not h, words


def test_create_rejects_fusion_without_interval():
    d = _descs()
    p = lbm.make_params(DecodeParams(), max_batch=1, max_frames=10, fusion_source=lbm.LB_FUSION_SYNTH_BIGRAM)
    p.fusion_interval = 0
    st, _ = _create(d, p)
    assert st == lbm.LB_ERR_INVALID_ARG


def test_null_arguments():
    L = lbm.lib()
    out = ctypes.c_void_p()
    assert L.lb_create(None, None, None, ctypes.byref(out)) == lbm.LB_ERR_INVALID_ARG
    assert L.lb_decode_batch(None, None, None, 1, 1, 3, None, None, None) == lbm.LB_ERR_INVALID_ARG
    assert L.lb_fusion_scores(None, None, None) == lbm.LB_ERR_INVALID_ARG
    assert L.lb_fusion_request(None, None, None, None) == lbm.LB_ERR_INVALID_ARG
    assert L.lb_get_status(None, None) == lbm.LB_ERR_INVALID_ARG
    L.lb_destroy(None)


def test_library_built_from_other_sources_is_refused(monkeypatch):
    """lib() loads the library only when its build id equals the hash of the
    sources in this tree."""
    import paper_2603_14002_amd.build as bld
    L = lbm.lib()
    assert L.lb_build_id().decode() == bld.source_hash()
    monkeypatch.setattr(lbm, "_lib", None)
    monkeypatch.setattr(bld, "source_hash", lambda: "0" * 64)
    with pytest.raises(ImportError, match="built from other sources"):
        lbm.lib()
