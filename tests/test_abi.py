"""CPU checks of the C ABI: the library loads, exports every call the header
declares, and rejects malformed input on the host before touching a GPU."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_14991_amd as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "fusion.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\**\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(F.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    return F.lib()


def test_header_declares_the_expected_calls():
    assert set(header_functions()) == set(F.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    raw = ctypes.CDLL(F.LIB_PATH)
    for name in header_functions():
        assert hasattr(raw, name), name


def _lm_args(tokens, logp, backoff):
    n = len(tokens)
    count = np.array([t.shape[0] for t in tokens], np.int64)
    VP = ctypes.c_void_p * n
    keep = [np.ascontiguousarray(t, np.int32) for t in tokens] + \
           [np.ascontiguousarray(p, np.float32) for p in logp] + \
           [None if b is None else np.ascontiguousarray(b, np.float32) for b in backoff]
    tp = VP(*[a.ctypes.data for a in keep[:n]])
    lp = VP(*[a.ctypes.data for a in keep[n:2 * n]])
    bp = VP(*[None if a is None else a.ctypes.data for a in keep[2 * n:]])
    return count, tp, lp, bp, keep


def _load(lib, order, V, blank, tokens, logp, backoff):
    count, tp, lp, bp, keep = _lm_args(tokens, logp, backoff)
    out = ctypes.c_void_p()
    rc = lib.ngram_load(order, V, blank, count.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                        tp, lp, bp, None, ctypes.byref(out))
    return rc, out


def _good_tables():
    uni = np.array([[1], [2], [3], [4], [5]], np.int32)  # V = 4, blank 0, <s> = 4, </s> = 5
    big = np.array([[1, 2], [4, 1]], np.int32)
    return [uni, big], [np.full(5, -1.5, np.float32), np.full(2, -0.5, np.float32)], \
           [np.zeros(5, np.float32), None]


def test_ngram_load_rejects_malformed_tables(lib):
    toks, lps, bos = _good_tables()
    rc, _ = _load(lib, 1, 4, 0, toks[:1], lps[:1], bos[:1])
    assert rc == F.FUSION_E_UNSUPPORTED
    rc, _ = _load(lib, 2, 9000, 0, toks, lps, bos)
    assert rc == F.FUSION_E_UNSUPPORTED
    bad = [toks[0], np.array([[1, 0], [4, 1]], np.int32)]  # blank inside an n-gram
    rc, _ = _load(lib, 2, 4, 0, bad, lps, bos)
    assert rc == F.FUSION_E_LM_FORMAT and "blank" in F.fusion_last_error()
    dup = [toks[0], np.array([[1, 2], [1, 2]], np.int32)]
    rc, _ = _load(lib, 2, 4, 0, dup, lps, bos)
    assert rc == F.FUSION_E_LM_FORMAT and "duplicate" in F.fusion_last_error()
    miss = [np.array([[1], [2], [4], [5]], np.int32), toks[1]]  # token 3 has no unigram
    rc, _ = _load(lib, 2, 4, 0, miss, [np.full(4, -1.0, np.float32), lps[1]], [None, None])
    assert rc == F.FUSION_E_LM_FORMAT and "unigram" in F.fusion_last_error()
    nan = [np.array([-1, np.nan, -1, -1, -1], np.float32), lps[1]]
    rc, _ = _load(lib, 2, 4, 0, toks, nan, bos)
    assert rc == F.FUSION_E_LM_FORMAT
    # trigram (1 2 3) without its suffix (2 3)
    t3 = [toks[0], toks[1], np.array([[1, 2, 3]], np.int32)]
    rc, _ = _load(lib, 3, 4, 0, t3, lps + [np.full(1, -0.1, np.float32)], [bos[0], np.zeros(2, np.float32), None])
    assert rc == F.FUSION_E_LM_FORMAT and "suffix" in F.fusion_last_error()
    # trigram (2 1 2) without its prefix (2 1)
    t3 = [toks[0], np.array([[1, 2], [4, 1]], np.int32), np.array([[2, 1, 2]], np.int32)]
    rc, _ = _load(lib, 3, 4, 0, t3, lps + [np.full(1, -0.1, np.float32)], [bos[0], np.zeros(2, np.float32), None])
    assert rc == F.FUSION_E_LM_FORMAT and "prefix" in F.fusion_last_error()


def test_boost_build_rejects_malformed_phrases(lib):
    def build(tokens, offsets, V=4, blank=0):
        t = np.ascontiguousarray(tokens, np.int32)
        o = np.ascontiguousarray(offsets, np.int64)
        out = ctypes.c_void_p()
        return lib.boost_build(V, blank, o.size - 1, ctypes.c_void_p(t.ctypes.data),
                               ctypes.c_void_p(o.ctypes.data), None, 1.0, None, ctypes.byref(out))

    assert build([1, 2], [0, 2, 2]) == F.FUSION_E_PHRASES  # empty phrase
    assert build([1, 0], [0, 2]) == F.FUSION_E_PHRASES  # blank inside
    assert build([1, 7], [0, 2]) == F.FUSION_E_PHRASES  # out of range
    assert build([1, 2], [1, 2]) == F.FUSION_E_PHRASES  # offsets[0] != 0


def test_fusion_calls_reject_bad_arguments(lib):
    out = [None] * 5
    rc = lib.fusion_step(None, None, None, None, None, 1, 4, 0.5, 0.5, 0, 1, 0, *out, None)
    assert rc == F.FUSION_E_ARG
    rc = lib.fusion_run(None, None, None, 1, 1, 1, 4, 1, 0.5, 0.5, 0, 0, None, None, None, None,
                        None, None, None, None)
    assert rc == F.FUSION_E_ARG
    assert "NULL" in F.fusion_last_error()
    # an empty batch still needs valid handles
    rc = lib.fusion_step(None, None, None, None, None, 0, 4, 0.5, 0.5, 0, 1, 0, *out, None)
    assert rc == F.FUSION_E_ARG
    rc = lib.fusion_run(None, None, None, 1, 0, 1, 4, 1, 0.5, 0.5, 0, 0, None, None, None, None,
                        None, None, None, None)
    assert rc == F.FUSION_E_ARG


def test_several_lm_calls_reject_bad_arguments(lib):
    out = [None] * 5
    al = (ctypes.c_float * 3)(0.5, 0.5, 0.5)
    hs = (ctypes.c_void_p * 3)(None, None, None)
    for n in (0, F.FUSION_MAX_LMS + 1):
        rc = lib.fusion_step_lms(ctypes.cast(hs, ctypes.c_void_p), ctypes.cast(al, ctypes.c_void_p), n,
                                 None, None, None, None, 1, 4, 0.5, 0, 1, 0, *out, None)
        assert rc == F.FUSION_E_ARG and "n_lm" in F.fusion_last_error()
    rc = lib.fusion_step_lms(None, None, 2, None, None, None, None, 1, 4, 0.5, 0, 1, 0, *out, None)
    assert rc == F.FUSION_E_ARG
    rc = lib.fusion_run_lms(ctypes.cast(hs, ctypes.c_void_p), ctypes.cast(al, ctypes.c_void_p), 2, None,
                            None, 1, 1, 1, 4, 1, 0.5, 0, 0, None, None, None, None, None, None, None,
                            0, None, None)
    assert rc == F.FUSION_E_ARG and "NULL" in F.fusion_last_error()
