"""CPU oracle for the shallow-fusion decode step (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  ``liboracle.so`` is built from ``oracle.c`` by plain gcc and
shares nothing with the product library; ``ref.py`` is a second, pure-Python
statement of the same definitions for tiny inputs.
"""

from __future__ import annotations

import ctypes
import os
import sys
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

GCC_CMD = ["gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", LIB, SRC, "-lm", "-lpthread"]


def build_oracle() -> str:
    """Compile liboracle.so (always; cheap)."""
    tmp = LIB + ".tmp"
    cmd = list(GCC_CMD)
    cmd[cmd.index(LIB)] = tmp
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("ORACLE_LIB", LIB)  # a sanitized build in the sanitizer test
        if path == LIB and not os.path.exists(LIB):
            build_oracle()
        L = ctypes.CDLL(path)
        vp, i32p, i64p, f32p, f64p = (ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                      ctypes.POINTER(ctypes.c_int64),
                                      ctypes.POINTER(ctypes.c_float),
                                      ctypes.POINTER(ctypes.c_double))
        c_int, c_float, c_double, c_i64 = ctypes.c_int, ctypes.c_float, ctypes.c_double, ctypes.c_int64
        L.or_last_error.restype = ctypes.c_char_p
        L.or_lm_new.restype = vp
        L.or_lm_new.argtypes = [c_int, c_int, c_int, i64p, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                ctypes.POINTER(vp)]
        L.or_lm_free.argtypes = [vp]
        L.or_lm_n_states.restype = c_i64
        L.or_lm_n_states.argtypes = [vp]
        L.or_lm_state_tuple.restype = c_int
        L.or_lm_state_tuple.argtypes = [vp, c_i64, i32p]
        L.or_lm_state_of_history.restype = c_i64
        L.or_lm_state_of_history.argtypes = [vp, i32p, c_int]
        L.or_lm_logp32.restype = c_float
        L.or_lm_logp32.argtypes = [vp, i32p, c_int, ctypes.c_int32]
        L.or_lm_logp64.restype = c_double
        L.or_lm_logp64.argtypes = [vp, i32p, c_int, ctypes.c_int32]
        L.or_lm_row64.restype = None
        L.or_lm_row64.argtypes = [vp, i32p, c_int, f64p]
        L.or_trie_new.restype = vp
        L.or_trie_new.argtypes = [c_int, c_int, c_i64, i32p, i64p, f32p, c_float]
        L.or_trie_free.argtypes = [vp]
        L.or_trie_n_nodes.restype = c_i64
        L.or_trie_n_nodes.argtypes = [vp]
        L.or_trie_max_len.restype = c_int
        L.or_trie_max_len.argtypes = [vp]
        L.or_trie_node_tuple.restype = c_int
        L.or_trie_node_tuple.argtypes = [vp, c_i64, i32p]
        L.or_trie_node_of.restype = c_i64
        L.or_trie_node_of.argtypes = [vp, i32p, c_int]
        L.or_trie_state_of_history.restype = c_i64
        L.or_trie_state_of_history.argtypes = [vp, i32p, c_int]
        L.or_trie_phi.restype = c_float
        L.or_trie_phi.argtypes = [vp, c_i64]
        L.or_trie_entry.restype = c_float
        L.or_trie_entry.argtypes = [vp, c_i64]
        L.or_step.restype = c_int
        L.or_step.argtypes = [vp, vp, f32p, i32p, i32p, c_int, c_int, c_float, c_float, c_int,
                              c_int, c_int, f32p, f64p, f64p, i32p, f64p, i32p, i32p]
        L.or_run.restype = c_int
        L.or_run.argtypes = [vp, vp, f32p, c_int, c_int, c_int, c_int, c_int, c_float, c_float,
                             c_int, c_int, i32p, i32p, f64p, i32p, i32p, f64p, i32p, i32p, f64p,
                             i32p, i32p, c_double, i64p, i64p, c_int]
        L.or_step_lms.restype = c_int
        L.or_step_lms.argtypes = [ctypes.POINTER(vp), f32p, c_int, vp, f32p, i32p, i32p, c_int,
                                  c_int, c_float, c_int, c_int, c_int, f32p, f64p, f64p, i32p,
                                  f64p, i32p, i32p]
        L.or_end_scores.restype = c_int
        L.or_end_scores.argtypes = [ctypes.POINTER(vp), f32p, c_int, i32p, c_int, f64p, f64p]
        L.or_run_lms.restype = c_int
        L.or_run_lms.argtypes = [ctypes.POINTER(vp), f32p, c_int, vp, f32p, c_int, c_int, c_int,
                                 c_int, c_int, c_float, c_int, c_int, i32p, i32p, f64p, i32p, i32p,
                                 f64p, i32p, i32p, f64p, i32p, i32p, c_double, i64p, i64p, c_int,
                                 c_int]
        _lib = L
    return _lib


def _p(a, ct):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ct))


class OracleError(RuntimeError):
    pass


def _err():
    return lib().or_last_error().decode()


class OracleLM:
    """The n-gram model as a set of sorted tuples (ARPA semantics)."""

    def __init__(self, lm):
        L = lib()
        self.N, self.V, self.blank = int(lm.order), int(lm.vocab), int(lm.blank)
        self._keep = []
        toks, lps, bos = [], [], []
        for k in range(self.N):
            t = np.ascontiguousarray(lm.tokens[k], dtype=np.int32)
            p = np.ascontiguousarray(lm.logp[k], dtype=np.float32)
            b = lm.backoff[k] if k < len(lm.backoff) else None
            b = None if b is None else np.ascontiguousarray(b, dtype=np.float32)
            self._keep += [t, p, b]
            toks.append(t.ctypes.data)
            lps.append(p.ctypes.data)
            bos.append(None if b is None else b.ctypes.data)
        counts = np.array([int(t.shape[0]) for t in lm.tokens], dtype=np.int64)
        VP = ctypes.c_void_p * self.N
        self.h = L.or_lm_new(self.N, self.V, self.blank, _p(counts, ctypes.c_int64),
                             VP(*toks), VP(*lps), VP(*bos))
        if not self.h:
            raise OracleError(_err())
        self._keep = None  # the oracle copied everything

    def __del__(self, _finalizing=sys.is_finalizing):
        if getattr(self, "h", None) and not _finalizing():  # at interpreter exit the memory goes anyway
            lib().or_lm_free(self.h)
            self.h = None

    @property
    def n_states(self):
        return int(lib().or_lm_n_states(self.h))

    def state_tuple(self, sid):
        out = np.zeros(32, dtype=np.int32)
        n = lib().or_lm_state_tuple(self.h, int(sid), _p(out, ctypes.c_int32))
        return None if n < 0 else tuple(out[:n].tolist())

    def state_of_history(self, hist):
        h = np.asarray(hist, dtype=np.int32)
        return int(lib().or_lm_state_of_history(self.h, _p(h, ctypes.c_int32), int(h.size)))

    def logp32(self, ctx, y):
        c = np.asarray(ctx, dtype=np.int32)
        c = c[max(0, c.size - (self.N - 1)):].copy()
        return np.float32(lib().or_lm_logp32(self.h, _p(c, ctypes.c_int32), int(c.size), int(y)))

    def row64(self, ctx):
        c = np.asarray(ctx, dtype=np.int32)
        c = c[max(0, c.size - (self.N - 1)):].copy()
        out = np.empty(self.V + 2, np.float64)
        lib().or_lm_row64(self.h, _p(c, ctypes.c_int32), int(c.size), _p(out, ctypes.c_double))
        return out

    def logp64(self, ctx, y):
        c = np.asarray(ctx, dtype=np.int32)
        c = c[max(0, c.size - (self.N - 1)):].copy()
        return float(lib().or_lm_logp64(self.h, _p(c, ctypes.c_int32), int(c.size), int(y)))


class OracleTrie:
    """The phrase list as sorted phrase and prefix sets (brute-force matching)."""

    def __init__(self, V, blank, phrases):
        L = lib()
        self.V, self.blank = int(V), int(blank)
        toks = np.ascontiguousarray(phrases.tokens, dtype=np.int32)
        offs = np.ascontiguousarray(phrases.offsets, dtype=np.int64)
        comp = None if phrases.completion is None else np.ascontiguousarray(phrases.completion,
                                                                            dtype=np.float32)
        self.h = L.or_trie_new(self.V, self.blank, int(offs.size - 1), _p(toks, ctypes.c_int32),
                               _p(offs, ctypes.c_int64), _p(comp, ctypes.c_float),
                               float(phrases.token_score))
        if not self.h:
            raise OracleError(_err())

    def __del__(self, _finalizing=sys.is_finalizing):
        if getattr(self, "h", None) and not _finalizing():  # at interpreter exit the memory goes anyway
            lib().or_trie_free(self.h)
            self.h = None

    @property
    def n_nodes(self):
        return int(lib().or_trie_n_nodes(self.h))

    @property
    def max_len(self):
        return int(lib().or_trie_max_len(self.h))

    def node_tuple(self, q):
        out = np.zeros(max(1, self.max_len), dtype=np.int32)
        n = lib().or_trie_node_tuple(self.h, int(q), _p(out, ctypes.c_int32))
        return None if n < 0 else tuple(out[:n].tolist())

    def node_of(self, prefix):
        p = np.asarray(prefix, dtype=np.int32)
        return int(lib().or_trie_node_of(self.h, _p(p, ctypes.c_int32), int(p.size)))

    def state_of_history(self, hist):
        h = np.asarray(hist, dtype=np.int32)
        return int(lib().or_trie_state_of_history(self.h, _p(h, ctypes.c_int32), int(h.size)))

    def phi(self, q):
        return np.float32(lib().or_trie_phi(self.h, int(q)))

    def entry(self, q):
        return np.float32(lib().or_trie_entry(self.h, int(q)))


def step(lm: OracleLM, trie: OracleTrie | None, logits, lm_state, boost_state, lam, beta,
         blank, k, mode, want_rows=True):
    """One decode step from state ids.  Returns a dict of numpy arrays."""
    x = np.ascontiguousarray(logits, dtype=np.float32)
    H, V = x.shape
    ls = np.ascontiguousarray(lm_state, dtype=np.int32)
    bs = np.ascontiguousarray(boost_state, dtype=np.int32)
    key = np.empty((H, V), np.float32) if want_rows else None
    fused = np.empty((H, V), np.float64) if want_rows else None
    lse = np.empty(H, np.float64)
    tok = np.empty((H, k), np.int32)
    sc = np.empty((H, k), np.float64)
    nl = np.empty((H, k), np.int32)
    nb = np.empty((H, k), np.int32)
    rc = lib().or_step(lm.h, trie.h if trie is not None else None, _p(x, ctypes.c_float),
                       _p(ls, ctypes.c_int32), _p(bs, ctypes.c_int32), H, V, float(lam),
                       float(beta), int(blank), int(k), int(mode), _p(key, ctypes.c_float),
                       _p(fused, ctypes.c_double), _p(lse, ctypes.c_double),
                       _p(tok, ctypes.c_int32), _p(sc, ctypes.c_double), _p(nl, ctypes.c_int32),
                       _p(nb, ctypes.c_int32))
    if rc != 0:
        raise OracleError(_err())
    return dict(key=key, fused=fused, lse=lse, tokens=tok, scores=sc, next_lm=nl, next_boost=nb)


def run(lm: OracleLM, trie: OracleTrie | None, logits, S, B, k, lam, beta, blank, mode,
        lm_state, boost_state, hyp_score=None, forced_tokens=None, forced_parents=None,
        tol=1e-4, threads=1):
    """Free-running decode over all frames of ``logits`` [T, S*B, V] from full
    token histories.  With ``forced_*`` the oracle replays those decisions and
    reports where they stop agreeing with its own (``mismatch_at`` per stream,
    -1 if never; near ties within ``tol`` are accepted and counted)."""
    x = np.ascontiguousarray(logits, dtype=np.float32)
    T, H, V = x.shape
    assert H == S * B
    ls = np.ascontiguousarray(lm_state, dtype=np.int32)
    bs = np.ascontiguousarray(boost_state, dtype=np.int32)
    hs = None
    if B > 1:
        hs = np.ascontiguousarray(hyp_score if hyp_score is not None else
                                  np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S),
                                  dtype=np.float64)
    tok = np.empty((T, H), np.int32)
    par = np.empty((T, H), np.int32) if B > 1 else None
    sel = np.empty((T, H), np.float64)
    lo = np.empty(H, np.int32)
    bo = np.empty(H, np.int32)
    so = np.empty(H, np.float64)
    ft = None if forced_tokens is None else np.ascontiguousarray(forced_tokens, dtype=np.int32)
    fp = None if forced_parents is None else np.ascontiguousarray(forced_parents, dtype=np.int32)
    near = np.zeros(max(S, 1), np.int64)
    mis = np.zeros(max(S, 1), np.int64)
    rc = lib().or_run(lm.h, trie.h if trie is not None else None, _p(x, ctypes.c_float), T, S, B,
                      V, int(k), float(lam), float(beta), int(blank), int(mode),
                      _p(ls, ctypes.c_int32), _p(bs, ctypes.c_int32), _p(hs, ctypes.c_double),
                      _p(tok, ctypes.c_int32), _p(par, ctypes.c_int32), _p(sel, ctypes.c_double),
                      _p(lo, ctypes.c_int32), _p(bo, ctypes.c_int32), _p(so, ctypes.c_double),
                      _p(ft, ctypes.c_int32), _p(fp, ctypes.c_int32), float(tol),
                      _p(near, ctypes.c_int64), _p(mis, ctypes.c_int64), int(threads))
    if rc != 0:
        raise OracleError(_err())
    return dict(tokens=tok, parents=par, sel_score=sel, lm_state=lo, boost_state=bo,
                hyp_score=so if B > 1 else None, near_ties=near[:S], mismatch_at=mis[:S])


MAX_LMS = 4


def _lm_list(lms, alphas):
    lms, alphas = list(lms), [float(a) for a in alphas]
    if not 1 <= len(lms) <= MAX_LMS or len(alphas) != len(lms):
        raise OracleError("need 1..4 LMs and one weight per LM")
    hs = (ctypes.c_void_p * len(lms))(*[m.h for m in lms])
    return hs, np.array(alphas, dtype=np.float32), len(lms)


def step_lms(lms, alphas, trie: OracleTrie | None, logits, lm_states, boost_state, beta, blank, k,
             mode, want_rows=True):
    """One decode step with several LMs (Eq. (1): one weighted term per LM, added
    in the given order).  ``lm_states`` is [n_lm, H]; ``next_lm`` comes back as
    [n_lm, H, k]."""
    hs, al, n = _lm_list(lms, alphas)
    x = np.ascontiguousarray(logits, dtype=np.float32)
    H, V = x.shape
    ls = np.ascontiguousarray(np.asarray(lm_states).reshape(n, H), dtype=np.int32)
    bs = np.ascontiguousarray(boost_state, dtype=np.int32)
    key = np.empty((H, V), np.float32) if want_rows else None
    fused = np.empty((H, V), np.float64) if want_rows else None
    lse = np.empty(H, np.float64)
    tok = np.empty((H, k), np.int32)
    sc = np.empty((H, k), np.float64)
    nl = np.empty((n, H, k), np.int32)
    nb = np.empty((H, k), np.int32)
    rc = lib().or_step_lms(hs, _p(al, ctypes.c_float), n, trie.h if trie is not None else None,
                           _p(x, ctypes.c_float), _p(ls, ctypes.c_int32), _p(bs, ctypes.c_int32), H,
                           V, float(beta), int(blank), int(k), int(mode), _p(key, ctypes.c_float),
                           _p(fused, ctypes.c_double), _p(lse, ctypes.c_double),
                           _p(tok, ctypes.c_int32), _p(sc, ctypes.c_double), _p(nl, ctypes.c_int32),
                           _p(nb, ctypes.c_int32))
    if rc != 0:
        raise OracleError(_err())
    return dict(key=key, fused=fused, lse=lse, tokens=tok, scores=sc, next_lm=nl, next_boost=nb)


def run_lms(lms, alphas, trie: OracleTrie | None, logits, S, B, k, beta, blank, mode, lm_states,
            boost_state, hyp_score=None, forced_tokens=None, forced_parents=None, tol=1e-4,
            threads=1, recombine=False):
    """``run`` with several LMs: ``lm_states`` is [n_lm, S*B] and the final LM
    states come back as [n_lm, S*B].  ``recombine`` (beam): candidates reaching
    the same token history merge into the first of them in candidate order,
    with the log-sum of their scores."""
    hs_, al, n = _lm_list(lms, alphas)
    x = np.ascontiguousarray(logits, dtype=np.float32)
    T, H, V = x.shape
    assert H == S * B
    ls = np.ascontiguousarray(np.asarray(lm_states).reshape(n, H), dtype=np.int32)
    bs = np.ascontiguousarray(boost_state, dtype=np.int32)
    hs = None
    if B > 1:
        hs = np.ascontiguousarray(hyp_score if hyp_score is not None else
                                  np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S),
                                  dtype=np.float64)
    tok = np.empty((T, H), np.int32)
    par = np.empty((T, H), np.int32) if B > 1 else None
    sel = np.empty((T, H), np.float64)
    lo = np.empty((n, H), np.int32)
    bo = np.empty(H, np.int32)
    so = np.empty(H, np.float64)
    ft = None if forced_tokens is None else np.ascontiguousarray(forced_tokens, dtype=np.int32)
    fp = None if forced_parents is None else np.ascontiguousarray(forced_parents, dtype=np.int32)
    near = np.zeros(max(S, 1), np.int64)
    mis = np.zeros(max(S, 1), np.int64)
    rc = lib().or_run_lms(hs_, _p(al, ctypes.c_float), n, trie.h if trie is not None else None,
                          _p(x, ctypes.c_float), T, S, B, V, int(k), float(beta), int(blank),
                          int(mode), _p(ls, ctypes.c_int32), _p(bs, ctypes.c_int32),
                          _p(hs, ctypes.c_double), _p(tok, ctypes.c_int32), _p(par, ctypes.c_int32),
                          _p(sel, ctypes.c_double), _p(lo, ctypes.c_int32), _p(bo, ctypes.c_int32),
                          _p(so, ctypes.c_double), _p(ft, ctypes.c_int32), _p(fp, ctypes.c_int32),
                          float(tol), _p(near, ctypes.c_int64), _p(mis, ctypes.c_int64),
                          int(threads), int(bool(recombine)))
    if rc != 0:
        raise OracleError(_err())
    return dict(tokens=tok, parents=par, sel_score=sel, lm_state=lo, boost_state=bo,
                hyp_score=so if B > 1 else None, near_ties=near[:S], mismatch_at=mis[:S])


def end_scores(lms, alphas, lm_states, hyp_score=None):
    """End of stream: per hypothesis the weighted LM terms of </s> (each LM's
    fp32 backoff value, fp32 product), added in LM order to ``hyp_score`` (a
    new array; None: zeros).  Returns (new scores, end terms)."""
    hs, al, n = _lm_list(lms, alphas)
    ls = np.ascontiguousarray(np.asarray(lm_states).reshape(n, -1), dtype=np.int32)
    H = ls.shape[1]
    sc = np.zeros(H, np.float64) if hyp_score is None else np.array(hyp_score, dtype=np.float64)
    term = np.empty(H, np.float64)
    rc = lib().or_end_scores(hs, _p(al, ctypes.c_float), n, _p(ls, ctypes.c_int32), H,
                             _p(sc, ctypes.c_double), _p(term, ctypes.c_double))
    if rc != 0:
        raise OracleError(_err())
    return sc, term
