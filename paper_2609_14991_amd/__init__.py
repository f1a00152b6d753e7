"""Python binding of the MI355X shallow-fusion library (libfusion.so).

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the C ABI declared in ``include/fusion.h``.  PyTorch supplies
device memory and the HIP stream.  The library must have been built
(``__graft_entry__.build()`` or ``python paper_2609_14991_amd/build.py``);
importing a function of this module without it raises an error, there is no
fallback.
"""

from __future__ import annotations

import atexit
import ctypes
import os
import sys
import weakref

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfusion.so")

FUSION_OK = 0
FUSION_E_ARG = -1
FUSION_E_NOMEM = -2
FUSION_E_HIP = -3
FUSION_E_LM_FORMAT = -4
FUSION_E_PHRASES = -5
FUSION_E_UNSUPPORTED = -6
FUSION_BLANK_AM = 0
FUSION_BLANK_COMPETE = 1
FUSION_STATUS_BAD_LM_STATE = 1
FUSION_STATUS_BAD_BOOST_STATE = 2

FUSION_MAX_LMS = 2
FUSION_RUN_RECOMBINE = 1

EXPORTS = ("ngram_load", "ngram_bos_state", "ngram_info", "ngram_free", "boost_build", "boost_info",
           "boost_free", "fusion_step", "fusion_run", "fusion_step_lms", "fusion_run_lms",
           "fusion_run_lms_noalloc", "fusion_run_projected",
           "fusion_end_scores", "joint_project", "fusion_last_error", "fusion_device_status")


class FusionError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"fusion error {code}: {msg}")
        self.code = code


_lib = None


def lib():
    """The loaded libfusion.so (raises if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                  ctypes.c_double)
        P = ctypes.POINTER
        L.ngram_load.restype = ctypes.c_int
        L.ngram_load.argtypes = [i32, i32, i32, P(i64), P(vp), P(vp), P(vp), vp, P(vp)]
        L.ngram_bos_state.restype = ctypes.c_int
        L.ngram_bos_state.argtypes = [vp, P(i32)]
        L.ngram_info.restype = ctypes.c_int
        L.ngram_info.argtypes = [vp, P(i64), P(i64)]
        L.ngram_free.restype = None
        L.ngram_free.argtypes = [vp]
        L.boost_build.restype = ctypes.c_int
        L.boost_build.argtypes = [i32, i32, i32, vp, vp, vp, f32, vp, P(vp)]
        L.boost_info.restype = ctypes.c_int
        L.boost_info.argtypes = [vp, P(i32), P(i32), P(i64)]
        L.boost_free.restype = None
        L.boost_free.argtypes = [vp]
        L.fusion_step.restype = ctypes.c_int
        L.fusion_step.argtypes = [vp, vp, vp, vp, vp, i32, i32, f32, f32, i32, i32, i32, vp, vp, vp,
                                  vp, vp, vp]
        L.fusion_run.restype = ctypes.c_int
        L.fusion_run.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, f32, f32, i32, i32, vp, vp, vp,
                                 vp, vp, vp, vp, vp]
        L.fusion_step_lms.restype = ctypes.c_int
        L.fusion_step_lms.argtypes = [vp, vp, i32, vp, vp, vp, vp, i32, i32, f32, i32, i32, i32, vp,
                                      vp, vp, vp, vp, vp]
        L.fusion_run_lms.restype = ctypes.c_int
        L.fusion_run_lms.argtypes = [vp, vp, i32, vp, vp, i32, i32, i32, i32, i32, f32, i32, i32, vp,
                                     vp, vp, vp, vp, vp, vp, i32, vp, vp]
        L.fusion_run_lms_noalloc.restype = ctypes.c_int
        L.fusion_run_lms_noalloc.argtypes = L.fusion_run_lms.argtypes
        L.fusion_run_projected.restype = ctypes.c_int
        L.fusion_run_projected.argtypes = [vp, vp, i32, vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, i32, i32, f32, i32,
                                           i32, vp, vp, vp, vp, vp, i32, vp, vp]
        L.fusion_end_scores.restype = ctypes.c_int
        L.fusion_end_scores.argtypes = [vp, vp, i32, vp, i32, vp, vp, vp]
        L.joint_project.restype = ctypes.c_int
        L.joint_project.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp]
        L.fusion_last_error.restype = ctypes.c_char_p
        L.fusion_last_error.argtypes = []
        L.fusion_device_status.restype = ctypes.c_int
        L.fusion_device_status.argtypes = [vp, P(i32)]
        _lib = L
    return _lib


def fusion_last_error() -> str:
    return lib().fusion_last_error().decode()


def _check(rc):
    if rc != FUSION_OK:
        raise FusionError(rc, fusion_last_error())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch

    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    """Device (or host numpy) pointer of a buffer, None for None."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return ctypes.c_void_p(t.ctypes.data)
    return ctypes.c_void_p(t.data_ptr())


# Device handles still alive when the interpreter begins to shut down are
# released by an atexit hook, while the HIP runtime is certainly still up;
# a handle's __del__ never calls into the library once shutdown has begun
_live = weakref.WeakSet()


def _release_all():
    for h in list(_live):
        h.close()


atexit.register(_release_all)


class _Handle:
    _free_fn = None

    def __init__(self, handle):
        self.h = ctypes.c_void_p(handle)
        _live.add(self)

    def close(self):
        """Release the device memory now (idempotent)."""
        if getattr(self, "h", None) is not None and self.h.value:
            getattr(lib(), self._free_fn)(self.h)
        self.h = None

    def __del__(self, _finalizing=sys.is_finalizing):
        if _finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


class NgramTables(_Handle):
    """Owning handle of device-resident n-gram tables."""

    _free_fn = "ngram_free"

    def __init__(self, handle, order, vocab, blank):
        super().__init__(handle)
        self.order, self.vocab, self.blank = order, vocab, blank


class BoostTrie(_Handle):
    """Owning handle of a device-resident phrase-boosting tree."""

    _free_fn = "boost_free"

    def __init__(self, handle, vocab, blank):
        super().__init__(handle)
        self.vocab, self.blank = vocab, blank


def ngram_load(order, vocab, blank_id, tokens, logp, backoff=None, stream=None) -> NgramTables:
    """tokens/logp/backoff: per-order host arrays (see include/fusion.h)."""
    L = lib()
    order = int(order)
    toks = [np.ascontiguousarray(t, dtype=np.int32) for t in tokens]
    lps = [np.ascontiguousarray(p, dtype=np.float32) for p in logp]
    bos = [None if (backoff is None or b is None) else np.ascontiguousarray(b, dtype=np.float32)
           for b in (backoff if backoff is not None else [None] * order)]
    count = np.array([t.shape[0] for t in toks], dtype=np.int64)
    VP = ctypes.c_void_p * order
    tp = VP(*[t.ctypes.data for t in toks])
    lp = VP(*[p.ctypes.data for p in lps])
    bp = VP(*[None if b is None else b.ctypes.data for b in bos])
    out = ctypes.c_void_p()
    _check(L.ngram_load(order, int(vocab), int(blank_id),
                        count.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), tp, lp, bp,
                        _stream(stream), ctypes.byref(out)))
    return NgramTables(out.value, order, int(vocab), int(blank_id))


def ngram_load_arrays(lm, stream=None) -> NgramTables:
    """ngram_load from an object with order/vocab/blank/tokens/logp/backoff."""
    return ngram_load(lm.order, lm.vocab, lm.blank, lm.tokens, lm.logp, lm.backoff, stream)


def ngram_bos_state(lm: NgramTables) -> int:
    v = ctypes.c_int32()
    _check(lib().ngram_bos_state(lm.h, ctypes.byref(v)))
    return v.value


def ngram_info(lm: NgramTables):
    n, b = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().ngram_info(lm.h, ctypes.byref(n), ctypes.byref(b)))
    return n.value, b.value


def boost_build(vocab, blank_id, tokens, offsets, completion=None, token_score=1.0,
                stream=None) -> BoostTrie:
    toks = np.ascontiguousarray(tokens, dtype=np.int32)
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    comp = None if completion is None else np.ascontiguousarray(completion, dtype=np.float32)
    out = ctypes.c_void_p()
    _check(lib().boost_build(int(vocab), int(blank_id), int(offs.size - 1), _ptr(toks), _ptr(offs),
                             _ptr(comp), float(token_score), _stream(stream), ctypes.byref(out)))
    return BoostTrie(out.value, int(vocab), int(blank_id))


def boost_build_phrases(vocab, blank_id, phrases, stream=None) -> BoostTrie:
    return boost_build(vocab, blank_id, phrases.tokens, phrases.offsets, phrases.completion,
                       phrases.token_score, stream)


def boost_info(trie: BoostTrie):
    n, d, b = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
    _check(lib().boost_info(trie.h, ctypes.byref(n), ctypes.byref(d), ctypes.byref(b)))
    return n.value, d.value, b.value


def _h(x):
    return None if x is None else x.h


def fusion_step(lm, trie, logits, lm_state, boost_state, H, V, lam, beta, blank_id, k, blank_mode,
                fused, tokens, scores, next_lm, next_boost, stream=None):
    """Same arguments as the C call; tensors are CUDA (HIP) tensors."""
    _check(lib().fusion_step(_h(lm), _h(trie), _ptr(logits), _ptr(lm_state), _ptr(boost_state),
                             int(H), int(V), float(lam), float(beta), int(blank_id), int(k),
                             int(blank_mode), _ptr(fused), _ptr(tokens), _ptr(scores),
                             _ptr(next_lm), _ptr(next_boost), _stream(stream)))


def fusion_run(lm, trie, logits, T, S, B, V, k, lam, beta, blank_id, blank_mode, lm_state,
               boost_state, hyp_score, tokens, parents, fused=None, traffic=None, stream=None):
    """Same arguments as the C call; tensors are CUDA (HIP) tensors."""
    _check(lib().fusion_run(_h(lm), _h(trie), _ptr(logits), int(T), int(S), int(B), int(V), int(k),
                            float(lam), float(beta), int(blank_id), int(blank_mode), _ptr(lm_state),
                            _ptr(boost_state), _ptr(hyp_score), _ptr(tokens), _ptr(parents),
                            _ptr(fused), _ptr(traffic), _stream(stream)))


def _lm_arrays(lms, alphas):
    """Host arrays of handles and weights for the several-LM calls."""
    lms, alphas = list(lms), [float(a) for a in alphas]
    if len(lms) != len(alphas):
        raise ValueError("one weight per LM")
    hs = (ctypes.c_void_p * max(1, len(lms)))(*[m.h.value for m in lms])
    al = np.array(alphas if alphas else [0.0], dtype=np.float32)
    return hs, al, len(lms)


def fusion_step_lms(lms, alphas, trie, logits, lm_state, boost_state, H, V, beta, blank_id, k,
                    blank_mode, fused, tokens, scores, next_lm, next_boost, stream=None):
    """Same arguments as the C call; lms and alphas are Python sequences,
    tensors are CUDA (HIP) tensors (lm_state [n_lm, H], next_lm [n_lm, H, k])."""
    hs, al, n = _lm_arrays(lms, alphas)
    _check(lib().fusion_step_lms(ctypes.cast(hs, ctypes.c_void_p), _ptr(al), n, _h(trie), _ptr(logits),
                                 _ptr(lm_state), _ptr(boost_state), int(H), int(V), float(beta),
                                 int(blank_id), int(k), int(blank_mode), _ptr(fused), _ptr(tokens),
                                 _ptr(scores), _ptr(next_lm), _ptr(next_boost), _stream(stream)))


def fusion_run_lms(lms, alphas, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                   boost_state, hyp_score, tokens, parents, fused=None, traffic=None, flags=0, hist=None,
                   stream=None):
    """Same arguments as the C call; lms and alphas are Python sequences,
    tensors are CUDA (HIP) tensors (lm_state [n_lm, S*B], hist [S*B] int64)."""
    hs, al, n = _lm_arrays(lms, alphas)
    _check(lib().fusion_run_lms(ctypes.cast(hs, ctypes.c_void_p), _ptr(al), n, _h(trie), _ptr(logits),
                                int(T), int(S), int(B), int(V), int(k), float(beta), int(blank_id),
                                int(blank_mode), _ptr(lm_state), _ptr(boost_state), _ptr(hyp_score),
                                _ptr(tokens), _ptr(parents), _ptr(fused), _ptr(traffic), int(flags),
                                _ptr(hist), _stream(stream)))


def fusion_run_lms_noalloc(lms, alphas, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                           boost_state, hyp_score, tokens, parents, fused=None, traffic=None, flags=0, hist=None,
                           stream=None):
    """fusion_run_lms through the entry point that allocates no device memory
    (its beam exchange lives in the library's static per-GPU scratch)."""
    hs, al, n = _lm_arrays(lms, alphas)
    _check(lib().fusion_run_lms_noalloc(ctypes.cast(hs, ctypes.c_void_p), _ptr(al), n, _h(trie), _ptr(logits),
                                        int(T), int(S), int(B), int(V), int(k), float(beta), int(blank_id),
                                        int(blank_mode), _ptr(lm_state), _ptr(boost_state), _ptr(hyp_score),
                                        _ptr(tokens), _ptr(parents), _ptr(fused), _ptr(traffic), int(flags),
                                        _ptr(hist), _stream(stream)))


def fusion_run_projected(lms, alphas, trie, A, W, bias, K, logits, chunk, T, S, B, V, k, beta, blank_id, blank_mode,
                         lm_state, boost_state, hyp_score, tokens, parents, flags=0, hist=None, stream=None):
    """Same arguments as the C call: A [T, S*B, K] and W [V, K] bf16 (int16 bit
    patterns), logits a [chunk, S*B, V] float32 workspace; CUDA (HIP) tensors."""
    hs, al, n = _lm_arrays(lms, alphas)
    _check(lib().fusion_run_projected(ctypes.cast(hs, ctypes.c_void_p), _ptr(al), n, _h(trie), _ptr(A), _ptr(W),
                                      _ptr(bias), int(K), _ptr(logits), int(chunk), int(T), int(S), int(B), int(V), int(k),
                                      float(beta), int(blank_id), int(blank_mode), _ptr(lm_state), _ptr(boost_state),
                                      _ptr(hyp_score), _ptr(tokens), _ptr(parents), int(flags), _ptr(hist),
                                      _stream(stream)))


def fusion_end_scores(lms, alphas, lm_state, H, hyp_score=None, end_term=None, stream=None):
    """Same arguments as the C call; lm_state [n_lm, H] int32, hyp_score / end_term
    [H] float64 CUDA tensors (either may be None, not both)."""
    hs, al, n = _lm_arrays(lms, alphas)
    _check(lib().fusion_end_scores(ctypes.cast(hs, ctypes.c_void_p), _ptr(al), n, _ptr(lm_state), int(H),
                                   _ptr(hyp_score), _ptr(end_term), _stream(stream)))


def joint_project(A, W, bias, M, N, K, out, stream=None):
    """Same arguments as the C call; A and W are int16/uint16 (bf16 bit patterns) or
    bfloat16 CUDA tensors, bias and out float32 CUDA tensors."""
    _check(lib().joint_project(_ptr(A), _ptr(W), _ptr(bias), int(M), int(N), int(K), _ptr(out),
                               _stream(stream)))


def fusion_device_status(stream=None) -> int:
    v = ctypes.c_int32()
    _check(lib().fusion_device_status(_stream(stream), ctypes.byref(v)))
    return v.value


# ---------------------------------------------------------------------------
# conveniences that allocate the outputs with torch (still no compute here)
# ---------------------------------------------------------------------------
def step(lm, trie, logits, lm_state, boost_state, lam, beta, blank_id, k, blank_mode,
         want_fused=False, stream=None):
    import torch

    H, V = logits.shape
    dev = logits.device
    out = dict(
        tokens=torch.empty((H, k), dtype=torch.int32, device=dev),
        scores=torch.empty((H, k), dtype=torch.float32, device=dev),
        next_lm=torch.empty((H, k), dtype=torch.int32, device=dev),
        next_boost=torch.empty((H, k), dtype=torch.int32, device=dev),
        fused=torch.empty((H, V), dtype=torch.float32, device=dev) if want_fused else None,
    )
    fusion_step(lm, trie, logits, lm_state, boost_state, H, V, lam, beta, blank_id, k, blank_mode,
                out["fused"], out["tokens"], out["scores"], out["next_lm"], out["next_boost"], stream)
    return out


def project(A, W, bias=None, stream=None):
    """logits [M, N] fp32 of A [M, K] and W [N, K] (bf16 CUDA tensors)."""
    import torch

    M, K = A.shape
    N = W.shape[0]
    out = torch.empty((M, N), dtype=torch.float32, device=A.device)
    joint_project(A, W, bias, M, N, K, out, stream)
    return out


def run(lm, trie, logits, S, B, k, lam, beta, blank_id, blank_mode, lm_state, boost_state,
        hyp_score=None, want_fused=False, traffic=None, stream=None):
    """Decode all frames of logits [T, S*B, V]; lm_state / boost_state /
    hyp_score are updated in place (they are the carried decoder state)."""
    import torch

    T, H, V = logits.shape
    dev = logits.device
    tokens = torch.empty((T, H), dtype=torch.int32, device=dev)
    parents = torch.empty((T, H), dtype=torch.int32, device=dev) if B > 1 else None
    fused = torch.zeros((T, H, V), dtype=torch.float32, device=dev) if want_fused else None
    fusion_run(lm, trie, logits, T, S, B, V, k, lam, beta, blank_id, blank_mode, lm_state,
               boost_state, hyp_score, tokens, parents, fused, traffic, stream)
    return dict(tokens=tokens, parents=parents, fused=fused)


def step_lms(lms, alphas, trie, logits, lm_state, boost_state, beta, blank_id, k, blank_mode,
             want_fused=False, stream=None):
    """``step`` with several LMs: lm_state [n_lm, H]; next_lm comes back [n_lm, H, k]."""
    import torch

    H, V = logits.shape
    dev = logits.device
    n = len(lms)
    out = dict(
        tokens=torch.empty((H, k), dtype=torch.int32, device=dev),
        scores=torch.empty((H, k), dtype=torch.float32, device=dev),
        next_lm=torch.empty((n, H, k), dtype=torch.int32, device=dev),
        next_boost=torch.empty((H, k), dtype=torch.int32, device=dev),
        fused=torch.empty((H, V), dtype=torch.float32, device=dev) if want_fused else None,
    )
    fusion_step_lms(lms, alphas, trie, logits, lm_state, boost_state, H, V, beta, blank_id, k,
                    blank_mode, out["fused"], out["tokens"], out["scores"], out["next_lm"],
                    out["next_boost"], stream)
    return out


def run_lms(lms, alphas, trie, logits, S, B, k, beta, blank_id, blank_mode, lm_state, boost_state,
            hyp_score=None, want_fused=False, traffic=None, recombine=False, hist=None, stream=None):
    """``run`` with several LMs: lm_state [n_lm, S*B] is updated in place;
    ``recombine`` merges beam candidates that reach the same history (``hist``,
    an int64 [S*B] tensor or None, carries the history hashes across calls)."""
    import torch

    T, H, V = logits.shape
    dev = logits.device
    tokens = torch.empty((T, H), dtype=torch.int32, device=dev)
    parents = torch.empty((T, H), dtype=torch.int32, device=dev) if B > 1 else None
    fused = torch.zeros((T, H, V), dtype=torch.float32, device=dev) if want_fused else None
    fusion_run_lms(lms, alphas, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                   boost_state, hyp_score, tokens, parents, fused, traffic,
                   FUSION_RUN_RECOMBINE if recombine else 0, hist, stream)
    return dict(tokens=tokens, parents=parents, fused=fused)
