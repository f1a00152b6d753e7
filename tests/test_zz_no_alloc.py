"""GPU check of fusion_run_lms_noalloc, the entry point that allocates no
device memory: on two calls in a row (the second with fewer streams, a
narrower beam and fewer frames, so the static scratch holds the first call's
records when it starts), its tokens, parents, final states and scores equal
those of fusion_run_lms on the same inputs, bit for bit, with and without
recombination; a greedy call (no scratch) agrees too."""

import numpy as np
import pytest
import torch

import paper_2609_14991_amd as F
from workloads import tiny_random_lm, tiny_random_phrases

pytestmark = pytest.mark.gpu


def dev():
    return torch.device("cuda:0")


def _decode(fn, glm, gtr, x, S, B, k, V, flags):
    H = S * B
    T = x.shape[0]
    ls = torch.full((1, H), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev()) if B > 1 else None
    hh = torch.zeros((H,), dtype=torch.int64, device=dev()) if flags else None
    tok = torch.full((T, H), -7, dtype=torch.int32, device=dev())
    par = torch.full((T, H), -7, dtype=torch.int32, device=dev()) if B > 1 else None
    mode = F.FUSION_BLANK_COMPETE if B > 1 else F.FUSION_BLANK_AM
    fn([glm], [0.5], gtr, x, T, S, B, V, k, 0.5, 0, mode, ls, bs, sc, tok, par, None, None, flags, hh)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    return [t.cpu() for t in (tok, par, ls, bs, sc, hh) if t is not None]


@pytest.mark.parametrize("flags", [0, F.FUSION_RUN_RECOMBINE])
def test_noalloc_equals_allocating_entry_point(flags):
    rng = np.random.default_rng(313)
    V = 300
    glm = F.ngram_load_arrays(tiny_random_lm(rng, V, 4, n_sent=3000))
    gtr = F.boost_build_phrases(V, 0, tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=30))
    for S, B, k, T in [(40, 4, 4, 30), (9, 2, 3, 11)]:
        x = torch.from_numpy((rng.standard_normal((T, S * B, V)) * 2).astype(np.float32)).to(dev())
        a = _decode(F.fusion_run_lms_noalloc, glm, gtr, x, S, B, k, V, flags)
        b = _decode(F.fusion_run_lms, glm, gtr, x, S, B, k, V, flags)
        for u, v in zip(a, b):
            assert torch.equal(u, v), (S, B, k, T)
        print(f"no-alloc beam S={S} B={B} k={k} T={T} flags={flags}: equal", flush=True)


def test_noalloc_greedy_equals_allocating_entry_point():
    rng = np.random.default_rng(314)
    V = 500
    glm = F.ngram_load_arrays(tiny_random_lm(rng, V, 3, n_sent=2000))
    gtr = F.boost_build_phrases(V, 0, tiny_random_phrases(rng, V, n=20, max_len=4, alphabet=40))
    x = torch.from_numpy((rng.standard_normal((25, 17, V)) * 2).astype(np.float32)).to(dev())
    a = _decode(F.fusion_run_lms_noalloc, glm, gtr, x, 17, 1, 1, V, 0)
    b = _decode(F.fusion_run_lms, glm, gtr, x, 17, 1, 1, V, 0)
    for u, v in zip(a, b):
        assert torch.equal(u, v)
