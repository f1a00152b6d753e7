"""GPU parity of the top-k selection on key patterns that stress how the
kernel narrows its candidates: every key equal, the best keys all in one
64-lane wave, equal wave maxima, equal keys at the boundary of the top k,
and random keys; at vocabularies of 16, 4 and 1 waves per hypothesis, k = 4
and 8, with and without the LM and boost terms.  Ties go to the lowest id on
both sides, so tokens must be equal."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from workloads import tiny_random_lm, tiny_random_phrases

pytestmark = pytest.mark.gpu

SCORE_TOL = 1e-5


def wave_tokens(V, w):
    """Token ids held by wave w of a hypothesis (one 4-token strip per lane)."""
    W = 1024 if V > 1024 else (256 if V > 256 else 64)
    lanes = np.arange(64)
    toks = ((w * 64 + lanes)[:, None] * 4 + np.arange(4)[None, :]).ravel()
    return toks[toks < V], W // 64


def patterns(V, k, rng):
    rows = []
    rows.append(np.zeros(V, np.float32))                                   # every key equal
    x = rng.standard_normal(V).astype(np.float32)
    t1, nw = wave_tokens(V, min(3, (V // 256) - 1) if V >= 512 else 0)
    x[t1[5:5 + k + 3]] = 9.0 + np.arange(k + 3, dtype=np.float32) * 0.25  # best keys in one wave
    rows.append(x)
    x = rng.standard_normal(V).astype(np.float32)
    x[t1[7:7 + k + 2]] = 9.0                                              # equal keys, one wave
    rows.append(x)
    x = (rng.standard_normal(V) * 0.1).astype(np.float32)
    for w in range(nw):                                                   # equal wave maxima
        tw, _ = wave_tokens(V, w)
        if tw.size:
            x[tw[(w * 7) % tw.size]] = 4.0
    rows.append(x)
    x = rng.integers(-3, 3, size=V).astype(np.float32)                    # many ties at the boundary
    rows.append(x)
    for _ in range(3):
        rows.append((rng.standard_normal(V) * 2).astype(np.float32))      # random
    return np.stack(rows)


@pytest.mark.parametrize("V", [4096, 1000, 200])
@pytest.mark.parametrize("k", [4, 8])
@pytest.mark.parametrize("terms", ["none", "lm_boost"])
def test_topk_patterns(V, k, terms):
    mode = 1  # blank competes (k > 1 needs it)
    rng = np.random.default_rng(V * 31 + k)
    lm = tiny_random_lm(rng, V, 3, n_sent=3000, len_range=(1, 10))
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=min(V - 1, 30), with_completion=True)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    x = patterns(V, k, rng)
    H = x.shape[0]
    lam, beta = (0.0, 0.0) if terms == "none" else (0.5, 0.5)
    ls = np.full(H, V, np.int32)
    bs = np.zeros(H, np.int32)
    g = F.step(glm, gtr, torch.from_numpy(x).to("cuda:0"), torch.from_numpy(ls).to("cuda:0"),
               torch.from_numpy(bs).to("cuda:0"), lam, beta, 0, k, mode)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.step(olm, otr, x, ls, bs, lam, beta, 0, k, mode)
    assert np.array_equal(g["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"])
    assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"])
    gs = g["scores"].cpu().numpy().astype(np.float64)
    fin = np.isfinite(r["scores"])
    assert np.array_equal(np.isfinite(gs), fin)
    assert np.abs(gs[fin] - r["scores"][fin]).max() <= SCORE_TOL
