"""GPU parity of the context rows (contexts of two or more tokens with many
successors, whose LM row is loaded whole instead of scattered arc by arc).

The C5 model has such contexts at its default threshold; here the threshold
is lowered with FUSION_CONTEXT_ROW_MIN_ARCS so that small models have many of
them at every level, and the fusion path must still agree with the oracle
(which knows nothing of the layout): step-wise at random states of every
order, free-running greedy, and a teacher-forced beam, with one and with two
LMs (context rows serve the first LM; the second scatters every level)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from workloads import tiny_random_lm, tiny_random_phrases

pytestmark = pytest.mark.gpu

SCORE_TOL = 1e-5
TIE_TOL = 1e-4


def dev():
    return torch.device("cuda:0")


def load_with_rows(lm, min_arcs, monkeypatch):
    """The model loaded twice: with context rows above min_arcs successors and
    without any (threshold above every fan-out); the first must hold more
    device memory, i.e. it really has rows."""
    monkeypatch.setenv("FUSION_CONTEXT_ROW_MIN_ARCS", str(min_arcs))
    g = F.ngram_load_arrays(lm)
    monkeypatch.setenv("FUSION_CONTEXT_ROW_MIN_ARCS", str(1 << 30))
    g0 = F.ngram_load_arrays(lm)
    monkeypatch.delenv("FUSION_CONTEXT_ROW_MIN_ARCS")
    assert F.ngram_info(g)[1] > F.ngram_info(g0)[1]
    g0.close()
    return g


def random_states(lm, n, rng):
    V = lm.vocab
    ids = [V] + [int(t) for t in rng.integers(1, V, size=n // 4)]
    off = V + 2
    for k in range(2, lm.order):
        nk = lm.tokens[k - 1].shape[0]
        ids += [off + int(i) for i in rng.integers(0, nk, size=n // 2)]
        off += nk
    return rng.choice(np.array(ids), size=n).astype(np.int32)


@pytest.mark.parametrize("V,N,min_arcs", [(300, 5, 6), (1500, 4, 12), (200, 6, 3)])
@pytest.mark.parametrize("mode,k", [(0, 1), (1, 4)])
def test_step_at_random_states(V, N, min_arcs, mode, k, monkeypatch):
    rng = np.random.default_rng(V + N + k)
    lm = tiny_random_lm(rng, V, N, n_sent=4000, cutoffs=tuple([1] * N))
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=20)
    glm, gtr = load_with_rows(lm, min_arcs, monkeypatch), F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    H = 300
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    x[:, 0] += 2
    ls = random_states(lm, H, rng)
    bs = rng.integers(0, otr.n_nodes, size=H).astype(np.int32)
    g = F.step(glm, gtr, torch.from_numpy(x).to(dev()), torch.from_numpy(ls).to(dev()),
               torch.from_numpy(bs).to(dev()), 0.5, 0.5, 0, k, mode, want_fused=True)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.step(olm, otr, x, ls, bs, 0.5, 0.5, 0, k, mode)
    assert np.array_equal(g["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"])
    assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"])
    assert np.abs(g["fused"].cpu().numpy().astype(np.float64) - r["fused"]).max() <= SCORE_TOL


@pytest.mark.parametrize("V,N,min_arcs", [(300, 5, 6), (1500, 4, 12)])
def test_greedy_free_running(V, N, min_arcs, monkeypatch):
    rng = np.random.default_rng(7 * V + N)
    lm = tiny_random_lm(rng, V, N, n_sent=4000, cutoffs=tuple([1] * N))
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=20)
    glm, gtr = load_with_rows(lm, min_arcs, monkeypatch), F.boost_build_phrases(V, 0, ph)
    S, T = 40, 60
    x = (rng.standard_normal((T, S, V)) * 2).astype(np.float32)
    x[:, :, 0] += 1
    ls = torch.full((S,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((S,), dtype=torch.int32, device=dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, 1, 1, 0.5, 0.5, 0, F.FUSION_BLANK_AM, ls, bs)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, S, 1, 1, 0.5, 0.5, 0, 0, [V] * S, [0] * S,
                   threads=8)
    assert np.array_equal(out["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])


@pytest.mark.parametrize("n_lm", [1, 2])
def test_teacher_forced_beam(n_lm, monkeypatch):
    rng = np.random.default_rng(41 + n_lm)
    V, S, B, k, T = 700, 16, 4, 4, 50
    lms = [tiny_random_lm(rng, V, 5, n_sent=5000, cutoffs=(1,) * 5), tiny_random_lm(rng, V, 4, n_sent=3000)][:n_lm]
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=30)
    glms = [load_with_rows(lms[0], 5, monkeypatch)] + [F.ngram_load_arrays(m) for m in lms[1:]]
    gtr = F.boost_build_phrases(V, 0, ph)
    H = S * B
    x = (rng.standard_normal((T, H, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    alphas = [0.5, 0.25][:n_lm]
    ls = torch.full((n_lm, H), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0, F.FUSION_BLANK_COMPETE,
                    ls, bs, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run_lms([oracle.OracleLM(m) for m in lms], alphas, oracle.OracleTrie(V, 0, ph), x, S, B, k, 0.5,
                       0, 1, [[V] * H] * n_lm, [0] * H, sc0, forced_tokens=out["tokens"].cpu().numpy(),
                       forced_parents=out["parents"].cpu().numpy(), tol=TIE_TOL, threads=8)
    assert (r["mismatch_at"] < 0).all(), f"diverge at {r['mismatch_at'][r['mismatch_at'] >= 0][:5]}"
    assert int(r["near_ties"].sum()) == 0
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
