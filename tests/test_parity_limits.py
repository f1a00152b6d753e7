"""GPU parity at the limits of the build, against the CPU oracle: the largest
vocabulary (V = 8190, two 4-token strips per lane), the largest candidate set
of a beam merge (B = 32 slots x k = 8), a vocabulary just above one strip per
lane (V = 4097), and empty runs."""

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


def states_of_every_order(lm, n, rng):
    V = lm.vocab
    ids = [V] + [int(t) for t in lm.tokens[0][:, 0] if t not in (V + 1, lm.blank)]
    off = V + 2
    for k in range(2, lm.order):
        nk = lm.tokens[k - 1].shape[0]
        ids += [off + i for i in range(nk) if lm.tokens[k - 1][i, -1] != V + 1]
        off += nk
    return rng.choice(np.array(ids, dtype=np.int64), size=n).astype(np.int32)


def models(V, seed):
    rng = np.random.default_rng(seed)
    lm = tiny_random_lm(rng, V, 4, n_sent=6000, len_range=(1, 12))
    ph = tiny_random_phrases(rng, V, n=60, max_len=5, alphabet=min(V - 1, 40), with_completion=True)
    return rng, lm, ph


@pytest.mark.parametrize("V", [4097, 8190])
def test_step_large_vocab(V):
    """Random states of every order, full fused rows, modes A and B."""
    rng, lm, ph = models(V, V)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    H = 40
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    x[:, 0] += 2
    ls = states_of_every_order(lm, H, rng)
    bs = rng.integers(0, otr.n_nodes, size=H).astype(np.int32)
    for mode, k in [(1, 8), (0, 1)]:
        g = F.step(glm, gtr, torch.from_numpy(x).to(dev()), torch.from_numpy(ls).to(dev()),
                   torch.from_numpy(bs).to(dev()), 0.5, 0.5, 0, k, mode, want_fused=True)
        torch.cuda.synchronize()
        assert F.fusion_device_status() == 0
        r = oracle.step(olm, otr, x, ls, bs, 0.5, 0.5, 0, k, mode)
        assert np.array_equal(g["tokens"].cpu().numpy(), r["tokens"])
        assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"])
        assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"])
        assert np.abs(g["fused"].cpu().numpy().astype(np.float64) - r["fused"]).max() <= SCORE_TOL
        assert np.abs(g["scores"].cpu().numpy().astype(np.float64) - r["scores"]).max() <= SCORE_TOL


def _beam_vs_oracle(V, S, B, k, T, seed):
    rng, lm, ph = models(V, seed)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    H = S * B
    x = (rng.standard_normal((T, H, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    ls = torch.full((H,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0.5, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, S, B, k, 0.5, 0.5, 0, 1, [V] * H,
                   [0] * H, sc0, forced_tokens=out["tokens"].cpu().numpy(),
                   forced_parents=out["parents"].cpu().numpy(), tol=TIE_TOL, threads=8)
    assert (r["mismatch_at"] < 0).all(), f"diverge at {r['mismatch_at'][r['mismatch_at'] >= 0][:5]}"
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.array_equal(np.isfinite(sc.cpu().numpy()), fin)
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
    return out


def test_beam_largest_vocab():
    """V = 8190 (two strips per lane), 8 streams x beam 4, top-4, 20 frames."""
    _beam_vs_oracle(8190, 8, 4, 4, 20, 3)


def test_beam_largest_candidate_set():
    """B = 32 slots x k = 8: 256 candidates per stream merge (four 64-lane
    chunks of the rendezvous), 4 streams, 16 frames."""
    out = _beam_vs_oracle(600, 4, 32, 8, 16, 5)
    par = out["parents"].cpu().numpy()
    assert (par[-1] >= 0).all()  # every slot alive at the end
    assert len(np.unique(par[-1])) > 1


def test_greedy_largest_vocab():
    """V = 8190, 6 streams, 60 frames of greedy mode A from <s>."""
    V, S, T = 8190, 6, 60
    rng, lm, ph = models(V, 9)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    x = (rng.standard_normal((T, S, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    ls = torch.full((S,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((S,), dtype=torch.int32, device=dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, 1, 1, 0.5, 0.5, 0, F.FUSION_BLANK_AM, ls, bs)
    torch.cuda.synchronize()
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, S, 1, 1, 0.5, 0.5, 0, 0, [V] * S,
                   [0] * S, threads=6)
    assert np.array_equal(out["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])


def test_zero_frames_change_nothing():
    rng, lm, ph = models(130, 2)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(130, 0, ph)
    ls = torch.full((4,), 130, dtype=torch.int32, device=dev())
    bs = torch.zeros((4,), dtype=torch.int32, device=dev())
    sc = torch.tensor([0.0, -np.inf, -1.5, -2.0], dtype=torch.float64, device=dev())
    x = torch.zeros((0, 4, 130), dtype=torch.float32, device=dev())
    out = F.run(glm, gtr, x, 1, 4, 4, 0.5, 0.5, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc)
    torch.cuda.synchronize()
    assert out["tokens"].numel() == 0
    assert (ls.cpu().numpy() == 130).all() and (bs.cpu().numpy() == 0).all()
    assert sc.cpu().numpy()[0] == 0.0 and sc.cpu().numpy()[2] == -1.5


def test_empty_batches_touch_nothing():
    """H == 0 (step) and S == 0 (run) check the handles and scalars, then
    return without reading or writing a buffer; bad scalars still fail."""
    rng, lm, ph = models(130, 4)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(130, 0, ph)
    e32 = torch.empty((0,), dtype=torch.int32, device=dev())
    g = F.step(glm, gtr, torch.empty((0, 130), device=dev()), e32, e32, 0.5, 0.5, 0, 4, 1)
    assert g["tokens"].shape == (0, 4)
    x = torch.empty((5, 0, 130), device=dev())
    out = F.run(glm, gtr, x, 0, 4, 4, 0.5, 0.5, 0, F.FUSION_BLANK_COMPETE, e32, e32,
                torch.empty((0,), dtype=torch.float64, device=dev()))
    assert out["tokens"].shape == (5, 0)
    with pytest.raises(F.FusionError):
        F.step(glm, gtr, torch.empty((0, 130), device=dev()), e32, e32, 0.5, 0.5, 0, 0, 1)  # k = 0
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0


@pytest.mark.parametrize("lam_beta", [(0.0, 0.0), (0.5, 0.5)])
def test_beam_exact_ties(lam_beta):
    """Integer-valued logits make many fused scores, and so many candidate
    totals, exactly equal: the beam's ranking must break them by candidate
    order (parent, then rank) and the top-k by token id, as the oracle does,
    in free-running decoding (no replay)."""
    lam, beta = lam_beta
    V, S, B, k, T = 130, 3, 4, 4, 12
    rng, lm, ph = models(V, 11)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    x = rng.integers(-2, 3, size=(T, S * B, V)).astype(np.float32)
    H = S * B
    ls = torch.full((H,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, B, k, lam, beta, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, S, B, k, lam, beta, 0, 1, [V] * H, [0] * H,
                   sc0)
    assert np.array_equal(out["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(out["parents"].cpu().numpy(), r["parents"])
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.array_equal(np.isfinite(sc.cpu().numpy()), fin)
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
