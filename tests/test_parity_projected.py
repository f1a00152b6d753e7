"""GPU parity of the frame loop with the joint projection as its producer
(fusion_run_projected): per chunk of frames (one frame, five frames with a
ragged last chunk, all frames), the MFMA projection of the hypotheses' joint
states feeds the chunk's fusion steps.  It must equal the joint projection of
all frames at once followed by one fusion_run bit for bit (tokens, parents,
final states and scores; the chunk's projection itself equals the batched
rows), and
the decode of those GPU-produced logits must be the oracle's: the oracle replays
every decision on the same logits (their own parity, against the fp64 product,
is tests/test_projection.py's)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from workloads import make_projection, tiny_random_lm, tiny_random_phrases
from workloads.gen import to_bf16_bits

pytestmark = pytest.mark.gpu

SCORE_TOL = 1e-5
TIE_TOL = 1e-4


def dev():
    return torch.device("cuda:0")


@pytest.mark.parametrize("chunk", [1, 5, 14])
@pytest.mark.parametrize("S,B,k", [(8, 4, 4), (24, 1, 1)])
def test_projected_loop_equals_batched(S, B, k, chunk):
    rng = np.random.default_rng(600 + B)
    V, K, T = 1024, 640, 14
    H = S * B
    lm = tiny_random_lm(rng, V, 4, n_sent=3000)
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=30)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    A = to_bf16_bits(rng.standard_normal((T * H, K), dtype=np.float32))
    W = to_bf16_bits(rng.standard_normal((V, K), dtype=np.float32) * np.float32(2.0 / np.sqrt(K)))
    bias = (rng.standard_normal(V, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
    bias[0] += 2.0
    a_d = torch.from_numpy(A.view(np.int16)).to(dev())
    w_d = torch.from_numpy(W.view(np.int16)).to(dev())
    b_d = torch.from_numpy(bias).to(dev())
    mode = F.FUSION_BLANK_COMPETE if B > 1 else F.FUSION_BLANK_AM
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)

    def fresh():
        return (torch.full((1, H), V, dtype=torch.int32, device=dev()), torch.zeros((H,), dtype=torch.int32, device=dev()),
                torch.from_numpy(sc0.copy()).to(dev()) if B > 1 else None)

    # batched: all frames' logits, then one decode
    logits = F.project(a_d, w_d, b_d).view(T, H, V)
    ls1, bs1, sc1 = fresh()
    one = F.run_lms([glm], [0.5], gtr, logits, S, B, k, 0.5, 0, mode, ls1, bs1, sc1)
    # per frame: projection of the frame, then the frame's fusion step
    ls2, bs2, sc2 = fresh()
    tok = torch.empty((T, H), dtype=torch.int32, device=dev())
    par = torch.empty((T, H), dtype=torch.int32, device=dev()) if B > 1 else None
    work = torch.empty((chunk, H, V), dtype=torch.float32, device=dev())
    F.fusion_run_projected([glm], [0.5], gtr, a_d.view(T, H, K), w_d, b_d, K, work, chunk, T, S, B, V, k, 0.5, 0,
                           mode, ls2, bs2, sc2, tok, par)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    last = T - (T - 1) % chunk - 1  # first frame of the last chunk
    assert torch.equal(work[:T - last], logits[last:])  # the chunk's projection equals the batched rows
    assert torch.equal(tok, one["tokens"])
    if B > 1:
        assert torch.equal(par, one["parents"]) and torch.equal(sc2, sc1)
    assert torch.equal(ls2, ls1) and torch.equal(bs2, bs1)
    # the oracle on the GPU-produced logits
    x = logits.cpu().numpy()
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    if B > 1:
        r = oracle.run(olm, otr, x, S, B, k, 0.5, 0.5, 0, 1, [V] * H, [0] * H, sc0,
                       forced_tokens=tok.cpu().numpy(), forced_parents=par.cpu().numpy(), tol=TIE_TOL, threads=8)
        assert (r["mismatch_at"] < 0).all() and int(r["near_ties"].sum()) == 0
        fin = np.isfinite(r["hyp_score"])
        assert np.abs(sc2.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
    else:
        r = oracle.run(olm, otr, x, S, 1, 1, 0.5, 0.5, 0, 0, [V] * H, [0] * H, threads=8)
        assert np.array_equal(tok.cpu().numpy(), r["tokens"])
    assert np.array_equal(ls2.cpu().numpy()[0], r["lm_state"])
    assert np.array_equal(bs2.cpu().numpy(), r["boost_state"])


def test_projected_loop_rejects_bad_arguments():
    rng = np.random.default_rng(1)
    V = 300
    glm = F.ngram_load_arrays(tiny_random_lm(rng, V, 3, n_sent=200))
    ls = torch.full((1, 4), V, dtype=torch.int32, device=dev())
    with pytest.raises(F.FusionError):
        F.fusion_run_projected([glm], [0.5], None, None, None, None, 64, None, 1, 3, 4, 1, V, 1, 0.5, 0, 0, ls, None,
                               None, torch.empty((3, 4), dtype=torch.int32, device=dev()), None)
    with pytest.raises(F.FusionError, match="chunk"):
        F.fusion_run_projected([glm], [0.5], None, None, None, None, 64, None, 0, 0, 4, 1, V, 1, 0.5, 0, 0, ls, None,
                               None, None, None)
    # nothing to do: no buffer is touched
    F.fusion_run_projected([glm], [0.5], None, None, None, None, 64, None, 1, 0, 4, 1, V, 1, 0.5, 0, 0, ls, None, None,
                           None, None)
