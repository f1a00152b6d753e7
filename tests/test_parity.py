"""GPU parity: the HIP fusion path against the CPU oracle on the same seeded
inputs.  Bar: tokens, top-k sets and orders, and next LM / phrase state ids
bit-exact; fp32 fused scores within 1e-5 of the oracle's fp64 reference;
beam merges exact except near ties (fp64 scores at the boundary within
1e-4), which are accepted and counted."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from workloads import Phrases, load_workload, tiny_random_lm, tiny_random_phrases

pytestmark = pytest.mark.gpu

SCORE_TOL = 1e-5
TIE_TOL = 1e-4


def dev():
    return torch.device("cuda:0")


class Env:
    """A workload with its GPU handles and oracle twins."""

    def __init__(self, w):
        self.w = w
        self.lm = F.ngram_load_arrays(w.lm)
        self.trie = F.boost_build_phrases(w.V, w.blank, w.phrases)
        self.olm = oracle.OracleLM(w.lm)
        self.otr = oracle.OracleTrie(w.V, w.blank, w.phrases)
        self.bos = F.ngram_bos_state(self.lm)


@pytest.fixture(scope="module")
def c1():
    return Env(load_workload(1))


@pytest.fixture(scope="module")
def c2():
    return Env(load_workload(2))


def context_states(env, n, rng):
    """n LM state ids drawn over every order of context (plus <s>)."""
    lm = env.w.lm
    V = lm.vocab
    ids = [V]
    ids += [int(t) for t in rng.choice(lm.tokens[0][:, 0], size=n // 3) if t not in (V + 1,)]
    off = V + 2
    for k in range(2, lm.order):
        nk = lm.tokens[k - 1].shape[0]
        if nk:
            ids += [off + int(i) for i in rng.integers(0, nk, size=n // 3)]
        off += nk
    ids = np.array(ids, dtype=np.int64)
    return rng.choice(ids, size=n).astype(np.int32)


def check_step(env, x, ls, bs, lam, beta, k, mode, label):
    w = env.w
    H, V = x.shape
    xd = torch.from_numpy(x).to(dev())
    lsd = torch.from_numpy(ls).to(dev())
    bsd = torch.from_numpy(bs).to(dev())
    g = F.step(env.lm, env.trie, xd, lsd, bsd, lam, beta, w.blank, k, mode, want_fused=True)
    torch.cuda.synchronize()
    r = oracle.step(env.olm, env.otr, x, ls, bs, lam, beta, w.blank, k, mode)
    tok = g["tokens"].cpu().numpy()
    assert np.array_equal(tok, r["tokens"]), f"{label}: tokens"
    assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"]), f"{label}: next LM states"
    assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"]), f"{label}: next phrase states"
    err = np.abs(g["fused"].cpu().numpy().astype(np.float64) - r["fused"]).max()
    assert err <= SCORE_TOL, f"{label}: fused max err {err}"
    serr = np.abs(g["scores"].cpu().numpy().astype(np.float64) - r["scores"]).max()
    assert serr <= SCORE_TOL, f"{label}: scores max err {serr}"
    assert F.fusion_device_status() == 0


@pytest.mark.parametrize("mode,k", [(0, 1), (1, 1), (1, 4), (1, 8)])
def test_step_random_states_c1(c1, mode, k):
    rng = np.random.default_rng(10 + k + mode)
    H = 300
    x = (rng.standard_normal((H, c1.w.V)) * 2).astype(np.float32)
    x[:, 0] += 2
    ls = context_states(c1, H, rng)
    bs = rng.integers(0, c1.otr.n_nodes, size=H).astype(np.int32)
    check_step(c1, x, ls, bs, c1.w.lam, c1.w.beta, k, mode, f"c1 mode {mode} k {k}")


@pytest.mark.parametrize("mode,k", [(0, 1), (1, 4)])
def test_step_random_states_c2(c2, mode, k):
    rng = np.random.default_rng(20 + k + mode)
    H = 257
    x = (rng.standard_normal((H, c2.w.V)) * 2).astype(np.float32)
    x[:, 0] += 2
    ls = context_states(c2, H, rng)
    bs = rng.integers(0, c2.otr.n_nodes, size=H).astype(np.int32)
    check_step(c2, x, ls, bs, 0.5, 0.5, k, mode, f"c2 mode {mode} k {k}")


def test_c1_greedy_free_running(c1):
    """C1 in full: one stream, 200 frames, greedy; the whole trajectory and the
    final states equal the oracle's, which decodes from full histories."""
    w = c1.w
    ls = torch.full((1,), c1.bos, dtype=torch.int32, device=dev())
    bs = torch.zeros((1,), dtype=torch.int32, device=dev())
    out = F.run(c1.lm, c1.trie, torch.from_numpy(w.logits).to(dev()), 1, 1, 1, w.lam, w.beta,
                w.blank, F.FUSION_BLANK_AM, ls, bs)
    r = oracle.run(c1.olm, c1.otr, w.logits, 1, 1, 1, w.lam, w.beta, w.blank, 0, [c1.bos], [0])
    tok = out["tokens"].cpu().numpy()
    assert np.array_equal(tok, r["tokens"])
    assert int(ls.cpu()[0]) == r["lm_state"][0] and int(bs.cpu()[0]) == r["boost_state"][0]
    assert (tok != 0).sum() > 100  # the LM state really advances


def test_c2_stream_in_13_frame_chunks(c2):
    """C2: 1000 frames fed in 13-frame chunks with the states carried across
    calls, against one oracle decode over all frames."""
    w = c2.w
    x = torch.from_numpy(w.logits).to(dev())
    ls = torch.full((1,), c2.bos, dtype=torch.int32, device=dev())
    bs = torch.zeros((1,), dtype=torch.int32, device=dev())
    toks = []
    for a in range(0, w.T, w.chunk):
        out = F.run(c2.lm, c2.trie, x[a:a + w.chunk], 1, 1, 1, w.lam, w.beta, w.blank,
                    F.FUSION_BLANK_AM, ls, bs)
        toks.append(out["tokens"])
    tok = torch.cat(toks).cpu().numpy()
    r = oracle.run(c2.olm, c2.otr, w.logits, 1, 1, 1, w.lam, w.beta, w.blank, 0, [c2.bos], [0])
    assert np.array_equal(tok, r["tokens"])
    assert int(ls.cpu()[0]) == r["lm_state"][0] and int(bs.cpu()[0]) == r["boost_state"][0]


def test_long_run_past_the_lds_stamp_period():
    """One launch of 33068 frames: the LDS rows of explicit arcs and phrase
    transitions carry a frame stamp that repeats every 32768 frames, so the run
    crosses the point where they are cleared; every token and the final states
    equal the oracle's."""
    rng = np.random.default_rng(91)
    V, S, T = 300, 2, 32768 + 300
    lm = tiny_random_lm(rng, V, 4, n_sent=2000)
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=20, with_completion=True)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    x = (rng.standard_normal((T, S, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    ls = torch.full((S,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((S,), dtype=torch.int32, device=dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, 1, 1, 0.5, 0.5, 0, F.FUSION_BLANK_AM, ls, bs)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run(olm, otr, x, S, 1, 1, 0.5, 0.5, 0, 0, [V] * S, [0] * S, threads=2)
    tok = out["tokens"].cpu().numpy()
    assert (tok[32768:] != 0).sum() > 100  # states keep moving after the wrap
    bad = np.argwhere(tok != r["tokens"])
    assert bad.size == 0, f"first mismatch (frame, stream) {bad[0]}"
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])


def test_c3_batched_greedy_prefix():
    """C3 (64 streams, 10% peaked rows): the first 60 frames of every stream."""
    w = load_workload(3, T=60)
    env = Env(w)
    x = torch.from_numpy(w.logits).to(dev())
    ls = torch.full((w.H,), env.bos, dtype=torch.int32, device=dev())
    bs = torch.zeros((w.H,), dtype=torch.int32, device=dev())
    out = F.run(env.lm, env.trie, x, w.S, 1, 1, w.lam, w.beta, w.blank, F.FUSION_BLANK_AM, ls, bs)
    r = oracle.run(env.olm, env.otr, w.logits, w.S, 1, 1, w.lam, w.beta, w.blank, 0,
                   [env.bos] * w.H, [0] * w.H, threads=8)
    assert np.array_equal(out["tokens"].cpu().numpy(), r["tokens"])
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    assert (bs.cpu().numpy() != 0).any()


def beam_stepwise(env, x, S, B, k, lam, beta, frames):
    """Chained single-frame beam launches, each checked against the oracle
    given the same incoming states and scores (teacher forcing); returns the
    GPU trajectory and the number of accepted near ties."""
    w = env.w
    H = S * B
    ls = torch.full((H,), env.bos, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0).to(dev())
    xd = torch.from_numpy(x).to(dev())
    toks, pars, near = [], [], 0
    for t in range(frames):
        ls_in, bs_in, sc_in = ls.cpu().numpy().copy(), bs.cpu().numpy().copy(), sc.cpu().numpy().copy()
        out = F.run(env.lm, env.trie, xd[t:t + 1], S, B, k, lam, beta, w.blank,
                    F.FUSION_BLANK_COMPETE, ls, bs, sc)
        gt, gp = out["tokens"].cpu().numpy(), out["parents"].cpu().numpy()
        r = oracle.run(env.olm, env.otr, x[t:t + 1], S, B, k, lam, beta, w.blank, 1, ls_in, bs_in,
                       sc_in, forced_tokens=gt, forced_parents=gp, tol=TIE_TOL, threads=8)
        bad = np.nonzero(r["mismatch_at"] >= 0)[0]
        assert bad.size == 0, f"frame {t}: streams {bad[:8]} disagree beyond near ties"
        near += int(r["near_ties"].sum())
        assert np.array_equal(ls.cpu().numpy(), r["lm_state"]), f"frame {t}: LM states"
        assert np.array_equal(bs.cpu().numpy(), r["boost_state"]), f"frame {t}: phrase states"
        gs = sc.cpu().numpy()
        live = np.isfinite(r["hyp_score"])
        assert np.array_equal(live, np.isfinite(gs))
        assert np.abs(gs[live] - r["hyp_score"][live]).max() <= SCORE_TOL
        toks.append(gt)
        pars.append(gp)
    return np.concatenate(toks), np.concatenate(pars), ls, bs, sc, near


def test_beam_teacher_forced_c2_lm(c2):
    """Beam of 4, top-4 per hypothesis, 8 streams, on the C2 model."""
    w = c2.w
    S, B, k, T = 8, 4, 4, 30
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((T, S * B, w.V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    toks, pars, ls, bs, sc, near = beam_stepwise(c2, x, S, B, k, 0.5, 0.5, T)
    # one launch over all frames reproduces the chained launches bit for bit
    ls2 = torch.full((S * B,), c2.bos, dtype=torch.int32, device=dev())
    bs2 = torch.zeros((S * B,), dtype=torch.int32, device=dev())
    sc2 = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev())
    out = F.run(c2.lm, c2.trie, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0.5, w.blank,
                F.FUSION_BLANK_COMPETE, ls2, bs2, sc2)
    assert np.array_equal(out["tokens"].cpu().numpy(), toks)
    assert np.array_equal(out["parents"].cpu().numpy(), pars)
    assert torch.equal(ls, ls2) and torch.equal(bs, bs2) and torch.equal(sc, sc2)


def test_exhaustive_beam_gpu():
    """V = 3, B = 27, k = 3: every path survives; final scores equal the
    oracle's sums over all 27 paths."""
    V, T, B, k = 3, 3, 27, 3
    rng = np.random.default_rng(11)
    lm = tiny_random_lm(rng, V, 3, n_sent=30)
    ph = Phrases(tokens=np.array([1, 2, 2, 1, 1], np.int32), offsets=np.array([0, 2, 5], np.int64))
    xs = (rng.standard_normal((T, 1, V)) * 2).astype(np.float32)
    x = np.repeat(xs, B, axis=1)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    ls = torch.full((B,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((B,), dtype=torch.int32, device=dev())
    sc = torch.from_numpy(np.array([0.0] + [-np.inf] * (B - 1))).to(dev())
    F.run(glm, gtr, torch.from_numpy(x).to(dev()), 1, B, k, 0.5, 0.5, 0, 1, ls, bs, sc)
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, 1, B, k, 0.5, 0.5, 0, 1,
                   [V] * B, [0] * B)
    got = np.sort(sc.cpu().numpy())[::-1]
    ref = np.sort(r["hyp_score"])[::-1]
    assert np.isfinite(got).all() and np.abs(got - ref).max() <= T * SCORE_TOL


@pytest.mark.parametrize("V", [3, 130, 1001])
def test_ragged_vocab_tiny_models(V):
    """Vocabularies that are not multiples of the 4-token lane strip or of
    the 1024-token slot width, with random small models and phrase lists."""
    rng = np.random.default_rng(V)
    lm = tiny_random_lm(rng, V, 4, n_sent=400 if V > 10 else 60)
    ph = tiny_random_phrases(rng, V, n=12, max_len=4, alphabet=min(V - 1, 6), with_completion=True)
    w = type("W", (), {})()
    w.lm, w.phrases, w.V, w.blank = lm, ph, V, 0
    env = Env(w)
    H = 70
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    ls = context_states(env, H, rng)
    bs = rng.integers(0, env.otr.n_nodes, size=H).astype(np.int32)
    for mode, k in [(0, 1), (1, min(V, 4))]:
        check_step(env, x, ls, bs, 0.7, 1.3, k, mode, f"V {V} mode {mode}")


def test_no_trie_and_empty_list(c1):
    w = c1.w
    rng = np.random.default_rng(3)
    H = 50
    x = (rng.standard_normal((H, w.V)) * 2).astype(np.float32)
    ls = context_states(c1, H, rng)
    xd, lsd = torch.from_numpy(x).to(dev()), torch.from_numpy(ls).to(dev())
    g = F.step(c1.lm, None, xd, lsd, None, w.lam, w.beta, 0, 4, 1, want_fused=True)
    empty = Phrases(tokens=np.zeros(0, np.int32), offsets=np.zeros(1, np.int64))
    etr = F.boost_build_phrases(w.V, 0, empty)
    z = torch.zeros(H, dtype=torch.int32, device=dev())
    g2 = F.step(c1.lm, etr, xd, lsd, z, w.lam, w.beta, 0, 4, 1, want_fused=True)
    r = oracle.step(c1.olm, None, x, ls, [0] * H, w.lam, w.beta, 0, 4, 1)
    for gg in (g, g2):
        assert np.array_equal(gg["tokens"].cpu().numpy(), r["tokens"])
        assert np.array_equal(gg["next_lm"].cpu().numpy(), r["next_lm"])
        assert np.abs(gg["fused"].cpu().numpy() - r["fused"]).max() <= SCORE_TOL
    assert (g2["next_boost"].cpu().numpy() == 0).all()


def test_invalid_states_flag_and_emit_blank(c1):
    w = c1.w
    x = np.zeros((3, w.V), np.float32)
    x[:, 5] = 3.0
    ls = torch.tensor([c1.bos, 10 ** 8, 0], dtype=torch.int32, device=dev())  # ok, out of range, blank id
    bs = torch.tensor([10 ** 6, 0, 0], dtype=torch.int32, device=dev())        # bad, ok, ok
    g = F.step(c1.lm, c1.trie, torch.from_numpy(x).to(dev()), ls, bs, w.lam, w.beta, 0, 1, 1)
    st = F.fusion_device_status()
    assert st == F.FUSION_STATUS_BAD_LM_STATE | F.FUSION_STATUS_BAD_BOOST_STATE
    assert (g["tokens"].cpu().numpy()[:, 0] == 0).all()
    assert np.array_equal(g["next_lm"].cpu().numpy()[:, 0], ls.cpu().numpy())
    assert F.fusion_device_status() == 0  # cleared by the read


def test_argument_errors_on_device(c1):
    w = c1.w
    x = torch.zeros((2, w.V), device=dev())
    s = torch.zeros(2, dtype=torch.int32, device=dev())
    with pytest.raises(F.FusionError) as e:
        F.step(c1.lm, c1.trie, x, s, s, 0.5, 0.5, 0, 4, F.FUSION_BLANK_AM)
    assert e.value.code == F.FUSION_E_ARG
    with pytest.raises(F.FusionError):
        F.step(c1.lm, c1.trie, torch.zeros((2, w.V + 1), device=dev()), s, s, 0.5, 0.5, 0, 1, 0)


def test_repeat_runs_are_identical(c2):
    w = c2.w
    S, B, k, T = 4, 4, 4, 20
    x = torch.from_numpy(np.ascontiguousarray(w.logits[:T, :1].repeat(S * B, axis=1))).to(dev())
    res = []
    for _ in range(2):
        ls = torch.full((S * B,), c2.bos, dtype=torch.int32, device=dev())
        bs = torch.zeros((S * B,), dtype=torch.int32, device=dev())
        sc = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev())
        out = F.run(c2.lm, c2.trie, x, S, B, k, 0.5, 0.5, 0, 1, ls, bs, sc, want_fused=True)
        res.append((out["tokens"].cpu(), out["parents"].cpu(), out["fused"].cpu(), ls.cpu(), sc.cpu()))
    for a, b in zip(*res):
        assert torch.equal(a, b)


def test_beam_in_several_launch_batches():
    """More streams than the device holds at once (160 x 4 workgroups of 1024
    lanes, 2.5 times the 256 CUs): the run is split into launch batches of
    what fits, whose rendezvous buffers and arrival counters are cleared in
    between.  Every decision is replayed by the oracle."""
    rng = np.random.default_rng(80)
    V, S, B, k, T = 1100, 160, 4, 4, 12
    lm = tiny_random_lm(rng, V, 4, n_sent=3000)
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=min(V - 1, 30), with_completion=True)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    x = (rng.standard_normal((T, S * B, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    H = S * B
    ls = torch.full((H,), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run(glm, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0.5, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run(olm, otr, x, S, B, k, 0.5, 0.5, 0, 1, [V] * H, [0] * H, sc0,
                   forced_tokens=out["tokens"].cpu().numpy(), forced_parents=out["parents"].cpu().numpy(),
                   tol=TIE_TOL, threads=8)
    assert (r["mismatch_at"] < 0).all()
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.array_equal(np.isfinite(sc.cpu().numpy()), fin)
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
