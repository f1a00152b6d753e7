"""GPU parity of the several-LM form of Eq. (1) (Sec. III-C: one weighted LM
term per model, each model with its own state) against the oracle's
``step_lms`` / ``run_lms``.  Same bar as the one-LM path: tokens, top-k sets
and every LM's next state bit-exact, fp32 fused scores within 1e-5, beam
merges exact except accepted near ties."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from workloads import load_workload, tiny_random_lm, tiny_random_phrases

pytestmark = pytest.mark.gpu

SCORE_TOL = 1e-5
TIE_TOL = 1e-4


def dev():
    return torch.device("cuda:0")


def random_states(lm, n, rng):
    """n LM state ids over every order of context (plus <s>)."""
    V = lm.vocab
    ids = [V] + [int(t) for t in lm.tokens[0][:, 0] if t != V + 1 and t != lm.blank]
    off = V + 2
    for k in range(2, lm.order):
        nk = lm.tokens[k - 1].shape[0]
        ids += [off + i for i in range(nk) if lm.tokens[k - 1][i, -1] != V + 1]
        off += nk
    return rng.choice(np.array(ids, dtype=np.int64), size=n).astype(np.int32)


def check_step(lms_arr, ph, x, states, bs, alphas, beta, k, mode, label):
    V = x.shape[1]
    glms = [F.ngram_load_arrays(m) for m in lms_arr]
    gtr = F.boost_build_phrases(V, 0, ph)
    olms = [oracle.OracleLM(m) for m in lms_arr]
    otr = oracle.OracleTrie(V, 0, ph)
    g = F.step_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), torch.from_numpy(states).to(dev()),
                   torch.from_numpy(bs).to(dev()), beta, 0, k, mode, want_fused=True)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.step_lms(olms, alphas, otr, x, states, bs, beta, 0, k, mode)
    assert np.array_equal(g["tokens"].cpu().numpy(), r["tokens"]), f"{label}: tokens"
    assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"]), f"{label}: next LM states"
    assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"]), f"{label}: next phrase states"
    err = np.abs(g["fused"].cpu().numpy().astype(np.float64) - r["fused"]).max()
    assert err <= SCORE_TOL, f"{label}: fused max err {err}"
    serr = np.abs(g["scores"].cpu().numpy().astype(np.float64) - r["scores"]).max()
    assert serr <= SCORE_TOL, f"{label}: scores max err {serr}"


@pytest.mark.parametrize("V,H", [(200, 40), (1000, 64), (4000, 48)])
def test_step_two_lms_random_states(V, H):
    """Two LMs of different orders in random states of every order, at the three
    workgroup shapes (64, 256 and 1024 lanes): full fused rows, top-4 in mode B
    and the acoustic-blank mode A."""
    rng = np.random.default_rng(V)
    lms = [tiny_random_lm(rng, V, 4, n_sent=3000), tiny_random_lm(rng, V, 3, n_sent=1500)]
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=min(V - 1, 30), with_completion=True)
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    x[:, 0] += 2
    states = np.stack([random_states(m, H, rng) for m in lms])
    nodes = oracle.OracleTrie(V, 0, ph).n_nodes
    bs = rng.integers(0, nodes, size=H).astype(np.int32)
    for mode, k in [(1, 4), (0, 1)]:
        check_step(lms, ph, x, states, bs, [0.5, 0.3], 0.5, k, mode, f"V {V} mode {mode} k {k}")


def test_second_lm_with_zero_weight_is_the_one_lm_kernel():
    """alpha_2 = 0: the two-LM kernel's keys, selections and first-LM states
    equal the one-LM kernel's bit for bit."""
    w = load_workload(2, T=1)
    rng = np.random.default_rng(4)
    other = tiny_random_lm(rng, w.V, 3, n_sent=2000)
    glm, glm2 = F.ngram_load_arrays(w.lm), F.ngram_load_arrays(other)
    gtr = F.boost_build_phrases(w.V, 0, w.phrases)
    H = 128
    x = torch.from_numpy((rng.standard_normal((H, w.V)) * 2).astype(np.float32)).to(dev())
    s1 = random_states(w.lm, H, rng)
    s2 = random_states(other, H, rng)
    bs = torch.zeros(H, dtype=torch.int32, device=dev())
    one = F.step(glm, gtr, x, torch.from_numpy(s1).to(dev()), bs, 0.5, 0.5, 0, 4, F.FUSION_BLANK_COMPETE,
                 want_fused=True)
    two = F.step_lms([glm, glm2], [0.5, 0.0], gtr, x, torch.from_numpy(np.stack([s1, s2])).to(dev()), bs,
                     0.5, 0, 4, F.FUSION_BLANK_COMPETE, want_fused=True)
    torch.cuda.synchronize()
    assert torch.equal(one["tokens"], two["tokens"])
    assert torch.equal(one["fused"], two["fused"])
    assert torch.equal(one["next_lm"], two["next_lm"][0])
    assert torch.equal(one["next_boost"], two["next_boost"])


def test_greedy_two_lms_free_running_c1():
    """C1 in full with a second LM: one stream, 200 frames, greedy mode A; the
    trajectory and both final LM states equal the oracle's."""
    w = load_workload(1)
    other = tiny_random_lm(np.random.default_rng(21), w.V, 4, n_sent=4000)
    glms = [F.ngram_load_arrays(w.lm), F.ngram_load_arrays(other)]
    gtr = F.boost_build_phrases(w.V, 0, w.phrases)
    ls = torch.full((2, 1), w.V, dtype=torch.int32, device=dev())
    bs = torch.zeros((1,), dtype=torch.int32, device=dev())
    alphas = [w.lam, 0.2]
    out = F.run_lms(glms, alphas, gtr, torch.from_numpy(w.logits).to(dev()), 1, 1, 1, w.beta, 0,
                    F.FUSION_BLANK_AM, ls, bs)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run_lms([oracle.OracleLM(w.lm), oracle.OracleLM(other)], alphas,
                       oracle.OracleTrie(w.V, 0, w.phrases), w.logits, 1, 1, 1, w.beta, 0, 0,
                       [[w.V], [w.V]], [0])
    tok = out["tokens"].cpu().numpy()
    assert np.array_equal(tok, r["tokens"])
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert int(bs.cpu()[0]) == r["boost_state"][0]
    assert (tok != 0).sum() > 100


@pytest.mark.parametrize("V,S", [(300, 24), (1100, 40)])
def test_beam_two_lms_teacher_forced(V, S):
    """Beam 4, top-4, 30 frames with two LMs: every decision is replayed by the
    oracle (near ties within 1e-4 accepted); both LMs' final states, the
    phrase states and the final scores match."""
    rng = np.random.default_rng(70 + V)
    B, k, T = 4, 4, 30
    lms = [tiny_random_lm(rng, V, 4, n_sent=3000), tiny_random_lm(rng, V, 3, n_sent=2000)]
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=min(V - 1, 30), with_completion=True)
    glms = [F.ngram_load_arrays(m) for m in lms]
    gtr = F.boost_build_phrases(V, 0, ph)
    x = (rng.standard_normal((T, S * B, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    H = S * B
    alphas = [0.5, 0.25]
    ls = torch.full((2, H), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0,
                    F.FUSION_BLANK_COMPETE, ls, bs, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run_lms([oracle.OracleLM(m) for m in lms], alphas, oracle.OracleTrie(V, 0, ph), x, S, B,
                       k, 0.5, 0, 1, [[V] * H, [V] * H], [0] * H, sc0,
                       forced_tokens=out["tokens"].cpu().numpy(),
                       forced_parents=out["parents"].cpu().numpy(), tol=TIE_TOL, threads=8)
    assert (r["mismatch_at"] < 0).all(), f"streams diverge at {r['mismatch_at'][r['mismatch_at'] >= 0][:5]}"
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.array_equal(np.isfinite(sc.cpu().numpy()), fin)
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL


def test_two_lms_above_4096_tokens_are_unsupported():
    rng = np.random.default_rng(1)
    V = 5000
    lms = [F.ngram_load_arrays(tiny_random_lm(rng, V, 2, n_sent=200)) for _ in range(2)]
    x = torch.zeros((1, V), dtype=torch.float32, device=dev())
    ls = torch.full((2, 1), V, dtype=torch.int32, device=dev())
    with pytest.raises(F.FusionError) as e:
        F.step_lms(lms, [0.5, 0.5], None, x, ls, None, 0.0, 0, 1, F.FUSION_BLANK_COMPETE)
    assert e.value.code == F.FUSION_E_UNSUPPORTED


def test_end_scores_random_states():
    """End-of-stream </s> terms at random states of every order, one and two
    LMs: the GPU adds exactly what the oracle adds (same fp32 recursion and
    product, same fp64 additions), dead slots stay -inf."""
    rng = np.random.default_rng(31)
    V, H = 1000, 300
    lms = [tiny_random_lm(rng, V, 5, n_sent=4000), tiny_random_lm(rng, V, 3, n_sent=2000)]
    glms = [F.ngram_load_arrays(m) for m in lms]
    olms = [oracle.OracleLM(m) for m in lms]
    states = np.stack([random_states(m, H, rng) for m in lms])
    sc0 = rng.standard_normal(H) * 10
    sc0[::7] = -np.inf
    for n, alphas in [(1, [0.5]), (2, [0.5, 0.3])]:
        sc = torch.from_numpy(sc0.copy()).to(dev())
        term = torch.empty(H, dtype=torch.float64, device=dev())
        F.fusion_end_scores(glms[:n], alphas, torch.from_numpy(states[:n].copy()).to(dev()), H, sc, term)
        torch.cuda.synchronize()
        assert F.fusion_device_status() == 0
        want_sc, want_term = oracle.end_scores(olms[:n], alphas, states[:n], sc0)
        assert np.array_equal(term.cpu().numpy(), want_term)
        assert np.array_equal(sc.cpu().numpy(), want_sc)


def test_end_scores_after_a_beam_run():
    """A 30-frame two-LM beam, then the end-of-stream terms on its final
    states: the completed scores equal the oracle's completion of its own
    replay (within the beam's score tolerance) and every slot's ranking by
    completed score is the oracle's."""
    rng = np.random.default_rng(33)
    V, S, B, k, T = 500, 8, 4, 4, 30
    lms = [tiny_random_lm(rng, V, 4, n_sent=3000), tiny_random_lm(rng, V, 3, n_sent=2000)]
    ph = tiny_random_phrases(rng, V, n=30, max_len=4, alphabet=30, with_completion=True)
    glms = [F.ngram_load_arrays(m) for m in lms]
    gtr = F.boost_build_phrases(V, 0, ph)
    H = S * B
    x = (rng.standard_normal((T, H, V)) * 2).astype(np.float32)
    x[:, :, 0] += 2
    alphas = [0.5, 0.25]
    ls = torch.full((2, H), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0, F.FUSION_BLANK_COMPETE,
                    ls, bs, sc)
    F.fusion_end_scores(glms, alphas, ls, H, sc)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    olms = [oracle.OracleLM(m) for m in lms]
    r = oracle.run_lms(olms, alphas, oracle.OracleTrie(V, 0, ph), x, S, B, k, 0.5, 0, 1, [[V] * H, [V] * H],
                       [0] * H, sc0, forced_tokens=out["tokens"].cpu().numpy(),
                       forced_parents=out["parents"].cpu().numpy(), tol=TIE_TOL, threads=8)
    assert (r["mismatch_at"] < 0).all()
    want, _ = oracle.end_scores(olms, alphas, r["lm_state"], r["hyp_score"])
    got = sc.cpu().numpy()
    assert np.abs(got - want).max() <= T * SCORE_TOL
    for s in range(S):
        assert np.array_equal(np.argsort(-got[s * B:(s + 1) * B], kind="stable"),
                              np.argsort(-want[s * B:(s + 1) * B], kind="stable"))


def test_end_scores_flag_invalid_states():
    rng = np.random.default_rng(35)
    V = 300
    glm = F.ngram_load_arrays(tiny_random_lm(rng, V, 3, n_sent=500))
    states = torch.tensor([[V, 0, V + 1, 5]], dtype=torch.int32, device=dev())  # <s>, blank, </s>, token 5
    term = torch.zeros(4, dtype=torch.float64, device=dev())
    F.fusion_end_scores([glm], [1.0], states, 4, None, term)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == F.FUSION_STATUS_BAD_LM_STATE
    t = term.cpu().numpy()
    assert t[1] == 0.0 and t[2] == 0.0 and t[0] < 0 and t[3] < 0
    assert F.fusion_device_status() == 0  # cleared by the read


def test_recombining_beam_exhaustive():
    """V = 3, T = 3, B = 27, k = 3 with recombination: every distinct history
    survives (15), and the GPU's merged scores equal the oracle's (the
    log-sum over each history's alignments)."""
    V, T, B, k = 3, 3, 27, 3
    rng = np.random.default_rng(14)
    lms = [tiny_random_lm(rng, V, 3, n_sent=30), tiny_random_lm(rng, V, 2, n_sent=30)]
    ph = tiny_random_phrases(rng, V, n=2, max_len=3, alphabet=2)
    xs = (rng.standard_normal((T, 1, V)) * 2).astype(np.float32)
    x = np.repeat(xs, B, axis=1)
    for n in (1, 2):
        glms = [F.ngram_load_arrays(m) for m in lms[:n]]
        ls = torch.full((n, B), V, dtype=torch.int32, device=dev())
        bs = torch.zeros((B,), dtype=torch.int32, device=dev())
        sc = torch.from_numpy(np.array([0.0] + [-np.inf] * (B - 1))).to(dev())
        F.run_lms(glms, [0.5, 0.25][:n], F.boost_build_phrases(V, 0, ph), torch.from_numpy(x).to(dev()), 1, B, k,
                  0.5, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc, recombine=True)
        torch.cuda.synchronize()
        assert F.fusion_device_status() == 0
        r = oracle.run_lms([oracle.OracleLM(m) for m in lms[:n]], [0.5, 0.25][:n], oracle.OracleTrie(V, 0, ph),
                           x, 1, B, k, 0.5, 0, 1, [[V] * B] * n, [0] * B, recombine=True)
        got = sc.cpu().numpy()
        assert np.isfinite(got).sum() == 15
        assert np.abs(np.sort(got[np.isfinite(got)]) - np.sort(r["hyp_score"][np.isfinite(r["hyp_score"])])).max() \
            <= T * SCORE_TOL


@pytest.mark.parametrize("n_lm", [1, 2])
def test_recombining_beam_teacher_forced(n_lm):
    """Beam 4, top-4, 40 frames with recombination: every decision (merged
    candidates included) is replayed by the oracle, which compares full
    histories; final states and scores match."""
    rng = np.random.default_rng(90 + n_lm)
    V, S, B, k, T = 300, 24, 4, 4, 40
    lms = [tiny_random_lm(rng, V, 4, n_sent=3000), tiny_random_lm(rng, V, 3, n_sent=2000)][:n_lm]
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=30, with_completion=True)
    glms = [F.ngram_load_arrays(m) for m in lms]
    gtr = F.boost_build_phrases(V, 0, ph)
    H = S * B
    x = (rng.standard_normal((T, H, V)) * 2).astype(np.float32)
    x[:, :, 0] += 3
    alphas = [0.5, 0.25][:n_lm]
    ls = torch.full((n_lm, H), V, dtype=torch.int32, device=dev())
    bs = torch.zeros((H,), dtype=torch.int32, device=dev())
    sc0 = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)
    sc = torch.from_numpy(sc0.copy()).to(dev())
    out = F.run_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), S, B, k, 0.5, 0, F.FUSION_BLANK_COMPETE,
                    ls, bs, sc, recombine=True)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    r = oracle.run_lms([oracle.OracleLM(m) for m in lms], alphas, oracle.OracleTrie(V, 0, ph), x, S, B, k, 0.5,
                       0, 1, [[V] * H] * n_lm, [0] * H, sc0, forced_tokens=out["tokens"].cpu().numpy(),
                       forced_parents=out["parents"].cpu().numpy(), tol=TIE_TOL, threads=8, recombine=True)
    assert (r["mismatch_at"] < 0).all(), f"diverge at {r['mismatch_at'][r['mismatch_at'] >= 0][:5]}"
    assert np.array_equal(ls.cpu().numpy(), r["lm_state"])
    assert np.array_equal(bs.cpu().numpy(), r["boost_state"])
    fin = np.isfinite(r["hyp_score"])
    assert np.array_equal(np.isfinite(sc.cpu().numpy()), fin)
    assert np.abs(sc.cpu().numpy()[fin] - r["hyp_score"][fin]).max() <= T * SCORE_TOL
    # recombination changed the search: the same run without it differs
    r0 = oracle.run_lms([oracle.OracleLM(m) for m in lms], alphas, oracle.OracleTrie(V, 0, ph), x, S, B, k, 0.5,
                        0, 1, [[V] * H] * n_lm, [0] * H, sc0, threads=8)
    assert not np.array_equal(r0["hyp_score"], r["hyp_score"])


def test_recombining_beam_chunked_equals_one_call():
    """A recombining beam decoded in 13-frame chunks, with the states, scores
    and history hashes carried from call to call (the streaming use of
    Sec. IV-A), gives exactly the tokens, parents, states and scores of one
    call over all frames; the one call is the oracle-checked decode above."""
    rng = np.random.default_rng(97)
    V, S, B, k, T = 300, 24, 4, 4, 40
    lm = tiny_random_lm(rng, V, 4, n_sent=3000)
    ph = tiny_random_phrases(rng, V, n=40, max_len=4, alphabet=30, with_completion=True)
    glm, gtr = F.ngram_load_arrays(lm), F.boost_build_phrases(V, 0, ph)
    H = S * B
    x = (rng.standard_normal((T, H, V)) * 2).astype(np.float32)
    x[:, :, 0] += 3
    xd = torch.from_numpy(x).to(dev())
    sc0 = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev())

    def fresh():
        return (torch.full((1, H), V, dtype=torch.int32, device=dev()), torch.zeros((H,), dtype=torch.int32, device=dev()),
                sc0.clone(), torch.zeros((H,), dtype=torch.int64, device=dev()))

    ls, bs, sc, hh = fresh()
    one = F.run_lms([glm], [0.5], gtr, xd, S, B, k, 0.5, 0, F.FUSION_BLANK_COMPETE, ls, bs, sc, recombine=True, hist=hh)
    ls2, bs2, sc2, hh2 = fresh()
    toks, pars = [], []
    for t0 in range(0, T, 13):
        o = F.run_lms([glm], [0.5], gtr, xd[t0:t0 + 13].contiguous(), S, B, k, 0.5, 0, F.FUSION_BLANK_COMPETE,
                      ls2, bs2, sc2, recombine=True, hist=hh2)
        toks.append(o["tokens"])
        pars.append(o["parents"])
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    assert torch.equal(torch.cat(toks), one["tokens"])
    assert torch.equal(torch.cat(pars), one["parents"])
    assert torch.equal(ls2, ls) and torch.equal(bs2, bs) and torch.equal(hh2, hh)
    assert torch.equal(sc2, sc)
    assert bool((hh != 0).all())
