"""Pins for the oracle's several-LM form of Eq. (1) (Sec. III-C: one weighted
log-probability term per LM, each LM with its own state): hand-worked
values, reduction to the one-LM case, an independent Python statement, and
brute force over every beam path."""

import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import ref
from workloads import Phrases, load_workload, tiny_random_lm, tiny_random_phrases

from test_oracle import _all_context_tuples, hand_lm


def test_two_lm_hand_values():
    """The hand example LM twice, each copy in its own state: the fp64 fused
    score minus the log-softmax term is a1 ln p(y|ctx1) + a2 ln p(y|ctx2), with
    p the values worked by hand.  Unequal weights catch a swapped state or a
    dropped term."""
    g, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    hv = {(tuple(v["ctx"]), v["y"]): v["p"] for v in g["hand_values"]}
    ids = {tuple(t): sid for t, sid in g["state_ids"]["tuples"]}
    ids[(3,)] = 3  # a one-token context w has id w
    # (context of LM 1, context of LM 2, token, hand key of LM 2 when its context is not a state)
    cases = [((4, 1), (1, 2), 3, (1, 2)), ((1, 2), (4,), 3, (4,)), ((1, 2), (3,), 1, (2, 3))]
    a1, a2 = 0.7, 0.2
    x = np.array([[0.3, -1.0, 0.5, 2.0], [1.0, 0.0, -0.5, 0.25], [0.0, 1.5, -2.0, 0.5]], np.float32)
    ls = np.array([[ids[c[0]] for c in cases], [ids[c[1]] for c in cases]], np.int32)
    r = oracle.step_lms([olm, olm], [a1, a2], None, x, ls, [0, 0, 0], 0.0, 0, 1, 1)
    for h, (c1, c2, y, key2) in enumerate(cases):
        ls_term = float(x[h, y]) - (math.log(np.exp(x[h].astype(np.float64)).sum()))
        want = a1 * math.log(hv[(c1, y)]) + a2 * math.log(hv[(key2, y)])
        got = r["fused"][h, y] - ls_term
        assert got == pytest.approx(want, rel=1e-6, abs=1e-7), (c1, c2, y)


def test_second_lm_with_zero_weight_is_the_one_lm_step():
    """alpha_2 = 0 adds fl(0 * l) = 0 to every key: keys, fused scores and
    selections equal the one-LM step exactly; the second LM's next states are
    its own states after the selected token (brute force)."""
    w = load_workload(1, T=2)
    other = tiny_random_lm(np.random.default_rng(5), w.V, 4, n_sent=400)
    olm, olm2 = oracle.OracleLM(w.lm), oracle.OracleLM(other)
    otr = oracle.OracleTrie(w.V, 0, w.phrases)
    rlm2 = ref.RefLM(other)
    rng = np.random.default_rng(9)
    H = 8
    x = (rng.standard_normal((H, w.V)) * 2).astype(np.float32)
    s1 = [w.V, 5, 17, 3, w.V, 60, 9, 11]
    pool = _all_context_tuples(other)
    c2 = [pool[i] for i in rng.integers(0, len(pool), size=H)]
    s2 = [rlm2.state_id(c) for c in c2]
    for mode, k in [(1, 4), (0, 1)]:
        one = oracle.step(olm, otr, x, s1, [0] * H, 0.5, 0.5, 0, k, mode)
        two = oracle.step_lms([olm, olm2], [0.5, 0.0], otr, x, [s1, s2], [0] * H, 0.5, 0, k, mode)
        assert np.array_equal(one["key"], two["key"])
        assert np.array_equal(one["fused"], two["fused"])
        assert np.array_equal(one["tokens"], two["tokens"])
        assert np.array_equal(one["next_lm"], two["next_lm"][0])
        assert np.array_equal(one["next_boost"], two["next_boost"])
        for h in range(H):
            for j in range(k):
                y = int(two["tokens"][h, j])
                want = s2[h] if y == 0 else rlm2.state_after(tuple(c2[h]) + (y,))
                assert two["next_lm"][1, h, j] == want


@pytest.mark.parametrize("seed", range(5))
def test_c_oracle_matches_python_statement_two_lms(seed):
    """Two (or three) random LMs of different orders, each in a random state:
    the C oracle equals the independent Python statement (keys bit-exact,
    fused within 1e-12, selections and every LM's next state)."""
    rng = np.random.default_rng(300 + seed)
    V = int(rng.integers(4, 9))
    n_lm = 2 + seed % 2
    lms = [tiny_random_lm(rng, V, int(rng.integers(2, 5)), n_sent=50) for _ in range(n_lm)]
    ph = tiny_random_phrases(rng, V, n=4, max_len=3, alphabet=V - 1, with_completion=bool(seed % 2))
    olms = [oracle.OracleLM(m) for m in lms]
    rlms = [ref.RefLM(m) for m in lms]
    otr, rtr = oracle.OracleTrie(V, 0, ph), ref.RefTrie(ph)
    H = 6
    lams = [float(a) for a in rng.uniform(0, 1, size=n_lm)]
    beta = float(rng.uniform(0, 2))
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    ctxs = []
    for m in lms:
        pool = _all_context_tuples(m)
        ctxs.append([pool[i] for i in rng.integers(0, len(pool), size=H)])
    qs = [rtr.nodes[i] for i in rng.integers(0, len(rtr.nodes), size=H)]
    k = min(3, V)
    states = [[rlms[i].state_id(c) for c in ctxs[i]] for i in range(n_lm)]
    r = oracle.step_lms(olms, lams, otr, x, states, [rtr.index[q] for q in qs], beta, 0, k, 1)
    for h in range(H):
        key, fused, _ = ref.score_row_lms(rlms, lams, rtr, x[h], [c[h] for c in ctxs], qs[h], beta, 0)
        assert np.array_equal(r["key"][h], key)
        assert np.abs(r["fused"][h] - fused).max() < 1e-12
        sel = ref.select(x[h], key, 0, k, 1)
        assert r["tokens"][h].tolist() == sel
        for j, y in enumerate(sel):
            for i in range(n_lm):
                want = states[i][h] if y == 0 else rlms[i].state_after(tuple(ctxs[i][h]) + (y,))
                assert r["next_lm"][i, h, j] == want
            if y != 0:
                assert r["next_boost"][h, j] == rtr.index[rtr.state(tuple(qs[h]) + (y,))]


def test_two_lm_greedy_run_matches_stepwise():
    """Free-running greedy from full histories equals chaining single steps
    from state ids, for every LM's state."""
    w = load_workload(1, T=40)
    other = tiny_random_lm(np.random.default_rng(6), w.V, 3, n_sent=800)
    olms = [oracle.OracleLM(w.lm), oracle.OracleLM(other)]
    otr = oracle.OracleTrie(w.V, 0, w.phrases)
    lams = [0.3, 0.4]
    r = oracle.run_lms(olms, lams, otr, w.logits, 1, 1, 1, w.beta, 0, 0, [[w.V], [w.V]], [0])
    ls, bs = np.array([[w.V], [w.V]]), [0]
    for t in range(w.T):
        s = oracle.step_lms(olms, lams, otr, w.logits[t], ls, bs, w.beta, 0, 1, 0, want_rows=False)
        assert s["tokens"][0, 0] == r["tokens"][t, 0]
        ls, bs = s["next_lm"][:, :, 0], [s["next_boost"][0, 0]]
    assert np.array_equal(ls[:, 0], r["lm_state"][:, 0]) and bs[0] == r["boost_state"][0]
    assert (r["tokens"] != 0).sum() > 5


def test_two_lm_exhaustive_beam_keeps_every_path():
    """V = 3, T = 3, k = 3, B = 27 with two LMs: the beam keeps all 27 paths,
    so its final scores are the brute-force sums over each path of the Python
    statement's fused scores, every LM evaluated from its own full history."""
    V, T, B, k = 3, 3, 27, 3
    rng = np.random.default_rng(12)
    lms = [tiny_random_lm(rng, V, 3, n_sent=30), tiny_random_lm(rng, V, 2, n_sent=30)]
    ph = Phrases(tokens=np.array([1, 2, 2, 1, 1], np.int32), offsets=np.array([0, 2, 5], np.int64))
    xs = rng.standard_normal((T, 1, V)).astype(np.float32) * 2
    x = np.repeat(xs, B, axis=1)
    lams, beta = [0.5, 0.25], 0.5
    r = oracle.run_lms([oracle.OracleLM(m) for m in lms], lams, oracle.OracleTrie(V, 0, ph), x, 1,
                       B, k, beta, 0, 1, [[V] * B, [V] * B], [0] * B)
    rlms, rtr = [ref.RefLM(m) for m in lms], ref.RefTrie(ph)
    brute = []
    for path in itertools.product(range(V), repeat=T):
        hists, phh, tot = [[V], [V]], [], 0.0
        for t, y in enumerate(path):
            _, fused, _ = ref.score_row_lms(rlms, lams, rtr, xs[t, 0], hists, phh, beta, 0)
            tot += fused[y]
            if y != 0:
                for hh in hists:
                    hh.append(y)
                phh.append(y)
        brute.append(tot)
    assert np.allclose(np.sort(r["hyp_score"])[::-1], sorted(brute, reverse=True), atol=1e-9, rtol=0)


def test_end_scores_hand_values():
    """End of stream on the hand example LM: the </s> term of a state is
    alpha ln p(</s> | state) with the hand-worked probabilities (context (3):
    0.1; context (1 2): bo(1 2) * P(</s>|2) = 0.625 * 0.1), and with two LMs the
    terms add in order onto the running score (dead slots stay -inf)."""
    g, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    ids = {tuple(t): sid for t, sid in g["state_ids"]["tuples"]}
    s3, s12 = 3, ids[(1, 2)]
    sc, term = oracle.end_scores([olm], [0.5], [[s3, s12]], [-1.0, 2.0])
    assert term[0] == pytest.approx(0.5 * math.log(0.1), rel=1e-6)
    assert term[1] == pytest.approx(0.5 * math.log(0.625 * 0.1), rel=1e-6)
    assert np.array_equal(sc, np.array([-1.0, 2.0]) + term)
    sc2, term2 = oracle.end_scores([olm, olm], [0.5, 0.25], [[s3, s3, s12], [s12, s3, s3]],
                                   [0.0, -np.inf, 1.0])
    want0 = 0.5 * math.log(0.1) + 0.25 * math.log(0.0625)
    assert term2[0] == pytest.approx(want0, rel=1e-6)
    assert sc2[1] == -np.inf
    assert sc2[2] == pytest.approx(1.0 + 0.5 * math.log(0.0625) + 0.25 * math.log(0.1), rel=1e-6)
    with pytest.raises(oracle.OracleError):
        oracle.end_scores([olm], [0.5], [[0]])  # the blank state


def test_end_scores_complete_the_sentence_probability():
    """Summed over a token path, the LM terms of every step plus the </s> term
    give ln P(<s> path </s>) (alpha = 1, beta = 0, logits 0): the chain rule of
    the LM, checked against the product of hand-worked conditionals."""
    g, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    # <s> 1 2 3 </s>: P(1|<s>) P(2|<s> 1) P(3|1 2) P(</s>|2 3)
    p = 0.5 * 0.6 * 0.5 * (1.0 * 0.1)  # (2 3) absent: bo = 1, (3 </s>) absent: bo(3) = 1, P(</s>) = 0.1
    V = g["V"]
    x = np.zeros((1, V), np.float32)
    ls, tot = [g["BOS"]], 0.0
    lse = math.log(V)  # log-softmax of zero logits
    for y in g["path"]["tokens"]:
        r = oracle.step_lms([olm], [1.0], None, x, [ls], [0], 0.0, 0, V, 1)
        tot += r["fused"][0, y] + lse
        ls = [int(r["next_lm"][0, 0, list(r["tokens"][0]).index(y)])]
    _, term = oracle.end_scores([olm], [1.0], [ls])
    assert tot + term[0] == pytest.approx(math.log(p), rel=1e-6)


@pytest.mark.parametrize("n_lm", [1, 2])
def test_recombining_beam_is_the_forward_sum_per_history(n_lm):
    """V = 3, T = 3, k = 3, B = 27 with recombination: no frame has more
    distinct histories than slots (1, 3, 7, 15), so the beam is exact and each
    surviving slot's score is the log-sum, over every alignment (token path
    with blanks) that emits its history, of the path's score; the path scores
    come from the Python statement, each LM evaluated from its own history."""
    V, T, B, k = 3, 3, 27, 3
    rng = np.random.default_rng(14)
    lms = [tiny_random_lm(rng, V, 3, n_sent=30), tiny_random_lm(rng, V, 2, n_sent=30)][:n_lm]
    ph = Phrases(tokens=np.array([1, 2, 2, 1, 1], np.int32), offsets=np.array([0, 2, 5], np.int64))
    xs = rng.standard_normal((T, 1, V)).astype(np.float32) * 2
    x = np.repeat(xs, B, axis=1)
    lams, beta = [0.5, 0.25][:n_lm], 0.5
    r = oracle.run_lms([oracle.OracleLM(m) for m in lms], lams, oracle.OracleTrie(V, 0, ph), x, 1, B, k,
                       beta, 0, 1, [[V] * B] * n_lm, [0] * B, recombine=True)
    rlms, rtr = [ref.RefLM(m) for m in lms], ref.RefTrie(ph)
    per_history = {}
    for path in itertools.product(range(V), repeat=T):
        hists, phh, tot = [[V] for _ in range(n_lm)], [], 0.0
        for t, y in enumerate(path):
            _, fused, _ = ref.score_row_lms(rlms, lams, rtr, xs[t, 0], hists, phh, beta, 0)
            tot += fused[y]
            if y != 0:
                for hh in hists:
                    hh.append(y)
                phh.append(y)
        per_history.setdefault(tuple(phh), []).append(tot)
    want = sorted((float(np.logaddexp.reduce(v)) for v in per_history.values()), reverse=True)
    got = np.sort(r["hyp_score"][np.isfinite(r["hyp_score"])])[::-1]
    assert len(want) == 15 and got.size == 15
    assert np.allclose(got, want, atol=1e-9, rtol=0)
    # without recombination the same beam keeps 27 paths, not 15 histories
    r0 = oracle.run_lms([oracle.OracleLM(m) for m in lms], lams, oracle.OracleTrie(V, 0, ph), x, 1, B, k,
                        beta, 0, 1, [[V] * B] * n_lm, [0] * B)
    assert np.isfinite(r0["hyp_score"]).sum() == 27
