"""Pins for the CPU oracle: hand-worked examples, invariants, special cases
that reduce to library routines, and brute force.  None of these compares the
oracle with a retyped copy of itself."""

import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import ref
from workloads import LMArrays, Phrases, load_workload, tiny_random_lm, tiny_random_phrases

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def hand_lm():
    g = _gold("lm_hand_example.json")
    V, N = g["V"], g["N"]
    uni_ids = sorted(int(k) for k in g["unigram_backoff"])
    up = {int(k): v for k, v in g["unigram_prob"].items()}
    ub = {int(k): v for k, v in g["unigram_backoff"].items()}
    t1 = np.array(uni_ids, dtype=np.int32).reshape(-1, 1)
    lp1 = np.array([math.log(up[w]) if w in up else -99.0 * math.log(10) for w in uni_ids],
                   dtype=np.float32)
    bo1 = np.array([math.log(ub[w]) for w in uni_ids], dtype=np.float32)
    big = sorted(g["bigrams"])
    t2 = np.array([b[0] for b in big], dtype=np.int32)
    lp2 = np.array([math.log(b[1]) for b in big], dtype=np.float32)
    bo2 = np.array([math.log(b[2]) for b in big], dtype=np.float32)
    t3 = np.array([t[0] for t in g["trigrams"]], dtype=np.int32)
    lp3 = np.array([math.log(t[1]) for t in g["trigrams"]], dtype=np.float32)
    return g, LMArrays(order=N, vocab=V, blank=g["blank"], tokens=[t1, t2, t3],
                       logp=[lp1, lp2, lp3], backoff=[bo1, bo2, None])


def hand_phrases():
    g = _gold("boost_hand_example.json")
    ph = g["phrases"]
    offs = np.zeros(len(ph) + 1, dtype=np.int64)
    np.cumsum([len(p) for p in ph], out=offs[1:])
    return g, Phrases(tokens=np.array(sum(ph, []), dtype=np.int32), offsets=offs,
                      completion=None, token_score=g["token_score"])


# ---------------------------------------------------------------- LM pins
def test_lm_hand_values_and_ids():
    g, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    rlm = ref.RefLM(lm)
    for hv in g["hand_values"]:
        p64 = math.exp(olm.logp64(hv["ctx"], hv["y"]))
        assert p64 == pytest.approx(hv["p"], rel=2e-6), hv["why"]
        p32 = math.exp(float(olm.logp32(hv["ctx"], hv["y"])))
        assert p32 == pytest.approx(hv["p"], rel=2e-6), hv["why"]
        assert math.exp(float(rlm.logp(hv["ctx"], hv["y"]))) == pytest.approx(hv["p"], rel=2e-6)
    for t, sid in g["state_ids"]["tuples"]:
        assert olm.state_tuple(sid) == tuple(t)
        assert rlm.state_id(t) == sid
    assert olm.n_states == g["V"] + 2 + 3
    hist = [g["BOS"]]
    states = [olm.state_of_history(hist)]
    for y in g["path"]["tokens"]:
        hist.append(y)
        states.append(olm.state_of_history(hist))
    assert states == g["path"]["states"]


def test_lm_hand_rows_sum_to_one():
    g, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    for ctx in g["row_sums"]["contexts"]:
        row = olm.row64(ctx)
        s = sum(math.exp(row[y]) for y in (1, 2, 3, g["EOS"]))
        assert s == pytest.approx(1.0, abs=1e-6), ctx


def _all_context_tuples(lm: LMArrays):
    out = []
    for k in range(1, lm.order):
        for row in lm.tokens[k - 1]:
            t = tuple(int(v) for v in row)
            if t[-1] == lm.vocab + 1:  # a context ending in </s> never occurs
                continue
            out.append(t)
    return out


def _check_normalised(lm: LMArrays, tol=1e-4, max_ctx=None):
    olm = oracle.OracleLM(lm)
    pred = [y for y in range(lm.vocab) if y != lm.blank] + [lm.vocab + 1]
    ctxs = _all_context_tuples(lm)
    if max_ctx is not None and len(ctxs) > max_ctx:
        idx = np.random.default_rng(0).choice(len(ctxs), size=max_ctx, replace=False)
        ctxs = [ctxs[i] for i in sorted(idx)]
    worst = 0.0
    for c in ctxs:
        row = olm.row64(c)
        s = float(np.exp(row[pred]).sum())
        worst = max(worst, abs(s - 1.0))
    assert worst < tol, worst


def test_lm_normalisation_c1():
    """Every context of the generated C1 model sums to one over the non-blank
    tokens plus </s> (a dropped backoff, a wrong suffix or a sign slip in the
    recursion breaks this)."""
    _check_normalised(load_workload(1, with_logits=False).lm)


@pytest.mark.parametrize("seed,V,N", [(1, 5, 2), (2, 6, 3), (3, 7, 4), (4, 5, 5), (5, 9, 3)])
def test_lm_normalisation_tiny(seed, V, N):
    rng = np.random.default_rng(seed)
    lm = tiny_random_lm(rng, V, N, n_sent=80)
    _check_normalised(lm, tol=1e-5)


def test_lm_without_bigrams_is_unigram():
    """A bigram model with no explicit bigrams: P(y|w) = bo(w) * P(y)."""
    V = 6
    ids = [1, 2, 3, 4, 5, V, V + 1]
    rng = np.random.default_rng(3)
    lp = np.log(rng.dirichlet(np.ones(len(ids)))).astype(np.float32)
    bo = np.array(rng.uniform(-1, 0.5, len(ids)), dtype=np.float32)
    lm = LMArrays(order=2, vocab=V, blank=0, tokens=[np.array(ids, np.int32).reshape(-1, 1),
                                                     np.zeros((0, 2), np.int32)],
                  logp=[lp, np.zeros(0, np.float32)], backoff=[bo, None])
    olm = oracle.OracleLM(lm)
    for i, w in enumerate(ids):
        for j, y in enumerate(ids):
            if y == V:
                continue
            assert olm.logp32([w], y) == np.float32(lp[j] + bo[i])
    lm0 = LMArrays(order=2, vocab=V, blank=0, tokens=lm.tokens, logp=lm.logp, backoff=[None, None])
    olm0 = oracle.OracleLM(lm0)
    for w in ids:
        for j, y in enumerate(ids):
            if y != V:
                assert olm0.logp32([w], y) == lp[j]


def test_lm_rejects_bad_tables():
    _, lm = hand_lm()
    bad = LMArrays(order=3, vocab=4, blank=0, tokens=[lm.tokens[0], np.vstack([lm.tokens[1],
                                                                              lm.tokens[1][:1]]),
                                                     lm.tokens[2]],
                   logp=[lm.logp[0], np.concatenate([lm.logp[1], lm.logp[1][:1]]), lm.logp[2]],
                   backoff=[lm.backoff[0], np.concatenate([lm.backoff[1], lm.backoff[1][:1]]), None])
    with pytest.raises(oracle.OracleError):
        oracle.OracleLM(bad)
    blank_in = LMArrays(order=3, vocab=4, blank=0,
                        tokens=[lm.tokens[0], np.array([[0, 1], [1, 2], [4, 1]], np.int32), lm.tokens[2]],
                        logp=lm.logp, backoff=lm.backoff)
    with pytest.raises(oracle.OracleError):
        oracle.OracleLM(blank_in)


# ---------------------------------------------------------------- boost pins
def _boost_row(olm, otr, V, lm_state, q):
    """boost(y|q) for all y, read off the fused key with lambda = 0, beta = 1
    and zero logits (key = 0 + 0*lm + 1*boost)."""
    x = np.zeros((1, V), np.float32)
    r = oracle.step(olm, otr, x, [lm_state], [q], 0.0, 1.0, 0, V, 1)
    return r["key"][0], r["fused"][0] + r["lse"][0]


def test_boost_hand_example():
    g, ph = hand_phrases()
    _, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    otr = oracle.OracleTrie(g["V"], g["blank"], ph)
    rtr = ref.RefTrie(ph)
    nodes = [tuple(t) for t in g["nodes"]["tuples"]]
    assert otr.n_nodes == len(nodes)
    for i, t in enumerate(nodes):
        assert otr.node_tuple(i) == t
        assert rtr.index[t] == i
        assert otr.phi(i) == g["phi"][i]
        assert otr.entry(i) - otr.phi(i) == g["out"]["values"][i]
    hist, q = [], 0
    for y, s_exp, b_exp in zip(g["sequence"]["tokens"], g["sequence"]["states"], g["sequence"]["boosts"]):
        row32, row64 = _boost_row(olm, otr, g["V"], 4, q)
        assert row32[y] == b_exp and row64[y] == b_exp
        hist.append(y)
        q = otr.state_of_history(hist)
        assert q == s_exp
        assert float(rtr.boost(hist[:-1], y)) == b_exp


def test_boost_empty_list_is_zero():
    _, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    empty = Phrases(tokens=np.zeros(0, np.int32), offsets=np.zeros(1, np.int64))
    otr = oracle.OracleTrie(4, 0, empty)
    row32, row64 = _boost_row(olm, otr, 4, 4, 0)
    assert np.all(row32[1:] == 0) and np.all(row64[1:] == 0)


def _occurrences(seq, p):
    L = len(p)
    return sum(1 for i in range(len(seq) - L + 1) if tuple(seq[i:i + L]) == tuple(p))


@pytest.mark.parametrize("seed", range(8))
def test_boost_telescopes_to_phrase_counts(seed):
    """Summed over any token sequence, the boost equals the final potential
    plus, for every distinct phrase, its bonus times its number of occurrences
    in the sequence (counted here by brute-force substring enumeration)."""
    rng = np.random.default_rng(100 + seed)
    V = 6
    ph = tiny_random_phrases(rng, V, n=int(rng.integers(1, 7)), max_len=4, alphabet=3,
                             with_completion=bool(seed % 2))
    lm = tiny_random_lm(np.random.default_rng(seed), V, 3, n_sent=40)
    olm = oracle.OracleLM(lm)
    otr = oracle.OracleTrie(V, 0, ph)
    seq = [int(v) for v in rng.integers(1, 4, size=30)]
    total, hist, q = 0.0, [], 0
    for y in seq:
        _, row64 = _boost_row(olm, otr, V, V, q)
        total += row64[y]
        hist.append(y)
        q = otr.state_of_history(hist)
    distinct = {}
    for i, p in enumerate(ph.as_lists()):
        t = tuple(p)
        if t not in distinct:
            distinct[t] = float(ph.completion[i]) if ph.completion is not None else float(len(t))
    phi_final = 0.0 if otr.node_tuple(q) in distinct else float(len(otr.node_tuple(q)))
    expect = phi_final + sum(c * _occurrences(seq, p) for p, c in distinct.items())
    assert total == pytest.approx(expect, abs=1e-9)


# ---------------------------------------------------------------- selection pins
def test_zero_weights_reduce_to_log_softmax_and_topk():
    w = load_workload(1, T=4, with_logits=True)
    olm = oracle.OracleLM(w.lm)
    otr = oracle.OracleTrie(w.V, 0, w.phrases)
    rng = np.random.default_rng(7)
    x = rng.standard_normal((6, w.V)).astype(np.float32) * 2
    states = [w.V, 5, 17, 3, w.V, 60]
    for mode, k in [(1, 1), (1, 5), (0, 1)]:
        r = oracle.step(olm, otr, x, states, [0] * 6, 0.0, 0.0, 0, k, mode)
        assert np.array_equal(r["key"], x)
        ref_ls = torch.log_softmax(torch.from_numpy(x).double(), dim=-1).numpy()
        assert np.abs(r["fused"] - ref_ls).max() < 1e-12
        if mode == 1:
            top = torch.topk(torch.from_numpy(x), k, dim=-1).indices.numpy()
            assert np.array_equal(r["tokens"], top)
        else:
            am = x.argmax(-1)
            nb = np.where(am == 0, 0, np.argmax(np.where(np.arange(w.V) == 0, -np.inf, x), -1))
            assert np.array_equal(r["tokens"][:, 0], nb)


def _path_scores_bruteforce(lm, ph, x, lam, beta, V):
    """Sum of reference fused scores of every token path, each evaluated from
    its own full history (pure-Python statement)."""
    rlm = ref.RefLM(lm)
    rtr = ref.RefTrie(ph)
    T = x.shape[0]
    out = {}
    for path in itertools.product(range(V), repeat=T):
        lmh, phh, tot = [V], [], 0.0
        for t, y in enumerate(path):
            _, fused, _ = ref.score_row(rlm, rtr, x[t], lmh, phh, lam, beta, 0)
            tot += fused[y]
            if y != 0:
                lmh.append(y)
                phh.append(y)
        out[path] = tot
    return out


@pytest.mark.parametrize("lam,beta", [(0.0, 0.0), (0.5, 0.5), (0.3, 1.5)])
def test_exhaustive_beam_keeps_every_path(lam, beta):
    """V = 3, T = 3, k = 3, B = 27: the beam keeps all 27 paths, so its final
    scores are exactly the brute-force path sums (with zero weights these are
    sums of torch log-softmax values)."""
    V, T, B, k = 3, 3, 27, 3
    rng = np.random.default_rng(11)
    lm = tiny_random_lm(rng, V, 3, n_sent=30)
    ph = Phrases(tokens=np.array([1, 2, 2, 1, 1], np.int32), offsets=np.array([0, 2, 5], np.int64))
    xs = rng.standard_normal((T, 1, V)).astype(np.float32) * 2
    x = np.repeat(xs, B, axis=1)  # every slot sees the same joint output
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    r = oracle.run(olm, otr, x, 1, B, k, lam, beta, 0, 1, [V] * B, [0] * B)
    final = np.sort(r["hyp_score"])[::-1]
    if lam == 0.0 and beta == 0.0:
        ls = torch.log_softmax(torch.from_numpy(xs[:, 0]).double(), -1).numpy()
        brute = sorted((sum(ls[t, y] for t, y in enumerate(p))
                        for p in itertools.product(range(V), repeat=T)), reverse=True)
    else:
        brute = sorted(_path_scores_bruteforce(lm, ph, xs[:, 0], lam, beta, V).values(), reverse=True)
    assert np.allclose(final, brute, atol=1e-9, rtol=0)


# ---------------------------------------------------------------- C oracle == Python statement
@pytest.mark.parametrize("seed", range(6))
def test_c_oracle_matches_python_statement(seed):
    rng = np.random.default_rng(200 + seed)
    V = int(rng.integers(4, 9))
    N = int(rng.integers(2, 5))
    lm = tiny_random_lm(rng, V, N, n_sent=50)
    ph = tiny_random_phrases(rng, V, n=4, max_len=3, alphabet=V - 1, with_completion=bool(seed % 2))
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    rlm, rtr = ref.RefLM(lm), ref.RefTrie(ph)
    H = 6
    lam, beta = float(rng.uniform(0, 1)), float(rng.uniform(0, 2))
    x = (rng.standard_normal((H, V)) * 2).astype(np.float32)
    ctx_pool = _all_context_tuples(lm)
    ctxs = [ctx_pool[i] for i in rng.integers(0, len(ctx_pool), size=H)]
    nodes = rtr.nodes
    qs = [nodes[i] for i in rng.integers(0, len(nodes), size=H)]
    k = min(3, V)
    r = oracle.step(olm, otr, x, [rlm.state_id(c) for c in ctxs], [rtr.index[q] for q in qs],
                    lam, beta, 0, k, 1)
    for h in range(H):
        key, fused, lse = ref.score_row(rlm, rtr, x[h], ctxs[h], qs[h], lam, beta, 0)
        assert np.array_equal(r["key"][h], key)
        assert np.abs(r["fused"][h] - fused).max() < 1e-12
        sel = ref.select(x[h], key, 0, k, 1)
        assert r["tokens"][h].tolist() == sel
        for j, y in enumerate(sel):
            if y == 0:
                continue
            assert r["next_lm"][h, j] == rlm.state_after(tuple(ctxs[h]) + (y,))
            assert r["next_boost"][h, j] == rtr.index[rtr.state(tuple(qs[h]) + (y,))]


def test_greedy_run_matches_stepwise():
    """Free-running greedy from full histories equals chaining single steps
    from state ids (the id encoding carries everything the history does)."""
    w = load_workload(1, T=40)
    olm = oracle.OracleLM(w.lm)
    otr = oracle.OracleTrie(w.V, 0, w.phrases)
    r = oracle.run(olm, otr, w.logits, 1, 1, 1, w.lam, w.beta, 0, 0, [w.V], [0])
    ls, bs = [w.V], [0]
    for t in range(w.T):
        s = oracle.step(olm, otr, w.logits[t], ls, bs, w.lam, w.beta, 0, 1, 0, want_rows=False)
        assert s["tokens"][0, 0] == r["tokens"][t, 0]
        ls, bs = [s["next_lm"][0, 0]], [s["next_boost"][0, 0]]
    assert ls[0] == r["lm_state"][0] and bs[0] == r["boost_state"][0]


def test_ties_go_to_lowest_id():
    """Equal keys rank by increasing token id (the stated tie rule), in both
    selection modes and in the acoustic argmax of mode A."""
    _, lm = hand_lm()
    olm = oracle.OracleLM(lm)
    x = np.array([[0.5, 2.0, 2.0, 2.0], [3.0, 1.0, 3.0, 1.0], [1.0, 1.0, 0.0, 1.0]], np.float32)
    r = oracle.step(olm, None, x, [4, 4, 4], [0, 0, 0], 0.0, 0.0, 0, 2, 1)
    assert r["tokens"].tolist() == [[1, 2], [0, 2], [0, 1]]
    r = oracle.step(olm, None, x, [4, 4, 4], [0, 0, 0], 0.0, 0.0, 0, 1, 0)
    # row 1: blank ties token 2 for the acoustic argmax -> blank (lower id)
    assert r["tokens"][:, 0].tolist() == [1, 0, 0]
    x2 = np.array([[0.0, 2.0, 2.0, 1.0]], np.float32)
    r = oracle.step(olm, None, x2, [4], [0], 0.0, 0.0, 0, 1, 0)
    assert r["tokens"][0, 0] == 1
