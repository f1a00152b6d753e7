"""CPU pins of the independent algorithmic-byte count (oracle/traffic.py).

Its two derived quantities are checked against their direct definitions on
small random models: fanout(c) against a count over the raw n-gram rows, and
n_delta(q) against the oracle's brute-force phrase state after every token
from q and from the empty prefix.  The visited states of a greedy decode are
checked against chaining the oracle's single steps."""

import numpy as np
import pytest

import oracle
from oracle import traffic
from workloads import load_workload, tiny_random_lm, tiny_random_phrases


@pytest.mark.parametrize("seed", range(4))
def test_fanout_is_the_number_of_one_token_extensions(seed):
    rng = np.random.default_rng(700 + seed)
    V, N = int(rng.integers(5, 40)), int(rng.integers(2, 6))
    lm = tiny_random_lm(rng, V, N, n_sent=200)
    ft = traffic.FanoutTable(lm)
    for L in range(1, N):
        ctxs = sorted({tuple(int(v) for v in r) for r in np.asarray(lm.tokens[L - 1])})
        got = ft.fanout(ctxs)
        rows = [tuple(int(v) for v in r) for r in np.asarray(lm.tokens[L])]
        for c, n in zip(ctxs, got):
            assert n == sum(1 for r in rows if r[:L] == c)


@pytest.mark.parametrize("seed", range(4))
def test_n_delta_counts_transitions_that_differ_from_the_root(seed):
    rng = np.random.default_rng(800 + seed)
    V = int(rng.integers(4, 12))
    ph = tiny_random_phrases(rng, V, n=int(rng.integers(1, 8)), max_len=5, alphabet=min(V - 1, 4))
    otr = oracle.OracleTrie(V, 0, ph)
    pd = traffic.PhraseDeltas(ph)
    root_next = [otr.state_of_history([y]) for y in range(V)]
    for q in range(otr.n_nodes):
        qt = otr.node_tuple(q)
        direct = sum(1 for y in range(1, V) if otr.state_of_history(list(qt) + [y]) != root_next[y])
        assert pd.n_delta(qt) == direct, (qt, direct)


def test_visited_states_follow_the_decode():
    w = load_workload(1, T=60)
    olm, otr = oracle.OracleLM(w.lm), oracle.OracleTrie(w.V, 0, w.phrases)
    r = oracle.run(olm, otr, w.logits, 1, 1, 1, w.lam, w.beta, 0, 0, [w.V], [0])
    visits = traffic.visited_states(olm, otr, w.V, 0, 1, r["tokens"])
    ls, bs = w.V, 0
    assert len(visits) == w.T
    for t, (tt, h, lt, qt) in enumerate(visits):
        assert (tt, h) == (t, 0)
        assert lt == olm.state_tuple(ls) and qt == otr.node_tuple(bs)
        s = oracle.step(olm, otr, w.logits[t], [ls], [bs], w.lam, w.beta, 0, 1, 0, want_rows=False)
        ls, bs = int(s["next_lm"][0, 0]), int(s["next_boost"][0, 0])


def test_beam_visits_skip_dead_slots():
    """At the first frame of a beam only slot 0 of each stream is live; a slot
    whose parent is -1 is dead at the next frame."""
    w = load_workload(1, T=3)
    olm, otr = oracle.OracleLM(w.lm), oracle.OracleTrie(w.V, 0, w.phrases)
    tok = np.array([[5, 6, -1, 0, 7, -1], [5, 5, 5, 0, 0, -1], [1, 1, 1, 1, 1, 1]], np.int32)
    par = np.array([[0, 0, -1, 0, 0, -1], [0, 1, 0, 0, 1, -1], [0, 0, 0, 0, 0, 0]], np.int32)
    visits = traffic.visited_states(olm, otr, w.V, 0, 3, tok, par)
    by_t = {}
    for t, h, _, _ in visits:
        by_t.setdefault(t, []).append(h)
    assert by_t[0] == [0, 3] and by_t[1] == [0, 1, 3, 4] and by_t[2] == [0, 1, 2, 3, 4]
    lt = {(t, h): l for t, h, l, _ in visits}
    assert lt[(2, 1)] == olm.state_tuple(olm.state_of_history([w.V, 6, 5]))
    assert lt[(2, 4)] == olm.state_tuple(olm.state_of_history([w.V, 7]))
