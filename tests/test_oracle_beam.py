"""CPU pins of the oracle's beam: truncation to B and the teacher-forced replay rule.

The beam of the fusion decoder (frame-synchronous, one symbol per frame) keeps,
per stream, the best B of the B*k candidates (each live slot's top-k of Eq. (1)
over the vocabulary, scored by running score + fused score), ties going to the
lower parent slot and then to the lower candidate rank.  Nothing in these tests
calls the C oracle's ranking: the kept sets are recomputed by brute force in
plain Python from ``oracle.ref`` (dictionaries and full token histories), and
the replay rule is probed with decisions built by hand.
"""

import itertools

import numpy as np
import pytest

import oracle
from oracle import ref
from workloads import Phrases, tiny_random_lm, tiny_random_phrases


def python_beam(lm, ph, x, S, B, k, lam, beta, blank=0):
    """Beam over logits x [T, S*B, V] from full token histories, every frame
    ranked by sorting all candidates on (total desc, parent asc, rank asc)."""
    rlm = ref.RefLM(lm)
    rtr = ref.RefTrie(ph) if ph is not None else None
    T, H, V = x.shape
    toks = np.full((T, H), -1, np.int64)
    pars = np.full((T, H), -1, np.int64)
    final = np.full(H, -np.inf)
    for s in range(S):
        hist = [[] for _ in range(B)]  # emitted tokens of each slot
        score = [0.0] + [-np.inf] * (B - 1)
        for t in range(T):
            cands = []
            for b in range(B):
                if score[b] == -np.inf:
                    continue
                row = x[t, s * B + b]
                key, fused, _ = ref.score_row(rlm, rtr, row, [V] + hist[b], hist[b], lam, beta, blank)
                for j, y in enumerate(ref.select(row, key, blank, k, 1)):
                    cands.append((score[b] + fused[y], b, j, y))
            cands.sort(key=lambda c: (-c[0], c[1], c[2]))
            kept = cands[:B]
            new_hist, new_score = [], []
            for i in range(B):
                if i < len(kept):
                    tot, b, _, y = kept[i]
                    new_hist.append(hist[b] + ([y] if y != blank else []))
                    new_score.append(tot)
                    toks[t, s * B + i], pars[t, s * B + i] = y, b
                else:
                    new_hist.append(hist[i])
                    new_score.append(-np.inf)
            hist, score = new_hist, new_score
        final[s * B:(s + 1) * B] = score
    return toks, pars, final


def _case(seed, V, N, integer_logits):
    rng = np.random.default_rng(900 + seed)
    lm = tiny_random_lm(rng, V, N, n_sent=40)
    ph = tiny_random_phrases(rng, V, n=3, max_len=3, alphabet=V - 1)
    return rng, lm, ph


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("integer_logits", [False, True])
def test_truncation_matches_brute_force_sort(seed, integer_logits):
    """V = 5, B = 2, k = 3 (six candidates for two slots), T = 4, two streams:
    tokens, parents and final scores equal the brute-force beam.  Integer
    logits with zero weights make many candidate totals exactly equal, so the
    parent-then-rank tie rule decides which ones survive."""
    V, N, S, B, k, T = 5, 3, 2, 2, 3, 4
    rng, lm, ph = _case(seed, V, N, integer_logits)
    if integer_logits:
        x = rng.integers(-1, 2, size=(T, S * B, V)).astype(np.float32)
        lam, beta = 0.0, 0.0
    else:
        x = (rng.standard_normal((T, S * B, V)) * 2).astype(np.float32)
        lam, beta = 0.5, 0.5
    r = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), x, S, B, k, lam, beta, 0, 1,
                   [V] * (S * B), [0] * (S * B))
    toks, pars, final = python_beam(lm, ph, x, S, B, k, lam, beta)
    assert np.array_equal(r["tokens"], toks)
    assert np.array_equal(r["parents"], pars)
    fin = np.isfinite(final)
    assert np.array_equal(np.isfinite(r["hyp_score"]), fin)
    assert np.abs(r["hyp_score"][fin] - final[fin]).max() < 1e-9


def test_truncation_drops_candidates():
    """The brute-force beam really truncates here: at frame 1 two slots
    propose six candidates and four are dropped; a beam wide enough for all
    of them keeps a path the narrow beam loses."""
    V, N, B, k, T = 5, 3, 2, 3, 3
    rng, lm, ph = _case(3, V, N, False)
    x1 = (rng.standard_normal((T, 1, V)) * 2).astype(np.float32)
    narrow = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), np.repeat(x1, B, axis=1), 1, B, k,
                        0.5, 0.5, 0, 1, [V] * B, [0] * B)
    wide = oracle.run(oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph), np.repeat(x1, 27, axis=1), 1, 27, k,
                      0.5, 0.5, 0, 1, [V] * 27, [0] * 27)
    # the wide beam keeps every path; the narrow one keeps the best two per frame
    assert np.isfinite(wide["hyp_score"]).sum() == 27
    assert np.isfinite(narrow["hyp_score"]).sum() == 2
    assert narrow["hyp_score"].max() <= wide["hyp_score"].max() + 1e-12


def _hand_lm():
    from test_oracle import hand_lm

    return hand_lm()[1]


def test_tie_rule_hand_example():
    """Hand-worked: V = 4 (blank 0), B = 2, k = 2, no LM or boost weight, all
    slots see the same logits.  Frame 0: x = (0, 3, 3, 0); only slot 0 is live
    and its top-2 is tokens 1, 2 (equal keys, lower id first), so slot 0 takes
    token 1 and slot 1 token 2, both from parent 0.  Frame 1: x = (0, 2, 2, 0);
    both slots hold equal scores and propose tokens 1, 2 with equal fused
    scores, so all four totals tie and the order (parent asc, rank asc) keeps
    parent 0's candidates: tokens 1, 2 from parent 0."""
    lm = _hand_lm()
    x = np.array([[[0, 3, 3, 0]] * 2, [[0, 2, 2, 0]] * 2], np.float32)
    r = oracle.run(oracle.OracleLM(lm), None, x, 1, 2, 2, 0.0, 0.0, 0, 1, [4, 4], [0, 0])
    assert r["tokens"].tolist() == [[1, 2], [1, 2]]
    assert r["parents"].tolist() == [[0, 0], [0, 0]]
    ls = np.log(np.exp([0, 3, 3, 0]) / np.exp([0, 3, 3, 0]).sum())
    ls2 = np.log(np.exp([0, 2, 2, 0]) / np.exp([0, 2, 2, 0]).sum())
    assert np.allclose(r["hyp_score"], [ls[1] + ls2[1], ls[1] + ls2[2]], atol=1e-12, rtol=0)


# ---------------------------------------------------------------- replay rule
def _replay(x, forced_tok, forced_par, B, k, tol=1e-4):
    lm = _hand_lm()
    H = x.shape[1]
    return oracle.run(oracle.OracleLM(lm), None, x, 1, B, k, 0.0, 0.0, 0, 1, [4] * H, [0] * H,
                      forced_tokens=np.array(forced_tok, np.int32), forced_parents=np.array(forced_par, np.int32),
                      tol=tol)


def test_replay_of_own_decisions_is_exact():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((6, 2, 4)) * 2).astype(np.float32)
    lm = _hand_lm()
    own = oracle.run(oracle.OracleLM(lm), None, x, 1, 2, 3, 0.0, 0.0, 0, 1, [4, 4], [0, 0])
    r = _replay(x, own["tokens"], own["parents"], 2, 3)
    assert r["mismatch_at"].tolist() == [-1]
    assert r["near_ties"].tolist() == [0]
    assert np.array_equal(r["tokens"], own["tokens"])


@pytest.mark.parametrize("gap,accepted", [(0.0, True), (2e-5, True), (1e-2, False)])
def test_replay_swapped_order(gap, accepted):
    """One frame: the beam keeps tokens 1, 2 (top-2 of slot 0) in slots 0, 1.
    A replay that puts them in the other order is accepted, and counted as a
    near tie, only when their totals differ by less than tol (1e-4)."""
    x = np.array([[[0, 3, 3 - gap, 0]] * 2], np.float32)
    lm = _hand_lm()
    own = oracle.run(oracle.OracleLM(lm), None, x, 1, 2, 2, 0.0, 0.0, 0, 1, [4, 4], [0, 0])
    assert own["tokens"][0].tolist() == [1, 2]
    ft, fp = own["tokens"].copy(), own["parents"].copy()
    ft[0] = [2, 1]
    r = _replay(x, ft, fp, 2, 2)
    if accepted:
        assert r["mismatch_at"].tolist() == [-1]
        assert r["near_ties"].tolist() == [1]
        assert r["tokens"][0].tolist() == [2, 1]  # the replay adopted the forced order
    else:
        assert r["mismatch_at"].tolist() == [0]


@pytest.mark.parametrize("gap,accepted", [(5e-6, True), (1.0, False)])
def test_replay_boundary_swap(gap, accepted):
    """One frame, B = 2, k = 3: slot 0 proposes tokens 1, 2, 3 and the beam keeps 1 and 2.
    A replay that keeps 1 and 3 instead is accepted only when token 3's total
    is within tol of the dropped token 2's."""
    x = np.array([[[0, 3, 2, 2 - gap]] * 2], np.float32)
    lm = _hand_lm()
    own = oracle.run(oracle.OracleLM(lm), None, x, 1, 2, 3, 0.0, 0.0, 0, 1, [4, 4], [0, 0])
    assert own["tokens"][0].tolist() == [1, 2]
    ft, fp = own["tokens"].copy(), own["parents"].copy()
    ft[0] = [1, 3]
    r = _replay(x, ft, fp, 2, 3)
    assert r["mismatch_at"].tolist() == ([-1] if accepted else [0])
    assert r["near_ties"].tolist() == ([1] if accepted else [0])


def test_replay_rejects_non_candidates():
    """A forced token outside the candidates (token 3 is not in slot 0's
    top-2), a forced parent that is dead, and a duplicated candidate are
    mismatches at their frame; later frames are still replayed."""
    x = np.array([[[0, 3, 3, 0]] * 2, [[0, 1, 0, 0]] * 2, [[0, 1, 0, 0]] * 2], np.float32)
    lm = _hand_lm()
    own = oracle.run(oracle.OracleLM(lm), None, x, 1, 2, 2, 0.0, 0.0, 0, 1, [4, 4], [0, 0])
    for frame, tok, par in [(0, [1, 3], [0, 0]), (0, [1, 2], [0, 1]), (0, [1, 1], [0, 0]),
                            (1, [1, 2], [0, -1])]:
        ft, fp = own["tokens"].copy(), own["parents"].copy()
        ft[frame], fp[frame] = tok, par
        r = _replay(x, ft, fp, 2, 2)
        assert r["mismatch_at"].tolist() == [frame], (frame, tok, par)


def test_replay_greedy_has_no_tolerance():
    """Greedy replay (B = 1): a forced token that differs from the oracle's
    pick is a mismatch even when the two keys are equal."""
    lm = _hand_lm()
    x = np.array([[[0, 3, 3, 0]], [[0, 1, 2, 0]]], np.float32)
    olm = oracle.OracleLM(lm)
    own = oracle.run(olm, None, x, 1, 1, 1, 0.0, 0.0, 0, 1, [4], [0])
    assert own["tokens"][:, 0].tolist() == [1, 2]
    r = oracle.run(olm, None, x, 1, 1, 1, 0.0, 0.0, 0, 1, [4], [0],
                   forced_tokens=np.array([[2], [2]], np.int32))
    assert r["mismatch_at"].tolist() == [0]
    r = oracle.run(olm, None, x, 1, 1, 1, 0.0, 0.0, 0, 1, [4], [0],
                   forced_tokens=np.array([[1], [2]], np.int32))
    assert r["mismatch_at"].tolist() == [-1]


def test_python_beam_is_exhaustive_when_wide():
    """Sanity of the brute-force beam itself: with B = V^T slots it keeps every
    path, and its final scores are the path sums of ref.score_row."""
    V, T = 3, 3
    rng = np.random.default_rng(12)
    lm = tiny_random_lm(rng, V, 3, n_sent=30)
    ph = Phrases(tokens=np.array([1, 2], np.int32), offsets=np.array([0, 2], np.int64))
    xs = (rng.standard_normal((T, 1, V)) * 2).astype(np.float32)
    B = V ** T
    _, _, final = python_beam(lm, ph, np.repeat(xs, B, axis=1), 1, B, V, 0.5, 0.5)
    rlm, rtr = ref.RefLM(lm), ref.RefTrie(ph)
    sums = []
    for path in itertools.product(range(V), repeat=T):
        h, tot = [], 0.0
        for t, y in enumerate(path):
            _, fused, _ = ref.score_row(rlm, rtr, xs[t, 0], [V] + h, h, 0.5, 0.5, 0)
            tot += fused[y]
            if y:
                h.append(y)
        sums.append(tot)
    assert np.allclose(np.sort(final)[::-1], np.sort(sums)[::-1], atol=1e-12, rtol=0)
