"""GPU parity at the kernel's overflow paths (the LDS side tables hold 256
entries): the state after a top-level arc at offset >= 256 of its context's
successor list is read from the device table, and so is the phrase state
(and, with two LMs, the entry value) after a transition at index >= 256 of a
phrase state's list.  Both models are built by hand so that the states really
have more than 256 such entries, which the test asserts on the CPU before
decoding; the selected tokens are steered onto those entries with peaked
logits."""

import numpy as np
import pytest
import torch

import oracle
import paper_2609_14991_amd as F
from oracle import traffic
from workloads import LMArrays, Phrases

SCORE_TOL = 1e-5
K_AUX = 256


def dev():
    return torch.device("cuda:0")


def closed_lm(V, N, grams, rng):
    """A backoff model over V tokens (blank 0, <s> = V, </s> = V+1) holding the
    given n-grams plus every prefix and suffix they need, every unigram, and
    random (finite) log-probabilities and backoffs."""
    orders = {k: set() for k in range(1, N + 1)}
    for t in range(1, V + 2):
        orders[1].add((t,))
    todo = [tuple(g) for g in grams]
    while todo:
        g = todo.pop()
        if g in orders[len(g)]:
            continue
        orders[len(g)].add(g)
        if len(g) > 1:
            todo += [g[:-1], g[1:]]
    toks, logp, backoff = [], [], []
    for k in range(1, N + 1):
        rows = np.array(sorted(orders[k]), dtype=np.int32).reshape(-1, k)
        toks.append(rows)
        logp.append(-rng.uniform(0.5, 8.0, size=rows.shape[0]).astype(np.float32))
        backoff.append(-rng.uniform(0.0, 2.0, size=rows.shape[0]).astype(np.float32) if k < N else None)
    return LMArrays(order=N, vocab=V, blank=0, tokens=toks, logp=logp, backoff=backoff)


def models():
    rng = np.random.default_rng(4242)
    V, N = 700, 4
    ctx = (1, 2, 3)
    succ = list(range(10, 10 + 400))  # 400 successors of the top-level context (1, 2, 3)
    grams = [ctx + (y,) for y in succ] + [(5, 6, 7, 8)]
    lm = closed_lm(V, N, grams, rng)
    first = 9  # the phrase state (9,) has 330 one-token extensions
    phr = [[first, y] for y in range(20, 20 + 330)] + [[4, 5, 6]]
    offs = np.zeros(len(phr) + 1, np.int64)
    np.cumsum([len(p) for p in phr], out=offs[1:])
    ph = Phrases(tokens=np.concatenate([np.array(p, np.int32) for p in phr]), offsets=offs)
    return V, N, ctx, succ, first, lm, ph


def test_the_states_exceed_the_side_tables():
    """CPU: the context has more than 256 successors and the phrase state more
    than 256 transitions that differ from the root's."""
    V, N, ctx, succ, first, lm, ph = models()
    assert traffic.FanoutTable(lm).fanout([ctx])[0] == len(succ) > K_AUX
    assert traffic.PhraseDeltas(ph).n_delta((first,)) == 330 > K_AUX


@pytest.mark.gpu
@pytest.mark.parametrize("rows", [False, True])
@pytest.mark.parametrize("n_lm", [1, 2])
def test_overflow_entries_select_and_advance(rows, n_lm, monkeypatch):
    V, N, ctx, succ, first, lm, ph = models()
    # rows=True: the context gets a context row (threshold below its 400
    # successors); rows=False: its arcs are scattered and resolved one by one
    monkeypatch.setenv("FUSION_CONTEXT_ROW_MIN_ARCS", "300" if rows else str(1 << 30))
    glms = [F.ngram_load_arrays(lm) for _ in range(n_lm)]
    monkeypatch.delenv("FUSION_CONTEXT_ROW_MIN_ARCS")
    gtr = F.boost_build_phrases(V, 0, ph)
    olm, otr = oracle.OracleLM(lm), oracle.OracleTrie(V, 0, ph)
    sid = olm.state_of_history([V] + list(ctx))
    assert olm.state_tuple(sid) == ctx
    q = otr.node_of([first])
    # hypotheses at (context, root phrase state) and at (<s>, the wide phrase
    # state); each row's logits peak on one token far down a long list
    targets_lm = succ[K_AUX:K_AUX + 40] + succ[-5:]
    targets_ph = list(range(20 + K_AUX, 20 + 330))[:45]
    H = len(targets_lm) + len(targets_ph)
    rng = np.random.default_rng(17)
    x = rng.standard_normal((H, V)).astype(np.float32)
    ls = np.array([sid] * len(targets_lm) + [V] * len(targets_ph), np.int32)
    bs = np.array([0] * len(targets_lm) + [q] * len(targets_ph), np.int32)
    for h, y in enumerate(targets_lm + targets_ph):
        x[h, y] += 30.0
    lsd = torch.from_numpy(np.stack([ls] * n_lm)).to(dev())
    alphas = [0.5, 0.25][:n_lm]
    for mode, k in ((0, 1), (1, 4)):
        g = F.step_lms(glms, alphas, gtr, torch.from_numpy(x).to(dev()), lsd, torch.from_numpy(bs).to(dev()), 0.5,
                       0, k, mode, want_fused=True)
        torch.cuda.synchronize()
        assert F.fusion_device_status() == 0
        r = oracle.step_lms([olm] * n_lm, alphas, otr, x, [ls] * n_lm, bs, 0.5, 0, k, mode)
        tok = g["tokens"].cpu().numpy()
        assert np.array_equal(tok, r["tokens"])
        assert (tok[:, 0] == np.array(targets_lm + targets_ph)).all()  # the steered entries won
        assert np.array_equal(g["next_lm"].cpu().numpy(), r["next_lm"])
        assert np.array_equal(g["next_boost"].cpu().numpy(), r["next_boost"])
        assert np.abs(g["fused"].cpu().numpy().astype(np.float64) - r["fused"]).max() <= SCORE_TOL
