"""Algorithmic bytes of a decode, recomputed from the states it visits.

TEST INFRASTRUCTURE ONLY (used by the tests and by the benchmark's CPU leg):
an independent count of the bytes the fusion method must move, so that the
roofline numerator does not rest on the counter inside the kernel under test.
It reads the raw n-gram tuples and phrase list and the oracle's state ids; it
shares nothing with the GPU library's tables.

Per live hypothesis-step (one hypothesis, one frame), for Eq. (1) of
Sec. III-C over the whole vocabulary of V tokens:

    4V                                  the logits row
    + min(8 fanout(c_1), 4V)            LM level 1 (last token): its explicit
                                        successors as (token, logp) pairs, or a
                                        dense V-row, whichever is smaller
    + sum over L = 2..m of
        min(8 fanout(c_L), 4V) + 12     each longer context of the state (m
                                        tokens): its successors, plus its
                                        backoff and arc range
    + 8 if m >= 2                       the state's record header
    + 16 + 16 n_delta(q)                with a phrase list: the phrase state's
                                        node, plus one entry per token whose
                                        transition differs from the root's
    + 8 (beam: token, parent) or 4 (greedy: token)
    + 4V if the fused rows are written

plus, with a phrase list, the root's row of V entries once per frame (shared
by all hypotheses).  fanout(c) is the number of n-grams that extend context c
by one token (</s> included); c_L is the state's last L tokens.  n_delta(q) is
the number of tokens y whose phrase state after y from q differs from the one
after y from the empty prefix: the union, over the suffixes of q that are
phrase prefixes, of their one-token extensions (a deeper match always differs
from a match of at most one token).
"""

from __future__ import annotations

import numpy as np


def _bits(V):
    return int(V + 2).bit_length()


def _pack(rows, b):
    """Each row of tokens (int) packed into one uint64, oldest token highest."""
    rows = np.asarray(rows, dtype=np.uint64)
    key = np.zeros(rows.shape[0], dtype=np.uint64)
    for j in range(rows.shape[1]):
        key = (key << np.uint64(b)) | rows[:, j]
    return key


class FanoutTable:
    """fanout(c) for contexts of 1..N-1 tokens, by binary search over the
    prefixes of each order's (lexicographically sorted) n-grams."""

    def __init__(self, lm):
        self.N, self.V = int(lm.order), int(lm.vocab)
        self.b = _bits(self.V)
        if self.b * (self.N - 1) > 64:
            raise ValueError("contexts too long to pack")
        self.pre = {}
        for k in range(2, self.N + 1):
            rows = np.asarray(lm.tokens[k - 1])
            pk = _pack(rows[:, :k - 1], self.b)
            order = np.argsort(pk, kind="stable")
            self.pre[k - 1] = pk[order]

    def fanout(self, ctxs):
        """ctxs: list of tuples, all of one length L (1 <= L <= N-1)."""
        if not ctxs:
            return np.zeros(0, np.int64)
        L = len(ctxs[0])
        pk = self.pre[L]
        q = _pack(np.array(ctxs, dtype=np.int64).reshape(len(ctxs), L), self.b)
        return (np.searchsorted(pk, q, side="right") - np.searchsorted(pk, q, side="left")).astype(np.int64)


class PhraseDeltas:
    """n_delta(q) from the phrase list itself (prefix set and one-token
    extensions), for phrase-state tuples."""

    def __init__(self, phrases):
        self.ext = {}
        for p in phrases.as_lists():
            p = tuple(int(v) for v in p)
            for L in range(len(p)):
                self.ext.setdefault(p[:L], set()).add(p[L])
        self.cache = {}

    def n_delta(self, q):
        q = tuple(q)
        if not q:
            return 0
        if q not in self.cache:
            ys = set()
            for i in range(len(q)):
                ys |= self.ext.get(q[i:], set())
            self.cache[q] = len(ys)
        return self.cache[q]


def visited_states(olm, otr, V, blank, B, tokens, parents=None):
    """(frame, hypothesis, LM state tuple, phrase state tuple) of every live
    hypothesis-step of a decode of streams of B slots (B = 1: greedy) from <s>
    and the empty phrase prefix, given its tokens [T, S*B] (and, for a beam,
    parents [T, S*B]: the slot of the previous frame each slot extends, -1 for
    a dead slot; slot 0 of each stream alone is live at the first frame).
    States come from the oracle's own suffix search over the full histories."""
    tokens = np.asarray(tokens)
    T, H = tokens.shape
    if B > 1:
        parents = np.asarray(parents)
    hist = [[] for _ in range(H)]
    live = [(h % B) == 0 for h in range(H)]
    out = []
    cache = {}
    for t in range(T):
        for h in range(H):
            if not live[h]:
                continue
            key = tuple(hist[h])
            if key not in cache:
                ls = olm.state_of_history([V] + list(key))
                qs = otr.state_of_history(list(key)) if otr is not None else 0
                cache[key] = (olm.state_tuple(ls), otr.node_tuple(qs) if otr is not None else ())
            lt, qt = cache[key]
            out.append((t, h, lt, qt))
        if B > 1:
            new_hist, new_live = [None] * H, [False] * H
            for h in range(H):
                p = int(parents[t, h])
                if p < 0:
                    new_hist[h] = hist[h]
                    continue
                y = int(tokens[t, h])
                new_hist[h] = hist[(h // B) * B + p] + ([y] if y != blank else [])
                new_live[h] = True
            hist, live = new_hist, new_live
        else:
            for h in range(H):
                y = int(tokens[t, h])
                if y != blank:
                    hist[h].append(y)
    return out


def algorithmic_bytes(lm, phrases, visits, T, beam, fused=False):
    """Total algorithmic bytes of the visited hypothesis-steps (see the module
    docstring) and their number.  ``lm`` is the raw n-gram arrays, ``phrases``
    the boost list or None, ``visits`` from visited_states, ``T`` the frames."""
    V = int(lm.vocab)
    row = 4 * V
    ft = FanoutTable(lm)
    pd = PhraseDeltas(phrases) if phrases is not None else None
    by_len = {}
    for (_, _, lt, _) in visits:
        for L in range(1, len(lt) + 1):
            by_len.setdefault(L, set()).add(tuple(lt[-L:]))
    fan = {}
    for L, ctxs in by_len.items():
        ctxs = sorted(ctxs)
        for c, n in zip(ctxs, ft.fanout(ctxs)):
            fan[c] = int(n)
    total = 0
    for (_, _, lt, qt) in visits:
        m = len(lt)
        b = row + (8 if beam else 4) + (row if fused else 0)
        b += min(8 * fan[tuple(lt[-1:])], row)
        for L in range(2, m + 1):
            b += min(8 * fan[tuple(lt[-L:])], row) + 12
        if m >= 2:
            b += 8
        if pd is not None:
            b += 16 + 16 * pd.n_delta(qt)
        total += b
    if pd is not None:
        total += row * T
    return total, len(visits)
