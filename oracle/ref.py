"""Pure-Python statement of the fusion step for tiny inputs (test infrastructure).

A second, independent implementation of the same definitions as ``oracle.c``
(Eq. (1) of the paper with one or several LMs, ARPA backoff, phrase prefixes
by direct suffix comparison), used to cross-check the C oracle on small random cases.
Dictionaries and tuples only; fp32 steps use numpy float32 scalars so every
operation rounds once.
"""

from __future__ import annotations

import math

import numpy as np

f32 = np.float32


class RefLM:
    def __init__(self, lm):
        self.N, self.V, self.blank = int(lm.order), int(lm.vocab), int(lm.blank)
        self.tab = {}
        self.rows = {}
        for k in range(1, self.N + 1):
            toks = np.asarray(lm.tokens[k - 1])
            lp = np.asarray(lm.logp[k - 1], dtype=np.float32)
            bo = lm.backoff[k - 1] if k < self.N and lm.backoff[k - 1] is not None else None
            rows = []
            for i in range(toks.shape[0]):
                t = tuple(int(v) for v in toks[i])
                self.tab[t] = (f32(lp[i]), f32(bo[i]) if bo is not None else f32(0.0))
                rows.append(t)
            self.rows[k] = sorted(rows)
        self.off = {2: self.V + 2}
        for k in range(2, self.N):
            self.off[k + 1] = self.off[k] + len(self.rows[k])

    def state_id(self, t):
        t = tuple(t)
        if len(t) == 1:
            return t[0]
        return self.off[len(t)] + self.rows[len(t)].index(t)

    def state_tuple(self, sid):
        if sid < self.V + 2:
            return (sid,)
        for k in range(2, self.N):
            if self.off[k] <= sid < self.off[k] + len(self.rows[k]):
                return self.rows[k][sid - self.off[k]]
        raise ValueError(sid)

    def logp(self, ctx, y, wide=False):
        ctx = tuple(ctx)[-(self.N - 1):] if self.N > 1 else ()
        t = ctx + (y,)
        if t in self.tab:
            v = self.tab[t][0]
            return float(v) if wide else v
        lower = self.logp(ctx[1:], y, wide)
        b = self.tab[ctx][1] if ctx in self.tab else f32(0.0)
        return lower + float(b) if wide else f32(lower + b)

    def state_after(self, hist):
        hist = tuple(hist)
        for L in range(min(len(hist), self.N - 1), 0, -1):
            if hist[-L:] in self.tab:
                return self.state_id(hist[-L:])
        raise ValueError(hist)


class RefTrie:
    def __init__(self, phrases):
        self.ts = f32(phrases.token_score)
        self.comp = {}
        plist = phrases.as_lists()
        for i, p in enumerate(plist):
            t = tuple(int(v) for v in p)
            if t in self.comp:
                continue
            c = (f32(phrases.completion[i]) if phrases.completion is not None
                 else f32(self.ts * f32(len(t))))
            self.comp[t] = c
        pref = {()}
        for t in self.comp:
            for L in range(1, len(t) + 1):
                pref.add(t[:L])
        self.nodes = sorted(pref, key=lambda p: (len(p), p))
        self.index = {p: i for i, p in enumerate(self.nodes)}
        self.maxlen = max([len(p) for p in self.nodes] + [1])

    def phi(self, p, wide=False):
        if p in self.comp:
            return 0.0 if wide else f32(0.0)
        return float(len(p)) * float(self.ts) if wide else f32(f32(len(p)) * self.ts)

    def out(self, p, wide=False):
        acc = 0.0 if wide else f32(0.0)
        for L in range(1, len(p) + 1):
            s = p[-L:]
            if s in self.comp:
                acc = float(self.comp[s]) + acc if wide else f32(self.comp[s] + acc)
        return acc

    def entry(self, p, wide=False):
        return self.phi(p, wide) + self.out(p, wide) if wide else f32(self.phi(p) + self.out(p))

    def state(self, hist):
        hist = tuple(hist)
        for L in range(min(len(hist), self.maxlen), 0, -1):
            if hist[-L:] in self.index:
                return hist[-L:]
        return ()

    def boost(self, hist, y, wide=False):
        q = self.state(hist)
        q2 = self.state(tuple(hist) + (y,))
        if wide:
            return self.entry(q2, True) - self.phi(q, True)
        return f32(self.entry(q2) - self.phi(q))


def score_row(lm: RefLM, trie: RefTrie | None, x, lm_hist, ph_hist, lam, beta, blank):
    """(key32[V], fused64[V], lse64) for one hypothesis."""
    V = len(x)
    m = max(float(v) for v in x)
    lse = m + math.log(sum(math.exp(float(v) - m) for v in x))
    lam, beta = f32(lam), f32(beta)
    key = np.empty(V, np.float32)
    fused = np.empty(V, np.float64)
    for y in range(V):
        xv = f32(x[y])
        if y == blank:
            key[y] = xv
            fused[y] = float(xv) - lse
            continue
        l32 = lm.logp(lm_hist, y)
        l64 = lm.logp(lm_hist, y, wide=True)
        b32 = trie.boost(ph_hist, y) if trie is not None else f32(0.0)
        b64 = trie.boost(ph_hist, y, wide=True) if trie is not None else 0.0
        key[y] = f32(f32(xv + f32(lam * l32)) + f32(beta * b32))
        fused[y] = float(xv) - lse + float(lam) * l64 + float(beta) * b64
    return key, fused, lse


def score_row_lms(lms, lams, trie: RefTrie | None, x, lm_hists, ph_hist, beta, blank):
    """score_row with several LMs, each with its own history and weight; the LM
    terms are added in the given order, then the boost term."""
    V = len(x)
    m = max(float(v) for v in x)
    lse = m + math.log(sum(math.exp(float(v) - m) for v in x))
    lams, beta = [f32(a) for a in lams], f32(beta)
    key = np.empty(V, np.float32)
    fused = np.empty(V, np.float64)
    for y in range(V):
        xv = f32(x[y])
        if y == blank:
            key[y] = xv
            fused[y] = float(xv) - lse
            continue
        u = xv
        acc = float(xv) - lse
        for lm, lam, hist in zip(lms, lams, lm_hists):
            u = f32(u + f32(lam * lm.logp(hist, y)))
            acc = acc + float(lam) * lm.logp(hist, y, wide=True)
        b32 = trie.boost(ph_hist, y) if trie is not None else f32(0.0)
        b64 = trie.boost(ph_hist, y, wide=True) if trie is not None else 0.0
        key[y] = f32(u + f32(beta * b32))
        fused[y] = acc + float(beta) * b64
    return key, fused, lse


def select(x, key, blank, k, mode):
    V = len(x)
    if mode == 0:
        a = int(np.argmax(x))
        if a == blank:
            return [blank]
        best = max((y for y in range(V) if y != blank), key=lambda y: (key[y], -y))
        return [best]
    order = sorted(range(V), key=lambda y: (-key[y], y))
    return order[:k]
