"""Seeded generators for the five fusion workloads and for tiny random cases.

Everything here is drawn from ``numpy.random`` PCG64 streams spawned from
``SeedSequence([2609, 14991, cfg])`` so that the CPU oracle and the GPU
library see byte-identical inputs.

Stand-ins: the paper fuses a 4-gram over sub-word tokens and a ~300-term
code-switch boost list into a Thai Transducer (Sec. III-C, Sec. IV-A); its
models, transcripts and word lists are not available, so a truncated-Zipf
token corpus, a Kneser-Ney model estimated from it, corpus-drawn plus rare
phrases and Gaussian joint logits stand in for them.

Token space: ASR ids ``0..V-1`` with ``blank`` (0) never entering the LM;
the LM adds ``BOS = V`` and ``EOS = V + 1``.
"""

from __future__ import annotations

import functools
import os
import sys
from dataclasses import dataclass, field

import numpy as np

LN10 = float(np.log(10.0))
# log-prob given to the <s> unigram, which is a context only (ARPA uses -99 in log10)
BOS_LOGP = np.float32(-99.0 * LN10)


# --------------------------------------------------------------------------
# data containers
# --------------------------------------------------------------------------
@dataclass
class LMArrays:
    """A backoff n-gram model in the raw per-order form ``ngram_load`` takes.

    ``tokens[k-1]`` is an int32 ``[n_k, k]`` array (oldest token first, rows
    in lexicographic order), ``logp[k-1]`` natural-log probabilities and
    ``backoff[k-1]`` natural-log backoff weights (``None`` for the top order).
    """

    order: int
    vocab: int
    blank: int
    tokens: list
    logp: list
    backoff: list

    @property
    def counts(self):
        return [int(t.shape[0]) for t in self.tokens]


@dataclass
class Phrases:
    """Boost list in CSR form: phrase ``i`` is ``tokens[offsets[i]:offsets[i+1]]``."""

    tokens: np.ndarray  # int32
    offsets: np.ndarray  # int64, n + 1
    completion: np.ndarray | None = None  # float32 [n] or None -> token_score * len
    token_score: float = 1.0

    @property
    def n(self):
        return int(self.offsets.shape[0] - 1)

    def as_lists(self):
        return [self.tokens[self.offsets[i]:self.offsets[i + 1]].tolist() for i in range(self.n)]


@dataclass
class Workload:
    cfg: int
    name: str
    V: int
    N: int
    blank: int
    lm: LMArrays
    phrases: Phrases
    S: int
    B: int
    T: int
    k: int
    lam: float
    beta: float
    chunk: int
    logits: np.ndarray  # float32 [T, S*B, V]
    meta: dict = field(default_factory=dict)

    @property
    def H(self):
        return self.S * self.B


# --------------------------------------------------------------------------
# configurations (shapes of the five workloads)
# --------------------------------------------------------------------------
# cutoffs[k-1] = minimum raw count kept at order k (order 1 is never pruned)
CONFIGS = {
    1: dict(name="c1_tiny_v128_3gram_greedy", V=128, N=3, lm_seed=1, n_sent=20_000, zipf=1.1,
            cutoffs=(1, 3, 10), n_phr=10, plen=(2, 5), S=1, B=1, T=200, k=1,
            lam=0.3, beta=1.5, chunk=0, peaked=0.0),
    2: dict(name="c2_stream_v1024_4gram_greedy_chunk13", V=1024, N=4, lm_seed=2, n_sent=2_000_000,
            zipf=1.05, cutoffs=(1, 1, 3, 3), n_phr=100, plen=(2, 8), S=1, B=1, T=1000, k=1,
            lam=0.5, beta=0.5, chunk=13, peaked=0.0),
    3: dict(name="c3_batched_greedy_v1024_4gram_s64", V=1024, N=4, lm_seed=2, n_sent=2_000_000,
            zipf=1.05, cutoffs=(1, 1, 3, 3), n_phr=1000, plen=(2, 8), S=64, B=1, T=1000, k=1,
            lam=0.5, beta=0.5, chunk=0, peaked=0.10),
    4: dict(name="c4_beam_v1024_6gram_s32b4_k4", V=1024, N=6, lm_seed=4, n_sent=20_000_000,
            zipf=1.05, cutoffs=(1, 1, 3, 3, 3, 3), n_phr=1000, plen=(2, 8), S=32, B=4, T=500,
            k=4, lam=0.5, beta=0.5, chunk=0, peaked=0.0),
    5: dict(name="c5_large_lm_v4096_5gram_s64b4_k4", V=4096, N=5, lm_seed=5, n_sent=2_500_000,
            zipf=1.05, cutoffs=(1, 1, 1, 1, 1), n_phr=10_000, plen=(2, 10), S=64, B=4, T=300,
            k=4, lam=0.5, beta=0.5, chunk=0, peaked=0.0),
}


def seed_streams(cfg: int):
    """Five independent PCG64 generators: corpus, phrases, logits, peaks, projection."""
    ss = np.random.SeedSequence([2609, 14991, int(cfg)])
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(5)]


# --------------------------------------------------------------------------
# corpus
# --------------------------------------------------------------------------
def make_corpus(rng, n_sent: int, V: int, s: float, blank: int = 0, len_range=(5, 30)):
    """Sentences of U{len_range} tokens, i.i.d. truncated Zipf(s) over the
    non-blank ids (rank r -> r-th non-blank id in increasing order)."""
    ids = np.array([t for t in range(V) if t != blank], dtype=np.int32)
    ranks = np.arange(1, ids.size + 1, dtype=np.float64)
    p = ranks ** (-s)
    cdf = np.cumsum(p / p.sum())
    lens = rng.integers(len_range[0], len_range[1] + 1, size=n_sent).astype(np.int64)
    offsets = np.zeros(n_sent + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    total = int(offsets[-1])
    toks = np.empty(total, dtype=np.int32)
    step = 1 << 24
    for a in range(0, total, step):
        b = min(total, a + step)
        r = np.searchsorted(cdf, rng.random(b - a), side="right")
        np.minimum(r, ids.size - 1, out=r)
        toks[a:b] = ids[r]
    return toks, offsets


# --------------------------------------------------------------------------
# Kneser-Ney estimation (workload tool: produces the LM the method consumes)
# --------------------------------------------------------------------------
def _progress(msg):
    """Progress of the slow estimation steps, when FUSION_WORKLOAD_PROGRESS=1."""
    if os.environ.get("FUSION_WORKLOAD_PROGRESS") == "1":
        print(f"[workloads] {msg}", file=sys.stderr, flush=True)


def _count_ngrams(tokens, offsets, V, N):
    """Distinct n-grams (as base-(V+2) packed keys, sorted) and raw counts per order."""
    base = V + 2
    BOS, EOS = V, V + 1
    n_sent = offsets.size - 1
    lens = np.diff(offsets)
    plen = lens + 2
    pstart = np.zeros(n_sent + 1, dtype=np.int64)
    np.cumsum(plen, out=pstart[1:])
    total = int(pstart[-1])
    seq = np.empty(total, dtype=np.int64)
    body = np.ones(total, dtype=bool)
    body[pstart[:-1]] = False
    body[pstart[1:] - 1] = False
    seq[pstart[:-1]] = BOS
    seq[pstart[1:] - 1] = EOS
    seq[body] = tokens
    del body
    # positions left in the sentence, counting the position itself
    rem = np.repeat(pstart[1:], plen) - np.arange(total, dtype=np.int64)
    key = seq.copy()
    uniq, raw = [None] * (N + 1), [None] * (N + 1)
    for k in range(1, N + 1):
        if k > 1:
            # key(i) <- key(i) * base + seq[i + k - 1] where the window fits
            ok = rem[: total - k + 1] >= k
            key[: total - k + 1][ok] = key[: total - k + 1][ok] * base + seq[k - 1:][ok]
        sel = key[rem >= k]
        u, c = np.unique(sel, return_counts=True)
        uniq[k], raw[k] = u, c.astype(np.int64)
        del sel
        _progress(f"order {k}: {u.size} distinct n-grams counted")
    return uniq, raw


def _discount(c):
    n1 = int(np.count_nonzero(c == 1))
    n2 = int(np.count_nonzero(c == 2))
    d = n1 / (n1 + 2.0 * n2) if (n1 > 0 and n2 > 0) else 0.5
    return float(min(max(d, 0.1), 0.9))


def _decode(keys, k, base):
    out = np.empty((keys.size, k), dtype=np.int32)
    rest = keys.copy()
    for j in range(k - 1, -1, -1):
        out[:, j] = rest % base
        rest //= base
    return out


def estimate_kn(tokens, offsets, V: int, N: int, cutoffs, blank: int = 0) -> LMArrays:
    """Interpolated Kneser-Ney with count cutoffs and renormalising backoffs.

    * Order N uses raw counts, lower orders continuation counts (raw counts
      for n-grams that start with <s>); one discount per order,
      D = n1 / (n1 + 2 n2).
    * Stored probability of a kept n-gram (h, w):
      max(c - D, 0) / c(h.) + gamma(h) * p_stored(w | h[1:]), where
      gamma(h) = D * N1+(h.) / c(h.).  Kept suffixes exist because the
      cutoffs never decrease with the order.
    * Backoff of h: gamma(h) + P(h) / (1 - B(h)) with P the discounted mass
      of pruned successors and B the lower-order mass of the kept ones, so
      every context sums to one over the non-blank tokens plus </s>.
    """
    base = V + 2
    assert base ** N < 2 ** 63, "packed n-gram keys need (V+2)^N < 2^63"
    BOS, EOS = V, V + 1
    uniq, raw = _count_ngrams(tokens, offsets, V, N)

    # Kneser-Ney counts
    kn = [None] * (N + 1)
    for k in range(1, N + 1):
        if k == N:
            kn[k] = raw[k].astype(np.float64)
            continue
        suf = uniq[k + 1] % (base ** k)
        su, sc = np.unique(suf, return_counts=True)
        idx = np.searchsorted(uniq[k], su)
        assert np.array_equal(uniq[k][idx], su)
        c = np.zeros(uniq[k].size, dtype=np.float64)
        c[idx] = sc
        bos_initial = (uniq[k] // (base ** (k - 1))) == BOS
        c[bos_initial] = raw[k][bos_initial]
        kn[k] = c

    # order 1: continuation unigram interpolated with a uniform floor
    predicted = np.array([t for t in range(V) if t != blank] + [EOS], dtype=np.int64)
    cont = np.zeros(base, dtype=np.float64)
    cont[uniq[1]] = kn[1]
    cw = cont[predicted]
    d1 = _discount(cw[cw > 0])
    tot = cw.sum()
    ntypes = float(np.count_nonzero(cw > 0))
    p_uni = np.zeros(base, dtype=np.float64)
    p_uni[predicted] = np.maximum(cw - d1, 0.0) / tot + (d1 * ntypes / tot) / predicted.size
    uni_ids = np.sort(np.concatenate([predicted, [BOS]]))

    kept_keys = {1: uni_ids.astype(np.int64)}
    kept_p = {1: p_uni[uni_ids]}
    bo = {}
    for k in range(2, N + 1):
        _progress(f"order {k}: estimating")
        u, c, r = uniq[k], kn[k], raw[k]
        d = _discount(c)
        ctx = u // base
        cu, cstart, ccount = np.unique(ctx, return_index=True, return_counts=True)
        csum = np.add.reduceat(c, cstart)
        gamma = d * ccount / csum
        gi = np.repeat(np.arange(cu.size), ccount)
        keep = r >= int(cutoffs[k - 1])
        suf = u[keep] % (base ** (k - 1))
        if k == 2:
            plow = p_uni[suf]
        else:
            idx = np.searchsorted(kept_keys[k - 1], suf)
            assert np.all(idx < kept_keys[k - 1].size)
            assert np.array_equal(kept_keys[k - 1][idx], suf), "suffix closure violated"
            plow = kept_p[k - 1][idx]
        disc = np.maximum(c - d, 0.0) / csum[gi]
        p_kept = disc[keep] + gamma[gi[keep]] * plow
        pruned_mass = np.bincount(gi[~keep], weights=disc[~keep], minlength=cu.size)
        low_mass = np.bincount(gi[keep], weights=plow, minlength=cu.size)
        with np.errstate(divide="ignore", invalid="ignore"):
            extra = np.where(pruned_mass > 0, pruned_mass / np.maximum(1.0 - low_mass, 1e-300), 0.0)
        bo_ctx = gamma + extra
        b = np.ones(kept_keys[k - 1].size, dtype=np.float64)
        pos = np.searchsorted(kept_keys[k - 1], cu)
        found = pos < kept_keys[k - 1].size
        found[found] = kept_keys[k - 1][pos[found]] == cu[found]
        b[pos[found]] = bo_ctx[found]
        bo[k - 1] = b
        kept_keys[k] = u[keep]
        kept_p[k] = p_kept

    toks, logp, backoff = [], [], []
    for k in range(1, N + 1):
        if k == 1:
            toks.append(uni_ids.astype(np.int32).reshape(-1, 1))
            with np.errstate(divide="ignore"):
                lp = np.log(kept_p[1]).astype(np.float32)
            lp[uni_ids == BOS] = BOS_LOGP
        else:
            toks.append(_decode(kept_keys[k], k, base))
            lp = np.log(kept_p[k]).astype(np.float32)
        logp.append(lp)
        backoff.append(np.log(bo[k]).astype(np.float32) if k < N else None)
    return LMArrays(order=N, vocab=V, blank=blank, tokens=toks, logp=logp, backoff=backoff)


# --------------------------------------------------------------------------
# phrases and logits
# --------------------------------------------------------------------------
def make_phrases(rng, n: int, plen, corpus_tokens, corpus_offsets, V: int, blank: int = 0,
                 token_score: float = 1.0) -> Phrases:
    """Half in-corpus substrings (frequent terms the LM has seen), half rare
    terms drawn from the upper half of the id range (Zipf tail)."""
    n_in = n // 2
    lens = rng.integers(plen[0], plen[1] + 1, size=n)
    n_sent = corpus_offsets.size - 1
    out = []
    sids = rng.integers(0, n_sent, size=n_in)
    for i in range(n_in):
        s0, s1 = int(corpus_offsets[sids[i]]), int(corpus_offsets[sids[i] + 1])
        L = int(min(lens[i], s1 - s0))
        st = int(rng.integers(s0, s1 - L + 1))
        out.append(np.asarray(corpus_tokens[st:st + L], dtype=np.int32))
    lo = V // 2 + 1
    for i in range(n_in, n):
        p = rng.integers(lo, V, size=int(lens[i])).astype(np.int32)
        p[p == blank] = lo
        out.append(p)
    offs = np.zeros(n + 1, dtype=np.int64)
    np.cumsum([len(p) for p in out], out=offs[1:])
    return Phrases(tokens=np.concatenate(out).astype(np.int32), offsets=offs,
                   completion=None, token_score=float(token_score))


def make_logits(rng, T: int, H: int, V: int, blank: int = 0, sigma: float = 2.0,
                blank_bias: float = 2.0, peaked: float = 0.0, peak: float = 8.0,
                peak_rng=None, phrase_tokens=None):
    """Joint logits N(0, sigma) with a blank bias; optionally a Bernoulli(peaked)
    share of (t, h) rows gets +peak on one token (a phrase token with
    probability 1/2, else a uniform non-blank token)."""
    x = np.empty((T, H, V), dtype=np.float32)
    for t in range(T):
        x[t] = rng.standard_normal((H, V), dtype=np.float32)
    x *= np.float32(sigma)
    x[:, :, blank] += np.float32(blank_bias)
    if peaked > 0.0:
        prng = peak_rng if peak_rng is not None else rng
        mask = prng.random((T, H)) < peaked
        rows = np.argwhere(mask)
        use_phrase = prng.random(rows.shape[0]) < 0.5
        nonblank = np.array([t for t in range(V) if t != blank], dtype=np.int64)
        uni_tok = nonblank[prng.integers(0, nonblank.size, size=rows.shape[0])]
        if phrase_tokens is not None and len(phrase_tokens) > 0:
            pt = np.asarray(phrase_tokens, dtype=np.int64)
            ph_tok = pt[prng.integers(0, pt.size, size=rows.shape[0])]
        else:
            ph_tok = uni_tok
        tok = np.where(use_phrase, ph_tok, uni_tok)
        x[rows[:, 0], rows[:, 1], tok] += np.float32(peak)
    return x


# --------------------------------------------------------------------------
# workload assembly
# --------------------------------------------------------------------------
def to_bf16_bits(x) -> np.ndarray:
    """float32 values -> bfloat16 bit patterns (uint16), rounded to nearest even.
    Input encoding only (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)).astype(np.uint16)


def make_projection(cfg: int = 5, M: int | None = None, K: int = 640, N: int | None = None,
                    blank: int = 0):
    """Inputs of the joint output projection: hidden states A ~ N(0, 1) [M, K]
    and weight W ~ N(0, (2 / sqrt(K))^2) [N, K] as bf16 bit patterns, fp32 bias
    N(0, 0.1^2) with +2 on blank.  M defaults to T * H of the config, N to V."""
    c = CONFIGS[cfg]
    M = c["T"] * c["S"] * c["B"] if M is None else int(M)
    N = c["V"] if N is None else int(N)
    r = seed_streams(cfg)[4]
    A = to_bf16_bits(r.standard_normal((M, K), dtype=np.float32))
    W = to_bf16_bits(r.standard_normal((N, K), dtype=np.float32) * np.float32(2.0 / np.sqrt(K)))
    bias = (r.standard_normal(N, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
    bias[blank] += np.float32(2.0)
    return A, W, bias


@functools.lru_cache(maxsize=2)
def _corpus_and_lm(lm_seed: int, n_sent: int):
    c = CONFIGS[lm_seed]
    rng = seed_streams(lm_seed)[0]
    toks, offs = make_corpus(rng, n_sent, c["V"], c["zipf"])
    lm = estimate_kn(toks, offs, c["V"], c["N"], c["cutoffs"])
    return toks, offs, lm


def load_workload(cfg: int, T: int | None = None, S: int | None = None,
                  with_logits: bool = True, n_sent: int | None = None) -> Workload:
    """Build workload ``cfg`` (1..5).  ``T``/``S`` shrink the frame or stream
    count (the LM and phrase list stay the full ones); ``n_sent`` replaces the
    corpus size the LM is estimated from (same order, cutoffs and seeds)."""
    c = CONFIGS[cfg]
    ns = c["n_sent"] if n_sent is None else int(n_sent)
    toks, offs, lm = _corpus_and_lm(c["lm_seed"], ns)
    _, r_phr, r_log, r_peak, _ = seed_streams(cfg)
    phr = make_phrases(r_phr, c["n_phr"], c["plen"], toks, offs, c["V"])
    T_full, S_full = c["T"], c["S"]
    T_ = T_full if T is None else int(T)
    S_ = S_full if S is None else int(S)
    H = S_ * c["B"]
    logits = None
    if with_logits:
        logits = make_logits(r_log, T_, H, c["V"], peaked=c["peaked"], peak_rng=r_peak,
                             phrase_tokens=phr.tokens)
    return Workload(cfg=cfg, name=c["name"], V=c["V"], N=c["N"], blank=0, lm=lm, phrases=phr,
                    S=S_, B=c["B"], T=T_, k=c["k"], lam=c["lam"], beta=c["beta"],
                    chunk=c["chunk"], logits=logits,
                    meta=dict(ngram_counts=lm.counts, n_sent=ns, zipf=c["zipf"],
                              cutoffs=list(c["cutoffs"]), n_phrases=c["n_phr"]))


def make_keyword_lm(cfg: int = 5, n_sent: int = 300_000, N: int = 4, len_range=(3, 12)) -> LMArrays:
    """A second LM over the vocabulary of workload ``cfg``, of the shape of the
    keyword LM of Sec. IV-A (an n = 4 model of synthesized text around the
    user's terms): short Zipf carrier sentences, each with one phrase of the
    workload's boost list inserted at a uniform position, estimated with
    interpolated KN and no cutoffs.  Synthetic tokens only."""
    c = CONFIGS[cfg]
    V = c["V"]
    w = load_workload(cfg, T=1, S=1, with_logits=False)
    phr = w.phrases.as_lists()
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([2609, 14991, int(cfg), 6])))
    toks, offs = make_corpus(rng, n_sent, V, c["zipf"], len_range=len_range)
    pick = rng.integers(0, len(phr), size=n_sent)
    lens = np.diff(offs)
    pos = (rng.random(n_sent) * (lens + 1)).astype(np.int64)
    out_lens = lens + np.array([len(phr[i]) for i in pick], dtype=np.int64)
    out_offs = np.zeros(n_sent + 1, dtype=np.int64)
    np.cumsum(out_lens, out=out_offs[1:])
    out = np.empty(int(out_offs[-1]), dtype=np.int32)
    for i in range(n_sent):
        a, b, o, q = int(offs[i]), int(offs[i + 1]), int(out_offs[i]), int(pos[i])
        p = phr[pick[i]]
        out[o:o + q] = toks[a:a + q]
        out[o + q:o + q + len(p)] = p
        out[o + q + len(p):int(out_offs[i + 1])] = toks[a + q:b]
    return estimate_kn(out, out_offs, V, N, tuple([1] * N))


# --------------------------------------------------------------------------
# tiny random cases for property tests
# --------------------------------------------------------------------------
def tiny_random_lm(rng, V: int, N: int, n_sent: int = 60, zipf: float = 1.0,
                   cutoffs=None, blank: int = 0, len_range=(1, 8)) -> LMArrays:
    toks, offs = make_corpus(rng, n_sent, V, zipf, blank=blank, len_range=len_range)
    if cutoffs is None:
        cutoffs = tuple([1] + [int(rng.integers(1, 3)) for _ in range(N - 1)])
        cutoffs = tuple(np.maximum.accumulate(np.array(cutoffs)))
    return estimate_kn(toks, offs, V, N, cutoffs, blank=blank)


def tiny_random_phrases(rng, V: int, n: int, max_len: int, blank: int = 0,
                        alphabet: int | None = None, token_score: float = 1.0,
                        with_completion: bool = False) -> Phrases:
    """Random short phrases over a small alphabet so that prefixes overlap."""
    hi = V if alphabet is None else min(V, alphabet + 1)
    ids = np.array([t for t in range(hi) if t != blank], dtype=np.int32)
    out = []
    for _ in range(n):
        L = int(rng.integers(1, max_len + 1))
        out.append(ids[rng.integers(0, ids.size, size=L)])
    offs = np.zeros(n + 1, dtype=np.int64)
    np.cumsum([len(p) for p in out], out=offs[1:])
    comp = None
    if with_completion:
        comp = rng.uniform(0.0, 4.0, size=n).astype(np.float32)
    return Phrases(tokens=np.concatenate(out).astype(np.int32) if out else np.zeros(0, np.int32),
                   offsets=offs, completion=comp, token_score=float(token_score))
