"""A keyword workload of the shape of the paper's fusion set-up (Sec. IV-A,
Table II), with synthetic tokens only.

Structure taken from the paper, none of its data:

* a list of 300 multi-token terms that doubles as the phrase-boost list;
* 90 carrier templates, each with one slot, and an in-domain corpus of 66k
  sentences made by putting a term into a template's slot;
* a *general* 4-gram estimated from ordinary transcripts only, in which the
  more frequent half of the terms occurs now and then and the rarer half
  never, and a *keyword-synth* 4-gram estimated from the same transcripts
  plus the in-domain corpus;
* a held-out test set (285 utterances, none of whose carriers is a template)
  whose acoustic logits hear every term but often prefer a variant spelling
  of it (one sub-word token swapped), with the right token a close second;
* an upper-bound 4-gram estimated from the test references themselves.

Scoring of decoded token sequences (keyword recall, token error rate) sits
here too: it evaluates what a decoder emitted and holds none of the fusion
arithmetic.  Everything is drawn from PCG64 streams spawned from
``SeedSequence([2609, 14991, 6])``.
"""

from __future__ import annotations

import functools
from dataclasses import dataclass

import numpy as np

from .gen import LMArrays, Phrases, estimate_kn, make_corpus

KEYWORD = dict(
    name="kw_terms300_templates90_v1024_4gram_greedy_s285",
    V=1024, N=4, blank=0, zipf=1.05,
    n_terms=300, term_len=(2, 5), term_ids=(256, 1024), n_frequent=150,
    n_templates=90, template_len=(4, 14), n_insert=66_000,
    n_general=200_000, general_len=(5, 30), general_term_share=0.05,
    n_test=285, test_len=(6, 20), two_term_share=0.3,
    sigma=1.0, am_margin=10.0, blank_margin=10.0, p_variant=0.5, gap=(0.3, 2.0), max_blanks=2,
    lam=0.5, beta=0.5,
)

# the rows of the steering table: (name, LM, alpha, beta); LM None = the
# general LM at alpha 0 (the LM term vanishes from every key)
CONDITIONS = (
    ("baseline", None, 0.0, 0.0),
    ("ngram_general", "general", 0.5, 0.0),
    ("ngram_keyword_synth", "keyword", 0.5, 0.0),
    ("phrase_boost", None, 0.0, 0.5),
    ("ngram_test_refs_upper_bound", "refs", 0.5, 0.0),
)


def _streams():
    ss = np.random.SeedSequence([2609, 14991, 6])
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(6)]


def _tail_ids(rng, n, lo, hi, blank):
    t = rng.integers(lo, hi, size=n).astype(np.int32)
    t[t == blank] = lo
    return t


def _insert(carrier, pos, term):
    return np.concatenate([carrier[:pos], np.asarray(term, dtype=np.int32), carrier[pos:]]).astype(np.int32)


def _csr(seqs):
    offs = np.zeros(len(seqs) + 1, dtype=np.int64)
    np.cumsum([len(s) for s in seqs], out=offs[1:])
    toks = np.concatenate(seqs).astype(np.int32) if seqs else np.zeros(0, np.int32)
    return toks, offs


def _split(toks, offs):
    return [toks[offs[i]:offs[i + 1]] for i in range(offs.size - 1)]


@dataclass
class KeywordWorkload:
    name: str
    V: int
    N: int
    blank: int
    terms: list            # 300 int32 arrays
    variants: list         # per term: the variant spelling (one token swapped)
    variant_pos: np.ndarray  # per term: position of the swapped token
    templates: list        # 90 int32 carriers
    template_slot: np.ndarray
    insert_corpus: tuple   # (tokens, offsets) of the 66k in-domain sentences
    insert_pairs: np.ndarray  # [n, 2] (template, term) of each in-domain sentence
    general_corpus: tuple  # (tokens, offsets)
    general_terms: np.ndarray  # per general sentence: inserted term or -1
    refs: list             # test references, int32 arrays
    ref_terms: list        # per utterance: list of (term, start) in the reference
    confused: list         # per utterance: list of bools, one per (term, start)
    emit_frame: list       # per utterance: frame of each reference token
    logits: np.ndarray     # float32 [T, n_test, V]
    lm_general: LMArrays
    lm_keyword: LMArrays
    lm_refs: LMArrays
    phrases: Phrases
    lam: float
    beta: float

    @property
    def S(self):
        return len(self.refs)

    @property
    def T(self):
        return int(self.logits.shape[0])

    def lm(self, which):
        return {"general": self.lm_general, "keyword": self.lm_keyword, "refs": self.lm_refs}[which]


@functools.lru_cache(maxsize=1)
def make_keyword_workload() -> KeywordWorkload:
    c = KEYWORD
    V, blank = c["V"], c["blank"]
    r_terms, r_tmpl, r_ins, r_gen, r_test, r_am = _streams()
    lo, hi = c["term_ids"]

    # terms (distinct token sequences from the Zipf tail) and their variant spellings
    terms, seen = [], set()
    while len(terms) < c["n_terms"]:
        L = int(r_terms.integers(c["term_len"][0], c["term_len"][1] + 1))
        t = _tail_ids(r_terms, L, lo, hi, blank)
        if tuple(t) not in seen:
            seen.add(tuple(t))
            terms.append(t)
    variants, vpos = [], np.zeros(c["n_terms"], dtype=np.int64)
    for i, t in enumerate(terms):
        p = int(r_terms.integers(0, len(t)))
        v = t.copy()
        while v[p] == t[p] or v[p] == blank:
            v[p] = int(r_terms.integers(lo, hi))
        variants.append(v)
        vpos[i] = p

    # carrier templates with one slot each, and the in-domain corpus
    tt, to = make_corpus(r_tmpl, c["n_templates"], V, c["zipf"], blank=blank, len_range=c["template_len"])
    templates = _split(tt, to)
    slot = np.array([int(r_tmpl.integers(0, len(s) + 1)) for s in templates], dtype=np.int64)
    pairs = np.stack([r_ins.integers(0, c["n_templates"], size=c["n_insert"]),
                      r_ins.integers(0, c["n_terms"], size=c["n_insert"])], axis=1)
    ins = [_insert(templates[a], int(slot[a]), terms[b]) for a, b in pairs]
    ins_corpus = _csr(ins)

    # general transcripts: Zipf sentences, a share of them carrying one of the
    # frequent terms (Zipf over the frequent half); the rare half never occurs
    gt, go = make_corpus(r_gen, c["n_general"], V, c["zipf"], blank=blank, len_range=c["general_len"])
    gen = _split(gt, go)
    nf = c["n_frequent"]
    w = 1.0 / np.arange(1, nf + 1)
    carry = r_gen.random(len(gen)) < c["general_term_share"]
    which = r_gen.choice(nf, size=len(gen), p=w / w.sum())
    gterms = np.where(carry, which, -1).astype(np.int64)
    for i in np.nonzero(carry)[0]:
        pos = int(r_gen.integers(0, len(gen[i]) + 1))
        gen[i] = _insert(gen[i], pos, terms[which[i]])
    gen_corpus = _csr(gen)

    # held-out test references: fresh carriers with one or two terms
    refs, ref_terms = [], []
    ct, co = make_corpus(r_test, c["n_test"], V, c["zipf"], blank=blank, len_range=c["test_len"])
    for u, car in enumerate(_split(ct, co)):
        n_t = 2 if r_test.random() < c["two_term_share"] else 1
        ids = r_test.integers(0, c["n_terms"], size=n_t)
        cuts = np.sort(r_test.integers(0, len(car) + 1, size=n_t))
        seq, occ, prev = [], [], 0
        for j in range(n_t):
            seq.append(car[prev:cuts[j]])
            start = sum(len(s) for s in seq)
            seq.append(terms[ids[j]])
            occ.append((int(ids[j]), int(start)))
            prev = int(cuts[j])
        seq.append(car[prev:])
        refs.append(np.concatenate(seq).astype(np.int32))
        ref_terms.append(occ)

    # acoustic logits: one emitting frame per reference token, then 0..max_blanks
    # blank frames; a confused term occurrence prefers its variant token by a gap
    lens, frames, confused = [], [], []
    for u, ref in enumerate(refs):
        f = int(r_am.integers(0, c["max_blanks"] + 1))
        fr = []
        for _ in ref:
            fr.append(f)
            f += 1 + int(r_am.integers(0, c["max_blanks"] + 1))
        frames.append(fr)
        lens.append(f)
        confused.append([bool(r_am.random() < c["p_variant"]) for _ in ref_terms[u]])
    T = max(lens) + 1
    S = len(refs)
    x = (r_am.standard_normal((T, S, V), dtype=np.float32) * np.float32(c["sigma"])).astype(np.float32)
    emitting = np.zeros((T, S), dtype=bool)
    for u, ref in enumerate(refs):
        for j, y in enumerate(ref):
            t = frames[u][j]
            emitting[t, u] = True
            x[t, u, y] += np.float32(c["am_margin"])
        for (term, start), conf in zip(ref_terms[u], confused[u]):
            if conf:
                t = frames[u][start + int(vpos[term])]
                gap = np.float32(r_am.uniform(c["gap"][0], c["gap"][1]))
                x[t, u, variants[term][vpos[term]]] += np.float32(c["am_margin"])
                x[t, u, terms[term][vpos[term]]] -= gap
    tb, ub = np.nonzero(~emitting)
    x[tb, ub, blank] += np.float32(c["blank_margin"])

    N = c["N"]
    lm_general = estimate_kn(gen_corpus[0], gen_corpus[1], V, N, (1,) * N, blank=blank)
    kw_t = np.concatenate([gen_corpus[0], ins_corpus[0]])
    kw_o = np.concatenate([gen_corpus[1], gen_corpus[1][-1] + ins_corpus[1][1:]])
    lm_keyword = estimate_kn(kw_t, kw_o, V, N, (1,) * N, blank=blank)
    rt, ro = _csr(refs)
    lm_refs = estimate_kn(rt, ro, V, N, (1,) * N, blank=blank)
    pt, po = _csr(terms)
    phrases = Phrases(tokens=pt, offsets=po, completion=None, token_score=1.0)
    return KeywordWorkload(
        name=c["name"], V=V, N=N, blank=blank, terms=terms, variants=variants, variant_pos=vpos,
        templates=templates, template_slot=slot, insert_corpus=ins_corpus, insert_pairs=pairs,
        general_corpus=gen_corpus, general_terms=gterms, refs=refs, ref_terms=ref_terms,
        confused=confused, emit_frame=frames, logits=x, lm_general=lm_general, lm_keyword=lm_keyword,
        lm_refs=lm_refs, phrases=phrases, lam=c["lam"], beta=c["beta"])


# --------------------------------------------------------------------------
# scoring of decoded outputs
# --------------------------------------------------------------------------
def hypotheses(tokens, blank):
    """Greedy decode output tokens [T, S] (one decision per frame) -> the
    emitted token sequence of each stream (blank decisions dropped)."""
    tok = np.asarray(tokens)
    return [tok[:, s][tok[:, s] != blank].astype(np.int32) for s in range(tok.shape[1])]


def count_occurrences(seq, pat):
    """Occurrences of the token sequence ``pat`` in ``seq`` (overlaps counted)."""
    seq, pat = list(seq), list(pat)
    n, m = len(seq), len(pat)
    return sum(1 for i in range(n - m + 1) if seq[i:i + m] == pat) if m else 0


def keyword_recall(hyps, ref_terms, terms):
    """Share of the reference term occurrences found in the hypotheses: per
    utterance and term, min(occurrences in the hypothesis, occurrences in
    the reference), summed over the test set, over all reference occurrences."""
    hit = tot = 0
    for hyp, occ in zip(hyps, ref_terms):
        ids = [t for t, _ in occ]
        for t in set(ids):
            n_ref = ids.count(t)
            hit += min(count_occurrences(hyp, terms[t]), n_ref)
            tot += n_ref
    return hit / tot if tot else 0.0, hit, tot


def edit_distance(a, b):
    """Levenshtein distance between two token sequences (unit costs)."""
    a, b = list(a), list(b)
    prev = list(range(len(b) + 1))
    for i, x in enumerate(a, 1):
        cur = [i] + [0] * len(b)
        for j, y in enumerate(b, 1):
            cur[j] = min(prev[j] + 1, cur[j - 1] + 1, prev[j - 1] + (x != y))
        prev = cur
    return prev[-1]


def token_error_rate(hyps, refs):
    """Sum of edit distances over the sum of reference lengths."""
    return sum(edit_distance(h, r) for h, r in zip(hyps, refs)) / max(1, sum(len(r) for r in refs))
