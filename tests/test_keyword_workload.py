"""The keyword workload (the structure of the paper's fusion set-up, Sec.
IV-A, on synthetic tokens) and its scoring, on the CPU: how the corpora and
the test logits are built, the recall and error-rate definitions on hand
cases, the oracle's no-fusion decode against the plain argmax of the
logits, and the ordering of the steering conditions that Table II reports."""

import itertools

import numpy as np
import pytest

import oracle
from workloads import (CONDITIONS, KEYWORD, count_occurrences, edit_distance, hypotheses, keyword_recall,
                       make_keyword_workload, token_error_rate)


@pytest.fixture(scope="module")
def kw():
    return make_keyword_workload()


def test_terms_and_variants(kw):
    c = KEYWORD
    assert len(kw.terms) == c["n_terms"] == kw.phrases.n
    assert len({tuple(t) for t in kw.terms}) == c["n_terms"]
    for t, v, p in zip(kw.terms, kw.variants, kw.variant_pos):
        assert c["term_len"][0] <= len(t) <= c["term_len"][1]
        assert (t >= c["term_ids"][0]).all() and (t < c["V"]).all() and (t != kw.blank).all()
        diff = np.nonzero(t != v)[0]
        assert diff.tolist() == [p] and v[p] != kw.blank
    assert [list(x) for x in kw.terms] == kw.phrases.as_lists()


def test_in_domain_corpus(kw):
    """66k sentences, each a template with one term put into its slot."""
    toks, offs = kw.insert_corpus
    assert offs.size - 1 == KEYWORD["n_insert"] == kw.insert_pairs.shape[0]
    assert len(kw.templates) == KEYWORD["n_templates"]
    for i in range(0, offs.size - 1, 997):
        a, b = kw.insert_pairs[i]
        tm, s = kw.templates[a], int(kw.template_slot[a])
        expect = list(tm[:s]) + list(kw.terms[b]) + list(tm[s:])
        assert toks[offs[i]:offs[i + 1]].tolist() == expect


def test_general_corpus_carries_frequent_terms_only(kw):
    toks, offs = kw.general_corpus
    carrying = np.nonzero(kw.general_terms >= 0)[0]
    assert (kw.general_terms[carrying] < KEYWORD["n_frequent"]).all()
    share = carrying.size / (offs.size - 1)
    assert abs(share - KEYWORD["general_term_share"]) < 0.01
    for i in carrying[::211]:
        assert count_occurrences(toks[offs[i]:offs[i + 1]], kw.terms[kw.general_terms[i]]) >= 1
    # the keyword-synth LM sees more n-grams than the general one at every order
    assert all(a >= b for a, b in zip(kw.lm_keyword.counts, kw.lm_general.counts))


def test_test_references_and_logits(kw):
    x = kw.logits
    assert x.shape == (kw.T, KEYWORD["n_test"], KEYWORD["V"])
    tmpl = {tuple(t) for t in kw.templates}
    n_conf = 0
    for u, ref in enumerate(kw.refs):
        for term, start in kw.ref_terms[u]:
            assert ref[start:start + len(kw.terms[term])].tolist() == kw.terms[term].tolist()
        fr = kw.emit_frame[u]
        assert all(b > a for a, b in zip(fr, fr[1:])) and fr[-1] < kw.T
        conf_frames = {}
        for (term, start), conf in zip(kw.ref_terms[u], kw.confused[u]):
            if conf:
                p = int(kw.variant_pos[term])
                conf_frames[fr[start + p]] = (kw.terms[term][p], kw.variants[term][p])
                n_conf += 1
        am = x[:, u, :].argmax(axis=1)
        emit = set(fr)
        for t in range(kw.T):
            if t in conf_frames:
                assert am[t] in conf_frames[t]
            elif t in emit:
                assert am[t] == ref[fr.index(t)]
            else:
                assert am[t] == kw.blank
        assert tuple(ref) not in tmpl
    total = sum(len(o) for o in kw.ref_terms)
    assert 0.4 < n_conf / total < 0.6


def test_recall_and_error_rate_hand_cases():
    terms = [np.array([5, 6]), np.array([7, 8, 9]), np.array([6, 6])]
    # one utterance with term 0 twice and term 1 once; the hypothesis has term 0 once
    ref_terms = [[(0, 0), (1, 3), (0, 6)]]
    hyps = [np.array([5, 6, 1, 7, 8, 4, 2, 2])]
    r, hit, tot = keyword_recall(hyps, ref_terms, terms)
    assert (hit, tot) == (1, 3) and r == pytest.approx(1 / 3)
    # occurrences overlap: 6 6 6 holds "6 6" twice
    assert count_occurrences([6, 6, 6], [6, 6]) == 2
    assert keyword_recall([np.array([6, 6, 6])], [[(2, 0), (2, 1)]], terms)[1:] == (2, 2)
    assert keyword_recall([np.array([6, 6, 6])], [[(2, 0)]], terms)[1:] == (1, 1)
    # Levenshtein distance: classic cases
    assert edit_distance("kitten", "sitting") == 3
    assert edit_distance([], [1, 2, 3]) == 3 and edit_distance([1, 2], []) == 2
    assert edit_distance([1, 2, 3], [1, 2, 3]) == 0
    assert token_error_rate([[1, 2, 4], [7]], [[1, 2, 3], [7, 8]]) == pytest.approx(2 / 5)
    tok = np.array([[0, 3], [4, 0], [0, 0], [5, 6]])
    assert [h.tolist() for h in hypotheses(tok, 0)] == [[4, 5], [3, 6]]


def test_edit_distance_brute_force():
    """Against the minimum over all alignments, enumerated, on tiny sequences."""

    def brute(a, b):
        if not a:
            return len(b)
        if not b:
            return len(a)
        return min(brute(a[1:], b) + 1, brute(a, b[1:]) + 1, brute(a[1:], b[1:]) + (a[0] != b[0]))

    rng = np.random.default_rng(3)
    for _ in range(200):
        a = rng.integers(0, 3, size=rng.integers(0, 6)).tolist()
        b = rng.integers(0, 3, size=rng.integers(0, 6)).tolist()
        assert edit_distance(a, b) == brute(a, b)
    for a, b in itertools.product([[], [1], [1, 2]], repeat=2):
        assert edit_distance(a, b) == brute(a, b)


def _oracle_decode(kw, which, alpha, beta):
    lm = oracle.OracleLM(kw.lm(which or "general"))
    tr = oracle.OracleTrie(kw.V, kw.blank, kw.phrases)
    return oracle.run(lm, tr, kw.logits, kw.S, 1, 1, alpha, beta, kw.blank, 0, [kw.V] * kw.S, [0] * kw.S,
                      threads=8)


def test_no_fusion_decode_is_the_argmax(kw):
    """With alpha = beta = 0 every key is the logit shifted by one row
    constant, so the greedy decode is the argmax of each frame's logits."""
    r = _oracle_decode(kw, None, 0.0, 0.0)
    assert np.array_equal(r["tokens"], kw.logits.argmax(axis=2))


def test_steering_conditions_order_as_in_table_ii(kw):
    """On this workload the oracle's decodes reproduce the ordering of Table
    II: each n-gram and the phrase boost raise recall over no fusion, the
    keyword-synth n-gram more than the general one, the n-gram of the test
    references most; the error rate does not rise."""
    rec, ter = {}, {}
    for name, which, a, b in CONDITIONS:
        r = _oracle_decode(kw, which, a, b)
        hy = hypotheses(r["tokens"], kw.blank)
        rec[name] = keyword_recall(hy, kw.ref_terms, kw.terms)[0]
        ter[name] = token_error_rate(hy, kw.refs)
    assert rec["baseline"] < rec["ngram_general"] < rec["ngram_keyword_synth"] < rec["ngram_test_refs_upper_bound"]
    assert rec["phrase_boost"] > rec["baseline"]
    assert all(ter[n] <= ter["baseline"] for n in rec)
