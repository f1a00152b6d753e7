"""Sanitizer build of the CPU-side code (CPU only).

The host table builders of the library (tables_host.cpp: validation,
canonical numbering and layouts of the n-gram tables and the phrase tree,
everything ngram_load / boost_build do before the upload) and the test
oracle (oracle.c) are compiled with -fsanitize=address,undefined.  The
builders run on the C1 and C2/C3 models and phrase lists and on malformed
input; the oracle runs its CPU pins in a child interpreter with the sanitized
library preloaded.  Any report from either sanitizer fails the test."""

import bisect
import os
import subprocess
import sys

import numpy as np
import pytest

from workloads import Phrases, load_workload, tiny_random_lm, tiny_random_phrases

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_14991_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("san") / "host_tables")
    cmd = ["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", "/opt/rocm/include",
           "-D__HIP_PLATFORM_AMD__", os.path.join(CSRC, "tables_host.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "host_tables_main.cpp"), "-o", out, "-lpthread"]
    subprocess.run(cmd, check=True)
    return out


def write_case(path, lm, ph):
    with open(path, "wb") as f:
        def put(a, dt):
            f.write(np.ascontiguousarray(a, dtype=dt).tobytes())
        put([lm.order, lm.vocab, lm.blank], np.int32)
        put([t.shape[0] for t in lm.tokens], np.int64)
        for k in range(1, lm.order + 1):
            put(lm.tokens[k - 1], np.int32)
            put(lm.logp[k - 1], np.float32)
            b = lm.backoff[k - 1] if k < lm.order else None
            put([0 if b is None else 1], np.int32)
            if b is not None:
                put(b, np.float32)
        put([ph.n], np.int32)
        put(ph.offsets, np.int64)
        put(ph.tokens, np.int32)
        put([0 if ph.completion is None else 1], np.int32)
        if ph.completion is not None:
            put(ph.completion, np.float32)
        put([ph.token_score], np.float32)


def run(driver, tmp_path, lm, ph, name):
    path = str(tmp_path / f"{name}.bin")
    write_case(path, lm, ph)
    r = subprocess.run([driver, path], capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0 and "ERROR" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-3000:]
    return r.stdout


@pytest.mark.parametrize("cfg", [1, 3])
def test_host_builders_on_workloads(driver, tmp_path, cfg):
    """C1 and the C2/C3 model (3.4M n-grams) with C3's 1000-phrase list."""
    w = load_workload(cfg, T=1, S=1, with_logits=False)
    out = run(driver, tmp_path, w.lm, w.phrases, f"c{cfg}")
    n_states = w.V + 2 + sum(w.lm.counts[1:w.N - 1])
    assert f"lm n_states={n_states} " in out, out
    assert "trie n_nodes=" in out and "error" not in out, out


def test_host_builders_on_random_and_malformed_input(driver, tmp_path):
    rng = np.random.default_rng(31)
    for i in range(6):
        V, N = int(rng.integers(3, 60)), int(rng.integers(2, 7))
        lm = tiny_random_lm(rng, V, N, n_sent=80)
        ph = tiny_random_phrases(rng, V, n=int(rng.integers(0, 12)), max_len=6, alphabet=min(V - 1, 5),
                                 with_completion=bool(i % 2))
        out = run(driver, tmp_path, lm, ph, f"rand{i}")
        assert "lm n_states=" in out and "trie n_nodes=" in out, out
    lm = tiny_random_lm(rng, 9, 3, n_sent=40)
    bad = [t.copy() for t in lm.tokens]
    bad[2] = np.concatenate([bad[2], bad[2][:1]])  # a duplicated trigram
    lm_bad = type(lm)(order=lm.order, vocab=lm.vocab, blank=lm.blank, tokens=bad,
                      logp=[lm.logp[0], lm.logp[1], np.concatenate([lm.logp[2], lm.logp[2][:1]])],
                      backoff=lm.backoff)
    ph_bad = Phrases(tokens=np.array([1, 0, 2], np.int32), offsets=np.array([0, 3], np.int64))  # blank in a phrase
    out = run(driver, tmp_path, lm_bad, ph_bad, "bad")
    assert "lm_error -4" in out and "trie_error -5" in out, out


def test_oracle_pins_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-std=c11", "-D_GNU_SOURCE", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    *SAN, "-o", lib, os.path.join(ROOT, "oracle", "oracle.c"), "-lm", "-lpthread"], check=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    env = dict(ENV, LD_PRELOAD=asan, ORACLE_LIB=lib)
    tests = [os.path.join(ROOT, "tests", f) for f in ("test_oracle.py", "test_oracle_beam.py",
                                                       "test_oracle_multi_lm.py", "test_traffic_checker.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        *tests], capture_output=True, text=True, env=env, cwd=ROOT, timeout=900)
    assert r.returncode == 0 and "ERROR: AddressSanitizer" not in r.stderr + r.stdout \
        and "runtime error" not in r.stderr + r.stdout, (r.stdout[-3000:], r.stderr[-3000:])


@pytest.mark.parametrize("seed,N,X", [(0, 4, 3), (1, 5, 2), (2, 6, 4), (3, 3, 5)])
def test_context_rows_equal_the_backoff_recursion(driver, tmp_path, seed, N, X):
    """With the threshold lowered (FUSION_CONTEXT_ROW_MIN_ARCS), every context
    of 2..N-1 tokens with more than X successors gets a row.  Each row entry
    must be the oracle's fp32 backoff recursion lm(y | c) bit for bit, each
    next-state record the oracle's state after c y (its longest present
    suffix), and each state record must name the deepest context of its chain
    that has a row."""
    import oracle

    rng = np.random.default_rng(950 + seed)
    V = 23
    lm = tiny_random_lm(rng, V, N, n_sent=400, cutoffs=tuple([1] * N))
    ph = tiny_random_phrases(rng, V, n=3, max_len=3)
    path, dump = str(tmp_path / "lm.bin"), str(tmp_path / "lm.dump")
    write_case(path, lm, ph)
    env = dict(ENV, FUSION_CONTEXT_ROW_MIN_ARCS=str(X))
    r = subprocess.run([driver, path, dump], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "runtime error" not in r.stderr, r.stderr[-2000:]
    olm = oracle.OracleLM(lm)
    # the contexts with rows, in row order: by length, then lexicographically
    ctxs = []
    for L in range(2, N):
        rows = [tuple(int(v) for v in t) for t in lm.tokens[L - 1]]
        nxt = [tuple(int(v) for v in t) for t in lm.tokens[L]]
        for c in sorted(rows):
            if sum(1 for t in nxt if t[:L] == c) > X:
                ctxs.append(c)
    with open(dump, "rb") as f:
        RS, n_ctx, n_rec, _ = (int(v) for v in np.frombuffer(f.read(32), np.int64))
        rec = np.frombuffer(f.read(4 * n_rec), np.int32).reshape(-1, RS)
        ctx_lm = np.frombuffer(f.read(4 * n_ctx * V), np.float32).reshape(n_ctx, V)
        ctx_rec = np.frombuffer(f.read(4 * n_ctx * V * RS), np.int32).reshape(n_ctx, V, RS)
    assert n_ctx == len(ctxs) and n_ctx > 0, (n_ctx, len(ctxs))
    for r_, c in enumerate(ctxs):
        for y in range(1, V):
            assert ctx_lm[r_, y] == olm.logp32(list(c), y), (c, y)
            assert ctx_rec[r_, y, 1] == olm.state_of_history(list(c) + [y]), (c, y)
    # state records: the deepest context of the chain with a row
    cw = 2 + 3 * (N - 2)
    index = {c: i for i, c in enumerate(ctxs)}
    for sid in range(V + 2, V + 2 + rec.shape[0]):
        t = olm.state_tuple(sid)
        want = 0
        for L in range(len(t), 1, -1):
            if t[-L:] in index:
                want = (L << 28) | index[t[-L:]]
                break
        assert rec[sid - V - 2, cw] == want, (t, rec[sid - V - 2, cw], want)


def _dump_tables(driver, tmp_path, lm, ph, name):
    """Both host layouts of a model and a phrase list, from the sanitized builders."""
    path, lmd, trd = (str(tmp_path / f"{name}.{s}") for s in ("bin", "lm", "tr"))
    write_case(path, lm, ph)
    r = subprocess.run([driver, path, lmd, trd], capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0 and "runtime error" not in r.stderr and "ERROR" not in r.stderr, r.stderr[-2000:]
    with open(lmd, "rb") as f:
        RS, _, n_rec, _ = (int(v) for v in np.frombuffer(f.read(32), np.int64))
        rec = np.frombuffer(f.read(4 * n_rec), np.int32).reshape(-1, RS)
    with open(trd, "rb") as f:
        n_nodes, n_delta, n_root, n_re = (int(v) for v in np.frombuffer(f.read(32), np.int64))
        node = np.frombuffer(f.read(16 * n_nodes), np.int32).reshape(-1, 4)
        delta = np.frombuffer(f.read(16 * n_delta), np.int32).reshape(-1, 4)
        root_node = np.frombuffer(f.read(16 * n_root), np.int32).reshape(-1, 4)
        root_E = np.frombuffer(f.read(4 * n_re), np.float32)
    return rec, (node, delta, root_node, root_E)


@pytest.mark.parametrize("seed,N", [(0, 3), (1, 4), (2, 5), (3, 6)])
def test_state_records_follow_the_oracle_numbering(driver, tmp_path, seed, N):
    """Every state record of the builders against the definitions: state sid
    is the oracle's context t = state_tuple(sid) (ids by order, then
    lexicographic rank, numbered by the oracle on its own); the record holds
    c_1 = t[-1], the order m = |t|, the id, and for each level L = 2..m the
    backoff of t's last L tokens read straight from the input tuples and
    their number of one-token extensions counted over the raw n-gram rows; the
    first-arc words of contexts with arcs advance with the number of arcs of
    the lexicographically smaller contexts."""
    import oracle

    rng = np.random.default_rng(970 + seed)
    V = 19
    lm = tiny_random_lm(rng, V, N, n_sent=300, cutoffs=tuple([1] * N))
    ph = tiny_random_phrases(rng, V, n=4, max_len=3)
    rec, _ = _dump_tables(driver, tmp_path, lm, ph, "rec")
    olm = oracle.OracleLM(lm)
    assert olm.n_states == V + 2 + rec.shape[0]
    bo, rows_by_len = {}, {}
    for k in range(1, N):
        toks = [tuple(int(v) for v in t) for t in lm.tokens[k - 1]]
        for t, b in zip(toks, lm.backoff[k - 1]):
            bo[t] = np.float32(b)
    for k in range(2, N + 1):
        rows_by_len[k - 1] = sorted(tuple(int(v) for v in t[:k - 1]) for t in lm.tokens[k - 1])
    offset_of_level = {}
    for sid in range(V + 2, V + 2 + rec.shape[0]):
        r, t = rec[sid - V - 2], olm.state_tuple(sid)
        m = len(t)
        assert 2 <= m <= N - 1
        assert r[0] == (t[-1] | (m << 16)) and r[1] == sid, (sid, t, r[:2])
        for L in range(2, m + 1):
            c = t[-L:]
            pre = rows_by_len[L]
            lo = bisect.bisect_left(pre, c)
            cnt = bisect.bisect_right(pre, c) - lo
            assert np.float32(r[2 + 3 * (L - 2)].view(np.float32)) == bo.get(c, np.float32(0.0)), (t, L)
            assert r[4 + 3 * (L - 2)] == cnt, (t, L, r[4 + 3 * (L - 2)], cnt)
            # first arc = a per-level base + the number of arcs of smaller
            # contexts (a context with no arcs has no first arc to check)
            if cnt:
                base = int(r[3 + 3 * (L - 2)]) - lo
                assert offset_of_level.setdefault(L, base) == base, (t, L)


def _prefix_numbering(phrases):
    """Phrase-tree node ids from the definition: every phrase prefix, the
    root first, ranked by (length, tokens)."""
    pre = {()}
    for p in phrases:
        for L in range(1, len(p) + 1):
            pre.add(tuple(p[:L]))
    nodes = sorted(pre, key=lambda t: (len(t), t))
    return nodes, {t: i for i, t in enumerate(nodes)}


@pytest.mark.parametrize("seed", range(4))
def test_phrase_transitions_are_the_longest_prefix_suffix(driver, tmp_path, seed):
    """The phrase tree with its failure links compiled out, against brute
    force: for every node q and token y, the transition (q's own list if y is
    in it, else the root's row) is the longest suffix of q y that is a phrase
    prefix; q's list holds exactly the tokens whose transition differs from
    the root's, sorted; every entry value is E = fl32(Phi + out) of R9 with
    Phi and out computed from the phrase list (out adding the completion
    bonuses of the phrases that end the prefix, shortest first).  The oracle's
    own node numbering is checked against the same definition."""
    import oracle

    rng = np.random.default_rng(990 + seed)
    V = 11
    lm = tiny_random_lm(rng, V, 3, n_sent=60)
    ph = tiny_random_phrases(rng, V, n=12, max_len=5, alphabet=4)
    plist = [tuple(int(v) for v in p) for p in ph.as_lists()]
    _, (node, delta, root_node, root_E) = _dump_tables(driver, tmp_path, lm, ph, "trie")
    nodes, nid = _prefix_numbering(plist)
    assert node.shape[0] == len(nodes)
    otr = oracle.OracleTrie(V, 0, ph)
    for q, t in enumerate(nodes):
        assert tuple(otr.node_tuple(q)) == t
    ts = np.float32(ph.token_score)
    bonus = {}
    for i, p in enumerate(plist):
        if p not in bonus:  # a repeated phrase keeps its first bonus
            bonus[p] = np.float32(ph.completion[i]) if ph.completion is not None else np.float32(ts * np.float32(len(p)))

    def E(t):
        phi = np.float32(0.0) if t in bonus else np.float32(np.float32(len(t)) * ts)
        out = np.float32(0.0)
        for L in range(1, len(t) + 1):
            if t[-L:] in bonus:
                out = np.float32(out + bonus[t[-L:]])
        return np.float32(phi + out)

    def target(t, y):
        s = t + (y,)
        for L in range(len(s), 0, -1):
            if s[-L:] in nid:
                return nid[s[-L:]]
        return 0

    for y in range(1, V):
        g = target((), y)
        assert root_node[y, 3] == g and root_E[y] == E(nodes[g]), y
    for q, t in enumerate(nodes):
        phi_bits, beg, cnt, qq = (int(v) for v in node[q])
        assert qq == q
        assert np.int32(phi_bits).view(np.float32) == (np.float32(0.0) if t in bonus else np.float32(np.float32(len(t)) * ts))
        own = {int(d[0]): (int(d[1]), np.int32(d[2]).view(np.float32)) for d in delta[beg:beg + cnt]}
        assert [int(d[0]) for d in delta[beg:beg + cnt]] == sorted(own)
        for y in range(1, V):
            want = target(t, y)
            if y in own:
                assert own[y][0] == want and own[y][0] != root_node[y, 3], (t, y)
                assert own[y][1] == E(nodes[want]), (t, y)
            else:
                assert root_node[y, 3] == want, (t, y, want)
