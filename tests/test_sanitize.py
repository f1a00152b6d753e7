"""Sanitizer build of the CPU-side code (CPU only).

The host table builders of the library (tables_host.cpp: validation,
canonical numbering and layouts of the n-gram tables and the phrase tree,
everything ngram_load / boost_build do before the upload) and the test
oracle (oracle.c) are compiled with -fsanitize=address,undefined.  The
builders run on the C1 and C2/C3 models and phrase lists and on malformed
input; the oracle runs its CPU pins in a child interpreter with the sanitized
library preloaded.  Any report from either sanitizer fails the test."""

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
