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
