"""Throughput of the shallow-fusion decode path on one MI355X.

One bench step = one fusion_run over the whole C5 batch: 64 streams x beam 4
(256 hypotheses) x 300 frames, V = 4096, a 5-gram Kneser-Ney model of ~97M
n-grams and a 10k-phrase boost list, top-4 per hypothesis plus the per-stream
beam merge (every step of the path, inputs resident in HBM).

Prints one JSON line: hyp x vocab scores/s (value), decode steps/s, the
roofline of the fusion kernel (algorithmic bytes per launch / mean launch
time from HIP events), and the CPU oracle timed on bounded samples of the
same workload (all host cores the run may use, and one thread), whose
decisions are also checked against the GPU trajectory.  Beside the main step
it reports, each in its own object: the other four workloads (C1-C4, C2 as
its 77 chunk calls), a single fusion_step call on C5 timed with its launch,
C5 with the fused rows written, a measured device-copy bandwidth, the joint
output projection (per frame and batched over all frames), the decode with a
second LM, the recombining beam and the keyword workload (the steering
conditions of Table II on synthetic terms and logits).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, vendor figure
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, vendor figure
METRIC = "fused hyp×vocab scores/sec + decode steps/sec; achieved HBM GB/s vs peak"
HOST_THREADS_CAP = 16  # the host-CPU share of one GPU on the measurement machines


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# sources that decide what the fusion kernel reads and writes; the HBM traffic
# recorded under profiles/ is reported only while they are unchanged
KERNEL_SOURCES = ("paper_2609_14991_amd/csrc/fusion_kernels.hip", "paper_2609_14991_amd/csrc/fusion_internal.h",
                  "paper_2609_14991_amd/csrc/ngram_tables.cpp", "paper_2609_14991_amd/csrc/boost_trie.cpp",
                  "paper_2609_14991_amd/csrc/tables_host.cpp", "paper_2609_14991_amd/csrc/tables_host.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fusion_kernel_c5_hbm_traffic.md")
TRAFFIC_FILE_TWO_LMS = os.path.join(ROOT, "profiles", "fusion_kernel_c5_two_lms_hbm_traffic.md")
TRAFFIC_FILE_RC = os.path.join(ROOT, "profiles", "fusion_kernel_c5_recombining_hbm_traffic.md")
TRAFFIC_FILE_KW = os.path.join(ROOT, "profiles", "fusion_kernel_keyword_hbm_traffic.md")


def kernel_sources_digest():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(workload, path=None):
    """(bytes per launch, source digest) from the committed PMC summary, or None."""
    path = TRAFFIC_FILE if path is None else path
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    fields = dict(re.findall(r"^- (\w+): `([^`]*)`", txt, re.M))
    if fields.get("workload") != workload or "traffic_bytes_per_launch" not in fields:
        return None
    return int(float(fields["traffic_bytes_per_launch"])), fields.get("kernel_sources_digest")


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_probe(nbytes):
    """A plain device copy of known size, for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch

    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copied {n * 4} bytes 3 times")


def copy_bandwidth(torch, stream, nbytes=1 << 31, reps=10):
    """Measured device-to-device copy rate (bytes read + bytes written per second)."""
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(reps):
        dst.copy_(src)
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    return {"bytes_per_copy": nbytes, "ms": ms, "gbs": 2.0 * nbytes / (ms / 1e3) / 1e9,
            "note": "torch device copy of 2 GiB fp32: bytes read + bytes written per second"}


def time_leg(F, torch, dev, stream, reset, launch, n_launch):
    """One launch with the kernel's byte count on (algorithmic bytes and
    hypothesis-steps), two warm-up launches, then the mean HIP-event time of
    n_launch launches on `stream`; `reset()` restores the carried state before
    each launch, outside the events."""
    traffic = torch.zeros(2, dtype=torch.int64, device=dev)
    reset()
    launch(traffic)
    torch.cuda.synchronize()
    assert F.fusion_device_status() == 0
    alg, steps = (int(v) for v in traffic.cpu())
    for _ in range(2):
        reset()
        launch(None)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_launch)]
    torch.cuda.synchronize()
    for a, b in ev:
        reset()
        a.record(stream)
        launch(None)
        b.record(stream)
    torch.cuda.synchronize()
    return alg, steps, float(np.mean([a.elapsed_time(b) for a, b in ev]))


def leg_roofline(alg, steps, kms, record, copy_gbs=None):
    """The roofline object of a leg; `record` is its PMC traffic record or None."""
    ach = alg / (kms / 1e3) / 1e9
    ok = record is not None and record[1] == kernel_sources_digest()
    out = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
           "algorithmic_bytes_per_launch": alg, "bytes_per_hyp_step": alg / max(steps, 1),
           "traffic": record[0] if ok else None,
           "traffic_note": ("HBM bytes per launch from the PMC record (FETCH_SIZE + WRITE_SIZE, scaled)" if ok
                            else "no PMC record for these kernel sources")}
    if ok:
        out["hbm_traffic_gbs"] = record[0] / (kms / 1e3) / 1e9
    if copy_gbs:
        out["frac_of_copy"] = ach / copy_gbs
    return out


def config_leg(F, torch, dev, stream, cfg, n_launch, copy_gbs):
    """Workload cfg (1-4) decoded on the GPU as the tests check it: µs per
    decode step (frame), decode steps/s, hyp x vocab scores/s and its roofline.
    C2 is its 1000 frames fed as 77 calls of 13 frames (the last of 12) with
    the states carried, timed as the sum of the calls."""
    from workloads import load_workload

    t0 = time.time()
    w = load_workload(cfg)
    lm = F.ngram_load_arrays(w.lm)
    trie = F.boost_build_phrases(w.V, w.blank, w.phrases)
    T, S, B, V, k, H = w.T, w.S, w.B, w.V, w.k, w.H
    x = torch.from_numpy(w.logits).to(dev)
    bos = F.ngram_bos_state(lm)
    ls = torch.full((H,), bos, dtype=torch.int32, device=dev)
    bs = torch.zeros((H,), dtype=torch.int32, device=dev)
    sc0 = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev)
    sc = sc0.clone()
    tokens = torch.empty((T, H), dtype=torch.int32, device=dev)
    parents = torch.empty((T, H), dtype=torch.int32, device=dev) if B > 1 else None
    mode = F.FUSION_BLANK_COMPETE if B > 1 else F.FUSION_BLANK_AM
    chunk = w.chunk if w.chunk else T
    log(f"{w.name}: built in {time.time() - t0:.1f}s")

    def reset():
        ls.fill_(bos)
        bs.zero_()
        sc.copy_(sc0)

    def launch(traffic):
        for t0_ in range(0, T, chunk):
            t1_ = min(T, t0_ + chunk)
            F.fusion_run(lm, trie, x[t0_:t1_], t1_ - t0_, S, B, V, k, w.lam, w.beta, w.blank, mode, ls, bs,
                         sc if B > 1 else None, tokens[t0_:t1_], parents[t0_:t1_] if B > 1 else None, None,
                         traffic, stream.cuda_stream)

    alg, steps, kms = time_leg(F, torch, dev, stream, reset, launch, n_launch)
    roof = leg_roofline(alg, steps, kms, None, copy_gbs)
    calls = (T + chunk - 1) // chunk
    out = {"workload": w.name, "V": V, "lm_order": w.N, "ngrams": int(sum(w.lm.counts)), "phrases": w.phrases.n,
           "streams": S, "beam": B, "hypotheses": H, "frames": T, "k": k, "calls": calls,
           "ms_per_run": kms, "us_per_step": kms * 1e3 / T, "decode_steps_per_s": T / (kms / 1e3),
           "value": float(T) * H * V / (kms / 1e3), "unit": "hyp×vocab scores/s", "roofline": roof}
    log(f"{w.name}: {kms:.3f} ms for {T} frames in {calls} call(s), {kms * 1e3 / T:.2f} us/step, "
        f"{alg / max(steps, 1):.0f} B/hyp-step, frac {roof['frac']:.4f}")
    lm.close()
    trie.close()
    return out


def keyword_leg(F, torch, dev, stream, n_launch):
    """The keyword workload: 285 test streams decoded greedily under each
    steering condition of Table II (keyword recall and token error rate from
    the GPU's tokens), then the deployed set-up (keyword-synth 4-gram and
    phrase boost together) timed with HIP events."""
    from workloads import CONDITIONS, hypotheses, keyword_recall, make_keyword_workload, token_error_rate

    t0 = time.time()
    kw = make_keyword_workload()
    glms = {k: F.ngram_load_arrays(kw.lm(k)) for k in ("general", "keyword", "refs")}
    gtr = F.boost_build_phrases(kw.V, kw.blank, kw.phrases)
    log(f"keyword workload {kw.name}: {kw.S} streams x {kw.T} frames, built in {time.time() - t0:.1f}s")
    x = torch.from_numpy(kw.logits).to(dev)
    S, T, V = kw.S, kw.T, kw.V
    ls = torch.empty((S,), dtype=torch.int32, device=dev)
    bs = torch.empty((S,), dtype=torch.int32, device=dev)
    tokens = torch.empty((T, S), dtype=torch.int32, device=dev)

    def reset(lm):
        ls.fill_(F.ngram_bos_state(lm))
        bs.zero_()

    def decode(lm, alpha, beta, traffic=None):
        F.fusion_run(lm, gtr, x, T, S, 1, V, 1, alpha, beta, kw.blank, F.FUSION_BLANK_AM, ls, bs, None, tokens,
                     None, None, traffic, stream.cuda_stream)

    conds = list(CONDITIONS) + [("ngram_keyword_synth+phrase_boost", "keyword", kw.lam, kw.beta)]
    table = {}
    for name, which, alpha, beta in conds:
        reset(glms[which or "general"])
        decode(glms[which or "general"], alpha, beta)
        torch.cuda.synchronize()
        assert F.fusion_device_status() == 0
        hy = hypotheses(tokens.cpu().numpy(), kw.blank)
        r, hit, tot = keyword_recall(hy, kw.ref_terms, kw.terms)
        table[name] = {"alpha": alpha, "beta": beta, "recall": r, "terms_found": hit, "terms": tot,
                       "token_error_rate": token_error_rate(hy, kw.refs)}
    lm = glms["keyword"]
    alg, steps, kms = time_leg(F, torch, dev, stream, lambda: reset(lm),
                               lambda tr: decode(lm, kw.lam, kw.beta, tr), n_launch)
    roof = leg_roofline(alg, steps, kms, recorded_traffic(kw.name, TRAFFIC_FILE_KW))
    log(f"keyword workload: {kms:.3f} ms kernel, {alg / max(steps, 1):.0f} B/hyp-step, {roof['achieved']:.1f} GB/s; "
        "recall " + ", ".join(f"{n} {v['recall']:.3f}" for n, v in table.items()))
    for h in list(glms.values()) + [gtr]:
        h.close()
    return {
        "workload": kw.name, "streams": S, "frames": T, "V": V, "lm_order": kw.N,
        "ngrams": {k: int(sum(kw.lm(k).counts)) for k in ("general", "keyword", "refs")},
        "terms": len(kw.terms), "data": "synthetic (terms, templates, transcripts and logits drawn from seeds)",
        "conditions": table,
        "timed": "ngram_keyword_synth+phrase_boost", "launches": n_launch, "kernel_ms_per_launch": kms,
        "value": float(T) * S * V / (kms / 1e3), "unit": "hyp×vocab scores/s",
        "decode_steps_per_s": T / (kms / 1e3),
        "roofline": roof,
    }


def projection_leg(F, torch, dev, stream, cfg, w=None, lm=None, trie=None):
    """The joint output projection (bf16 MFMA) that would produce C5's logits:
    the per-frame shape [256, 640] x [640, 4096] (one frame of all hypotheses)
    and the batch of all 300 frames [76800, 640] x [640, 4096], each timed with
    HIP events over back-to-back launches."""
    from workloads import make_projection

    A, Wt, bias = make_projection(cfg)
    M, K = A.shape
    N = Wt.shape[0]
    a_d = torch.from_numpy(A.view(np.int16)).to(dev)
    w_d = torch.from_numpy(Wt.view(np.int16)).to(dev)
    b_d = torch.from_numpy(bias).to(dev)
    o_d = torch.empty((M, N), dtype=torch.float32, device=dev)
    out = {"kernel": "joint_proj_kernel"}
    H = M // 300
    for name, m, n_rep in (("per_frame", H, 200), ("batched", M, 10)):
        for _ in range(3):
            F.joint_project(a_d, w_d, b_d, m, N, K, o_d, stream.cuda_stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n_rep):
            F.joint_project(a_d, w_d, b_d, m, N, K, o_d, stream.cuda_stream)
        e1.record(stream)
        torch.cuda.synchronize()
        pms = e0.elapsed_time(e1) / n_rep
        flops = 2.0 * m * N * K
        pbytes = 2.0 * m * K + 2.0 * N * K + 4.0 * N + 4.0 * m * N
        out[name] = {
            "shape": [m, N, K], "ms_per_launch": pms, "launches": n_rep,
            "tflops": flops / (pms / 1e3) / 1e12, "peak_tflops_bf16": BF16_PEAK_TFLOPS,
            "frac_of_peak": flops / (pms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
            "min_hbm_bytes": pbytes, "hbm_gbs_at_min_bytes": pbytes / (pms / 1e3) / 1e9,
        }
        log(f"joint projection {m}x{N}x{K}: {pms * 1e3:.1f} us, {flops / (pms / 1e3) / 1e12:.1f} TFLOP/s")
        out[name]["vendor_gemm"] = vendor_gemm(torch, stream, a_d, w_d, b_d, o_d, m, n_rep, flops)
    if w is not None:
        out["producer_loop"] = producer_leg(F, torch, dev, stream, w, lm, trie, a_d, w_d, b_d, o_d, K)
    del a_d, w_d, b_d, o_d
    return out


def vendor_gemm(torch, stream, a_d, w_d, b_d, o_d, m, n_rep, flops):
    """The same product from the vendor GEMM library (hipBLASLt through torch,
    fp32 output) on the same inputs, for context: with the bias
    (torch.addmm, the same work as joint_project) and without it (torch.mm,
    less work), each with its largest difference from joint_project's output."""
    a = a_d[:m].view(torch.bfloat16)
    wt = w_d.view(torch.bfloat16).t()
    forms = {"addmm_with_bias": lambda: torch.addmm(b_d, a, wt, out_dtype=torch.float32),
             "mm_without_bias": lambda: torch.mm(a, wt, out_dtype=torch.float32)}
    out = {"library": "hipBLASLt (through torch, out_dtype float32)"}
    with torch.cuda.stream(stream):
        for name, fn in forms.items():
            for _ in range(3):
                y = fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(n_rep):
                y = fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / n_rep
            ref = o_d[:m] if name == "addmm_with_bias" else o_d[:m] - b_d
            out[name] = {"ms_per_launch": ms, "tflops": flops / (ms / 1e3) / 1e12,
                         "max_abs_diff_vs_joint_project": float((y - ref).abs().max())}
            del y, ref
    return out


def producer_leg(F, torch, dev, stream, w, lm, trie, a_d, w_d, b_d, o_d, K, n_launch=5):
    """C5 decoded with the joint projection as the producer of its logits:
    fusion_run_projected per frame (chunk 1: the [256, 640] x [640, 4096]
    projection, then the frame's fusion step), per 13-frame chunk (a streaming
    encoder chunk) and over all 300 frames at once, against the batched order
    (one joint_project of all frames, then one fusion_run), each timed end to
    end with HIP events; every decode's decisions must equal the batched one's."""
    T, S, B, V, k, H = w.T, w.S, w.B, w.V, w.k, w.H
    bos = F.ngram_bos_state(lm)
    sc0 = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev)
    mode = F.FUSION_BLANK_COMPETE
    runs = {"chunk_1": 1, "chunk_13": 13, f"chunk_{T}": T, "batched": None}
    st = {n: (torch.empty((H,), dtype=torch.int32, device=dev), torch.empty((H,), dtype=torch.int32, device=dev),
              torch.empty((H,), dtype=torch.float64, device=dev),
              torch.empty((T, H), dtype=torch.int32, device=dev), torch.empty((T, H), dtype=torch.int32, device=dev))
          for n in runs}

    def reset(n):
        ls, bs, sc = st[n][:3]
        ls.fill_(bos)
        bs.zero_()
        sc.copy_(sc0)

    def run(n):
        ls, bs, sc, tok, par = st[n]
        if runs[n] is None:
            F.joint_project(a_d, w_d, b_d, T * H, V, K, o_d, stream.cuda_stream)
            F.fusion_run(lm, trie, o_d, T, S, B, V, k, w.lam, w.beta, w.blank, mode, ls, bs, sc, tok, par, None, None,
                         stream.cuda_stream)
        else:
            F.fusion_run_projected([lm], [w.lam], trie, a_d, w_d, b_d, K, o_d, runs[n], T, S, B, V, k, w.beta,
                                   w.blank, mode, ls, bs, sc, tok, par, stream=stream.cuda_stream)

    res = {}
    for name in runs:
        for _ in range(2):
            reset(name)
            run(name)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_launch)]
        torch.cuda.synchronize()
        for a, b in ev:
            reset(name)
            a.record(stream)
            run(name)
            b.record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
        res[name] = {"frames_per_projection": runs[name] or T, "ms": ms, "us_per_frame": ms * 1e3 / T}
    assert F.fusion_device_status() == 0
    same = all(torch.equal(x, y) for n in runs for x, y in zip(st[n], st["batched"]))
    res["decisions_equal"] = bool(same)
    res["note"] = ("chunk_c: fusion_run_projected with c frames per projection ([c*H, K] x [K, V] into a [c, H, V] "
                   "workspace, then one decode launch of those c frames); batched: one [T*H, K] x [K, V] projection "
                   "then one fusion_run")
    log("producer loop (C5): " + ", ".join(f"{n} {res[n]['ms']:.3f} ms" for n in runs) + f", decisions equal {same}")
    return res


def step_leg(F, torch, dev, stream, w, lm, trie, x, n_calls=300):
    """One fusion_step over C5's 256 hypotheses at a frame of its decode: the
    host-side time per call including its launch (calls back to back, one
    synchronisation at the end), and the HIP-event time of one call."""
    H, V = w.H, w.V
    rng = np.random.default_rng(5)
    ls = torch.from_numpy(rng.integers(1, V, size=H).astype(np.int32)).to(dev)
    bs = torch.zeros((H,), dtype=torch.int32, device=dev)
    out = {n: torch.empty((H, w.k), dtype=dt, device=dev)
           for n, dt in (("tokens", torch.int32), ("scores", torch.float32), ("next_lm", torch.int32),
                         ("next_boost", torch.int32))}
    row = x[w.T // 2]

    def call():
        F.fusion_step(lm, trie, row, ls, bs, H, V, w.lam, w.beta, w.blank, w.k, F.FUSION_BLANK_COMPETE, None,
                      out["tokens"], out["scores"], out["next_lm"], out["next_boost"], stream.cuda_stream)

    for _ in range(10):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n_calls):
        call()
    torch.cuda.synchronize()
    host_us = (time.perf_counter() - t0) / n_calls * 1e6
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(50)]
    for a, b in ev:
        a.record(stream)
        call()
        b.record(stream)
    torch.cuda.synchronize()
    ev_us = float(np.mean([a.elapsed_time(b) for a, b in ev])) * 1e3
    assert F.fusion_device_status() == 0
    log(f"fusion_step (C5, 256 hypotheses, top-4): {host_us:.2f} us per call with launch, {ev_us:.2f} us events")
    return {"hypotheses": H, "V": V, "k": w.k, "calls": n_calls, "us_per_call_launch_inclusive": host_us,
            "us_per_call_events": ev_us, "note": "random one-token LM states, root phrase state; states not "
            "advanced between calls"}


def cpu_leg(w, ref_tokens, ref_parents, bos, n_threads, streams, frames):
    """The oracle on the first `frames` frames of `streams` streams of the
    workload, replaying the GPU's decisions, on n_threads threads."""
    import oracle

    olm = oracle.OracleLM(w.lm)
    otr = oracle.OracleTrie(w.V, w.blank, w.phrases)
    B, k, V = w.B, w.k, w.V
    Sc, Tc = min(streams, w.S), min(frames, w.T)
    xs = np.ascontiguousarray(w.logits[:Tc, :Sc * B])
    sc_init = np.tile(np.array([0.0] + [-np.inf] * (B - 1)), Sc)
    tc = time.perf_counter()
    r = oracle.run(olm, otr, xs, Sc, B, k, w.lam, w.beta, w.blank, 1 if B > 1 else 0,
                   [bos] * (Sc * B), [0] * (Sc * B), sc_init,
                   forced_tokens=ref_tokens[:Tc, :Sc * B],
                   forced_parents=ref_parents[:Tc, :Sc * B] if B > 1 else None,
                   tol=1e-4, threads=n_threads)
    sec = time.perf_counter() - tc
    agree = bool((r["mismatch_at"] < 0).all())
    near = int(r["near_ties"].sum())
    return olm, otr, r, sec, Sc, Tc, agree, near


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--fused", action="store_true", help="time the main step with the full fused score rows written")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--no-projection", action="store_true", help="skip the joint-projection measurement")
    ap.add_argument("--no-recombine", action="store_true", help="skip the recombining-beam measurement")
    ap.add_argument("--no-second-lm", action="store_true",
                    help="skip the two-LM measurement (C5 with a second, keyword 4-gram LM)")
    ap.add_argument("--no-keyword", action="store_true",
                    help="skip the keyword workload (steering conditions of Table II, synthetic)")
    ap.add_argument("--no-configs", action="store_true", help="skip the C1-C4 rows")
    ap.add_argument("--cpu-frames", type=int, default=300)
    ap.add_argument("--cpu-streams", type=int, default=64)
    ap.add_argument("--cpu-streams-single", type=int, default=4,
                    help="streams of the single-thread oracle sample")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of this size (counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the fusion path would shard by stream, with no exchange between GPUs per step)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_14991_amd as F
    from workloads import load_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    t0 = time.time()
    w = load_workload(args.config)
    log(f"workload {w.name}: n-grams {w.lm.counts} built in {time.time() - t0:.1f}s")
    t1 = time.time()
    lm = F.ngram_load_arrays(w.lm)
    trie = F.boost_build_phrases(w.V, w.blank, w.phrases)
    n_states, lm_bytes = F.ngram_info(lm)
    n_nodes, max_depth, trie_bytes = F.boost_info(trie)
    t_load = time.time() - t1
    log(f"tables on device: LM {lm_bytes / 1e9:.2f} GB ({n_states} states), trie {n_nodes} nodes, {t_load:.1f}s")

    T, S, B, V, k = w.T, w.S, w.B, w.V, w.k
    H = S * B
    x = torch.from_numpy(w.logits).to(dev)
    bos = F.ngram_bos_state(lm)
    ls0 = torch.full((H,), bos, dtype=torch.int32, device=dev)
    bs0 = torch.zeros((H,), dtype=torch.int32, device=dev)
    sc0 = torch.from_numpy(np.tile(np.array([0.0] + [-np.inf] * (B - 1)), S)).to(dev)
    ls, bs, sc = ls0.clone(), bs0.clone(), sc0.clone()
    tokens = torch.empty((T, H), dtype=torch.int32, device=dev)
    parents = torch.empty((T, H), dtype=torch.int32, device=dev)
    fused = torch.empty((T, H, V), dtype=torch.float32, device=dev) if args.fused else None
    mode = F.FUSION_BLANK_COMPETE if B > 1 else F.FUSION_BLANK_AM

    def reset():
        ls.copy_(ls0)
        bs.copy_(bs0)
        sc.copy_(sc0)

    def run_once(traffic=None, fused_rows=fused):
        F.fusion_run(lm, trie, x, T, S, B, V, k, w.lam, w.beta, w.blank, mode, ls, bs, sc, tokens,
                     parents if B > 1 else None, fused_rows, traffic, stream.cuda_stream)

    # algorithmic bytes of one launch (visited states), counted by the kernel
    traffic = torch.zeros(2, dtype=torch.int64, device=dev)
    reset()
    run_once(traffic)
    torch.cuda.synchronize()
    alg_bytes, hyp_steps = (int(v) for v in traffic.cpu())
    ref_tokens = tokens.cpu().numpy().copy()
    ref_parents = parents.cpu().numpy().copy()
    assert F.fusion_device_status() == 0

    for _ in range(args.warmup):
        reset()
        run_once()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    tw = time.perf_counter()
    for i in range(args.steps):
        reset()
        starts[i].record(stream)
        run_once()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - tw
    kern_ms = float(np.mean([s.elapsed_time(e) for s, e in zip(starts, ends)]))
    assert np.array_equal(tokens.cpu().numpy(), ref_tokens), "non-deterministic decode"
    ms_per_step = wall * 1e3 / args.steps
    scores = float(T) * H * V
    value = scores / (ms_per_step / 1e3)
    achieved = alg_bytes / (kern_ms / 1e3) / 1e9
    log(f"fusion_run: {ms_per_step:.3f} ms/step wall, {kern_ms:.3f} ms kernel, {kern_ms * 1e3 / T:.2f} us/frame, "
        f"{alg_bytes / hyp_steps:.0f} B/hyp-step, {achieved:.1f} GB/s")

    copy = copy_bandwidth(torch, stream)
    log(f"device copy: {copy['gbs']:.0f} GB/s")
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "hyp×vocab scores/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "V": V, "lm_order": w.N, "ngrams": int(sum(w.lm.counts)),
            "ngrams_per_order": w.lm.counts, "lm_states": n_states, "lm_device_bytes": lm_bytes,
            "phrases": w.phrases.n, "trie_nodes": n_nodes, "streams": S, "beam": B,
            "hypotheses": H, "frames": T, "k": k, "lambda": w.lam, "beta": w.beta,
            "fused_rows_written": bool(args.fused),
        },
        "step_unit": "one fusion_run launch: all 300 frames of the 256 hypotheses (ms_per_step); "
                     "one decode step is one frame (us_per_frame)",
        "ms_per_launch_kernel": kern_ms,
        "us_per_frame": kern_ms * 1e3 / T,
        "decode_steps_per_s": T / (kern_ms / 1e3),
        "decode_steps_per_s_wall": T / (ms_per_step / 1e3),
        "table_build_s": t_load,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": None,
            "traffic_note": None,
            "algorithmic_bytes_per_launch": alg_bytes,
            "algorithmic_bytes_source": "kernel counter over the visited states (checked against an independent "
                                        "count in the tests and in cpu_baseline)",
            "bytes_per_hyp_step": alg_bytes / max(hyp_steps, 1),
            "hyp_steps_per_launch": hyp_steps,
            "kernel": "fusion_kernel",
            "copy_gbs": copy["gbs"],
            "frac_of_copy": achieved / copy["gbs"],
        },
        "copy_bandwidth": copy,
        "cpu_baseline": None,
    }

    # C5 with the full fused rows written (full-score mode), beside select-only
    if not args.fused:
        fz = torch.empty((T, H, V), dtype=torch.float32, device=dev)
        alg_f, steps_f, kms_f = time_leg(F, torch, dev, stream, reset, lambda tr: run_once(tr, fz),
                                         max(3, args.steps // 4))
        out["full_score"] = {"kernel": "fusion_kernel (fused rows written)", "kernel_ms_per_launch": kms_f,
                             "us_per_frame": kms_f * 1e3 / T, "value": scores / (kms_f / 1e3),
                             "unit": "hyp×vocab scores/s",
                             "roofline": leg_roofline(alg_f, steps_f, kms_f, None, copy["gbs"])}
        log(f"full-score mode: {kms_f:.3f} ms kernel, frac {alg_f / (kms_f / 1e3) / 1e9 / HBM_PEAK_GBS:.4f}")
        del fz
    out["fusion_step"] = step_leg(F, torch, dev, stream, w, lm, trie, x)

    if not args.no_projection:
        out["projection"] = projection_leg(F, torch, dev, stream, args.config, w, lm, trie)

    # Eq. (1) with two LMs: the same decode with a second, keyword 4-gram LM
    # (weights lambda, lambda), timed the same way; not part of the step above
    if not args.no_second_lm and args.config == 5:
        from workloads import make_keyword_lm

        t3 = time.time()
        lm2_arrays = make_keyword_lm(args.config)
        lm2 = F.ngram_load_arrays(lm2_arrays)
        n2_states, lm2_bytes = F.ngram_info(lm2)
        log(f"second LM: {lm2_arrays.counts} n-grams, {lm2_bytes / 1e9:.2f} GB, {time.time() - t3:.1f}s")
        lms2, alphas2 = [lm, lm2], [w.lam, w.lam]
        ls2_0 = torch.stack([ls0, torch.full((H,), F.ngram_bos_state(lm2), dtype=torch.int32, device=dev)])
        ls2 = ls2_0.clone()

        def reset2():
            ls2.copy_(ls2_0)
            bs.copy_(bs0)
            sc.copy_(sc0)

        def run2(traffic):
            F.fusion_run_lms(lms2, alphas2, trie, x, T, S, B, V, k, w.beta, w.blank, mode, ls2, bs, sc,
                             tokens, parents if B > 1 else None, None, traffic, stream=stream.cuda_stream)

        n2 = max(3, args.steps // 4)
        alg2, steps2, k2 = time_leg(F, torch, dev, stream, reset2, run2, n2)
        roof2 = leg_roofline(alg2, steps2, k2, recorded_traffic(w.name + "+keyword4", TRAFFIC_FILE_TWO_LMS))
        out["two_lms"] = {
            "kernel": "fusion_kernel (two LMs)", "launches": n2, "kernel_ms_per_launch": k2,
            "value": float(T) * H * V / (k2 / 1e3), "unit": "hyp×vocab scores/s",
            "decode_steps_per_s": T / (k2 / 1e3), "alphas": alphas2,
            "second_lm": {"kind": "keyword 4-gram (inserted phrases in Zipf carriers)",
                          "ngrams": int(sum(lm2_arrays.counts)), "ngrams_per_order": lm2_arrays.counts,
                          "lm_states": n2_states, "lm_device_bytes": lm2_bytes},
            "roofline": roof2,
        }
        log(f"two LMs: {k2:.3f} ms kernel, {alg2 / max(steps2, 1):.0f} B/hyp-step, {roof2['achieved']:.1f} GB/s")
        lm2.close()

    # the same decode with beam recombination (candidates that reach the same
    # history merge, log-summed): the kernel's recombining beam variant
    if not args.no_recombine and B > 1:
        ls1 = ls0.view(1, H)
        lsr = ls1.clone()

        def reset_rc():
            lsr.copy_(ls1)
            bs.copy_(bs0)
            sc.copy_(sc0)

        def run_rc(traffic):
            F.fusion_run_lms([lm], [w.lam], trie, x, T, S, B, V, k, w.beta, w.blank, mode, lsr, bs, sc, tokens,
                             parents, None, traffic, flags=F.FUSION_RUN_RECOMBINE, stream=stream.cuda_stream)

        n3 = max(3, args.steps // 4)
        alg3, steps3, k3 = time_leg(F, torch, dev, stream, reset_rc, run_rc, n3)
        roof3 = leg_roofline(alg3, steps3, k3, recorded_traffic(w.name + "+recombine", TRAFFIC_FILE_RC))
        out["recombining_beam"] = {
            "kernel": "fusion_kernel (beam with recombination)", "launches": n3, "kernel_ms_per_launch": k3,
            "value": float(T) * H * V / (k3 / 1e3), "unit": "hyp×vocab scores/s",
            "decode_steps_per_s": T / (k3 / 1e3),
            "roofline": roof3,
        }
        log(f"recombining beam: {k3:.3f} ms kernel, {alg3 / max(steps3, 1):.0f} B/hyp-step, {roof3['achieved']:.1f} GB/s")

    if not args.no_keyword:
        out["keyword_workload"] = keyword_leg(F, torch, dev, stream, max(3, args.steps // 4))

    rec = recorded_traffic(w.name)
    digest = kernel_sources_digest()
    if rec is None:
        out["roofline"]["traffic_note"] = "no PMC record for this workload under profiles/"
    elif rec[1] != digest:
        out["roofline"]["traffic_note"] = f"PMC record is for kernel sources {rec[1]}, these are {digest}"
    elif args.fused:
        out["roofline"]["traffic_note"] = "PMC record is for the run without fused rows"
    else:
        out["roofline"]["traffic"] = rec[0]
        out["roofline"]["hbm_traffic_gbs"] = rec[0] / (kern_ms / 1e3) / 1e9
        out["roofline"]["traffic_note"] = ("HBM bytes per launch: rocprofv3 FETCH_SIZE + WRITE_SIZE, each scaled "
                                           "by the counter's reading for a plain copy of known size; "
                                           "hbm_traffic_gbs is that over the kernel time")

    # the main step's tables are released before the other workloads are built
    lm.close()
    trie.close()
    del x, tokens, parents, fused, ls, bs, sc, ls0, bs0, sc0
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    if not args.no_configs:
        out["configs"] = {}
        for cfg in (1, 2, 3, 4):
            if cfg == args.config:
                continue
            out["configs"][f"c{cfg}"] = config_leg(F, torch, dev, stream, cfg, 5, copy["gbs"])
            torch.cuda.empty_cache()

    if not args.no_cpu:
        from oracle import traffic as checker

        n_thr = min(len(os.sched_getaffinity(0)), HOST_THREADS_CAP)
        olm, otr, r, sec, Sc, Tc, agree, near = cpu_leg(w, ref_tokens, ref_parents, bos, n_thr, args.cpu_streams,
                                                      args.cpu_frames)
        cpu_scores = float(Tc) * Sc * B * V / sec
        log(f"oracle on {n_thr} threads: {sec:.1f}s, {cpu_scores:.3g} scores/s, agrees={agree}")
        # the independent count of the algorithmic bytes, from the states the
        # oracle's (replayed) decode visits
        chk = None
        if Sc == S and Tc == T:
            visits = checker.visited_states(olm, otr, V, w.blank, B, r["tokens"], r["parents"])
            chk, chk_steps = checker.algorithmic_bytes(w.lm, w.phrases, visits, T, beam=B > 1)
            out["roofline"]["algorithmic_bytes_checker"] = chk
            out["roofline"]["algorithmic_bytes_agree"] = bool(chk == alg_bytes and chk_steps == hyp_steps)
            log(f"checker: {chk} algorithmic bytes over {chk_steps} hyp-steps (kernel {alg_bytes}, {hyp_steps})")
        _, _, _, sec1, Sc1, Tc1, agree1, _ = cpu_leg(w, ref_tokens, ref_parents, bos, 1, args.cpu_streams_single,
                                                     args.cpu_frames)
        cpu1 = float(Tc1) * Sc1 * B * V / sec1
        log(f"oracle on 1 thread: {sec1:.1f}s, {cpu1:.3g} scores/s")
        out["cpu_baseline"] = {
            "value": cpu_scores, "unit": "hyp×vocab scores/s", "cores": n_thr, "kind": "oracle",
            "sample": f"first {Tc} frames of {Sc} of the {S} streams (beam {B}), {Sc * B * Tc} hyp-steps, "
                      f"{sec:.1f}s on {n_thr} threads (host threads capped at {HOST_THREADS_CAP}, the CPU share "
                      f"of one GPU; {os.cpu_count()} logical CPUs visible); GPU decisions on the sample agree "
                      f"with the oracle: {agree} (near ties accepted: {near})",
            "cpu_model": cpu_model(),
            "single_thread": {"value": cpu1, "unit": "hyp×vocab scores/s", "cores": 1,
                              "sample": f"first {Tc1} frames of {Sc1} streams (beam {B}), {Sc1 * B * Tc1} hyp-steps, "
                                        f"{sec1:.1f}s; agree: {agree1}"},
        }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
