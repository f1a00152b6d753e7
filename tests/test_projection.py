"""Joint output projection: the oracle pinned on the CPU, the MFMA kernel
against the oracle on the GPU.

The projection produces the logits whose log-softmax is the acoustic term of
Eq. (1) (Sec. III-C).  Parity bar: every output within the fp32 error bound
of the oracle (``oracle.projection.fp32_error_bound``: exact products, K-1
roundings of the sum in any order, one rounding for the bias).
"""

from __future__ import annotations

import ctypes

import numpy as np
import pytest

from oracle.projection import U32, bf16_to_f64, fp32_error_bound, joint_project
from workloads import make_projection, to_bf16_bits


# ---------------------------------------------------------------------------
# pins of the oracle (CPU)
# ---------------------------------------------------------------------------
def test_bf16_decoding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint32).astype(np.uint16)
    # drop NaN patterns (exponent all ones, nonzero mantissa): compare values only
    finite = ((bits >> 7) & 0xFF) != 0xFF
    bits = bits[finite]
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    assert np.array_equal(bf16_to_f64(bits), ref)


def test_bf16_encoding_rounds_to_nearest_even_like_torch():
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(3).standard_normal(20000).astype(np.float32) * 7
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(to_bf16_bits(x), ref)


def test_projection_on_exact_integers_equals_brute_force():
    # small integers are exact in bf16 and every sum is exact, so the oracle
    # must equal integer arithmetic; M != N != K catches a transposed operand
    rng = np.random.default_rng(11)
    M, N, K = 5, 7, 24
    a = rng.integers(-8, 9, size=(M, K))
    w = rng.integers(-8, 9, size=(N, K))
    bias = rng.integers(-50, 51, size=N)
    got = joint_project(to_bf16_bits(a.astype(np.float32)), to_bf16_bits(w.astype(np.float32)),
                        bias.astype(np.float32))
    for m in range(M):
        for n in range(N):
            s = sum(int(a[m, k]) * int(w[n, k]) for k in range(K)) + int(bias[n])
            assert got[m, n] == s


def test_bias_is_per_output_column():
    A, W, _ = make_projection(5, M=3, N=9, K=16)
    bias = np.arange(9, dtype=np.float32)
    d = joint_project(A, W, bias) - joint_project(A, W, None)
    assert np.array_equal(d, np.tile(np.arange(9, dtype=np.float64), (3, 1)))


def test_error_bound_covers_sequential_fp32_and_is_tight_enough():
    A, W, bias = make_projection(5, M=16, N=64, K=640)
    exact = joint_project(A, W, bias)
    bound = fp32_error_bound(A, W, bias)
    a32 = bf16_to_f64(A).astype(np.float32)
    w32 = bf16_to_f64(W).astype(np.float32)
    seq = np.zeros((16, 64), dtype=np.float32)
    for k in range(640):  # one fp32 rounding per addition, in index order
        seq = seq + a32[:, k:k + 1] * w32[None, :, k]
    seq = seq + bias[None, :]
    assert np.all(np.abs(seq.astype(np.float64) - exact) <= bound)
    # the bound is a few hundred ulps of the sum of |products|, no looser
    assert np.all(bound <= 700 * U32 * (np.abs(bf16_to_f64(A)) @ np.abs(bf16_to_f64(W)).T) + 1e-6)


# ---------------------------------------------------------------------------
# GPU parity through the C ABI
# ---------------------------------------------------------------------------
def _run(A, W, bias):
    import torch

    import paper_2609_14991_amd as F

    dev = torch.device("cuda:0")
    a = torch.from_numpy(A.view(np.int16)).to(dev)
    w = torch.from_numpy(W.view(np.int16)).to(dev)
    b = None if bias is None else torch.from_numpy(bias).to(dev)
    out = torch.full((A.shape[0], W.shape[0]), float("nan"), dtype=torch.float32, device=dev)
    F.joint_project(a, w, b, A.shape[0], W.shape[0], A.shape[1], out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check(A, W, bias, rows=None):
    got = _run(A, W, bias)
    if rows is not None:
        got, A = got[rows], A[rows]
    exact = joint_project(A, W, bias)
    bound = fp32_error_bound(A, W, bias)
    err = np.abs(got.astype(np.float64) - exact)
    assert np.all(np.isfinite(got))
    bad = np.argwhere(err > bound)
    assert bad.size == 0, f"{bad.shape[0]} outputs outside the bound, first {bad[:3]}"
    return float((err / np.maximum(bound, 1e-300)).max())


@pytest.mark.gpu
def test_projection_one_c5_frame():
    A, W, bias = make_projection(5, M=256)
    print("max error / bound", _check(A, W, bias))


@pytest.mark.gpu
@pytest.mark.parametrize("M,N,K", [(100, 1000, 40), (1, 16, 8), (129, 130, 648), (300, 4096, 64),
                                   (257, 1024, 640)])
def test_projection_ragged_shapes(M, N, K):
    A, W, bias = make_projection(5, M=M, N=N, K=K)
    _check(A, W, bias)
    _check(A, W, None)


@pytest.mark.gpu
def test_projection_full_c5_run_sampled_rows():
    # all 300 frames x 256 hypotheses in one launch (the shape bench.py times);
    # the oracle checks a sample of rows, every column
    A, W, bias = make_projection(5)
    rows = np.random.default_rng(5).choice(A.shape[0], size=384, replace=False)
    rows.sort()
    _check(A, W, bias, rows=rows)


@pytest.mark.gpu
def test_projection_argument_errors():
    import torch

    import paper_2609_14991_amd as F

    dev = torch.device("cuda:0")
    a = torch.zeros((4, 64), dtype=torch.int16, device=dev)
    w = torch.zeros((8, 64), dtype=torch.int16, device=dev)
    out = torch.zeros((4, 8), dtype=torch.float32, device=dev)
    L = F.lib()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = ctypes.c_void_p
    assert L.joint_project(P(a.data_ptr()), P(w.data_ptr()), None, 4, 8, 60, P(out.data_ptr()), s) == F.FUSION_E_UNSUPPORTED
    assert L.joint_project(P(a.data_ptr()), P(w.data_ptr()), None, 4, 8, 4, P(out.data_ptr()), s) == F.FUSION_E_ARG
    assert L.joint_project(P(a.data_ptr() + 2), P(w.data_ptr()), None, 4, 8, 64, P(out.data_ptr()), s) == F.FUSION_E_ARG
    assert L.joint_project(None, P(w.data_ptr()), None, 4, 8, 64, P(out.data_ptr()), s) == F.FUSION_E_ARG
    assert L.joint_project(None, None, None, 0, 8, 64, None, s) == F.FUSION_OK  # M = 0: nothing to do
    torch.cuda.synchronize()
