"""Oracle of the joint output projection (test infrastructure only).

TEST INFRASTRUCTURE ONLY: used by the tests and the benchmark; the product
path never imports it.

The joint network of the Transducer produces, per hypothesis-frame, the
logits whose log-softmax is the acoustic term of Eq. (1) (Sec. III-C).  Its
output projection is the plain matrix product

    out[m, n] = sum_k A[m, k] * W[n, k] + bias[n]

evaluated here exactly in fp64 from the bf16 inputs (every bf16 value and
every product of two of them is exact in fp64; the K-term sums of the
workloads stay far inside fp64's exact range for the bound below to hold).
"""

from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24  # unit roundoff of fp32


def bf16_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns -> float64: the pattern is the top half of an fp32."""
    b = np.ascontiguousarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def joint_project(A_bits, W_bits, bias=None) -> np.ndarray:
    """fp64 out[m, n] = sum_k A[m, k] W[n, k] + bias[n]."""
    A = bf16_to_f64(A_bits)
    W = bf16_to_f64(W_bits)
    out = A @ W.T
    if bias is not None:
        out = out + np.asarray(bias, dtype=np.float64)[None, :]
    return out


def fp32_error_bound(A_bits, W_bits, bias=None) -> np.ndarray:
    """Largest |fp32 result - exact| of any fp32 evaluation that forms the K
    products exactly (8-bit significands: exact in fp32), sums them in any
    order with one rounding per addition, then adds the bias:

        |s^ - s| <= g * sum_k |a_k w_k|,   g = (K-1) u / (1 - (K-1) u)
        |r^ - (s + b)| <= |s^ - s| + u * (|s + b| + |s^ - s|)
    """
    A = np.abs(bf16_to_f64(A_bits))
    W = np.abs(bf16_to_f64(W_bits))
    K = A.shape[1]
    g = (K - 1) * U32 / (1.0 - (K - 1) * U32)
    e_sum = g * (A @ W.T)
    exact = joint_project(A_bits, W_bits, bias)
    return e_sum + U32 * (np.abs(exact) + e_sum)
