"""Dense projections of the attention block (test infrastructure only).

Alg. 1 and Alg. 6 form Q = X W_Q, K = X W_K, V = X W_V before the operator
and return O_head W_O after it; the paper keeps these matrices dense.  The
reference is the definition: float64 matrix products (numpy's matmul as the
library primitive) of the logical matrices, with the head-major storage of
attention tensors spelled out element by element.

Head-major storage: a [B*S, H*dh] matrix whose row b*S + n and column
h*dh + e is kept at [b, h, n, e] of a [B, H, S, dh] tensor.
"""
from __future__ import annotations

import numpy as np


def heads_to_matrix(t) -> np.ndarray:
    """[B, H, S, dh] head-major tensor -> the [B*S, H*dh] matrix it stores."""
    t = np.asarray(t, dtype=np.float64)
    B, H, S, dh = t.shape
    X = np.empty((B * S, H * dh))
    for b in range(B):
        for h in range(H):
            X[b * S:(b + 1) * S, h * dh:(h + 1) * dh] = t[b, h]
    return X


def matrix_to_heads(X, H: int, S: int) -> np.ndarray:
    """[B*S, H*dh] matrix -> its [B, H, S, dh] head-major tensor."""
    X = np.asarray(X, dtype=np.float64)
    R, Cc = X.shape
    B, dh = R // S, Cc // H
    t = np.empty((B, H, S, dh))
    for b in range(B):
        for h in range(H):
            t[b, h] = X[b * S:(b + 1) * S, h * dh:(h + 1) * dh]
    return t


def gemm(A, B, trans_a: bool = False, trans_b: bool = False) -> np.ndarray:
    """op(A) op(B) in float64, op(X) = X^T when trans_x."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    return (A.T if trans_a else A) @ (B.T if trans_b else B)
