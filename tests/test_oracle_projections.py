"""Pins of the projection reference (oracle/projections.py) against what the
definitions fix independently: brute-force sums, the head-major index map
written per element, and algebraic identities of the matrix product."""
import itertools

import numpy as np
import pytest

import oracle


def _brute(A, B, ta, tb):
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    M = A.shape[1] if ta else A.shape[0]
    K = A.shape[0] if ta else A.shape[1]
    N = B.shape[0] if tb else B.shape[1]
    C = [[0.0] * N for _ in range(M)]
    for i in range(M):
        for j in range(N):
            s = 0.0
            for k in range(K):
                a = A[k][i] if ta else A[i][k]
                b = B[j][k] if tb else B[k][j]
                s += a * b
            C[i][j] = s
    return np.array(C)


@pytest.mark.parametrize("ta,tb", list(itertools.product([False, True], repeat=2)))
def test_gemm_matches_brute_force(ta, tb):
    rng = np.random.default_rng([7, int(ta), int(tb)])
    M, N, K = 5, 7, 6
    A = rng.standard_normal((K, M) if ta else (M, K))
    B = rng.standard_normal((N, K) if tb else (K, N))
    np.testing.assert_allclose(oracle.gemm(A, B, ta, tb), _brute(A, B, ta, tb), rtol=1e-13, atol=1e-13)


def test_gemm_transpose_identity():
    # (A B)^T = B^T A^T, computed through the trans flags only
    rng = np.random.default_rng(3)
    A, B = rng.standard_normal((6, 4)), rng.standard_normal((4, 9))
    np.testing.assert_allclose(oracle.gemm(A, B).T, oracle.gemm(B, A, True, True), rtol=1e-13, atol=1e-13)
    np.testing.assert_array_equal(oracle.gemm(A, np.eye(4)), A)


def test_head_major_map_per_element():
    rng = np.random.default_rng(11)
    B, H, S, dh = 2, 3, 5, 4
    t = rng.standard_normal((B, H, S, dh))
    X = oracle.heads_to_matrix(t)
    assert X.shape == (B * S, H * dh)
    for b, h, n, e in itertools.product(range(B), range(H), range(S), range(dh)):
        assert X[b * S + n, h * dh + e] == t[b, h, n, e]
    np.testing.assert_array_equal(oracle.matrix_to_heads(X, H, S), t)
    # the same map as a reshape / transpose chain
    np.testing.assert_array_equal(X, t.transpose(0, 2, 1, 3).reshape(B * S, H * dh))


def test_projection_of_heads_is_per_head_product():
    # (X W)[:, head h] = X W[:, head h]: a head-major output stores each head's
    # own projection
    rng = np.random.default_rng(5)
    S, dm, H = 6, 8, 2
    X, W = rng.standard_normal((S, dm)), rng.standard_normal((dm, dm))
    Q = oracle.matrix_to_heads(oracle.gemm(X, W), H, S)
    for h in range(H):
        np.testing.assert_allclose(Q[0, h], _brute(X, W[:, h * 4:(h + 1) * 4], False, False), rtol=1e-13, atol=1e-13)
