"""Token-wise rules of the fusion: the gate network and the query-dependent
lambda (test infrastructure only).

Sec. 3.3 and Alg. 1 take the two gates as sigmoid(G_theta(q_i)); the setup
of the experiments makes G_theta a two-layer MLP with a SiLU between the
layers and two independent sigmoid outputs (one per branch), unnormalised,
with hidden width 64 (text) or 128 (vision).  The appendix on the ELSAA
configuration gives the query-dependent coefficient
    lambda_i = c + sigmoid(w^T q_i + b),
with c >= 0 learnable, q_i detached from this path and a floor
lambda_min = 1e-6.  Readings taken here:
  * the gate input is the head's query q_i and every head has its own
    parameters (W1 [G, d_h], b1 [G], W2 [2, G], b2 [2]), so that the gates
    are token- and head-wise like the fusion they feed;
  * the floor is applied as lambda_i = max(lambda_min, c + sigmoid(.)), and
    its gradient passes where c + sigmoid(.) >= lambda_min (zero below);
  * c is used as given (the caller keeps it nonnegative).
Arithmetic is float64 numpy; numpy's matmul is the only library primitive.
The backward is derived by hand from the chain rule, step by step in the
reverse order of the forward.
"""
from __future__ import annotations

import numpy as np


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def gate_forward(q, W1, b1, W2, b2) -> np.ndarray:
    """Gates (g_sparse, g_lr) = sigmoid(W2 silu(W1 q_i + b1) + b2) of every row
    of q [n, d]; returns [n, 2]."""
    q = np.asarray(q, np.float64)
    z1 = q @ np.asarray(W1, np.float64).T + np.asarray(b1, np.float64)
    a = z1 * _sigmoid(z1)
    z2 = a @ np.asarray(W2, np.float64).T + np.asarray(b2, np.float64)
    return _sigmoid(z2)


def gate_backward(q, W1, b1, W2, b2, dg) -> dict:
    """Gradients of sum(dg * gates) with respect to q, W1, b1, W2, b2."""
    q = np.asarray(q, np.float64)
    W1 = np.asarray(W1, np.float64)
    W2 = np.asarray(W2, np.float64)
    dg = np.asarray(dg, np.float64)
    z1 = q @ W1.T + np.asarray(b1, np.float64)
    s1 = _sigmoid(z1)
    a = z1 * s1
    g = _sigmoid(a @ W2.T + np.asarray(b2, np.float64))
    dz2 = dg * g * (1.0 - g)                      # through the output sigmoid
    da = dz2 @ W2                                 # through the second layer
    dz1 = da * (s1 * (1.0 + z1 * (1.0 - s1)))     # SiLU'(z) = s (1 + z (1 - s))
    return {"dq": dz1 @ W1, "dW1": dz1.T @ q, "db1": dz1.sum(0),
            "dW2": dz2.T @ a, "db2": dz2.sum(0)}


def lambda_forward(q, w, b: float, c: float, lambda_min: float = 1e-6) -> np.ndarray:
    """lambda_i = max(lambda_min, c + sigmoid(w^T q_i + b)) of every row of q."""
    z = np.asarray(q, np.float64) @ np.asarray(w, np.float64) + b
    return np.maximum(lambda_min, c + _sigmoid(z))


def lambda_backward(q, w, b: float, c: float, dlam, lambda_min: float = 1e-6) -> dict:
    """Gradients of sum(dlam * lambda) with respect to w, b and c (q is
    detached from this path, so it receives none)."""
    q = np.asarray(q, np.float64)
    s = _sigmoid(q @ np.asarray(w, np.float64) + b)
    e = np.asarray(dlam, np.float64) * (c + s >= lambda_min)
    t = e * s * (1.0 - s)
    return {"dw": q.T @ t, "db": float(t.sum()), "dc": float(e.sum())}
