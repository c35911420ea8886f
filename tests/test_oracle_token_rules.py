"""Pins of the oracle's gate network and query-dependent lambda.

Closed forms from the definitions (SiLU and sigmoid at points with exact
values), the initial value the paper states for lambda_i, the floor, central
finite differences of the hand-derived gradients, and torch autograd through
torch's own SiLU and sigmoid (an implementation independent of the oracle's).
"""
import math

import numpy as np
import torch

from oracle import token_rules as TR


def _params(rng, n, d, G):
    return (rng.standard_normal((n, d)), rng.standard_normal((G, d)) * 0.4, rng.standard_normal(G) * 0.3,
            rng.standard_normal((2, G)) * 0.4, rng.standard_normal(2) * 0.3)


def test_gate_closed_form_with_zero_first_layer():
    # W1 = 0 leaves z1 = b1.  b1 = (ln 3, 0): SiLU(ln 3) = ln 3 * 3/4, SiLU(0) = 0.
    # W2 = I, b2 = (0, ln 2): z2 = (0.75 ln 3, ln 2), so
    # g_sparse = 3^0.75 / (1 + 3^0.75) and g_lr = 2/3 for every token.
    q = np.random.default_rng(0).standard_normal((5, 4))
    g = TR.gate_forward(q, np.zeros((2, 4)), [math.log(3.0), 0.0], np.eye(2), [0.0, math.log(2.0)])
    t = 3.0 ** 0.75
    assert np.allclose(g[:, 0], t / (1.0 + t), rtol=0, atol=1e-15)
    assert np.allclose(g[:, 1], 2.0 / 3.0, rtol=0, atol=1e-15)


def test_gate_second_layer_picks_hidden_units():
    # One-hot W2 rows read single hidden units: g = sigmoid(SiLU(z1_j)).
    rng = np.random.default_rng(1)
    q, W1, b1, _, _ = _params(rng, 6, 5, 3)
    W2 = np.array([[0.0, 1.0, 0.0], [0.0, 0.0, 1.0]])
    g = TR.gate_forward(q, W1, b1, W2, np.zeros(2))
    for i in range(6):
        for o, j in ((0, 1), (1, 2)):
            z = float(np.dot(W1[j], q[i]) + b1[j])
            silu = z / (1.0 + math.exp(-z))
            assert abs(g[i, o] - 1.0 / (1.0 + math.exp(-silu))) < 1e-15


def test_gates_lie_in_the_open_unit_interval():
    rng = np.random.default_rng(2)
    g = TR.gate_forward(*_params(rng, 200, 16, 8))
    assert np.all(g > 0.0) and np.all(g < 1.0)


def test_gate_backward_matches_finite_differences():
    rng = np.random.default_rng(3)
    q, W1, b1, W2, b2 = _params(rng, 7, 6, 4)
    dg = rng.standard_normal((7, 2))
    got = TR.gate_backward(q, W1, b1, W2, b2, dg)
    args = {"dq": q, "dW1": W1, "db1": b1, "dW2": W2, "db2": b2}
    h = 1e-6
    for name, x in args.items():
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + h
            fp = float(np.sum(dg * TR.gate_forward(q, W1, b1, W2, b2)))
            x[idx] = old - h
            fm = float(np.sum(dg * TR.gate_forward(q, W1, b1, W2, b2)))
            x[idx] = old
            fd[idx] = (fp - fm) / (2 * h)
        assert np.max(np.abs(got[name] - fd)) < 1e-8, name


def test_gate_backward_matches_torch_autograd():
    rng = np.random.default_rng(4)
    q, W1, b1, W2, b2 = _params(rng, 33, 16, 8)
    dg = rng.standard_normal((33, 2))
    got = TR.gate_backward(q, W1, b1, W2, b2, dg)
    T = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, W1, b1, W2, b2)]
    g = torch.sigmoid(torch.nn.functional.silu(T[0] @ T[1].T + T[2]) @ T[3].T + T[4])
    assert np.max(np.abs(g.detach().numpy() - TR.gate_forward(q, W1, b1, W2, b2))) < 1e-14
    (g * torch.tensor(dg)).sum().backward()
    for t, name in zip(T, ("dq", "dW1", "db1", "dW2", "db2")):
        assert np.max(np.abs(t.grad.numpy() - got[name])) < 1e-12, name


def test_lambda_initial_value_is_the_stated_average_target():
    # c = 0.3 and a zero bias give 0.3 + sigmoid(0) = 0.8 (the stated initial
    # average target); w ~ N(0, 1e-3^2) keeps every lambda_i within 1e-2 of it.
    rng = np.random.default_rng(5)
    q = rng.standard_normal((4096, 128))
    assert np.all(TR.lambda_forward(q, np.zeros(128), 0.0, 0.3) == 0.8)
    lam = TR.lambda_forward(q, rng.standard_normal(128) * 1e-3, 0.0, 0.3)
    assert abs(lam.mean() - 0.8) < 1e-3 and np.max(np.abs(lam - 0.8)) < 1e-2


def test_lambda_floor_and_its_zero_gradient():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((9, 4))
    w = rng.standard_normal(4) * 0.1
    lam = TR.lambda_forward(q, w, -60.0, 0.0)
    assert np.all(lam == 1e-6)
    g = TR.lambda_backward(q, w, -60.0, 0.0, rng.standard_normal(9))
    assert g["dc"] == 0.0 and g["db"] == 0.0 and np.all(g["dw"] == 0.0)


def test_lambda_backward_matches_finite_differences_and_autograd():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((11, 5))
    w, b, c = rng.standard_normal(5) * 0.5, 0.2, 0.3
    dl = rng.standard_normal(11)
    got = TR.lambda_backward(q, w, b, c, dl)
    f = lambda w_, b_, c_: float(np.sum(dl * TR.lambda_forward(q, w_, b_, c_)))   # noqa: E731
    h = 1e-6
    fd_w = np.array([(f(w + h * e, b, c) - f(w - h * e, b, c)) / (2 * h) for e in np.eye(5)])
    assert np.max(np.abs(got["dw"] - fd_w)) < 1e-8
    assert abs(got["db"] - (f(w, b + h, c) - f(w, b - h, c)) / (2 * h)) < 1e-8
    assert abs(got["dc"] - (f(w, b, c + h) - f(w, b, c - h)) / (2 * h)) < 1e-8
    T = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (w, [b], [c])]
    lam = torch.clamp(T[2] + torch.sigmoid(torch.tensor(q) @ T[0] + T[1]), min=1e-6)
    (lam * torch.tensor(dl)).sum().backward()
    assert np.max(np.abs(T[0].grad.numpy() - got["dw"])) < 1e-12
    assert abs(T[1].grad.item() - got["db"]) < 1e-12 and abs(T[2].grad.item() - got["dc"]) < 1e-12
