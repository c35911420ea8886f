"""Pins of the oracle's variants of the operator that the paper names:
r neighbouring sorted blocks (Sec. 6 cost discussion, "Neighbor blocks" in the
hyper-parameter table), a per-token coefficient lambda_i in Eq. (m_sparse) with
its gradient (the learned and query-dependent lambda of the appendix), and the
Sort_Lsh_RACE ablation m_sparse = 1 (Sec. 7).  Checked against brute force
(explicit supports, materialised passes), PyTorch float64 autograd of the
materialised forward, finite differences and closed forms.  CPU only."""
import numpy as np
import pytest
import torch

import bruteforce as bf
import oracle
from test_oracle_pins import _csr_to_mask, _pad_key, _rng, _tiny


@pytest.mark.parametrize("N,k,r", [(40, 8, 1), (48, 8, 2), (37, 6, 1)])
def test_neighbor_blocks_noncausal_support(N, k, r):
    cfg, Q, K, V, Ws, Wr = _tiny(31, N, 8, k, 32, False)
    cfg.neighbors = r
    rp, cols = oracle.support(cfg, Q, K, Ws)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    np.testing.assert_array_equal(_csr_to_mask(N, rp, cols), bf.noncausal_support_mask(N, k, kq, kk, r))
    # closed form: query at sorted block t sees key positions [max(0,(t-r)k), min(N,(t+r+1)k))
    nb = (N + k - 1) // k
    want = sum(min(N, (t + r + 1) * k) - max(0, (t - r) * k) for t in range(nb)
               for _ in range(min(k, N - t * k)))
    assert rp[-1] == want


@pytest.mark.parametrize("N,n0,k,r", [(64, 16, 8, 1), (96, 12, 4, 2)])
def test_neighbor_blocks_causal_support_equals_literal_recursion(N, n0, k, r):
    cfg, Q, K, V, Ws, Wr = _tiny(32, N, 8, k, 32, True, n0=n0)
    cfg.neighbors = r
    rp, cols = oracle.support(cfg, Q, K, Ws)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    want = bf.causal_support_mask(N, n0, k, kq, kk, _pad_key(Ws), r)
    np.testing.assert_array_equal(_csr_to_mask(N, rp, cols), want)


def test_zero_neighbors_is_the_main_setting():
    cfg, Q, K, V, Ws, Wr = _tiny(33, 64, 8, 8, 32, True, n0=16)
    a = oracle.forward(cfg, Q, K, V, Ws, Wr)
    cfg.neighbors = 0
    b = oracle.forward(cfg, Q, K, V, Ws, Wr)
    np.testing.assert_array_equal(a["O"], b["O"])


@pytest.mark.parametrize("causal,m_one", [(True, False), (False, False), (True, True)])
def test_per_token_lambda_and_m_one_forward_equal_materialised(causal, m_one):
    N = 48
    rng = _rng(34, int(causal), int(m_one))
    cfg, Q, K, V, Ws, Wr = _tiny(34, N, 8, 8, 32, causal, n0=12 if causal else None, beta=0.8)
    cfg.m_one = m_one
    lam = rng.uniform(0.05, 3.0, N).astype(np.float32)
    gates = rng.uniform(0.1, 0.9, (N, 2)).astype(np.float32)
    got = oracle.forward(cfg, Q, K, V, Ws, Wr, gates=gates, lam_rows=lam)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    mask = (bf.causal_support_mask(N, 12, 8, kq, kk, _pad_key(Ws)) if causal
            else bf.noncausal_support_mask(N, 8, kq, kk))
    phq = bf.race_features_sigmoid(Q, Wr, cfg.beta)
    phk = bf.race_features_sigmoid(K, Wr, cfg.beta)
    ref = bf.dense_forward_np(Q, K, V, mask, phq, phk, Wr.shape[0], causal, cfg.eps, lam.astype(np.float64),
                              1 / np.sqrt(8), gates, m_one=m_one)
    for key in ("O", "m", "O_s", "O_lr"):
        np.testing.assert_allclose(got[key], ref[key], rtol=1e-10, atol=1e-12, err_msg=key)


@pytest.mark.parametrize("causal,m_one", [(True, False), (False, False), (True, True)])
def test_backward_with_per_token_lambda_matches_torch_autograd(causal, m_one):
    N = 40
    rng = _rng(35, int(causal), int(m_one))
    cfg, Q, K, V, Ws, Wr = _tiny(35, N, 8, 8, 32, causal, n0=10 if causal else None, beta=0.9)
    cfg.m_one = m_one
    lam = rng.uniform(0.05, 3.0, N).astype(np.float32)
    gates = rng.uniform(0.1, 0.9, (N, 2)).astype(np.float32)
    dO = rng.standard_normal((N, 8)).astype(np.float32)
    g = oracle.backward(cfg, Q, K, V, Ws, Wr, dO, gates=gates, lam_rows=lam)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    mask = (bf.causal_support_mask(N, 10, 8, kq, kk, _pad_key(Ws)) if causal
            else bf.noncausal_support_mask(N, 8, kq, kk))
    tQ, tK, tV = (torch.tensor(a.astype(np.float64), requires_grad=True) for a in (Q, K, V))
    tG = torch.tensor(gates.astype(np.float64), requires_grad=True)
    tL = torch.tensor(lam.astype(np.float64), requires_grad=True)
    O = bf.dense_forward_torch(tQ, tK, tV, mask, Wr, cfg.beta, causal, cfg.eps, tL, 1 / np.sqrt(8), tG,
                               m_one=m_one)
    (O * torch.tensor(dO.astype(np.float64))).sum().backward()
    for t, key in ((tQ, "dQ"), (tK, "dK"), (tV, "dV"), (tG, "dgates"), (tL, "dlambda")):
        ref = t.grad.numpy() if t.grad is not None else np.zeros_like(g[key])
        assert np.max(np.abs(g[key] - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref))), key
    if m_one:
        assert np.all(g["dlambda"] == 0.0)


def test_scalar_lambda_gradient_is_sum_of_per_token_gradients_by_finite_differences():
    # d/dlambda of sum(O * dO) for the scalar lambda, by central differences of
    # the oracle forward, equals the sum of the per-token gradients
    N = 48
    rng = _rng(36)
    cfg, Q, K, V, Ws, Wr = _tiny(36, N, 8, 8, 32, True, n0=12, lam=0.7)
    dO = rng.standard_normal((N, 8)).astype(np.float32)
    g = oracle.backward(cfg, Q, K, V, Ws, Wr, dO)
    h = 1e-5
    vals = []
    for lam in (0.7 + h, 0.7 - h):
        cfg.lam = lam
        vals.append(float(np.sum(oracle.forward(cfg, Q, K, V, Ws, Wr)["O"] * dO.astype(np.float64))))
    fd = (vals[0] - vals[1]) / (2 * h)
    assert abs(g["dlambda"].sum() - fd) <= 1e-6 * max(1.0, abs(fd))
