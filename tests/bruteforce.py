"""Independent brute-force checks used to pin the CPU reference.

Written separately from ``oracle/`` (no shared code): a literal Python
run of the causal divide-and-conquer of Alg. 5 that builds an explicit
N x N support mask, NumPy float64 hash projections, RACE features in their
product-of-sigmoids form, and materialised N x N forward passes (NumPy and
PyTorch float64, the latter differentiable).  Only for tiny inputs.
"""
from __future__ import annotations

import numpy as np
import torch


def gray(n: int) -> int:
    """Reflected Gray code of n."""
    return n ^ (n >> 1)


def sign_codes64(X: np.ndarray, W: np.ndarray):
    """Sign code of every row (bit t = <W_t, x> > 0) in float64, with margins."""
    P = X.astype(np.float64) @ W.astype(np.float64).T
    scale = np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T
    code = ((P > 0).astype(np.int64) << np.arange(W.shape[0])).sum(axis=1)
    margin = np.min(np.abs(P) / np.maximum(scale, 1e-300), axis=1)
    return code, margin


def bucket_from_code(code: int, bits: int) -> int:
    """Position of ``code`` in the reflected Gray sequence (searched, not inverted)."""
    for p in range(1 << bits):
        if gray(p) == code:
            return p
    raise ValueError(code)


def keys64(X, W):
    code, margin = sign_codes64(X, W)
    bits = W.shape[0]
    return np.array([bucket_from_code(int(c), bits) for c in code]), margin


def with_margin(rng, shape, W, min_margin=1e-3, scale=1.0):
    """Draw rows ~ N(0, scale^2) whose projections on W all clear ``min_margin``."""
    X = (rng.standard_normal(shape) * scale).astype(np.float32)
    for _ in range(1000):
        _, m = sign_codes64(X, W)
        bad = m < min_margin
        if not bad.any():
            return X
        X[bad] = (rng.standard_normal((int(bad.sum()), shape[1])) * scale).astype(np.float32)
    raise RuntimeError("could not draw rows with hash margin")


# --------------------------------------------------------------------------
# Alg. 5 run literally on Python lists
# --------------------------------------------------------------------------

PAD = None


def _sortlsh_pairs(qs, ks, kq, kk, pad_key, b, r=0):
    """Pairs (query, key) of SortLSH(qs, ks; b): sort by (hash, position), equal
    blocks; query block t sees key blocks t - r .. t + r (those that exist)."""
    def hk(tok, table):
        return pad_key if tok is PAD else table[tok]
    oq = sorted(range(len(qs)), key=lambda p: (hk(qs[p], kq), p))
    ok = sorted(range(len(ks)), key=lambda p: (hk(ks[p], kk), p))
    bb = min(b, len(qs))
    key_blocks = [ok[t0:t0 + bb] for t0 in range(0, len(ks), bb)]
    out = []
    for t, t0 in enumerate(range(0, len(qs), bb)):
        seen = [q for u in range(t - r, t + r + 1) if 0 <= u < len(key_blocks) for q in key_blocks[u]]
        for p in oq[t0:t0 + bb]:
            for q in seen:
                out.append((qs[p], ks[q]))
    return out


def causal_support_mask(N, n0, b, kq, kk, pad_key=0, r=0):
    """N x N boolean support of Alg. 5's CausalSparse (padding tokens dropped);
    r neighbouring blocks per SortLSH call."""
    M = np.zeros((N, N), dtype=np.int64)

    def rec(toks):
        n = len(toks)
        if n <= n0:
            for p in range(n):
                for q in range(p + 1):
                    if toks[p] is not PAD and toks[q] is not PAD:
                        M[toks[p], toks[q]] += 1
            return
        if n % 2:
            toks = toks + [PAD]
        m = len(toks) // 2
        rec(toks[:m])
        rec(toks[m:])
        for i, j in _sortlsh_pairs(toks[m:], toks[:m], kq, kk, pad_key, b, r):
            if i is not PAD and j is not PAD:
                M[i, j] += 1

    rec(list(range(N)))
    return M


def noncausal_support_mask(N, b, kq, kk, r=0):
    M = np.zeros((N, N), dtype=np.int64)
    for i, j in _sortlsh_pairs(list(range(N)), list(range(N)), kq, kk, 0, b, r):
        M[i, j] += 1
    return M


def causal_literal_forward(Q, K, V, n0, b, kq, kk, eps, tau, pad_key=0):
    """O_s and log d_s of Alg. 5 exactly as printed: leaf exact causal attention,
    SortLSH with O = A V / (d + eps), MergeLSE with eps inside each merge."""
    d = Q.shape[1]
    Qd, Kd, Vd = (np.asarray(a, np.float64) for a in (Q, K, V))

    def row(tok, M):
        return np.zeros(d) if tok is PAD else M[tok]

    def exact_causal(toks):
        n = len(toks)
        O = np.zeros((n, d))
        ld = np.full(n, -np.inf)
        for p in range(n):
            z = np.array([tau * row(toks[p], Qd) @ row(toks[q], Kd) for q in range(p + 1)])
            w = np.exp(z - z.max())
            vs = np.array([row(toks[q], Vd) for q in range(p + 1)])
            O[p] = (w @ vs) / w.sum()
            ld[p] = z.max() + np.log(w.sum())
        return O, ld

    def sortlsh(qs, ks):
        n = len(qs)
        O = np.zeros((n, d))
        ld = np.full(n, -np.inf)
        pairs = _sortlsh_pairs(list(range(n)), list(range(len(ks))),
                               [pad_key if t is PAD else kq[t] for t in qs],
                               [pad_key if t is PAD else kk[t] for t in ks], pad_key, b)
        groups = {}
        for p, q in pairs:
            groups.setdefault(p, []).append(q)
        for p, qlist in groups.items():
            z = np.array([tau * row(qs[p], Qd) @ row(ks[q], Kd) for q in qlist])
            A = np.exp(z)
            vs = np.array([row(ks[q], Vd) for q in qlist])
            dd = A.sum()
            O[p] = (A @ vs) / (dd + eps)
            ld[p] = np.log(dd)
        return O, ld

    def merge(O1, l1, O2, l2):
        mu = np.maximum(l1, l2)
        w1, w2 = np.exp(l1 - mu), np.exp(l2 - mu)
        s = w1 + w2
        return (w1[:, None] * O1 + w2[:, None] * O2) / (s + eps)[:, None], mu + np.log(s + eps)

    def rec(toks):
        n = len(toks)
        if n <= n0:
            return exact_causal(toks)
        padded = n % 2 == 1
        if padded:
            toks = toks + [PAD]
        m = len(toks) // 2
        Ot, lt = rec(toks[:m])
        Od, ldg = rec(toks[m:])
        Oo, lo = sortlsh(toks[m:], toks[:m])
        Ob, lb = merge(Od, ldg, Oo, lo)
        O = np.concatenate([Ot, Ob])
        ld = np.concatenate([lt, lb])
        if padded:
            O, ld = O[:n], ld[:n]
        return O, ld

    return rec(list(range(Q.shape[0])))


# --------------------------------------------------------------------------
# RACE features in product-of-sigmoids form, and materialised forward passes
# --------------------------------------------------------------------------

def _vertex_signs(g):
    return np.array([[1.0 if (c >> b) & 1 else -1.0 for b in range(g)] for c in range(1 << g)])


def race_features_sigmoid(X, Wrace, beta):
    """phi[n, L*2^g]: product over bits of sigmoid(2 beta v_cb tanh(u_b))."""
    L, g, d = Wrace.shape
    U = np.einsum("lgd,nd->nlg", Wrace.astype(np.float64), X.astype(np.float64))
    T = np.tanh(U)                                             # [n, L, g]
    Vs = _vertex_signs(g)                                      # [R, g]
    S = 1.0 / (1.0 + np.exp(-2.0 * beta * T[:, :, None, :] * Vs[None, None]))   # [n, L, R, g]
    return S.prod(axis=-1).reshape(X.shape[0], L << g)


def dense_forward_np(Q, K, V, mask, phq, phk, L, causal, eps, lam, tau, gates=None, m_one=False):
    """Materialised forward from an explicit support mask and explicit features
    (lam: scalar or per-row array; m_one: the m_sparse = 1 ablation)."""
    Q, K, V = (np.asarray(a, np.float64) for a in (Q, K, V))
    N = Q.shape[0]
    Z = tau * Q @ K.T
    E = np.where(mask > 0, np.exp(Z), 0.0)
    ds = E.sum(axis=1)
    Os = (E @ V) / (ds + eps)[:, None]
    M = (phq @ phk.T) / L
    if causal:
        M = np.tril(M)
    Den = M.sum(axis=1)
    Olr = (M @ V) / (Den + eps)[:, None]
    m = np.ones(N) if m_one else ds / (ds + np.asarray(lam, np.float64) * Den + eps)
    gs = np.ones(N) if gates is None else gates[:, 0].astype(np.float64)
    gl = np.ones(N) if gates is None else gates[:, 1].astype(np.float64)
    O = (gs * m)[:, None] * Os + gl[:, None] * Olr
    return dict(O=O, O_s=Os, O_lr=Olr, lse=np.log(ds), d_lr=Den, m=m)


def dense_forward_torch(Q, K, V, mask, Wrace, beta, causal, eps, lam, tau, gates=None, m_one=False):
    """Same materialised forward in PyTorch float64 (features from Wrace),
    differentiable (lam: a float or a per-row float64 tensor)."""
    L, g, d = Wrace.shape
    Wr = torch.as_tensor(np.asarray(Wrace, np.float64))
    Vs = torch.as_tensor(_vertex_signs(g))

    def feats(X):
        T = torch.tanh(torch.einsum("lgd,nd->nlg", Wr, X))
        S = torch.sigmoid(2.0 * beta * T[:, :, None, :] * Vs[None, None])
        return S.prod(dim=-1).reshape(X.shape[0], L << g)

    Z = tau * Q @ K.T
    msk = torch.as_tensor(mask > 0)
    E = torch.where(msk, torch.exp(Z), torch.zeros_like(Z))
    ds = E.sum(dim=1)
    Os = (E @ V) / (ds + eps)[:, None]
    M = feats(Q) @ feats(K).T / L
    if causal:
        M = torch.tril(M)
    Den = M.sum(dim=1)
    Olr = (M @ V) / (Den + eps)[:, None]
    m = torch.ones_like(ds) if m_one else ds / (ds + lam * Den + eps)
    N = Q.shape[0]
    if gates is None:
        gs = torch.ones(N, dtype=torch.float64)
        gl = torch.ones(N, dtype=torch.float64)
    else:
        gs, gl = gates[:, 0], gates[:, 1]
    return (gs * m)[:, None] * Os + gl[:, None] * Olr
