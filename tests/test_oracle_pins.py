"""Pins of the CPU reference against what the paper and the mathematics fix.

Each test checks the reference (``oracle``) against something other than
itself: the paper's printed interaction counts (App. E), brute force on tiny
inputs (``bruteforce``: literal Alg. 5 recursion, explicit masks,
materialised N x N passes), closed forms, invariants and finite
differences.  CPU only.
"""
import json
import os

import numpy as np
import pytest
import torch

import bruteforce as bf
import oracle
from oracle import HeadCfg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(*seed):
    return np.random.default_rng([7, *seed])


def _tiny(seed, N, d, k, r, causal, n0=None, g=4, gs=5, beta=1.0, lam=1.0, eps=1e-6, qk_scale=1.0,
          margin=1e-3):
    rng = _rng(seed, N, d)
    Ws = rng.standard_normal((gs, d)).astype(np.float32)
    Wr = rng.standard_normal((r >> g, g, d)).astype(np.float32)
    Q = bf.with_margin(rng, (N, d), Ws, margin, qk_scale)
    K = bf.with_margin(rng, (N, d), Ws, margin, qk_scale)
    V = rng.standard_normal((N, d)).astype(np.float32)
    cfg = HeadCfg(N=N, d=d, k=k, r=r, causal=causal, race_bits=g, sort_bits=gs, n0=n0, beta=beta,
                  lam=lam, eps=eps)
    return cfg, Q, K, V, Ws, Wr


def _csr_to_mask(N, rp, cols):
    M = np.zeros((N, N), np.int64)
    for i in range(N):
        for j in cols[rp[i]:rp[i + 1]]:
            M[i, j] += 1
    return M


def _pad_key(Ws):
    return int(oracle.hash_keys(np.zeros((1, Ws.shape[1]), np.float32), Ws, Ws.shape[0])[0])


# --------------------------------------------------------------------------
# Hash (Alg. 4 "Hash"; sorted Hamming LSH, Sec. 3)
# --------------------------------------------------------------------------

def test_hash_sign_bits_match_float64_where_margin_is_clear():
    rng = _rng(1)
    X = rng.standard_normal((4000, 64)).astype(np.float32)
    W = rng.standard_normal((5, 64)).astype(np.float32)
    key = oracle.hash_keys(X, W, 5)
    code64, margin = bf.sign_codes64(X, W)
    clear = margin > 1e-5
    assert clear.mean() > 0.99
    # the Gray code of the bucket key must reproduce the sign code
    gray_of_key = key.astype(np.int64) ^ (key.astype(np.int64) >> 1)
    assert np.array_equal(gray_of_key[clear], code64[clear])


def test_hash_bucket_order_is_reflected_gray():
    # x = +-1 pattern with W = identity gives every code; keys must be a
    # bijection onto [0, 32) and adjacent keys must differ in exactly one bit
    bits = 5
    W = np.eye(bits, dtype=np.float32)
    codes = np.arange(1 << bits)
    X = np.array([[1.0 if (c >> t) & 1 else -1.0 for t in range(bits)] for c in codes], np.float32)
    key = oracle.hash_keys(X, W, bits)
    assert sorted(key.tolist()) == list(range(1 << bits))
    code_of_key = np.empty(1 << bits, np.int64)
    code_of_key[key] = codes
    for p in range(31):
        assert bin(int(code_of_key[p] ^ code_of_key[p + 1])).count("1") == 1
    for c, kk in zip(codes, key):
        assert bf.bucket_from_code(int(c), bits) == kk


def test_hash_zero_and_negative_zero_map_to_bucket_zero():
    W = _rng(2).standard_normal((5, 16)).astype(np.float32)
    X = np.zeros((2, 16), np.float32)
    X[1] = -0.0
    assert oracle.hash_keys(X, W, 5).tolist() == [0, 0]


# --------------------------------------------------------------------------
# Sort and blocks (Alg. 4 "Sort", "Partition"; Alg. 5 per level)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("N,k", [(64, 8), (100, 16), (37, 64)])
def test_select_noncausal_is_stable_sort_by_key(N, k):
    cfg, Q, K, V, Ws, Wr = _tiny(3, N, 16, k, 32, False)
    pq, pk = oracle.select(cfg, Q, K, Ws)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    assert pq.tolist() == sorted(range(N), key=lambda i: (kq[i], i))
    assert pk.tolist() == sorted(range(N), key=lambda i: (kk[i], i))


def test_select_causal_levels_partition_halves():
    N, n0, k = 256, 32, 16
    cfg, Q, K, V, Ws, Wr = _tiny(4, N, 16, k, 32, True, n0=n0)
    pq, pk = oracle.select(cfg, Q, K, Ws)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    lv = oracle.num_levels(cfg)
    assert lv == 3 and pq.shape == (3, N // 2)
    for l in range(lv):
        seg = N >> l
        h = seg // 2
        for s in range(1 << l):
            a = s * seg
            fut = list(range(a + h, a + seg))
            past = list(range(a, a + h))
            assert pq[l, s * h:(s + 1) * h].tolist() == sorted(fut, key=lambda i: (kq[i], i))
            assert pk[l, s * h:(s + 1) * h].tolist() == sorted(past, key=lambda i: (kk[i], i))


def test_num_levels():
    assert oracle.num_levels(HeadCfg(N=16384, d=8, k=128, r=16, causal=True)) == 6
    assert oracle.num_levels(HeadCfg(N=65536, d=8, k=256, r=16, causal=True)) == 7
    assert oracle.num_levels(HeadCfg(N=768, d=8, k=128, r=16, causal=True)) == 2
    assert oracle.num_levels(HeadCfg(N=200, d=8, k=128, r=16, causal=True)) == 0
    # 300, 150, 75 (padded to 76), 38 <= 64: Alg. 5's zero token
    assert oracle.num_levels(HeadCfg(N=300, d=8, k=32, r=16, causal=True)) == 3
    assert oracle.num_levels(HeadCfg(N=16386, d=8, k=128, r=16, causal=True)) == 7
    # 5 -> 3 + 3 (one zero token) -> the future half 2 real + 1 zero, padded to
    # 4: its past half would be 2 entries with 1 real token -> no layout
    assert oracle.num_levels(HeadCfg(N=5, d=8, k=1, r=16, causal=True, n0=1)) == -1


def _padded_lists_support(N, n0, k, pq, pk):
    """Support mask implied by sorted lists in the padded layout: level by
    level, segment by segment (lists of ceil(L / 2) entries, L_0 = N), query
    block t of a list sees key block t; every leaf segment's real tokens attend
    causally.  Segment geometry written out here from the recursion itself:
    an odd list gets one zero token at its end, the past half is the first
    half of the (padded) list and the future half the rest."""
    M = np.zeros((N, N), dtype=np.int64)
    segs = [(0, N)]                       # (first real token, real tokens) per segment
    L, off = N, 0
    while L > n0:
        m = (L + 1) // 2
        b = min(k, m)
        nxt = []
        for s, (a, r) in enumerate(segs):
            q = pq[off + s * m: off + (s + 1) * m]
            kl = pk[off + s * m: off + (s + 1) * m]
            assert sorted(kl.tolist()) == list(range(a, a + m)), "past half = first m real tokens"
            fut = sorted(t for t in q.tolist() if t >= 0)
            assert fut == list(range(a + m, a + r)), "future half = the remaining real tokens"
            assert (q < 0).sum() == m - (r - m), "zero tokens fill the future list"
            for p, tq in enumerate(q.tolist()):
                if tq >= 0:
                    t = p // b
                    for tk in kl[t * b:(t + 1) * b].tolist():
                        M[tq, tk] += 1
            nxt += [(a, m), (a + m, r - m)]
        off += m * len(segs)
        segs, L = nxt, m
    for a, r in segs:
        for i in range(a, a + r):
            M[i, a:i + 1] += 1
    return M


@pytest.mark.parametrize("N,n0,k", [(37, 8, 4), (45, 7, 3), (50, 6, 5), (101, 16, 8), (300, 64, 32),
                                    (129, 32, 16), (64, 8, 4)])
def test_select_lists_reproduce_the_literal_recursion(N, n0, k):
    """The sorted lists (with Alg. 5's zero tokens, -1 in perm_q) define the
    same supports as the literal recursion, padding included."""
    cfg, Q, K, V, Ws, Wr = _tiny(10, N, 8, k, 16, True, n0=n0)
    pq, pk = oracle.select(cfg, Q, K, Ws)
    pq, pk = pq.reshape(-1), pk.reshape(-1)
    assert pq.size == oracle.perm_length(cfg)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    want = bf.causal_support_mask(N, n0, k, kq, kk, pad_key=_pad_key(Ws))
    assert np.array_equal(_padded_lists_support(N, n0, k, pq, pk), want)


def test_zero_tokens_sort_after_the_real_tokens_of_their_bucket():
    N, n0, k = 45, 7, 3
    cfg, Q, K, V, Ws, Wr = _tiny(11, N, 8, k, 16, True, n0=n0)
    pq, _ = oracle.select(cfg, Q, K, Ws)
    kq, _ = bf.keys64(Q, Ws)
    zk = _pad_key(Ws)
    L, off, nseg, zeros = N, 0, 1, 0
    while L > n0:
        m = (L + 1) // 2
        for s in range(nseg):
            q = pq[off + s * m: off + (s + 1) * m].tolist()
            keys = [zk if t < 0 else kq[t] for t in q]
            assert keys == sorted(keys), "lists ascend by bucket"
            for p in range(1, m):
                if q[p - 1] < 0 and q[p] >= 0:
                    assert keys[p] > keys[p - 1], "a zero token follows the real tokens of its bucket"
            zeros += sum(t < 0 for t in q)
        off += m * nseg
        L, nseg = m, 2 * nseg
    assert zeros > 0


# --------------------------------------------------------------------------
# Support S(i) (Alg. 4 blocks; Alg. 5 recursion with padding)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("N,n0,k", [(64, 8, 4), (37, 8, 4), (50, 6, 5), (96, 16, 16), (33, 40, 8),
                                    (45, 7, 3)])
def test_causal_support_equals_literal_recursion(N, n0, k):
    cfg, Q, K, V, Ws, Wr = _tiny(5, N, 8, k, 16, True, n0=n0)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    ref = bf.causal_support_mask(N, n0, k, kq, kk, pad_key=_pad_key(Ws))
    rp, cols = oracle.support(cfg, Q, K, Ws)
    got = _csr_to_mask(N, rp, cols)
    assert ref.max() <= 1, "Alg. 5 supports are disjoint unions"
    assert np.array_equal(got, ref)
    assert not np.triu(got, 1).any(), "causal"
    assert np.all(np.diag(got) == 1), "every query sees itself (leaf)"


@pytest.mark.parametrize("N,k", [(64, 8), (70, 16), (20, 64)])
def test_noncausal_support_equals_blocks(N, k):
    cfg, Q, K, V, Ws, Wr = _tiny(6, N, 8, k, 16, False)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    ref = bf.noncausal_support_mask(N, k, kq, kk)
    rp, cols = oracle.support(cfg, Q, K, Ws)
    assert np.array_equal(_csr_to_mask(N, rp, cols), ref)
    # block sizes: every query sees min(k, N) keys except the ragged last block
    sizes = np.diff(rp)
    b = min(k, N)
    nfull = N // b
    assert (sizes == b).sum() >= nfull * b


def test_causal_support_size_closed_form():
    # N = n0 * 2^Lv, b | halves: |S(i)| = (i mod n0) + 1 + b * #{l : bit (log2 N - 1 - l) of i}
    N, n0, b = 512, 32, 16
    cfg, Q, K, V, Ws, Wr = _tiny(7, N, 8, b, 16, True, n0=n0)
    rp, _ = oracle.support(cfg, Q, K, Ws)
    lv = oracle.num_levels(cfg)
    logn = int(np.log2(N))
    want = np.array([(i % n0) + 1 + b * sum((i >> (logn - 1 - l)) & 1 for l in range(lv))
                     for i in range(N)])
    assert np.array_equal(np.diff(rp), want)
    assert rp[-1] == N * (n0 + 1) // 2 + lv * N * b // 2


def test_causal_support_base_length_k_or_2k_identical():
    N, k = 256, 16
    cfg1, Q, K, V, Ws, Wr = _tiny(8, N, 8, k, 16, True, n0=k)
    cfg2 = HeadCfg(**{**cfg1.__dict__, "n0": 2 * k})
    a = oracle.support(cfg1, Q, K, Ws)
    b = oracle.support(cfg2, Q, K, Ws)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_interaction_counts_of_the_paper_example():
    g = json.load(open(os.path.join(GOLDEN, "app_e_interaction_counts.json")))
    N, s, L, gam = g["N"], g["s"], g["L_s"], g["gamma"]
    rng = _rng(9)
    d = 8
    Ws = rng.standard_normal((5, d)).astype(np.float32)
    Q = rng.standard_normal((N, d)).astype(np.float32)
    K = rng.standard_normal((N, d)).astype(np.float32)
    cfg = HeadCfg(N=N, d=d, k=s, r=L << gam, causal=False, race_bits=gam)
    c = cfg.c()
    import ctypes
    lib = oracle._load()
    sparse = lib.ora_support_size(ctypes.byref(c), oracle._ptr(Q), oracle._ptr(K), oracle._ptr(Ws))
    Wr = rng.standard_normal((L, gam, d)).astype(np.float32)
    race = oracle.features(Q[:10], Wr, gam, 1.0).shape[1] * N
    assert sparse == g["sortlsh_interactions"]
    assert race == g["race_bucket_interactions"]
    assert sparse + race == g["elsaa_interactions"]
    assert N * N == g["dense_interactions"]
    assert abs((sparse + race) / (N * N) - g["elsaa_fraction_of_dense"]) < 1e-12
    assert abs(sparse / (N * N) - g["sortlsh_fraction_of_dense"]) < 1e-12


# --------------------------------------------------------------------------
# RACE features and sums (Alg. 2, Alg. 3)
# --------------------------------------------------------------------------

def test_features_softmax_equals_product_of_sigmoids():
    rng = _rng(10)
    X = rng.standard_normal((200, 16)).astype(np.float32)
    for g, beta in [(4, 1.0), (2, 0.5), (3, 2.0)]:
        Wr = rng.standard_normal((3, g, 16)).astype(np.float32)
        phi = oracle.features(X, Wr, g, beta)
        ref = bf.race_features_sigmoid(X, Wr, beta)
        assert np.max(np.abs(phi - ref)) < 1e-14
        assert np.allclose(phi.reshape(200, 3, 1 << g).sum(-1), 1.0, atol=1e-14)
        assert phi.min() > 0


@pytest.mark.parametrize("causal", [False, True])
def test_race_matches_materialised_kernel_matrix(causal):
    cfg, Q, K, V, Ws, Wr = _tiny(11, 48, 8, 8, 48, causal, n0=16, beta=0.8)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr)
    phq = bf.race_features_sigmoid(Q, Wr, cfg.beta)
    phk = bf.race_features_sigmoid(K, Wr, cfg.beta)
    M = phq @ phk.T / cfg.L
    if causal:
        M = np.tril(M)
    Den = M.sum(1)
    Olr = M @ V.astype(np.float64) / (Den + cfg.eps)[:, None]
    assert np.max(np.abs(out["d_lr"] - Den)) < 1e-12 * Den.max()
    assert np.max(np.abs(out["O_lr"] - Olr)) < 1e-12
    vis = np.arange(1, 49) if causal else np.full(48, 48)
    assert np.all(out["d_lr"] > 0) and np.all(out["d_lr"] <= vis + 1e-12)


@pytest.mark.parametrize("C", [1, 7, 64, 48])
def test_causal_race_equals_chunked_prefix_form(C):
    # Alg. 3 run with chunk size C: strict prefix states + masked intra-chunk part
    cfg, Q, K, V, Ws, Wr = _tiny(12, 48, 8, 8, 32, True, n0=16)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr)
    N, L = 48, cfg.L
    phq = bf.race_features_sigmoid(Q, Wr, cfg.beta)
    phk = bf.race_features_sigmoid(K, Wr, cfg.beta)
    Np = -(-N // C) * C
    pq = np.zeros((Np, phq.shape[1])); pq[:N] = phq
    pk = np.zeros((Np, phk.shape[1])); pk[:N] = phk
    Vp = np.zeros((Np, 8)); Vp[:N] = V
    num = np.zeros((Np, 8)); den = np.zeros(Np)
    sA = np.zeros(phk.shape[1]); sB = np.zeros((phk.shape[1], 8))
    for n in range(Np // C):
        sl = slice(n * C, (n + 1) * C)
        inum = pq[sl] @ sB / L
        iden = pq[sl] @ sA / L
        Mn = np.tril(pq[sl] @ pk[sl].T / L)
        num[sl] = inum + Mn @ Vp[sl]
        den[sl] = iden + Mn.sum(1)
        sA = sA + pk[sl].sum(0)
        sB = sB + pk[sl].T @ Vp[sl]
    Olr = num[:N] / (den[:N] + cfg.eps)[:, None]
    assert np.max(np.abs(out["O_lr"] - Olr)) < 1e-12
    assert np.max(np.abs(out["d_lr"] - den[:N])) < 1e-12 * den.max()


@pytest.mark.parametrize("causal", [False, True])
def test_race_zero_temperature_is_mean_of_visible_values(causal):
    cfg, Q, K, V, Ws, Wr = _tiny(13, 40, 8, 8, 32, causal, n0=16, beta=1e-9)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr)
    R = 16
    V64 = V.astype(np.float64)
    for i in range(40):
        vis = np.arange(i + 1) if causal else np.arange(40)
        n = len(vis)
        assert abs(out["d_lr"][i] - n / R) < 1e-7 * n
        want = V64[vis].sum(0) / (n + R * cfg.eps)
        assert np.max(np.abs(out["O_lr"][i] - want)) < 1e-7


# --------------------------------------------------------------------------
# Sparse sums, fusion, reductions (Alg. 4-6, Eq. m_sparse, Eq. fusion)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("N,n0,k,causal", [(64, 8, 4, True), (45, 7, 3, True), (40, 0, 8, False),
                                           (37, 0, 16, False)])
def test_forward_equals_materialised_brute_force(N, n0, k, causal):
    rng = _rng(14, N)
    cfg, Q, K, V, Ws, Wr = _tiny(14, N, 8, k, 32, causal, n0=n0 or None, lam=0.7, beta=0.9)
    gates = rng.uniform(0.1, 0.9, (N, 2)).astype(np.float32)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr, gates=gates)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    mask = (bf.causal_support_mask(N, n0, k, kq, kk, _pad_key(Ws)) if causal
            else bf.noncausal_support_mask(N, k, kq, kk))
    phq = bf.race_features_sigmoid(Q, Wr, cfg.beta)
    phk = bf.race_features_sigmoid(K, Wr, cfg.beta)
    ref = bf.dense_forward_np(Q, K, V, mask, phq, phk, cfg.L, causal, cfg.eps, cfg.lam,
                              1 / np.sqrt(8), gates)
    for name in ("O", "O_s", "O_lr", "lse", "d_lr", "m"):
        a, b = out[name], ref[name]
        assert np.max(np.abs(a - b)) <= 1e-12 * max(1.0, np.max(np.abs(b))), name
    assert np.all((out["m"] > 0) & (out["m"] < 1))


@pytest.mark.parametrize("causal", [False, True])
def test_full_support_reduces_to_dense_softmax_attention(causal):
    # sparse budget covering every key (b >= N, or N_0 >= N), lambda = 0,
    # gates (1, 0): the fused output is dense softmax attention up to eps/d
    N, d = 96, 16
    cfg, Q, K, V, Ws, Wr = _tiny(15, N, d, 128 if not causal else 8, 32, causal,
                                 n0=128 if causal else None, lam=0.0)
    gates = np.tile(np.array([1.0, 0.0], np.float32), (N, 1))
    out = oracle.forward(cfg, Q, K, V, Ws, Wr, gates=gates)
    Z = (Q.astype(np.float64) @ K.astype(np.float64).T) / np.sqrt(d)
    if causal:
        Z = np.where(np.tril(np.ones((N, N))) > 0, Z, -np.inf)
    P = np.exp(Z - Z.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    dense = P @ V.astype(np.float64)
    # O_s = N_s/(d_s+eps) and m = d_s/(d_s+eps): each row is off by at most 2 eps/d_s
    tol = 2.5 * cfg.eps / np.exp(out["lse"]) * np.abs(dense).max(1) + 1e-13
    assert np.all(np.abs(out["O"] - dense).max(1) <= tol)
    assert np.all(np.abs(out["O_s"] - dense).max(1) <= tol)
    rowsum = np.log(np.exp(Z - Z.max(1, keepdims=True)).sum(1)) + Z.max(1)
    assert np.max(np.abs(out["lse"] - rowsum)) < 1e-12


def test_sparse_denominator_is_bounded_by_dense_row_sum():
    N, d = 128, 8
    cfg, Q, K, V, Ws, Wr = _tiny(16, N, d, 8, 16, True, n0=16)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr)
    Z = (Q.astype(np.float64) @ K.astype(np.float64).T) / np.sqrt(d)
    Z = np.where(np.tril(np.ones((N, N))) > 0, Z, -np.inf)
    dense_lse = np.log(np.exp(Z).sum(1))
    assert np.all(out["lse"] <= dense_lse + 1e-12)
    leaf_only = np.arange(N) < 16          # these rows see every earlier key
    assert np.max(np.abs(out["lse"][leaf_only] - dense_lse[leaf_only])) < 1e-12
    assert np.all(out["lse"][~leaf_only] < dense_lse[~leaf_only])


def test_fusion_limits():
    cfg, Q, K, V, Ws, Wr = _tiny(17, 64, 8, 8, 32, True, n0=16)
    g0 = np.tile(np.array([0.0, 0.6], np.float32), (64, 1))
    out = oracle.forward(cfg, Q, K, V, Ws, Wr, gates=g0)
    assert np.max(np.abs(out["O"] - np.float64(np.float32(0.6)) * out["O_lr"])) < 1e-15
    big = HeadCfg(**{**cfg.__dict__, "lam": 1e12})
    assert oracle.forward(big, Q, K, V, Ws, Wr)["m"].max() < 1e-8
    zero = HeadCfg(**{**cfg.__dict__, "lam": 0.0})
    o = oracle.forward(zero, Q, K, V, Ws, Wr)
    ds = np.exp(o["lse"])
    assert np.max(np.abs(o["m"] - ds / (ds + cfg.eps))) < 1e-15


@pytest.mark.parametrize("N,n0,k", [(64, 8, 4), (45, 7, 3), (128, 16, 8)])
def test_single_eps_reading_matches_literal_merge_lse(N, n0, k):
    # Alg. 5 applies eps inside SortLSH and inside every MergeLSE; the
    # reference applies one eps to the union-support denominator.  The two
    # differ by a relative (levels + 2) * eps / min(1, d_s) at most.
    cfg, Q, K, V, Ws, Wr = _tiny(18, N, 8, k, 16, True, n0=n0)
    out = oracle.forward(cfg, Q, K, V, Ws, Wr)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    O_lit, ld_lit = bf.causal_literal_forward(Q, K, V, n0, k, kq, kk, cfg.eps, 1 / np.sqrt(8),
                                              _pad_key(Ws))
    levels = int(np.ceil(np.log2(N / n0))) + 1
    bound = (levels + 2) * cfg.eps / min(1.0, np.exp(out["lse"]).min())
    assert np.max(np.abs(out["O_s"] - O_lit)) <= bound * np.max(np.abs(O_lit))
    assert np.max(np.abs(out["lse"] - ld_lit)) <= bound


# --------------------------------------------------------------------------
# Backward (exact gradient with the selection held fixed)
# --------------------------------------------------------------------------

def _fd_grads(cfg, Q, K, V, Ws, Wr, gates, R, which, h=2.0 ** -11):
    """Central differences with Richardson extrapolation of L = sum(O * R)."""
    base = {"Q": Q, "K": K, "V": V, "G": gates}
    X = base[which]
    G = np.zeros(X.shape)
    sup0 = oracle.support(cfg, Q, K, Ws)

    def loss(Xp):
        args = dict(base)
        args[which] = Xp
        if which in ("Q", "K"):
            s = oracle.support(cfg, args["Q"], args["K"], Ws)
            assert np.array_equal(s[0], sup0[0]) and np.array_equal(s[1], sup0[1])
        o = oracle.forward(cfg, args["Q"], args["K"], args["V"], Ws, Wr, gates=args["G"])["O"]
        return float((o * R).sum())

    for idx in np.ndindex(X.shape):
        est = []
        for hh in (h, h / 2):
            Xp = X.copy(); Xp[idx] += hh
            Xm = X.copy(); Xm[idx] -= hh
            # the float32 steps actually taken (x +- h rounds for tiny |x|)
            hp = float(Xp[idx]) - float(X[idx])
            hm = float(X[idx]) - float(Xm[idx])
            est.append((loss(Xp) - loss(Xm)) / (hp + hm))
        G[idx] = (4 * est[1] - est[0]) / 3
    return G


@pytest.mark.parametrize("causal,N,n0,k", [(True, 24, 4, 3), (False, 20, 0, 6), (True, 21, 5, 2)])
def test_backward_matches_finite_differences(causal, N, n0, k):
    rng = _rng(19, N)
    cfg, Q, K, V, Ws, Wr = _tiny(19, N, 4, k, 32, causal, n0=n0 or None, lam=0.8, beta=0.7,
                                 eps=1e-3, margin=1e-2)
    cfg.race_bits = 2
    Wr = rng.standard_normal((2, 2, 4)).astype(np.float32)
    cfg.r = 8
    gates = rng.uniform(0.2, 0.9, (N, 2)).astype(np.float32)
    R = rng.standard_normal((N, 4))
    g = oracle.backward(cfg, Q, K, V, Ws, Wr, R.astype(np.float32), gates=gates)
    R32 = R.astype(np.float32).astype(np.float64)
    for which, key in (("Q", "dQ"), ("K", "dK"), ("V", "dV"), ("G", "dgates")):
        fd = _fd_grads(cfg, Q, K, V, Ws, Wr, gates, R32, which)
        err = np.max(np.abs(fd - g[key])) / np.max(np.abs(fd))
        assert err < 1e-6, (which, err)


@pytest.mark.parametrize("causal,N,n0,k", [(True, 64, 8, 4), (False, 48, 0, 8), (True, 45, 7, 3)])
def test_backward_matches_torch_autograd_of_materialised_forward(causal, N, n0, k):
    rng = _rng(20, N)
    cfg, Q, K, V, Ws, Wr = _tiny(20, N, 8, k, 32, causal, n0=n0 or None, lam=0.6, beta=0.9)
    gates = rng.uniform(0.1, 0.9, (N, 2)).astype(np.float32)
    dO = rng.standard_normal((N, 8)).astype(np.float32)
    g = oracle.backward(cfg, Q, K, V, Ws, Wr, dO, gates=gates)
    kq, _ = bf.keys64(Q, Ws)
    kk, _ = bf.keys64(K, Ws)
    mask = (bf.causal_support_mask(N, n0, k, kq, kk, _pad_key(Ws)) if causal
            else bf.noncausal_support_mask(N, k, kq, kk))
    tQ, tK, tV = (torch.tensor(a.astype(np.float64), requires_grad=True) for a in (Q, K, V))
    tG = torch.tensor(gates.astype(np.float64), requires_grad=True)
    O = bf.dense_forward_torch(tQ, tK, tV, mask, Wr, cfg.beta, causal, cfg.eps, cfg.lam,
                               1 / np.sqrt(8), tG)
    (O * torch.tensor(dO.astype(np.float64))).sum().backward()
    for t, key in ((tQ, "dQ"), (tK, "dK"), (tV, "dV"), (tG, "dgates")):
        ref = t.grad.numpy()
        assert np.max(np.abs(g[key] - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref))), key


def test_backward_row_masks_restrict_only_the_sparse_part():
    cfg, Q, K, V, Ws, Wr = _tiny(21, 64, 8, 4, 32, True, n0=8)
    dO = _rng(21).standard_normal((64, 8)).astype(np.float32)
    full = oracle.backward(cfg, Q, K, V, Ws, Wr, dO)
    qm = np.zeros(64, np.uint8); qm[::5] = 1
    km = np.zeros(64, np.uint8); km[3::7] = 1
    part = oracle.backward(cfg, Q, K, V, Ws, Wr, dO, q_mask=qm, k_mask=km)
    assert np.array_equal(part["dQ"][qm > 0], full["dQ"][qm > 0])
    assert np.array_equal(part["dK"][km > 0], full["dK"][km > 0])
    assert np.array_equal(part["dV"][km > 0], full["dV"][km > 0])


def test_dense_reduction_gradient_is_textbook_attention_gradient():
    N, d = 40, 8
    cfg, Q, K, V, Ws, Wr = _tiny(22, N, d, 64, 16, False, lam=0.0)
    gates = np.tile(np.array([1.0, 0.0], np.float32), (N, 1))
    dO = _rng(22).standard_normal((N, d)).astype(np.float32)
    g = oracle.backward(cfg, Q, K, V, Ws, Wr, dO, gates=gates)
    tQ, tK, tV = (torch.tensor(a.astype(np.float64), requires_grad=True) for a in (Q, K, V))
    O = torch.softmax(tQ @ tK.T / np.sqrt(d), dim=1) @ tV
    (O * torch.tensor(dO.astype(np.float64))).sum().backward()
    for t, key in ((tQ, "dQ"), (tK, "dK"), (tV, "dV")):
        ref = t.grad.numpy()
        assert np.max(np.abs(g[key] - ref)) < 1e-6 * np.max(np.abs(ref)), key
