"""GPU parity of the dense projections (elsaa_gemm) against the float64
reference of oracle/projections.py on the same bf16 inputs.

Bars: float32 output within 1e-4 of max|ref| (float32 accumulation of exact
bf16 products); bf16 output within 2e-2 of max|ref|, and per element within
one bf16 rounding step (2^-8 |ref|) plus 1e-4 max|ref|."""
import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2607_20214_amd as E
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV).to(torch.bfloat16)


def _check(got, ref, out_dtype, what=""):
    got = got.float().cpu().numpy().astype(np.float64) if torch.is_tensor(got) else got
    scale = np.abs(ref).max()
    err = np.abs(got - ref)
    if out_dtype == torch.float32:
        assert err.max() <= 1e-4 * scale, f"{what}: {err.max() / scale:.3e}"
    else:
        assert err.max() <= 2e-2 * scale, f"{what}: {err.max() / scale:.3e}"
        bound = 2.0 ** -8 * np.abs(ref) + 1e-4 * scale
        assert (err <= bound).all(), f"{what}: worst element ratio {(err / bound).max():.3f}"


# ragged and small shapes (128 x 128 tiles) and whole 256 x 256 tiles with K
# a multiple of 64 (the large-tile kernel)
SHAPES = [(200, 136, 72), (384, 256, 320), (8, 8, 8), (512, 256, 128), (256, 768, 192)]


@pytest.mark.parametrize("shape,ta,tb,od", [
    (s, ta, tb, od) for s in SHAPES for ta, tb in itertools.product([0, 1], repeat=2)
    for od in (torch.bfloat16, torch.float32)])
def test_gemm_plain(shape, ta, tb, od):
    M, N, K = shape
    seed = M * 7 + N * 3 + K + 10 * ta + 20 * tb
    A = W.random_matrix(seed, 1, (K, M) if ta else (M, K))
    B = W.random_matrix(seed, 2, (N, K) if tb else (K, N))
    got = E.gemm(_t(A), _t(B), bool(ta), bool(tb), out_dtype=od)
    torch.cuda.synchronize()
    _check(got, oracle.gemm(A, B, ta, tb), od, f"{shape} ta={ta} tb={tb}")


@pytest.mark.parametrize("ta,od", [(1, torch.float32), (1, torch.bfloat16), (0, torch.float32)])
def test_gemm_split_k(ta, od):
    M, N, K = 256, 264, 4096
    A = W.random_matrix(40 + ta, 1, (K, M) if ta else (M, K))
    B = W.random_matrix(40 + ta, 2, (K, N))
    got = E.gemm(_t(A), _t(B), bool(ta), False, out_dtype=od)
    torch.cuda.synchronize()
    desc = E._GemmDesc(M, N, K, ta, 0, M if ta else K, N, N, 0, 0, 0, 0, 0)
    assert E.gemm_workspace_bytes(desc) > 0          # this case runs split over K
    _check(got, oracle.gemm(A, B, ta, False), od, "split-K")


@pytest.mark.parametrize("ta,tb,od", [(1, 0, torch.float32), (1, 1, torch.bfloat16), (0, 1, torch.float32)])
def test_gemm_split_k_large_tiles(ta, tb, od):
    """Whole 256 x 256 tiles with a long K: the large-tile kernel split over K."""
    M, N, K = 256, 512, 8192
    A = W.random_matrix(45 + ta, 1, (K, M) if ta else (M, K))
    B = W.random_matrix(45 + tb, 2, (N, K) if tb else (K, N))
    got = E.gemm(_t(A), _t(B), bool(ta), bool(tb), out_dtype=od)
    torch.cuda.synchronize()
    desc = E._GemmDesc(M, N, K, ta, tb, M if ta else K, K if tb else N, N, 0, 0, 0, 0, 0)
    assert E.gemm_workspace_bytes(desc) > 0
    _check(got, oracle.gemm(A, B, ta, tb), od, "split-K large tiles")


def test_gemm_repeatable():
    A = _t(W.random_matrix(50, 1, (4096, 512)))
    B = _t(W.random_matrix(50, 2, (4096, 256)))
    r1 = E.gemm(A, B, True, False, out_dtype=torch.float32)
    r2 = E.gemm(A, B, True, False, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(r1, r2)


@pytest.mark.parametrize("Bb,S,H,dh", [(2, 96, 4, 16), (2, 256, 4, 64)])
def test_block_projections_head_major(Bb, S, H, dh):
    """Every product of one attention block (fwd and bwd) with the attention
    tensors in head-major [B, H, S, dh] storage (the second size takes the
    large-tile kernel for all six products)."""
    dm = H * dh
    X = W.random_matrix(60, 1, (Bb * S, dm))
    Wqkv = W.random_matrix(60, 2, (dm, 3 * dm), 0.1)
    Wo = W.random_matrix(60, 3, (dm, dm), 0.1)
    O = W.random_matrix(60, 4, (Bb, H, S, dh))
    dY = W.random_matrix(60, 5, (Bb * S, dm))
    dQKV = W.random_matrix(60, 6, (Bb, 3 * H, S, dh))
    bf = torch.bfloat16
    # QKV = X W_qkv, written head-major with 3H heads
    qkv = torch.empty(Bb, 3 * H, S, dh, dtype=bf, device=DEV)
    E.gemm(_t(X), _t(Wqkv), out=qkv)
    # Y = O W_O with O read head-major
    y = E.gemm(_t(O), _t(Wo), out_dtype=torch.float32)
    # dO = dY W_O^T written head-major
    do = torch.empty(Bb, H, S, dh, dtype=torch.float32, device=DEV)
    E.gemm(_t(dY), _t(Wo), trans_b=True, out=do)
    # dW_O = O^T dY with O read head-major and transposed
    dwo = E.gemm(_t(O), _t(dY), trans_a=True, out_dtype=torch.float32)
    # dX = dQKV W_qkv^T with dQKV read head-major
    dx = E.gemm(_t(dQKV), _t(Wqkv), trans_b=True, out_dtype=torch.float32)
    # dW_qkv = X^T dQKV with dQKV read head-major
    dwqkv = E.gemm(_t(X), _t(dQKV), trans_a=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    Om, dQm = oracle.heads_to_matrix(O), oracle.heads_to_matrix(dQKV)
    ref_qkv = oracle.matrix_to_heads(oracle.gemm(X, Wqkv), 3 * H, S)
    _check(qkv, ref_qkv, bf, "qkv")
    _check(y, oracle.gemm(Om, Wo), torch.float32, "y")
    _check(do, oracle.matrix_to_heads(oracle.gemm(dY, Wo, False, True), H, S), torch.float32, "do")
    _check(dwo, oracle.gemm(Om, dY, True, False), torch.float32, "dwo")
    _check(dx, oracle.gemm(dQm, Wqkv, False, True), torch.float32, "dx")
    _check(dwqkv, oracle.gemm(X, dQm, True, False), torch.float32, "dwqkv")


def test_block_projections_full_size_sampled():
    """The 32768-token, d_model 1024 block's products at full size (the launch
    configuration the benchmark times), checked on sampled rows / columns."""
    w = W.BLOCK_32K
    S, dm, H = w.N, w.d_model, w.H
    dh = dm // H
    X = W.random_matrix(70, 1, (S, dm))
    Wqkv = W.random_matrix(70, 2, (dm, 3 * dm), 0.02)
    dQKV = W.random_matrix(70, 3, (1, 3 * H, S, dh))
    qkv = torch.empty(1, 3 * H, S, dh, dtype=torch.bfloat16, device=DEV)
    E.gemm(_t(X), _t(Wqkv), out=qkv)
    dwqkv = E.gemm(_t(X), _t(dQKV), trans_a=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    rng = np.random.default_rng(71)
    rows = np.sort(rng.choice(S, 48, replace=False))
    ref = oracle.gemm(X[rows], Wqkv)                                   # [48, 3 dm]
    got = qkv[0].permute(1, 0, 2).reshape(S, 3 * dm)[torch.from_numpy(rows).to(DEV)]
    _check(got, ref, torch.bfloat16, "qkv rows")
    dQm = dQKV[0].transpose(1, 0, 2).reshape(S, 3 * dm)
    r2 = np.sort(rng.choice(dm, 16, replace=False))
    c2 = np.sort(rng.choice(3 * dm, 16, replace=False))
    ref2 = oracle.gemm(X[:, r2], dQm[:, c2], True, False)
    got2 = dwqkv.cpu().numpy()[np.ix_(r2, c2)].astype(np.float64)
    _check(got2, ref2, torch.float32, "dW rows/cols")


def test_block_projections_full_size_other_products():
    """The block's other four products at full size (32768 tokens, d_model
    1024, head-major attention tensors), as the benchmark launches them:
    Y = O W_O, dO = dY W_O^T (head-major bf16 out), dW_O = O^T dY (split
    over K) and dX = dQKV W_qkv^T, checked on sampled rows / columns."""
    w = W.BLOCK_32K
    S, dm, H = w.N, w.d_model, w.H
    dh = dm // H
    O = W.random_matrix(80, 1, (1, H, S, dh))
    Wo = W.random_matrix(80, 2, (dm, dm), 0.02)
    dY = W.random_matrix(80, 3, (S, dm))
    dQKV = W.random_matrix(80, 4, (1, 3 * H, S, dh))
    Wqkv = W.random_matrix(80, 5, (dm, 3 * dm), 0.02)
    y = E.gemm(_t(O), _t(Wo), out_dtype=torch.float32)
    do = torch.empty(1, H, S, dh, dtype=torch.bfloat16, device=DEV)
    E.gemm(_t(dY), _t(Wo), trans_b=True, out=do)
    dwo = E.gemm(_t(O), _t(dY), trans_a=True, out_dtype=torch.float32)
    dx = E.gemm(_t(dQKV), _t(Wqkv), trans_b=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    Om = O[0].transpose(1, 0, 2).reshape(S, dm)
    dQm = dQKV[0].transpose(1, 0, 2).reshape(S, 3 * dm)
    rng = np.random.default_rng(81)
    rows = np.sort(rng.choice(S, 48, replace=False))
    ridx = torch.from_numpy(rows).to(DEV)
    _check(y[ridx], oracle.gemm(Om[rows], Wo), torch.float32, "Y rows")
    got = do[0].permute(1, 0, 2).reshape(S, dm)[ridx]
    _check(got, oracle.gemm(dY[rows], Wo, False, True), torch.bfloat16, "dO rows")
    _check(dx[ridx], oracle.gemm(dQm[rows], Wqkv, False, True), torch.float32, "dX rows")
    r2 = np.sort(rng.choice(dm, 16, replace=False))
    c2 = np.sort(rng.choice(dm, 16, replace=False))
    ref2 = oracle.gemm(Om[:, r2], dY[:, c2], True, False)
    got2 = dwo.cpu().numpy()[np.ix_(r2, c2)].astype(np.float64)
    _check(got2, ref2, torch.float32, "dW_O rows/cols")
