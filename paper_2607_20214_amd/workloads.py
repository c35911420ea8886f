"""Seeded synthetic inputs for the ELSAA operator.

This module only draws tensors; it contains none of the operator's
arithmetic.  It is the one module that both the CPU reference and the
GPU library's tests, benchmark and smoke check read their inputs from.

Every array is produced by ``numpy.random.default_rng([42, seed, tensor_id])``
(seed 42 as in the paper's training setup, App. D), drawn in float32, and
for bf16 workloads rounded to bfloat16 with round-to-nearest-even and
returned as float32 holding the exact bf16 value.

Value recipes (they stand in for the paper's datasets, which are not used):

``iid``        Q, K, V ~ N(0,1); Q and K multiplied by ``qk_scale``
               (d^-1/4 for the "scores are O(1)" workloads).
``clustered``  per (batch, head): ``centres`` cluster centres ~ N(0,1)^d;
               key j = centre[c_j] + 0.3 N(0,1) with c_j uniform;
               query i = K[pi_i] + 0.3 N(0,1) with pi_i uniform over all N
               keys.  Attention is peaked (the vision-like regime of Sec. 7).
``mixed``      heads 0..H/2-1 follow ``clustered``; the remaining heads are
               i.i.d. N(0,1) * 0.1 (diffuse attention, the long-text regime).
V and the upstream gradient dO are i.i.d. N(0,1) in every recipe.

The hash projections are per head, i.i.d. N(0,1) in float32:
``W_sort`` [H, sort_bits, d] (sortLSH sign hash, Alg. 4) and
``W_race`` [H, L, race_bits, d] with L = r / 2^race_bits (RACE tables, Alg. 2).
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

# tensor ids inside one seed
_T_Q, _T_K, _T_V, _T_DO = 1, 2, 3, 4
_T_CENTRES, _T_ASSIGN, _T_KNOISE, _T_PICK, _T_QNOISE = 10, 11, 12, 13, 14
_T_X, _T_WQ, _T_WK, _T_WV, _T_WO, _T_DY = 20, 21, 22, 23, 24, 25
_T_WSORT, _T_WRACE, _T_GATES, _T_LAMBDA = 100, 101, 102, 103
_T_RULES, _T_RULE_GRADS = 110, 111


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(x.shape)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic operator workload (shapes, settings and value recipe)."""
    name: str
    B: int
    H: int
    N: int
    d: int
    k: int                      # sortLSH block size b (keys per sorted block)
    r: int                      # RACE features = L * 2^race_bits
    causal: bool
    dtype: str                  # "f32" or "bf16"
    recipe: str = "iid"         # "iid" | "clustered" | "mixed"
    qk_scale: float = 1.0       # multiplier on Q and K for the iid recipe
    centres: int = 64
    backward: bool = True
    race_bits: int = 4
    sort_bits: int = 5
    n0: Optional[int] = None    # causal base length; None -> 2k
    seed: int = 0
    # attention-block workloads (dense projections around the operator)
    d_model: int = 0

    @property
    def L(self) -> int:
        return self.r // (1 << self.race_bits)

    @property
    def base_len(self) -> int:
        return self.n0 if self.n0 is not None else 2 * self.k


def _rng(seed: int, tid: int) -> np.random.Generator:
    return np.random.default_rng([42, seed, tid])


def _normal(seed: int, tid: int, shape) -> np.ndarray:
    return _rng(seed, tid).standard_normal(shape, dtype=np.float32)


def _clustered_qk(seed: int, B: int, H: int, N: int, d: int, centres: int, heads):
    """Clustered keys and noisy-copy queries for the given head indices."""
    Q = np.empty((B, len(heads), N, d), np.float32)
    K = np.empty((B, len(heads), N, d), np.float32)
    cen = _normal(seed, _T_CENTRES, (B, H, centres, d))
    asg = _rng(seed, _T_ASSIGN).integers(0, centres, size=(B, H, N))
    kno = _normal(seed, _T_KNOISE, (B, H, N, d))
    pick = _rng(seed, _T_PICK).integers(0, N, size=(B, H, N))
    qno = _normal(seed, _T_QNOISE, (B, H, N, d))
    for b in range(B):
        for t, h in enumerate(heads):
            kk = cen[b, h][asg[b, h]] + np.float32(0.3) * kno[b, h]
            K[b, t] = kk
            Q[b, t] = kk[pick[b, h]] + np.float32(0.3) * qno[b, h]
    return Q, K


def make_inputs(w: Workload, with_grad: Optional[bool] = None) -> dict:
    """Draw Q, K, V (and dO), W_sort and W_race for workload ``w``.

    Returns float32 numpy arrays; for bf16 workloads every tensor the
    operator reads in its storage dtype (Q, K, V, dO) holds bf16 values.
    """
    B, H, N, d, s = w.B, w.H, w.N, w.d, w.seed
    if w.recipe == "iid":
        Q = _normal(s, _T_Q, (B, H, N, d)) * np.float32(w.qk_scale)
        K = _normal(s, _T_K, (B, H, N, d)) * np.float32(w.qk_scale)
    elif w.recipe == "clustered":
        Q, K = _clustered_qk(s, B, H, N, d, w.centres, list(range(H)))
    elif w.recipe == "mixed":
        hc = H // 2
        Q = _normal(s, _T_Q, (B, H, N, d)) * np.float32(0.1)
        K = _normal(s, _T_K, (B, H, N, d)) * np.float32(0.1)
        qc, kc = _clustered_qk(s, B, H, N, d, w.centres, list(range(hc)))
        Q[:, :hc] = qc
        K[:, :hc] = kc
    else:
        raise ValueError(f"unknown recipe {w.recipe!r}")
    V = _normal(s, _T_V, (B, H, N, d))
    out = {"Q": Q, "K": K, "V": V}
    if with_grad if with_grad is not None else w.backward:
        out["dO"] = _normal(s, _T_DO, (B, H, N, d))
    if w.dtype == "bf16":
        out = {k_: bf16_round(v) for k_, v in out.items()}
    out["W_sort"] = _normal(s, _T_WSORT, (H, w.sort_bits, d))
    out["W_race"] = _normal(s, _T_WRACE, (H, w.L, w.race_bits, d))
    return out


def make_gates(w: Workload) -> np.ndarray:
    """Token-wise gate values (g_sparse, g_lr) in (0.05, 0.95), shape [B,H,N,2]."""
    g = _rng(w.seed, _T_GATES).uniform(0.05, 0.95, size=(w.B, w.H, w.N, 2))
    return g.astype(np.float32)


def make_lambda_rows(w: Workload, lo: float = 0.05, hi: float = 3.0) -> np.ndarray:
    """Token-wise fusion coefficients lambda_i in (lo, hi), shape [B,H,N]."""
    lam = _rng(w.seed, _T_LAMBDA).uniform(lo, hi, size=(w.B, w.H, w.N))
    return lam.astype(np.float32)


def make_rule_params(w: Workload, G: int, lam: bool = True) -> dict:
    """Parameters of the token-wise rules for every head: gate network
    W1 [H,G,d] ~ N(0, 1/d), b1 [H,G] ~ N(0, 0.1^2), W2 [H,2,G] ~ N(0, 1/G),
    b2 [H,2] ~ N(0, 0.1^2); lambda rule w [H,d] ~ N(0, 0.05^2), b [H] ~
    N(0, 0.1^2), c [H] uniform in (0.2, 0.4).  float32."""
    rng = _rng(w.seed, _T_RULES)
    H, d = w.H, w.d
    out = {}
    if G:
        out["W1"] = (rng.standard_normal((H, G, d)) / np.sqrt(d)).astype(np.float32)
        out["b1"] = (rng.standard_normal((H, G)) * 0.1).astype(np.float32)
        out["W2"] = (rng.standard_normal((H, 2, G)) / np.sqrt(G)).astype(np.float32)
        out["b2"] = (rng.standard_normal((H, 2)) * 0.1).astype(np.float32)
    if lam:
        out["lam_w"] = (rng.standard_normal((H, d)) * 0.05).astype(np.float32)
        out["lam_b"] = (rng.standard_normal(H) * 0.1).astype(np.float32)
        out["lam_c"] = rng.uniform(0.2, 0.4, size=H).astype(np.float32)
    return out


def make_rule_grads(w: Workload) -> dict:
    """Upstream gradients of the rules' outputs: dgates [B,H,N,2] and
    dlambda [B,H,N], N(0,1) float32."""
    rng = _rng(w.seed, _T_RULE_GRADS)
    return {"dgates": rng.standard_normal((w.B, w.H, w.N, 2)).astype(np.float32),
            "dlambda": rng.standard_normal((w.B, w.H, w.N)).astype(np.float32)}


def make_block_inputs(w: Workload) -> dict:
    """Inputs of an attention-block step: X [B,N,d_model], W_{Q,K,V,O}, dY.

    Weights are N(0, 0.02^2) with no bias; activations and the upstream
    gradient are N(0,1); all rounded to bf16 for bf16 workloads.
    """
    dm = w.d_model
    out = {
        "X": _normal(w.seed, _T_X, (w.B, w.N, dm)),
        "W_Q": _normal(w.seed, _T_WQ, (dm, dm)) * np.float32(0.02),
        "W_K": _normal(w.seed, _T_WK, (dm, dm)) * np.float32(0.02),
        "W_V": _normal(w.seed, _T_WV, (dm, dm)) * np.float32(0.02),
        "W_O": _normal(w.seed, _T_WO, (dm, dm)) * np.float32(0.02),
        "dY": _normal(w.seed, _T_DY, (w.B, w.N, dm)),
    }
    if w.dtype == "bf16":
        out = {k_: bf16_round(v) for k_, v in out.items()}
    out["W_sort"] = _normal(w.seed, _T_WSORT, (w.H, w.sort_bits, w.d))
    out["W_race"] = _normal(w.seed, _T_WRACE, (w.H, w.L, w.race_bits, w.d))
    return out


# The five operator workloads measured and parity-tested by this repository.
TINY_FP32 = Workload("tiny-fwd-noncausal-fp32", 1, 1, 512, 64, 32, 32, False, "f32",
                     recipe="iid", qk_scale=64 ** -0.25, backward=False, seed=1)
CLUSTERED_4K = Workload("clustered-4k-noncausal-bf16", 2, 8, 4096, 64, 64, 64, False, "bf16",
                        recipe="clustered", centres=64, seed=2)
CAUSAL_16K = Workload("causal-16k-d128-bf16", 1, 16, 16384, 128, 128, 128, True, "bf16",
                      recipe="iid", qk_scale=128 ** -0.25, seed=3)
CAUSAL_64K_MIXED = Workload("causal-64k-mixed-bf16", 1, 8, 65536, 128, 256, 256, True, "bf16",
                            recipe="mixed", centres=256, seed=4)
BLOCK_32K = Workload("block-32k-dmodel1024-bf16", 1, 16, 32768, 64, 128, 128, True, "bf16",
                     recipe="iid", seed=5, d_model=1024)

# the paper's causal text setting (block size 256, base length 4096, RACE
# with 4 tables of 4 bits) at its ArXiv length N = 32000: three levels of
# 16000 / 8000 / 4000 sorted queries and leaves of 4000 tokens
TEXT_32K = Workload("causal-32k-text-b256-n04096-bf16", 1, 16, 32000, 128, 256, 64, True, "bf16",
                    recipe="iid", qk_scale=128 ** -0.25, n0=4096, seed=6)
WORKLOADS = {w.name: w for w in (TINY_FP32, CLUSTERED_4K, CAUSAL_16K, CAUSAL_64K_MIXED, BLOCK_32K, TEXT_32K)}


def random_matrix(seed: int, tid: int, shape, scale: float = 1.0) -> np.ndarray:
    """Seeded N(0, scale^2) float32 array rounded to bf16 values (matrix-core
    operands of the projection tests)."""
    return bf16_round(_normal(seed, tid, shape) * np.float32(scale))
