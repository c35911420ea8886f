"""Helpers of the GPU parity tests: run the HIP library and the CPU oracle
on the same seeded inputs and compare them.

Tolerances: selected indices bit-exact; floating outputs
max|gpu - oracle| / max|oracle| per head <= 1e-4 (float32 storage) or
2e-2 (bfloat16 storage with float32 accumulation)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2607_20214_amd as E
from paper_2607_20214_amd import workloads as W

TOL = {"f32": 1e-4, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def cfg_of(w: W.Workload, **over) -> E.Config:
    kw = dict(B=w.B, H=w.H, N=w.N, d_h=w.d, k=w.k, r=w.r, causal=w.causal, dtype=w.dtype,
              race_bits=w.race_bits, sort_bits=w.sort_bits, n0=w.n0 or 0)
    kw.update(over)
    return E.Config(**kw)


def head_cfg_of(cfg: E.Config) -> oracle.HeadCfg:
    return oracle.HeadCfg(N=cfg.N, d=cfg.d_h, k=cfg.k, r=cfg.r, causal=cfg.causal,
                          race_bits=cfg.race_bits, sort_bits=cfg.sort_bits,
                          n0=cfg.n0 if cfg.n0 > 0 else None, beta=cfg.beta, lam=cfg.lam,
                          eps=cfg.eps, scale=cfg.scale, neighbors=cfg.neighbors, m_one=cfg.m_one)


def to_dev(x: np.ndarray, dtype) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(dtype).contiguous()


def run_gpu_fwd(cfg: E.Config, inp: dict, gates=None, lam_rows=None):
    dt = cfg.torch_dtype
    q, k, v = (to_dev(inp[n], dt) for n in ("Q", "K", "V"))
    ws = to_dev(inp["W_sort"], torch.float32)
    wr = to_dev(inp["W_race"], torch.float32)
    g = None if gates is None else to_dev(gates, torch.float32)
    lr = None if lam_rows is None else to_dev(lam_rows, torch.float32)
    o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, gates=g, lam_rows=lr)
    torch.cuda.synchronize()
    sv = E.saved_views(cfg, saved)
    out = {"O": o, "lse": lse, "d_lr": dlr, "m": sv["m"], "O_s": sv["o_sparse"],
           "O_lr": sv["o_lowrank"], "perm_q": sv["perm_q"], "perm_k": sv["perm_k"]}
    return {k_: t.float().cpu().numpy() if t.is_floating_point() else t.cpu().numpy()
            for k_, t in out.items()}, (q, k, v, ws, wr, g, saved, lse, dlr, lr)


def elem_stats(got, ref) -> dict:
    """Error figures of one tensor against the oracle:
      rel   max|d| / max|ref|            (the bar the tests assert)
      l2    ||d|| / ||ref||
      elem  max over elements of |d| / (|ref| + rms(ref)): each element
            against its own size, the tensor's rms as the floor."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    d = np.abs(g - r)
    mx = float(np.max(np.abs(r))) if r.size else 0.0
    nr = float(np.linalg.norm(r))
    rms = nr / np.sqrt(max(r.size, 1))
    return {"rel": float(d.max()) / (mx if mx > 0 else 1.0) if d.size else 0.0,
            "l2": float(np.linalg.norm(d)) / (nr if nr > 0 else 1.0),
            "elem": float(np.max(d / (np.abs(r) + (rms if rms > 0 else 1.0)))) if d.size else 0.0}


def rel_err(a, b) -> float:
    den = float(np.max(np.abs(b)))
    return float(np.max(np.abs(a.astype(np.float64) - b))) / (den if den > 0 else 1.0)


def compare_heads(name, got, want, tol, heads=None):
    """max|got - want| / max|want| for each (b, h) slice; returns the worst."""
    worst = 0.0
    B, H = got.shape[:2]
    for b in range(B):
        for h in range(H):
            if heads is not None and (b, h) not in heads:
                continue
            e = rel_err(got[b, h], want[b, h])
            worst = max(worst, e)
            assert e <= tol, f"{name} (b={b}, h={h}): relative error {e:.3e} > {tol:.1e}"
    return worst


def run_gpu_fwd_bwd(cfg: E.Config, inp: dict, gates=None, want_dgates=False, lam_rows=None,
                    want_dlambda=False):
    """Forward then backward on the GPU; returns numpy dQ, dK, dV (and dgates,
    dlambda when asked for)."""
    got, (q, k, v, ws, wr, g, saved, lse, dlr, lr) = run_gpu_fwd(cfg, inp, gates, lam_rows)
    do = to_dev(inp["dO"], cfg.torch_dtype)
    res = E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, gates=g, want_dgates=want_dgates,
                lam_rows=lr, want_dlambda=want_dlambda)
    torch.cuda.synchronize()
    names = ["dQ", "dK", "dV"] + (["dgates"] if want_dgates else []) + (["dlambda"] if want_dlambda else [])
    return got, {n: t.float().cpu().numpy() for n, t in zip(names, res)}
