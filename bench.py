#!/usr/bin/env python3
"""ELSAA forward + backward throughput on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step = elsaa_fwd + elsaa_bwd over one batch of the workload (all inputs
already resident in HBM).  Prints one JSON line with tokens/s, the roofline
of the dominant kernel (timed with HIP events on the library's stream over
the timed region) and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # fp32 matrix


def kernel_model(w, Lv: int) -> dict:
    """Algorithmic bytes and flops per launch of each kernel (name -> (bytes, flops)).

    Counts what the method must move or compute: every input row it needs is
    read once per pass that needs it, outputs are written once at their
    storage precision; scratch partials between kernels are not counted.
    """
    s = 2 if w.dtype == "bf16" else 4
    bh = w.B * w.H
    N, D, k, r, L = w.N, w.d, w.k, w.r, w.L
    P = 4 * L                      # RACE projections per row
    gs = w.sort_bits
    n0 = w.base_len
    n_leaf = N >> Lv
    seg_states = 0                 # RACE segment states are reported with race_state/scan
    half = N // 2
    m = {}
    m["project"] = (bh * N * (D * s + 1 + P * 4), bh * N * 2 * D * (gs + P))
    m["sort"] = (bh * (Lv if w.causal else 2) * N * 5, 0)
    # RACE: features, chunk states (r x d per 64-token chunk), readout
    C = 64
    m["race_state"] = (bh * N * (P * 4 + D * s), bh * N * 2 * r * D)
    m["race_out"] = (bh * N * (2 * P * 4 + D * s + D * s + 4),
                     bh * N * (2 * r * D * (2 if w.causal else 1) + (C * (r + D) if w.causal else 0)))
    m["race_dq"] = (bh * N * (2 * P * 4 + 2 * D * s + 8 + D * s),
                    bh * N * (2 * r * D * 2 + C * (D + r) + 2 * P * D))
    m["race_dk"] = m["race_dq"]
    m["race_dv"] = (bh * N * (2 * P * 4 + D * s + 4 + D * s), bh * N * (2 * r * D * 2 + C * (r + D)))
    # sparse branch: interactions per query, 4D flops each forward (QK^T, PV)
    lvl_inter = half * min(k, half) if w.causal else 0
    m["sparse_fwd_levels"] = (Lv * bh * half * (3 * D * s + 8), Lv * bh * lvl_inter * 4 * D)
    m["sparse_fwd_leaf"] = (bh * N * (3 * D * s + D * 4 + 4 + D * s + 12),
                            bh * (N // n_leaf) * (n_leaf * (n_leaf + 1) // 2) * 4 * D)
    m["sparse_fwd_blocks"] = (bh * N * (3 * D * s + 8 + D * 4 + 4 + D * s + 12), bh * N * min(k, N) * 4 * D)
    m["bwd_rows"] = (bh * N * (D * s + 2 * D * 4 + 12 + 20), bh * N * 4 * D)
    m["sparse_dq_levels"] = (Lv * bh * half * (4 * D * s + 8 + D * 4), Lv * bh * lvl_inter * 6 * D)
    m["sparse_dkv_levels"] = (Lv * bh * half * (4 * D * s + 8 + 2 * D * 4), Lv * bh * lvl_inter * 8 * D)
    leaf_inter = bh * (N // n_leaf) * (n_leaf * (n_leaf + 1) // 2)
    m["sparse_dq_leaf"] = (bh * N * (4 * D * s + D * s + 12), leaf_inter * 6 * D)
    m["sparse_dkv_leaf"] = (bh * N * (4 * D * s + 2 * D * s + 12), leaf_inter * 8 * D)
    m["sparse_dq_blocks"] = (bh * N * (4 * D * s + D * s + 12), bh * N * min(k, N) * 6 * D)
    m["sparse_dkv_blocks"] = (bh * N * (4 * D * s + 2 * D * s + 12), bh * N * min(k, N) * 8 * D)
    del seg_states, n0
    return m


def source_digest(names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_20214_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "project": ["select.hip", "common.hpp"], "sort": ["select.hip"],
    "race_state": ["race_fwd.hip", "race_common.hpp", "common.hpp"],
    "race_scan": ["race_fwd.hip"], "race_out": ["race_fwd.hip", "race_common.hpp", "common.hpp"],
    "race_dq": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "race_dk": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "race_dv": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "bwd_rows": ["bwd_rows.hip", "common.hpp"],
}


def sources_of(kernel: str):
    if kernel in KERNEL_SOURCES:
        return KERNEL_SOURCES[kernel]
    if kernel.startswith("sparse_fwd"):
        return ["sparse_fwd.hip", "common.hpp"]
    return ["sparse_bwd.hip", "common.hpp"]


def read_traffic(kernel: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 --pmc summary, if it
    was taken on the current source of that kernel (else None)."""
    path = os.path.join(ROOT, "profiles", f"{kernel}.{workload}.pmc.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                key, v = line.split(":", 1)
                vals[key.strip()] = v.strip()
    if vals.get("source_digest") != source_digest(sources_of(kernel)):
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, inp, min_seconds: float = 10.0) -> dict:
    """Oracle forward + backward over the full sequence of as many heads as
    fit in about min_seconds (at least one), scaled to whole-job tokens/s
    (the job is B * H such heads)."""
    import oracle

    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    hc = oracle.head_cfg(w)
    heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    done = 0
    t0 = time.perf_counter()
    for b, h in heads:
        args = (inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h], inp["W_race"][h])
        oracle.forward(hc, *args)
        oracle.backward(hc, *args, inp["dO"][b, h])
        done += 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = time.perf_counter() - t0
    total = len(heads)
    return {"value": w.B * w.N * done / (dt * total), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{done} of {total} heads, all {w.N} tokens each, forward + backward in "
                      f"{dt:.1f} s, scaled to {total} heads"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="causal-16k-d128-bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the ELSAA operator on one GPU only; multi-GPU runs are not "
              "part of this build (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_20214_amd as E
    from paper_2607_20214_amd import workloads as W

    w = W.WORKLOADS[args.workload]
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    cfg = E.Config(B=w.B, H=w.H, N=w.N, d_h=w.d, k=w.k, r=w.r, causal=w.causal, dtype=w.dtype,
                   race_bits=w.race_bits, sort_bits=w.sort_bits, n0=w.n0 or 0)
    inp = W.make_inputs(w, with_grad=True)
    dt = cfg.torch_dtype

    def to(x, t):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(t).contiguous()

    q, k, v, do = (to(inp[n], dt) for n in ("Q", "K", "V", "dO"))
    ws, wr = to(inp["W_sort"], torch.float32), to(inp["W_race"], torch.float32)
    bufs = E.Buffers(cfg, dev, backward=True)
    Lv = E.num_levels(cfg)

    def step():
        o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, buffers=bufs)
        E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, buffers=bufs)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    E.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = E.profile_read()
    E.profile_enable(False)

    elapsed = t1 - t0
    tokens = w.B * w.N * args.steps
    per_step = {name: ms / args.steps for name, (ms, n) in prof.items()}
    dom = max(per_step, key=per_step.get)
    ms_total, launches = prof[dom]
    avg_s = ms_total / launches / 1e3
    model = kernel_model(w, Lv)
    nbytes, nflops = model.get(dom, (0, 0))
    t_hbm = nbytes / (PEAK_HBM_GBS * 1e9)
    peak_tf = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    t_mma = nflops / (peak_tf * 1e12)
    if t_hbm >= t_mma:
        ach = nbytes / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4)}
    else:
        ach = nflops / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak_tf, "unit": "TFLOP/s",
                "frac": round(ach / peak_tf, 4)}
    roof["traffic"] = read_traffic(dom, w.name)
    roof["kernel"] = dom
    roof["avg_launch_ms"] = round(avg_s * 1e3, 4)
    roof["algorithmic_bytes_per_launch"] = nbytes
    roof["algorithmic_flops_per_launch"] = nflops

    result = {
        "metric": "ELSAA fwd+bwd tokens/sec at N=16k,d_h=128; % HBM/MFMA roofline",
        "value": tokens / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "d_h": w.d, "k": w.k, "r": w.r,
                   "causal": w.causal, "levels": Lv},
        "roofline": roof,
        "kernel_ms_per_step": {n: round(t, 4) for n, t in sorted(per_step.items(), key=lambda x: -x[1])},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, inp)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
