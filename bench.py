#!/usr/bin/env python3
"""ELSAA forward + backward throughput on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step = elsaa_fwd + elsaa_bwd over one batch of the workload (all inputs
already resident in HBM).  After W warm-up steps, K steps are timed as a user
runs them (value, ms_per_step); then K more steps are timed with the library's
per-kernel HIP events on (each launch bracketed on its own stream), which give
the kernel durations behind the roofline of the dominant kernel and of every
kernel (their step time is reported as profiled_ms_per_step).  Last, K calls
of the forward and of the backward are timed on their own (medians, in
fwd_bwd_split), and K replays of one step captured as a HIP graph (graph_replay:
the same kernels without per-launch host overhead).  Prints one JSON line, with
the CPU oracle timed on a bounded sample.
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


def survey_units(w, Lv: int, rules_G: int = 0, rules_lam: bool = False, rules_part_bytes: int = 0) -> dict:
    """Algorithmic bytes and flops per step of each unit of the hot path, in
    the accounting of the method's complexity (the Theta(N s) sparse term and
    the Theta(N L_s 2^gamma) RACE term turned into bytes): every input the
    step must read is counted once, every output written once; partial
    results that one kernel hands to the next are NOT counted.

    Returns {unit: (bytes, flops, kernels)}; a unit is one kernel or the few
    kernels that together compute one step of the path.  Per head, with s the
    element size, N tokens, d = d_h, Lv causal levels:
      selection      2Nds + 2N (hash: Q, K read, keys written) and the perm
                     writes, 8N non-causal or 4N per level
      sparse fwd     3Nds + 4Nd + 12N (leaf / blocks) and 1.5Nds + 4N per level
      low-rank fwd   N (3ds + 4d + 4)
      sparse bwd     4Nds + 12Nd + 8N (leaf / blocks) and 2Nds + 4N per level
      low-rank bwd   2 N (3ds + 4d + 4)
      fusion         N (ds + 4d + 8), fused into the sparse leaf / blocks kernel
                     (O_lr and d_lr read, O and m written; O_s never leaves it)
      bwd rows       N (ds + 8d + 12)  (dO, O_s and O_lr read, row scalars)
    Flops: 4d per sparse interaction forward, 10d backward (recompute
    included); low-rank forward 4r(d+1) + 4dL gamma per token plus
    2C(r+d+1) causal (C = 64), backward 2.25 times that; bwd rows 4d per row.
    """
    s = 2 if w.dtype == "bf16" else 4
    bh = w.B * w.H
    N, D, k, r, L = w.N, w.d, w.k, w.r, w.L
    gs, g = w.sort_bits, w.race_bits
    C = 64
    u = {}
    u["project"] = (bh * (2 * N * D * s + 2 * N), bh * N * 2 * 2 * D * gs, ["project"])
    u["sort"] = (bh * (4 * N * Lv if w.causal else 8 * N), 0, ["sort"])
    lr_tok_bytes = 3 * D * s + 4 * D + 4
    lr_tok_flops = 4 * r * (D + 1) + 4 * D * L * g + (2 * C * (r + D + 1) if w.causal else 0)
    u["lowrank_fwd"] = (bh * N * lr_tok_bytes, bh * N * lr_tok_flops,
                        ["race_state_fwd", "race_scan_fwd", "race_out"])
    u["lowrank_bwd"] = (2 * bh * N * lr_tok_bytes, int(2.25 * bh * N * lr_tok_flops),
                        ["race_state_bwd", "race_scan_bwd", "race_dq", "race_dk", "race_dv", "race_wt"])
    u["bwd_rows"] = (bh * N * (D * s + 8 * D + 12), bh * N * 4 * D, ["bwd_rows"])
    base_fwd = bh * (3 * N * D * s + 4 * N * D + 12 * N) + bh * N * (D * s + 4 * D + 8)
    base_bwd = bh * (4 * N * D * s + 12 * N * D + 8 * N)
    if w.causal:
        half = N // 2
        n_leaf = N >> Lv
        lvl_inter = bh * Lv * half * min(k, half)
        leaf_inter = bh * (N // n_leaf) * (n_leaf * (n_leaf + 1) // 2)
        u["sparse_fwd_levels"] = (bh * Lv * (3 * half * D * s + 4 * N), lvl_inter * 4 * D, ["sparse_fwd_levels"])
        u["sparse_fwd_leaf"] = (base_fwd, leaf_inter * 4 * D, ["sparse_fwd_leaf"])
        u["sparse_bwd_levels"] = (bh * Lv * (2 * N * D * s + 4 * N), lvl_inter * 10 * D,
                                  ["sparse_bwd_levels", "sparse_dq_levels", "sparse_dkv_levels"])
        u["sparse_bwd_leaf"] = (base_bwd, leaf_inter * 10 * D,
                                ["sparse_leaf_bwd", "sparse_dq_leaf", "sparse_dkv_leaf"])
    else:
        inter = bh * N * min(k, N)
        u["sparse_fwd_blocks"] = (base_fwd, inter * 4 * D, ["sparse_fwd_blocks"])
        u["sparse_bwd_blocks"] = (base_bwd, inter * 10 * D,
                                  ["sparse_bwd_blocks", "sparse_dq_blocks", "sparse_dkv_blocks"])
    if rules_G or rules_lam:
        # token-wise rules (outside the operator): q read once; gates (8 B) and
        # lambda (4 B) per row; the backward also reads dgates / dlambda and
        # adds into dQ (read + write); the reduction reads the partial records
        G = rules_G
        gx = G + (1 if rules_lam else 0)
        out_b = (8 if G else 0) + (4 if rules_lam else 0)
        u["token_rules_fwd"] = (bh * N * (D * s + out_b), bh * N * (2 * D * gx + 4 * G), ["token_rules_fwd"])
        u["token_rules_bwd"] = (bh * N * (D * s + out_b + (2 * D * s if G else 0)),
                                bh * N * (2 * D * gx * 2 + (2 * D * G) + 8 * G),
                                ["token_rules_bwd", "token_rules_reduce"])
    if w.d_model:
        # the six dense products of one block step (bf16 operands; QKV and dO
        # written bf16, Y and the gradients of X and of the weights float32)
        T, dm = w.B * w.N, w.d_model
        prods = [(T, 3 * dm, dm, 2), (T, dm, dm, 4), (T, dm, dm, 2),
                 (dm, dm, T, 4), (T, dm, 3 * dm, 4), (dm, 3 * dm, T, 4)]
        u["gemm"] = (sum(2 * (M * K + K * N_) + o * M * N_ for M, N_, K, o in prods),
                     sum(2 * M * N_ * K for M, N_, K, _ in prods), ["gemm", "gemm_reduce"])
    return u


def kernel_model(w, Lv: int) -> dict:
    """Bytes each sparse-branch kernel actually has to move as the path is
    split into kernels (name -> bytes per step): the survey accounting above
    plus the level partials (storage dtype), which the level kernels write and the
    leaf kernels read back, with every tensor at the size the path stores it
    (O_s float32; O_lr and the gradients in the storage dtype).  Reported beside the
    algorithmic figure so the cost of the split is visible; not a roofline
    numerator."""
    s = 2 if w.dtype == "bf16" else 4
    bh = w.B * w.H
    N, D = w.N, w.d
    if not w.causal:
        return {}
    half = N // 2
    ps = s                          # level partials are kept in the storage dtype
    lvl_pos = Lv * bh * half        # (level, position) slots of the partials
    wk = max(32, 4 * w.L)
    return {
        "sparse_fwd_levels": lvl_pos * (3 * D * s + 8 + D * ps + 4),
        "sparse_fwd_leaf": bh * N * (3 * D * s + 4 * D + D * s + 4 + D * s + 8) + lvl_pos * (D * ps + 4),
        "sparse_bwd_levels": lvl_pos * (4 * D * s + 20 + 3 * D * ps),
        "sparse_leaf_bwd": bh * N * (4 * D * s + 12 + 2 * wk * s + D * s + 3 * D * s) + lvl_pos * 3 * D * ps,
    }



def source_digest(names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_20214_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "project": ["select.hip", "common.hpp"], "sort": ["select.hip", "causal.hpp"],
    "race_state_fwd": ["race_fwd.hip", "race_common.hpp", "common.hpp"],
    "race_state_bwd": ["race_fwd.hip", "race_common.hpp", "common.hpp"],
    "race_scan_fwd": ["race_fwd.hip"], "race_scan_bwd": ["race_fwd.hip"],
    "race_out": ["race_fwd.hip", "race_common.hpp", "common.hpp"],
    "race_dq": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "race_dk": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "race_dv": ["race_bwd.hip", "race_common.hpp", "common.hpp"],
    "bwd_rows": ["bwd_rows.hip", "common.hpp"],
    "gemm": ["gemm.hip", "common.hpp"], "gemm_reduce": ["gemm.hip"],
    "token_rules_fwd": ["token_rules.hip", "tile.hpp", "common.hpp"],
    "token_rules_bwd": ["token_rules.hip", "tile.hpp", "common.hpp"],
    "token_rules_reduce": ["token_rules.hip"],
}


def sources_of(kernel: str):
    if kernel in KERNEL_SOURCES:
        return KERNEL_SOURCES[kernel]
    if kernel.startswith("sparse_fwd"):
        return ["sparse_fwd.hip", "tile.hpp", "causal.hpp", "internal.hpp", "common.hpp"]
    return ["sparse_bwd.hip", "tile.hpp", "causal.hpp", "internal.hpp", "common.hpp"]


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


def cpu_model() -> str:
    """Model name of the host CPU (first 'model name' line of /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_heads(w, inp, hc, backward: bool, min_seconds: float):
    """Run the oracle on whole heads until about min_seconds have passed (at
    least one head); returns (heads done, seconds).  The oracle's backward
    computes the forward state itself, so one backward call is a complete
    forward + backward of the head."""
    import oracle

    done, t0 = 0, time.perf_counter()
    for b in range(w.B):
        for h in range(w.H):
            args = (inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h], inp["W_race"][h])
            if backward:
                oracle.backward(hc, *args, inp["dO"][b, h])
            else:
                oracle.forward(hc, *args)
            done += 1
            if time.perf_counter() - t0 >= min_seconds:
                return done, time.perf_counter() - t0
    return done, time.perf_counter() - t0


def cpu_baseline(w, inp, min_seconds: float = 10.0) -> dict:
    """The fp64 oracle on the host cores, on a bounded sample of whole heads,
    scaled to whole-job tokens/s (the job is B * H heads).  The forward and
    the forward + backward (one oracle backward call, which computes its
    forward state itself) are timed separately; value is the latter, or the
    forward alone for forward-only workloads.  Small workloads also get a
    single-thread figure."""
    import oracle

    threads = oracle.threads()
    hc = oracle.head_cfg(w)
    total = w.B * w.H
    nf, tf = _oracle_heads(w, inp, hc, False, min_seconds / 3)
    fwd_tps = w.B * w.N * nf / (tf * total)
    out = {"unit": "tokens/s", "cores": threads, "kind": "oracle", "cpu": cpu_model(),
           "fwd_value": fwd_tps}
    if w.backward:
        nb, tb = _oracle_heads(w, inp, hc, True, min_seconds)
        out["value"] = w.B * w.N * nb / (tb * total)
        # the backward alone: a head's forward + backward less its forward
        t_bwd = tb / nb - tf / nf
        if t_bwd > 0:
            out["bwd_value"] = w.B * w.N / (t_bwd * total)
        out["sample"] = (f"forward alone on {nf} of {total} heads ({tf:.1f} s); forward + backward (one "
                         f"oracle backward call per head) on {nb} of {total} heads ({tb:.1f} s); all "
                         f"{w.N} tokens of each head; {threads} threads; scaled to {total} heads")
    else:
        out["value"] = fwd_tps
        out["sample"] = (f"forward on {nf} of {total} heads, all {w.N} tokens each ({tf:.1f} s); "
                         f"{threads} threads; scaled to {total} heads")
    if w.B * w.N * w.H <= 65536:
        oracle.threads(1)
        try:
            n1, t1 = _oracle_heads(w, inp, hc, w.backward, min_seconds / 2)
        finally:
            oracle.threads(threads)
        out["single_thread_value"] = w.B * w.N * n1 / (t1 * total)
    return out


def cpu_baseline_block(w, inp, blk, min_seconds: float = 10.0) -> dict:
    """Oracle of one attention-block step on a bounded sample: the six
    float64 products on a slice of the tokens and the operator forward +
    backward on whole heads, each scaled to the full step."""
    import numpy as np
    import oracle

    threads = oracle.threads()
    T, dm = w.B * w.N, w.d_model
    rows = 2048
    X = blk["X"].reshape(T, dm)[:rows]
    dY = blk["dY"].reshape(T, dm)[:rows]
    Wqkv = np.concatenate([blk["W_Q"], blk["W_K"], blk["W_V"]], axis=1)
    t0 = time.perf_counter()
    qkv = oracle.gemm(X, Wqkv)
    O = qkv[:, :dm]
    oracle.gemm(O, blk["W_O"])
    oracle.gemm(dY, blk["W_O"], False, True)
    oracle.gemm(O, dY, True, False)
    oracle.gemm(qkv, Wqkv, False, True)
    oracle.gemm(X, qkv, True, False)
    t_gemm = (time.perf_counter() - t0) * T / rows
    hc = oracle.head_cfg(w)
    done, dt = _oracle_heads(w, inp, hc, True, min_seconds)
    t_att = dt * (w.B * w.H) / done
    return {"value": T / (t_gemm + t_att), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"projections on {rows} of {T} tokens and the operator forward + backward (one "
                      f"oracle backward call per head) on {done} of {w.B * w.H} heads, scaled to the "
                      f"full step"}


def roofline_entry(nbytes, nflops, seconds, peak_tf):
    """Roofline of work (bytes, flops) done in `seconds`: bound by whichever
    of HBM and the matrix cores would take longer at peak."""
    if nbytes / (PEAK_HBM_GBS * 1e9) >= nflops / (peak_tf * 1e12):
        a = nbytes / seconds / 1e9
        return {"bound": "hbm", "achieved": round(a, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(a / PEAK_HBM_GBS, 4)}
    a = nflops / seconds / 1e12
    return {"bound": "mfma", "achieved": round(a, 2), "peak": peak_tf, "unit": "TFLOP/s",
            "frac": round(a / peak_tf, 4)}


def dominant_unit(unit_rows: dict, per_step: dict) -> str:
    """The unit of the kernel with the largest time per step.  unit_rows:
    {unit: (ms, bytes, flops, kernels that ran)}; per_step: {kernel: ms}."""
    unit_of = {kn: name for name, row in unit_rows.items() for kn in row[3]}
    return unit_of[max(unit_of, key=lambda kn: per_step[kn])]


def graph_replay(step, steps: int, warmup: int) -> dict:
    """Capture one step as a HIP graph (after a warm-up call on a side stream,
    as capture needs) and time `steps` replays; a refused capture is
    reported instead of ending the run."""
    import torch
    try:
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            step()
        torch.cuda.current_stream().wait_stream(cap)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            g.replay()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        del g
        return {"ms_per_step": round((t1 - t0) / steps * 1e3, 4), "steps": steps}
    except RuntimeError as exc:
        torch.cuda.synchronize()
        return {"error": str(exc)[:200]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="causal-16k-d128-bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rules", action="store_true",
                    help="add the token-wise rules (gate network of hidden width 64 and the "
                         "query-dependent lambda) around the operator in every step")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of 1 GiB (reference for HBM byte counters)")
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
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 4, "copy_bytes_written": dst.numel() * 4}))
        return
    cfg = E.Config(B=w.B, H=w.H, N=w.N, d_h=w.d, k=w.k, r=w.r, causal=w.causal, dtype=w.dtype,
                   race_bits=w.race_bits, sort_bits=w.sort_bits, n0=w.n0 or 0)
    inp = W.make_inputs(w, with_grad=w.backward)
    dt = cfg.torch_dtype

    def to(x, t):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(t).contiguous()

    q, k, v = (to(inp[n], dt) for n in ("Q", "K", "V"))
    do = to(inp["dO"], dt) if w.backward else None
    ws, wr = to(inp["W_sort"], torch.float32), to(inp["W_race"], torch.float32)
    bufs = E.Buffers(cfg, dev, backward=w.backward)
    Lv = E.num_levels(cfg)

    def step():
        o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, buffers=bufs)
        E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, buffers=bufs)

    if not w.backward:
        def step():
            E.fwd(cfg, q, k, v, ws, wr, buffers=bufs)

    rules_G, rules_part = 0, 0
    if args.rules:
        if not w.backward:
            raise SystemExit("--rules needs a forward + backward workload")
        rules_G = 64
        rp = W.make_rule_params(w, rules_G, True)
        rules = E.TokenRules(**{n: to(a, torch.float32) for n, a in rp.items()})
        rules_part = E.token_rules_workspace_bytes(cfg, rules)

        def step():
            gates, lam = E.token_rules_fwd(cfg, rules, q)
            o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, gates=gates, buffers=bufs, lam_rows=lam)
            dq, _, _, dg, dl = E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, gates=gates, want_dgates=True,
                                     buffers=bufs, lam_rows=lam, want_dlambda=True)
            E.token_rules_bwd(cfg, rules, q, dg, dl, dq=dq)

    blk = None
    if w.d_model:
        # one attention-block step: projections on the matrix cores around the
        # operator, every attention tensor head-major [1, 3H or H, N, d_h]
        from paper_2607_20214_amd.block import AttentionBlock

        blk = W.make_block_inputs(w)
        Tn, dm = w.B * w.N, w.d_model
        bf = torch.bfloat16
        block = AttentionBlock(cfg, to(blk["X"].reshape(Tn, dm), bf), to(blk["dY"].reshape(Tn, dm), bf),
                               to(np.concatenate([blk["W_Q"], blk["W_K"], blk["W_V"]], axis=1), bf),
                               to(blk["W_O"], bf), ws, wr)
        del bufs, q, k, v, do
        step = block.step

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # timed region 1: the steps as a user runs them (throughput, ms_per_step)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # timed region 2: the same steps with the library's per-kernel HIP events
    # recorded on each launch's stream (kernel durations for the roofline);
    # the events cost time of their own, so this region's step time is
    # reported separately
    E.profile_enable(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    prof = E.profile_read()
    E.profile_enable(False)
    # timed region 3: forward and backward each on their own, every call
    # bracketed by events on torch's current stream (the library's side
    # stream joins that stream before each call returns); medians over the
    # calls
    split = None
    if w.backward and blk is None and not args.rules:
        cur = torch.cuda.current_stream()
        tf, tb = [], []
        for _ in range(args.steps):
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(cur)
            o_, lse_, dlr_, saved_ = E.fwd(cfg, q, k, v, ws, wr, buffers=bufs)
            e1.record(cur)
            E.bwd(cfg, q, k, v, wr, do, lse_, dlr_, saved_, buffers=bufs)
            e2.record(cur)
            e2.synchronize()
            tf.append(e0.elapsed_time(e1))
            tb.append(e1.elapsed_time(e2))
        split = {"fwd_ms_median": round(float(np.median(tf)), 4), "bwd_ms_median": round(float(np.median(tb)), 4),
                 "calls": args.steps}

    # timed region 4: one step captured as a HIP graph (the library enqueues
    # only kernels and event record / wait pairs), replayed K times
    graph = graph_replay(step, args.steps, args.warmup) if blk is None and not args.rules else None

    elapsed = t1 - t0
    ms_step = elapsed / args.steps * 1e3
    tokens = w.B * w.N * args.steps
    per_step = {name: ms / args.steps for name, (ms, n) in prof.items()}
    units = survey_units(w, Lv, rules_G, bool(args.rules), rules_part)
    peak_tf = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS

    # per-unit roofline: algorithmic bytes / flops of the unit per step over
    # the summed per-step time of its kernels
    unit_rows = {}
    for name, (nb, nf, kernels) in units.items():
        ran = [kn for kn in kernels if kn in prof]
        if not ran:
            continue
        ms = sum(per_step[kn] for kn in ran)
        unit_rows[name] = (ms, nb, nf, ran)
    # the dominant kernel (largest time per step) and its unit; for a unit of
    # one kernel the figures are per launch over that kernel's average launch
    # duration, for a unit of several the unit's per step
    dom = dominant_unit(unit_rows, per_step)
    ms, nb, nf, ran = unit_rows[dom]
    if len(ran) == 1:
        tot_ms, n = prof[ran[0]]
        per = n // args.steps
        avg_s = tot_ms / n / 1e3
        nb, nf = nb / per, nf / per
        roof = roofline_entry(nb, nf, avg_s, peak_tf)
        roof["traffic"] = read_traffic(ran[0], w.name)
        roof["kernel"] = ran[0]
        roof["avg_launch_ms"] = round(avg_s * 1e3, 4)
        roof["algorithmic_bytes_per_launch"] = nb
        roof["algorithmic_flops_per_launch"] = nf
    else:
        roof = roofline_entry(nb, nf, ms / 1e3, peak_tf)
        roof["traffic"] = None
        roof["kernel"] = dom
        roof["kernels"] = ran
        roof["ms_per_step"] = round(ms, 4)
        roof["algorithmic_bytes_per_step"] = nb
        roof["algorithmic_flops_per_step"] = nf
    # the whole step against the same accounting
    step_b = sum(r_[1] for r_ in unit_rows.values())
    step_f = sum(r_[2] for r_ in unit_rows.values())
    step_roof = roofline_entry(step_b, step_f, ms_step / 1e3, peak_tf)
    step_roof["algorithmic_bytes_per_step"] = step_b
    step_roof["algorithmic_flops_per_step"] = step_f
    # what the split into kernels moves (the sparse kernels' level partials)
    km = kernel_model(w, Lv)
    kmodel = {}
    for kn, b_ in km.items():
        if kn in prof:
            tot_ms, n = prof[kn]
            kmodel[kn] = {"bytes_per_launch": b_ / (n // args.steps),
                          "frac": round(b_ / (n // args.steps) / (tot_ms / n / 1e3) / 1e9 / PEAK_HBM_GBS, 4),
                          "traffic": read_traffic(kn, w.name)}

    if blk is not None:
        metric = "ELSAA attention-block step (projections + operator) fwd+bwd tokens/sec"
    elif not w.backward:
        metric = "ELSAA forward tokens/sec (forward-only workload)"
    else:
        metric = "ELSAA fwd+bwd tokens/sec at N=16k,d_h=128; % HBM/MFMA roofline"
    result = {
        "metric": metric,
        "value": tokens / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "profiled_ms_per_step": (t3 - t2) / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "d_h": w.d, "k": w.k, "r": w.r,
                   "causal": w.causal, "levels": Lv, "backward": w.backward,
                   **({"d_model": w.d_model} if blk is not None else {})},
        "roofline": roof,
        "roofline_step": step_roof,
        "roofline_units": {n: {**roofline_entry(r_[1], r_[2], r_[0] / 1e3, peak_tf), "ms_per_step": round(r_[0], 4)}
                           for n, r_ in sorted(unit_rows.items(), key=lambda x: -x[1][0])},
        "roofline_kernel_model": kmodel,
        "kernel_ms_per_step": {n: round(t, 4) for n, t in sorted(per_step.items(), key=lambda x: -x[1])},
    }
    if split is not None:
        result["fwd_bwd_split"] = split
    if graph is not None:
        result["graph_replay"] = graph
    if args.rules:
        result["config"]["rules"] = {"gate_hidden": rules_G, "lambda_rule": True}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_block(w, inp, blk) if blk is not None else cpu_baseline(w, inp)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
