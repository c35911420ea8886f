"""The operator under HIP graph capture: elsaa_fwd and elsaa_bwd enqueue only
kernels and event record / wait pairs (the forward's sort runs on the
library's second stream between a fork and a join), so a caller can capture
a whole step and replay it.  Each replay is checked, bit for bit, against
the eager call on the same inputs, with other eager work and host
synchronisation between the replays."""
import pytest
import torch

import paper_2607_20214_amd as E
from gpu_util import cfg_of, say, to_dev
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, r, causal, dtype, seed):
    qs = d ** -0.25
    return W.Workload(name, B, H, N, d, k, r, causal, dtype, recipe="iid", qk_scale=qs, seed=seed, centres=16)


CASES = [
    (_w("c-bf16-d128-2048", 1, 2, 2048, 128, 128, 128, True, "bf16", 70), True),
    (_w("nc-bf16-d64-1000", 2, 1, 1000, 64, 64, 64, False, "bf16", 71), True),
    (W.TINY_FP32, False),
]


def _step(cfg, bufs, q, k, v, ws, wr, do, backward):
    """One step; returns its outputs and the saved state's typed views (the
    regions the library documents; alignment gaps between them are never
    written)."""
    o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, buffers=bufs)
    out = [o, lse, dlr] + list(E.saved_views(cfg, saved).values())
    if backward:
        out += list(E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, buffers=bufs))
    return out


@pytest.mark.parametrize("w,backward", CASES, ids=[w.name for w, _ in CASES])
def test_step_replays_as_a_graph(w, backward):
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=True)
    dt = cfg.torch_dtype
    q, k, v, do = (to_dev(inp[n], dt) for n in ("Q", "K", "V", "dO"))
    ws, wr = to_dev(inp["W_sort"], torch.float32), to_dev(inp["W_race"], torch.float32)
    say(f"[graph] {w.name}: B={w.B} H={w.H} N={w.N} causal={w.causal} backward={backward}")
    bufs = E.Buffers(cfg, q.device, backward=backward)
    # eager reference (also creates the library's second stream and caches
    # its launch geometry before capture)
    ref = [t.clone() for t in _step(cfg, bufs, q, k, v, ws, wr, do, backward)]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                     # warm-up on a non-default stream, as capture needs
        _step(cfg, bufs, q, k, v, ws, wr, do, backward)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = _step(cfg, bufs, q, k, v, ws, wr, do, backward)
    for rep in range(4):
        for t in outs:
            t.zero_()                                 # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(outs, ref)):
            assert torch.equal(got, want), f"replay {rep}: output {i} differs from the eager call"
    say(f"   {len(outs)} outputs bit-identical over 4 replays")
    del g
