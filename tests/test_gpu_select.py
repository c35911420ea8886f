"""GPU parity of the standalone selection entry point (elsaa_select: Alg. 4
steps Hash / Sort / Partition, one SortLSH call per node of Alg. 5) against
the oracle: the sorted index lists must be identical, bit for bit.

Cases: lists longer than the 16384 keys the sort stages in LDS (non-causal
N = 40000; causal N = 65536 whose first level sorts 32768-key halves),
ragged lengths, fp32 and bf16 storage, d_h 64 and 128, 3 to 8 hash bits,
clustered inputs (many equal keys: the tie order decides), and the lists
elsaa_fwd writes into `saved` for the same inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20214_amd as E
from gpu_util import cfg_of, head_cfg_of, say, to_dev
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, causal, dtype, recipe="iid", sort_bits=5, seed=70, **kw):
    qs = d ** -0.25 if recipe == "iid" else 1.0
    return W.Workload(name, B, H, N, d, k, 16, causal, dtype, recipe=recipe, qk_scale=qs, seed=seed,
                      sort_bits=sort_bits, centres=kw.pop("centres", 16), **kw)


CASES = [
    _w("nc-bf16-d64-40000", 1, 2, 40000, 64, 64, False, "bf16"),
    _w("c-bf16-d128-65536-k256", 1, 1, 65536, 128, 256, True, "bf16"),
    _w("nc-f32-d128-777-bits3", 2, 1, 777, 128, 32, False, "f32", sort_bits=3),
    _w("c-f32-d64-3072-bits8", 1, 2, 3072, 64, 128, True, "f32", sort_bits=8),
    _w("c-bf16-d64-2048-clustered", 1, 2, 2048, 64, 64, True, "bf16", recipe="clustered", centres=4),
    _w("nc-bf16-d128-5000-clustered-bits1", 1, 1, 5000, 128, 128, False, "bf16", recipe="clustered",
       sort_bits=1, centres=3),
]


def _run(w):
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    say(f"[select] {w.name}: B={w.B} H={w.H} N={w.N} d={w.d} k={w.k} causal={w.causal} bits={w.sort_bits}")
    dt = cfg.torch_dtype
    q, k = to_dev(inp["Q"], dt), to_dev(inp["K"], dt)
    ws = to_dev(inp["W_sort"], torch.float32)
    pq, pk = E.select(cfg, q, k, ws)
    torch.cuda.synchronize()
    return cfg, inp, pq.cpu().numpy(), pk.cpu().numpy()


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_select_matches_oracle(w):
    cfg, inp, pq, pk = _run(w)
    hc = head_cfg_of(cfg)
    for b in range(w.B):
        for h in range(w.H):
            rq, rk = oracle.select(hc, inp["Q"][b, h], inp["K"][b, h], inp["W_sort"][h])
            assert np.array_equal(pq[b, h], rq), f"perm_q (b={b}, h={h})"
            assert np.array_equal(pk[b, h], rk), f"perm_k (b={b}, h={h})"


def test_select_equals_forward_selection():
    """elsaa_select and the selection elsaa_fwd keeps in `saved` agree."""
    w = _w("c-bf16-d128-4096", 1, 2, 4096, 128, 128, True, "bf16", seed=71)
    cfg, inp, pq, pk = _run(w)
    dt = cfg.torch_dtype
    q, k, v = (to_dev(inp[n], dt) for n in ("Q", "K", "V"))
    ws, wr = to_dev(inp["W_sort"], torch.float32), to_dev(inp["W_race"], torch.float32)
    _, _, _, saved = E.fwd(cfg, q, k, v, ws, wr)
    torch.cuda.synchronize()
    sv = E.saved_views(cfg, saved)
    assert np.array_equal(sv["perm_q"].cpu().numpy(), pq)
    assert np.array_equal(sv["perm_k"].cpu().numpy(), pk)
