"""The selection entry point that allocates nothing (elsaa_select_noalloc,
keys in the library's fixed device scratch) against the existing entry point
(elsaa_select, keys in a caller workspace): identical index lists, bit for
bit, on two calls in a row, the second on a smaller input, so the second
call reuses scratch the first left behind; and the oracle agrees with both."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20214_amd as E
from gpu_util import cfg_of, head_cfg_of, say, to_dev
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, causal, seed):
    return W.Workload(name, B, H, N, d, k, 64, causal, "bf16", recipe="iid", qk_scale=d ** -0.25, seed=seed)


def _both(w):
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    q, k = to_dev(inp["Q"], torch.bfloat16), to_dev(inp["K"], torch.bfloat16)
    ws = to_dev(inp["W_sort"], torch.float32)
    ref_q, ref_k = E.select(cfg, q, k, ws)
    pq = torch.full_like(ref_q, -7)
    pk = torch.full_like(ref_k, -7)
    E.select_noalloc(cfg, q, k, ws, pq, pk)
    torch.cuda.synchronize()
    return cfg, inp, ref_q.cpu().numpy(), ref_k.cpu().numpy(), pq.cpu().numpy(), pk.cpu().numpy()


@pytest.mark.parametrize("causal", [True, False])
def test_select_noalloc_matches_select_twice(causal):
    big = _w("noalloc-big", 2, 4, 16384, 128, 128, causal, 80)
    small = _w("noalloc-small", 1, 2, 1000 if not causal else 2048, 64, 64, causal, 81)
    for w in (big, small):
        say(f"[noalloc] {w.name}: B={w.B} H={w.H} N={w.N} d={w.d} causal={causal}")
        cfg, inp, rq, rk, gq, gk = _both(w)
        assert np.array_equal(gq, rq), "perm_q differs from elsaa_select"
        assert np.array_equal(gk, rk), "perm_k differs from elsaa_select"
        hc = head_cfg_of(cfg)
        for b in range(w.B):
            for h in range(w.H):
                oq, ok = oracle.select(hc, inp["Q"][b, h], inp["K"][b, h], inp["W_sort"][h])
                assert np.array_equal(gq[b, h], oq) and np.array_equal(gk[b, h], ok), f"oracle (b={b}, h={h})"


def test_select_noalloc_rejects_more_tokens_than_the_scratch_holds():
    # 2 * align256(B*H*N) > 32 MiB: rejected on the host, nothing launched
    cfg = E.Config(B=1, H=256, N=65600, d_h=64, k=64, r=64, causal=False)
    q = torch.empty(16, dtype=torch.bfloat16, device="cuda")
    c = cfg.c()
    rc = E.load().elsaa_select_noalloc(E.C.byref(c), E._p(q), E._p(q), E._p(q), E._p(q), E._p(q), None)
    assert rc == -3
    assert "scratch" in E.load().elsaa_last_error().decode()
