"""GPU parity of the causal recursion when segment and leaf lengths are not
multiples of the 64-row tile, and of the paper's causal text setting
(block size 256, base length 4096), against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, cfg_of, head_cfg_of, rel_err, run_gpu_fwd_bwd, say
import paper_2607_20214_amd as E
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, r, dtype, n0, recipe="iid", seed=80):
    qs = d ** -0.25 if recipe == "iid" else 1.0
    return W.Workload(name, B, H, N, d, k, r, True, dtype, recipe=recipe, qk_scale=qs, seed=seed,
                      centres=16, n0=n0)


CASES = [
    # levels of 1000 / 500 / 250 sorted queries, leaves of 250 tokens
    _w("c-bf16-d128-2000-leaf250", 1, 2, 2000, 128, 64, 128, "bf16", 300),
    # odd leaves of 125 tokens
    _w("c-f32-d64-1000-leaf125", 1, 1, 1000, 64, 32, 32, "f32", 130),
    _w("c-bf16-d64-1000-leaf125-clustered", 1, 2, 1000, 64, 64, 64, "bf16", 130, recipe="clustered"),
    # leaf shorter than one tile
    _w("c-bf16-d128-800-leaf50", 2, 1, 800, 128, 32, 64, "bf16", 60),
    # the text setting's block and base length, scaled: levels 4000 / 2000 / 1000, leaves 1000
    _w("c-bf16-text-8000-b256-leaf1000", 1, 1, 8000, 128, 256, 64, "bf16", 1000),
    # leaves of 9 tiles (odd: the last workgroup of a long leaf holds one query tile), d_h 64
    _w("c-bf16-d64-2080-leaf520", 1, 2, 2080, 64, 64, 64, "bf16", 520),
    # the text setting's own leaf of 4096 tokens
    _w("c-bf16-text-8192-b256-n04096", 1, 1, 8192, 128, 256, 64, "bf16", 4096),
]


def _check(w, neighbors=0, heads=None, q_mask=None):
    cfg = cfg_of(w, neighbors=neighbors)
    Lv = E.num_levels(cfg)
    say(f"[ragged] {w.name}: N={w.N} k={w.k} n0={w.n0} levels={Lv} leaf={w.N >> Lv} {w.dtype} nbr={neighbors}")
    inp = W.make_inputs(w, with_grad=True)
    fwd, bwd = run_gpu_fwd_bwd(cfg, inp)
    tol = TOL[w.dtype]
    hc = head_cfg_of(cfg)
    errs = {}
    for b in range(w.B):
        for h in range(w.H):
            if heads is not None and (b, h) not in heads:
                continue
            args = (inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h], inp["W_race"][h])
            pq, pk = oracle.select(hc, args[0], args[1], args[3])
            assert np.array_equal(fwd["perm_q"][b, h], pq) and np.array_equal(fwd["perm_k"][b, h], pk)
            ref = oracle.forward(hc, *args, row_mask=q_mask)
            rows = slice(None) if q_mask is None else (q_mask > 0)
            for name in ("O", "O_s", "m"):
                e = rel_err(fwd[name][b, h][rows], ref[name][rows])
                errs[name] = max(errs.get(name, 0.0), e)
                assert e <= tol, f"{name} (b={b}, h={h}): {e:.3e}"
            rb = oracle.backward(hc, *args, inp["dO"][b, h], q_mask=q_mask, k_mask=q_mask)
            for name in ("dQ", "dK", "dV"):
                e = rel_err(bwd[name][b, h][rows], rb[name][rows])
                errs[name] = max(errs.get(name, 0.0), e)
                assert e <= tol, f"{name} (b={b}, h={h}): {e:.3e}"
    say("   errors:", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_ragged_causal(w):
    _check(w)


def test_ragged_causal_with_neighbours():
    _check(_w("c-bf16-d128-2000-leaf250-nbr1", 1, 1, 2000, 128, 64, 128, "bf16", 300, seed=81), neighbors=1)


@pytest.mark.timeout(900)
def test_text_setting_full_size_sampled_rows():
    """All 16 heads of the text setting at N = 32000 on 368 sampled rows each."""
    # N = 32000 (the ArXiv length): the oracle computes sampled rows only
    w = W.TEXT_32K
    mask = np.zeros(w.N, np.uint8)
    rng = np.random.default_rng(8)
    mask[rng.choice(w.N, 200, replace=False)] = 1
    mask[:64] = 1
    mask[-64:] = 1
    mask[3990:4010] = 1        # across the first leaf boundary
    mask[15990:16010] = 1      # across the top-level halves
    _check(w, q_mask=mask)
