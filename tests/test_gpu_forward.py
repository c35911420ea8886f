"""GPU parity of the forward (selection, both branches, fusion) against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, cfg_of, elem_stats, head_cfg_of, run_gpu_fwd, say
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, r, causal, dtype, recipe="iid", seed=50, **kw):
    qs = d ** -0.25 if recipe == "iid" else 1.0
    return W.Workload(name, B, H, N, d, k, r, causal, dtype, recipe=recipe, qk_scale=qs, seed=seed,
                      centres=kw.pop("centres", 16), **kw)


SMALL = [
    _w("nc-f32-512", 1, 1, 512, 64, 32, 32, False, "f32"),
    _w("nc-bf16-ragged-300", 1, 2, 300, 64, 64, 64, False, "bf16", recipe="clustered"),
    _w("nc-bf16-d128-1000", 2, 1, 1000, 128, 128, 128, False, "bf16"),
    _w("nc-bf16-k48-ragged-777", 1, 2, 777, 64, 48, 48, False, "bf16"),
    _w("nc-bf16-dense-k256-200", 1, 1, 200, 128, 256, 16, False, "bf16"),
    _w("c-bf16-d128-1024", 1, 2, 1024, 128, 64, 128, True, "bf16"),
    _w("c-bf16-d64-2048-clustered", 1, 2, 2048, 64, 128, 64, True, "bf16", recipe="clustered"),
    _w("c-f32-d64-512", 1, 1, 512, 64, 32, 32, True, "f32"),
    _w("c-f32-d128-512", 1, 1, 512, 128, 32, 64, True, "f32"),
    _w("c-bf16-leaf-only-256", 2, 1, 256, 64, 128, 48, True, "bf16"),
    _w("c-bf16-r256-1024", 1, 1, 1024, 128, 128, 256, True, "bf16", recipe="mixed", centres=8),
    # degenerate lengths: one token, two, three; 65 = one padded level
    _w("nc-f32-n1", 1, 1, 1, 64, 32, 32, False, "f32"),
    _w("c-bf16-n1-d128", 1, 2, 1, 128, 64, 128, True, "bf16"),
    _w("c-bf16-n2-d64", 2, 1, 2, 64, 64, 64, True, "bf16"),
    _w("nc-bf16-n3-d128", 1, 1, 3, 128, 128, 128, False, "bf16"),
    _w("c-bf16-n65-k32-padded", 1, 2, 65, 64, 32, 64, True, "bf16"),
    # 256 features: the state, dQ and dK passes split the tables over two
    # workgroups; r = 192 leaves the second one 4 live tables of 8
    _w("nc-bf16-d64-r256-700", 1, 2, 700, 64, 64, 256, False, "bf16"),
    _w("c-bf16-d64-r256-ragged-900", 1, 1, 900, 64, 128, 256, True, "bf16"),
    _w("c-bf16-d128-r192-ragged-1300", 1, 1, 1300, 128, 128, 192, True, "bf16", recipe="clustered"),
    _w("c-bf16-n0-3x-768", 1, 1, 768, 64, 128, 64, True, "bf16"),
    # Alg. 5's zero-token padding of odd lists: 1001 -> 501 -> 251 -> 126
    _w("c-bf16-d64-padded-1001", 1, 2, 1001, 64, 64, 64, True, "bf16"),
    _w("c-bf16-d128-padded-777-k32", 1, 1, 777, 128, 32, 64, True, "bf16", recipe="clustered"),
    _w("c-f32-d64-padded-300-k32", 1, 1, 300, 64, 32, 32, True, "f32"),
]


def _check_case(w, gates=None, lam=1.0, heads=None, row_mask=None):
    cfg = cfg_of(w, lam=lam)
    inp = W.make_inputs(w, with_grad=False)
    say(f"[fwd] {w.name}: B={w.B} H={w.H} N={w.N} d={w.d} k={w.k} r={w.r} causal={w.causal} {w.dtype}")
    got, _ = run_gpu_fwd(cfg, inp, gates)
    tol = TOL[w.dtype]
    hc = head_cfg_of(cfg)
    errs = {}
    for b in range(w.B):
        for h in range(w.H):
            if heads is not None and (b, h) not in heads:
                continue
            args = (inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h], inp["W_race"][h])
            pq, pk = oracle.select(hc, *args[:2], args[3])
            assert np.array_equal(got["perm_q"][b, h], pq), f"perm_q (b={b}, h={h})"
            assert np.array_equal(got["perm_k"][b, h], pk), f"perm_k (b={b}, h={h})"
            ref = oracle.forward(hc, *args, gates=None if gates is None else gates[b, h],
                                 row_mask=row_mask)
            rows = slice(None) if row_mask is None else (row_mask > 0)
            for name in ("O", "O_s", "O_lr", "d_lr", "m"):
                r_ = rows if name not in ("O_lr", "d_lr") else slice(None)
                st = elem_stats(got[name][b, h][r_], ref[name][r_])
                for key, v in st.items():
                    errs[f"{name}.{key}"] = max(errs.get(f"{name}.{key}", 0.0), v)
                assert st["rel"] <= tol, f"{name} (b={b}, h={h}): {st['rel']:.3e} > {tol}"
            e = float(np.max(np.abs(got["lse"][b, h][rows] - ref["lse"][rows])))
            errs["lse(abs)"] = max(errs.get("lse(abs)", 0.0), e)
            assert e <= tol, f"lse (b={b}, h={h}): {e:.3e}"
    say("   errors:", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_forward_small(w):
    _check_case(w)


def test_forward_gates_and_lambda():
    w = _w("c-bf16-gates", 1, 2, 1024, 64, 64, 64, True, "bf16", seed=51)
    _check_case(w, gates=W.make_gates(w), lam=0.37)
    w2 = _w("nc-f32-gates", 1, 1, 512, 64, 32, 32, False, "f32", seed=52)
    _check_case(w2, gates=W.make_gates(w2), lam=0.0)


def test_forward_tiny_fp32_workload():
    _check_case(W.TINY_FP32)


def test_forward_clustered_4k_workload():
    """All 16 heads (B = 2, H = 8) of the clustered 4K workload."""
    _check_case(W.CLUSTERED_4K)


@pytest.mark.timeout(600)
def test_forward_causal_16k_workload_all_heads():
    """All 16 heads of the 16K causal workload (the measured one), every row."""
    _check_case(W.CAUSAL_16K)


@pytest.mark.timeout(600)
def test_forward_causal_64k_mixed_workload_sampled_rows():
    """All 8 heads of the 64K mixed workload (heads 0-3 peaked, 4-7
    diffuse) on 428 sampled rows each."""
    w = W.CAUSAL_64K_MIXED
    mask = np.zeros(w.N, np.uint8)
    rng = np.random.default_rng(5)
    mask[rng.choice(w.N, 300, replace=False)] = 1
    mask[:64] = 1
    mask[-64:] = 1
    _check_case(w, row_mask=mask)


@pytest.mark.timeout(600)
def test_forward_block_32k_attention_sampled_rows():
    """The attention of the 32768-token, d_model 1024 block (16 heads of 64,
    seven levels) at full size, on sampled rows of every head."""
    w = W.BLOCK_32K
    mask = np.zeros(w.N, np.uint8)
    rng = np.random.default_rng(7)
    mask[rng.choice(w.N, 300, replace=False)] = 1
    mask[:64] = 1
    mask[-64:] = 1
    _check_case(w, row_mask=mask)


def test_forward_padded_16386_sampled_rows():
    """N = 16386 (odd lists from the second level on: seven levels, up to six
    zero tokens per list) and the same N with n0 = 4096 (three levels, leaves
    of 2049 entries), every row of two heads."""
    for n0, k in ((None, 128), (4096, 256)):
        w = _w(f"c-bf16-padded-16386-n0-{n0}", 1, 2, 16386, 128, k, 128, True, "bf16", seed=54, n0=n0)
        _check_case(w)


def test_forward_is_deterministic():
    w = _w("c-bf16-det", 1, 2, 2048, 128, 128, 128, True, "bf16", seed=53)
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    say(f"[fwd-det] {w.name}")
    a, _ = run_gpu_fwd(cfg, inp)
    b, _ = run_gpu_fwd(cfg, inp)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
