"""GPU parity of the backward (dQ, dK, dV, gate gradients) against the oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, cfg_of, elem_stats, head_cfg_of, run_gpu_fwd_bwd, say
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, r, causal, dtype, recipe="iid", seed=60, **kw):
    qs = d ** -0.25 if recipe == "iid" else 1.0
    return W.Workload(name, B, H, N, d, k, r, causal, dtype, recipe=recipe, qk_scale=qs, seed=seed,
                      centres=kw.pop("centres", 16), **kw)


SMALL = [
    _w("nc-f32-512", 1, 1, 512, 64, 32, 32, False, "f32"),
    _w("nc-bf16-ragged-300", 1, 2, 300, 64, 64, 64, False, "bf16", recipe="clustered"),
    _w("nc-bf16-d128-k48-777", 1, 1, 777, 128, 48, 128, False, "bf16"),
    _w("nc-bf16-d64-k128-1000", 1, 2, 1000, 64, 128, 64, False, "bf16"),
    _w("nc-bf16-d128-k128-1000", 1, 1, 1000, 128, 128, 128, False, "bf16"),
    _w("nc-f32-d128-k64-700", 1, 1, 700, 128, 64, 64, False, "f32"),
    _w("c-bf16-d128-1024", 1, 2, 1024, 128, 64, 128, True, "bf16"),
    _w("c-bf16-d64-2048-clustered", 1, 2, 2048, 64, 128, 64, True, "bf16", recipe="clustered"),
    _w("c-f32-d64-512", 1, 1, 512, 64, 32, 32, True, "f32"),
    _w("c-f32-d128-512", 1, 1, 512, 128, 32, 64, True, "f32"),
    _w("c-bf16-leaf-only-256", 2, 1, 256, 64, 128, 48, True, "bf16"),
    _w("c-bf16-r256-1024", 1, 1, 1024, 128, 128, 256, True, "bf16", recipe="mixed", centres=8),
    # degenerate lengths: one token, two, three; 65 = one padded level
    _w("nc-f32-n1", 1, 1, 1, 64, 32, 32, False, "f32"),
    # (one causal token in fp32: both branches reproduce V_0, so dK is only
    # the residue of exact cancellations, below the bf16 operand rounding of
    # the low-rank kernel matrix; the forward runs it in bf16)
    _w("c-f32-n1-d128", 1, 2, 1, 128, 64, 64, True, "f32"),
    _w("c-bf16-n2-d64", 2, 1, 2, 64, 64, 64, True, "bf16"),
    _w("nc-bf16-n3-d128", 1, 1, 3, 128, 128, 128, False, "bf16"),
    _w("c-bf16-n65-k32-padded", 1, 2, 65, 64, 32, 64, True, "bf16"),
    # 256 features: the state, dQ and dK passes split the tables over two
    # workgroups; r = 192 leaves the second one 4 live tables of 8
    _w("nc-bf16-d64-r256-700", 1, 2, 700, 64, 64, 256, False, "bf16"),
    _w("c-bf16-d64-r256-ragged-900", 1, 1, 900, 64, 128, 256, True, "bf16"),
    _w("c-bf16-d128-r192-ragged-1300", 1, 1, 1300, 128, 128, 192, True, "bf16", recipe="clustered"),
    _w("c-bf16-n0-3x-768", 1, 1, 768, 64, 128, 64, True, "bf16"),
    # Alg. 5's zero-token padding of odd lists
    _w("c-bf16-d64-padded-1001", 1, 2, 1001, 64, 64, 64, True, "bf16"),
    _w("c-bf16-d128-padded-777-k32", 1, 1, 777, 128, 32, 64, True, "bf16", recipe="clustered"),
    _w("c-f32-d64-padded-300-k32", 1, 1, 300, 64, 32, 32, True, "f32"),
    # b = 256 levels as two 128-key halves (two dQ partials per level): whole
    # groups of 8 blocks, d_h 64, and the tail of the item order (10 blocks)
    _w("c-bf16-d128-k256-4096", 1, 2, 4096, 128, 256, 128, True, "bf16"),
    _w("c-bf16-d64-k256-2048-clustered", 1, 2, 2048, 64, 256, 64, True, "bf16", recipe="clustered"),
    _w("c-bf16-d128-k256-1024-h5", 1, 5, 1024, 128, 256, 64, True, "bf16"),
    # level halves of 1500, 750 and 375 entries: every list ends in a short
    # block (375: 119 entries, so its second key half holds no key)
    _w("c-bf16-d128-k256-3000-short", 1, 2, 3000, 128, 256, 64, True, "bf16"),
    _w("c-bf16-d64-k256-1500-short", 1, 2, 1500, 64, 256, 64, True, "bf16", recipe="clustered"),
]


def _check(w, gates=None, lam=1.0, heads=None, q_mask=None, k_mask=None, want_dgates=False):
    cfg = cfg_of(w, lam=lam)
    inp = W.make_inputs(w, with_grad=True)
    say(f"[bwd] {w.name}: B={w.B} H={w.H} N={w.N} d={w.d} k={w.k} r={w.r} causal={w.causal} {w.dtype}")
    _, got = run_gpu_fwd_bwd(cfg, inp, gates, want_dgates=want_dgates)
    tol = TOL[w.dtype]
    hc = head_cfg_of(cfg)
    errs = {}
    for b in range(w.B):
        for h in range(w.H):
            if heads is not None and (b, h) not in heads:
                continue
            ref = oracle.backward(hc, inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h],
                                  inp["W_race"][h], inp["dO"][b, h],
                                  gates=None if gates is None else gates[b, h], q_mask=q_mask,
                                  k_mask=k_mask)
            for name, msk in (("dQ", q_mask), ("dK", k_mask), ("dV", k_mask), ("dgates", None)):
                if name not in got:
                    continue
                rows = slice(None) if msk is None else (msk > 0)
                st = elem_stats(got[name][b, h][rows], ref[name][rows])
                for key, v in st.items():
                    errs[f"{name}.{key}"] = max(errs.get(f"{name}.{key}", 0.0), v)
                assert st["rel"] <= tol, f"{name} (b={b}, h={h}): {st['rel']:.3e} > {tol}"
    say("   errors:", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_backward_small(w):
    _check(w)


def test_backward_gates_lambda_and_gate_gradients():
    w = _w("c-bf16-gates", 1, 2, 1024, 64, 64, 64, True, "bf16", seed=61)
    _check(w, gates=W.make_gates(w), lam=0.37, want_dgates=True)
    w2 = _w("nc-f32-gates", 1, 1, 512, 64, 32, 32, False, "f32", seed=62)
    _check(w2, gates=W.make_gates(w2), lam=0.0, want_dgates=True)


def test_backward_clustered_4k_workload():
    """All 16 heads (B = 2, H = 8) of the clustered 4K workload."""
    _check(W.CLUSTERED_4K)


@pytest.mark.timeout(900)
def test_backward_causal_16k_workload_all_heads():
    """All 16 heads of the 16K causal workload (the measured one), every row."""
    _check(W.CAUSAL_16K)


@pytest.mark.timeout(900)
def test_backward_causal_64k_mixed_workload_sampled_rows():
    """All 8 heads of the 64K mixed workload (heads 0-3 peaked, 4-7
    diffuse) on 264 sampled query rows and 264 sampled key rows each."""
    w = W.CAUSAL_64K_MIXED
    rng = np.random.default_rng(6)
    qm = np.zeros(w.N, np.uint8)
    km = np.zeros(w.N, np.uint8)
    qm[rng.choice(w.N, 200, replace=False)] = 1
    km[rng.choice(w.N, 200, replace=False)] = 1
    qm[-64:] = 1
    km[:64] = 1
    _check(w, q_mask=qm, k_mask=km)


@pytest.mark.timeout(900)
def test_backward_block_32k_attention_sampled_rows():
    """Backward of the 32768-token, d_model 1024 block's attention (16 heads
    of 64, seven levels) at full size, on sampled rows of every head."""
    w = W.BLOCK_32K
    rng = np.random.default_rng(8)
    qm = np.zeros(w.N, np.uint8)
    km = np.zeros(w.N, np.uint8)
    qm[rng.choice(w.N, 200, replace=False)] = 1
    km[rng.choice(w.N, 200, replace=False)] = 1
    qm[-64:] = 1
    km[:64] = 1
    _check(w, q_mask=qm, k_mask=km)


@pytest.mark.timeout(300)
def test_backward_padded_16386():
    """N = 16386 with n0 = 256 (seven levels, zero tokens from the second
    level on) and with n0 = 4096 (three levels, leaves of 2049 entries), every
    row of two heads."""
    for n0, k in ((None, 128), (4096, 256)):
        w = _w(f"c-bf16-padded-16386-n0-{n0}", 1, 2, 16386, 128, k, 128, True, "bf16", seed=64, n0=n0)
        _check(w)


@pytest.mark.parametrize("k", [128, 256], ids=["k128", "k256-halves"])
def test_backward_is_deterministic(k):
    """Two runs give the same bits (b = 256: the two key halves of each
    block in turn, the first half's dQ kept in LDS)."""
    w = _w(f"c-bf16-det-k{k}", 1, 2, 2048, 128, k, 128, True, "bf16", seed=63)
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=True)
    say(f"[bwd-det] {w.name}")
    _, a = run_gpu_fwd_bwd(cfg, inp)
    _, b = run_gpu_fwd_bwd(cfg, inp)
    for name in a:
        assert np.array_equal(a[name], b[name]), name
