"""GPU parity of the operator variants against the oracle: neighbouring
sorted blocks (r >= 1 blocks on each side of a query's own block, the
(2r+1)s-key variant of Sec. 6), token-wise lambda_i with its gradient
(learned and query-dependent lambda), and the m_sparse = 1 ablation (Sec. 7)."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, cfg_of, head_cfg_of, rel_err, run_gpu_fwd_bwd, say
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu


def _w(name, B, H, N, d, k, r, causal, dtype, recipe="iid", seed=70, **kw):
    qs = d ** -0.25 if recipe == "iid" else 1.0
    return W.Workload(name, B, H, N, d, k, r, causal, dtype, recipe=recipe, qk_scale=qs, seed=seed,
                      centres=kw.pop("centres", 16), **kw)


def _check(w, neighbors=0, m_one=False, lam_rows=None, gates=None, lam=1.0, heads=None):
    cfg = cfg_of(w, lam=lam, neighbors=neighbors, m_one=m_one)
    inp = W.make_inputs(w, with_grad=True)
    say(f"[variant] {w.name}: N={w.N} d={w.d} k={w.k} r={w.r} causal={w.causal} {w.dtype} "
        f"neighbors={neighbors} m_one={m_one} lam_rows={lam_rows is not None} gates={gates is not None}")
    fwd, bwd = run_gpu_fwd_bwd(cfg, inp, gates, want_dgates=gates is not None, lam_rows=lam_rows,
                               want_dlambda=True)
    tol = TOL[w.dtype]
    hc = head_cfg_of(cfg)
    errs = {}
    for b in range(w.B):
        for h in range(w.H):
            if heads is not None and (b, h) not in heads:
                continue
            args = (inp["Q"][b, h], inp["K"][b, h], inp["V"][b, h], inp["W_sort"][h], inp["W_race"][h])
            g = None if gates is None else gates[b, h]
            lr = None if lam_rows is None else lam_rows[b, h]
            pq, pk = oracle.select(hc, args[0], args[1], args[3])
            assert np.array_equal(fwd["perm_q"][b, h], pq) and np.array_equal(fwd["perm_k"][b, h], pk)
            ref = oracle.forward(hc, *args, gates=g, lam_rows=lr)
            for name in ("O", "O_s", "m"):
                e = rel_err(fwd[name][b, h], ref[name])
                errs[name] = max(errs.get(name, 0.0), e)
                assert e <= tol, f"{name} (b={b}, h={h}): {e:.3e} > {tol}"
            if m_one:
                assert np.all(fwd["m"][b, h] == 1.0)
            e = float(np.max(np.abs(fwd["lse"][b, h] - ref["lse"])))
            assert e <= tol, f"lse (b={b}, h={h}): {e:.3e}"
            rb = oracle.backward(hc, *args, inp["dO"][b, h], gates=g, lam_rows=lr)
            for name in ("dQ", "dK", "dV", "dgates", "dlambda"):
                if name not in bwd:
                    continue
                if name == "dlambda" and m_one:
                    assert np.all(bwd[name][b, h] == 0.0)
                    continue
                e = rel_err(bwd[name][b, h], rb[name])
                errs[name] = max(errs.get(name, 0.0), e)
                assert e <= tol, f"{name} (b={b}, h={h}): {e:.3e} > {tol}"
    say("   errors:", {k: f"{v:.2e}" for k, v in errs.items()})


NEIGHBOUR_CASES = [
    (_w("nc-f32-n1-512", 1, 1, 512, 64, 32, 32, False, "f32"), 1),
    (_w("nc-bf16-n2-ragged-777", 1, 2, 777, 64, 48, 48, False, "bf16"), 2),
    (_w("nc-bf16-n1-d128-1000", 1, 1, 1000, 128, 128, 128, False, "bf16"), 1),
    (_w("c-f32-n1-512", 1, 1, 512, 64, 32, 32, True, "f32"), 1),
    (_w("c-bf16-n1-d128-1024", 1, 2, 1024, 128, 64, 128, True, "bf16"), 1),
    (_w("c-bf16-n2-clustered-2048", 1, 1, 2048, 64, 128, 64, True, "bf16", recipe="clustered"), 2),
    (_w("c-bf16-n3-saturating-512", 1, 1, 512, 64, 64, 64, True, "bf16"), 3),
]


@pytest.mark.parametrize("w,nbr", NEIGHBOUR_CASES, ids=[c[0].name for c in NEIGHBOUR_CASES])
def test_neighbouring_blocks(w, nbr):
    _check(w, neighbors=nbr)


@pytest.mark.parametrize("causal", [False, True])
def test_token_lambda_with_gradient(causal):
    w = _w(f"{'c' if causal else 'nc'}-bf16-lambda-1024", 1, 2, 1024, 128, 64, 128, causal, "bf16", seed=71)
    _check(w, lam_rows=W.make_lambda_rows(w), gates=W.make_gates(w))


def test_token_lambda_f32():
    w = _w("c-f32-lambda-512", 1, 1, 512, 64, 32, 32, True, "f32", seed=72)
    _check(w, lam_rows=W.make_lambda_rows(w))


def test_scalar_lambda_gradient():
    w = _w("c-bf16-scalar-lambda-1024", 1, 2, 1024, 64, 64, 64, True, "bf16", seed=73)
    _check(w, lam=0.6, gates=W.make_gates(w))


@pytest.mark.parametrize("causal", [False, True])
def test_m_one_ablation(causal):
    w = _w(f"{'c' if causal else 'nc'}-bf16-m1-1024", 1, 2, 1024, 128, 128, 128, causal, "bf16", seed=74)
    _check(w, m_one=True, gates=W.make_gates(w))


def test_all_variants_together():
    w = _w("c-bf16-all-2048", 1, 1, 2048, 128, 128, 128, True, "bf16", recipe="mixed", centres=8, seed=75)
    _check(w, neighbors=1, lam_rows=W.make_lambda_rows(w), gates=W.make_gates(w))


def test_neighbours_at_full_size_sampled_head():
    w = W.CAUSAL_16K
    _check(w, neighbors=1, heads={(0, 3)})
