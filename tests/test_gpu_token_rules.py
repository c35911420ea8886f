"""GPU parity of the token-wise rules (gate network and query-dependent
lambda) against the oracle, alone and chained with the operator."""
import numpy as np
import pytest
import torch

import oracle
from oracle import token_rules as TR
from gpu_util import TOL, cfg_of, head_cfg_of, rel_err, say, to_dev
import paper_2607_20214_amd as E
from paper_2607_20214_amd import workloads as W

pytestmark = pytest.mark.gpu

FWD_TOL = 1e-4      # float32 outputs of exactly representable inputs


def _w(name, B, H, N, d, causal, dtype, k=64, r=64, seed=90):
    return W.Workload(name, B, H, N, d, k, r, causal, dtype, recipe="iid", qk_scale=1.0, seed=seed, centres=16)


def _rules_dev(p: dict) -> E.TokenRules:
    return E.TokenRules(**{k: to_dev(v, torch.float32) for k, v in p.items()})


def _oracle_fwd(q, p, h):
    g = TR.gate_forward(q, p["W1"][h], p["b1"][h], p["W2"][h], p["b2"][h]) if "W1" in p else None
    lam = TR.lambda_forward(q, p["lam_w"][h], float(p["lam_b"][h]), float(p["lam_c"][h])) if "lam_w" in p else None
    return g, lam


CASES = [
    (_w("bf16-d128-g64-lam-ragged-777", 2, 2, 777, 128, False, "bf16"), 64, True),
    (_w("bf16-d64-g128-lam-1024", 1, 3, 1024, 64, True, "bf16"), 128, True),
    (_w("bf16-d128-g128-300", 1, 2, 300, 128, False, "bf16"), 128, False),
    (_w("bf16-d64-lam-only-63", 1, 2, 63, 64, False, "bf16"), 0, True),
    (_w("bf16-d128-g64-1", 1, 1, 1, 128, False, "bf16", k=1, r=16), 64, True),
    (_w("f32-d128-g64-lam-512", 1, 2, 512, 128, True, "f32", k=32, r=32), 64, True),
    (_w("f32-d64-g128-lam-ragged-333", 2, 1, 333, 64, False, "f32"), 128, True),
    (_w("f32-d128-g128-lam-200", 1, 1, 200, 128, False, "f32"), 128, True),
]


@pytest.mark.parametrize("w,G,lam", CASES, ids=[c[0].name for c in CASES])
def test_token_rules_forward_and_backward(w, G, lam):
    say(f"[rules] {w.name}: B={w.B} H={w.H} N={w.N} d={w.d} G={G} lambda={lam} {w.dtype}")
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    p = W.make_rule_params(w, G, lam)
    up = W.make_rule_grads(w)
    rules = _rules_dev(p)
    q = to_dev(inp["Q"], cfg.torch_dtype)
    gates, lam_rows = E.token_rules_fwd(cfg, rules, q)
    dq0 = W.bf16_round(np.random.default_rng(3).standard_normal(inp["Q"].shape).astype(np.float32))
    dq = to_dev(dq0, cfg.torch_dtype)
    grads = E.token_rules_bwd(cfg, rules, q, to_dev(up["dgates"], torch.float32),
                              to_dev(up["dlambda"], torch.float32), dq=dq)
    torch.cuda.synchronize()
    tol = TOL[w.dtype]
    H, d = w.H, w.d
    want = {"dW1": np.zeros((H, G, d)), "db1": np.zeros((H, G)), "dW2": np.zeros((H, 2, G)),
            "db2": np.zeros((H, 2)), "dlam_w": np.zeros((H, d)), "dlam_b": np.zeros(H), "dlam_c": np.zeros(H)}
    errs = {}
    for b in range(w.B):
        for h in range(w.H):
            qn = inp["Q"][b, h]
            g_ref, l_ref = _oracle_fwd(qn, p, h)
            if G:
                e = rel_err(gates[b, h].cpu().numpy(), g_ref)
                errs["gates"] = max(errs.get("gates", 0.0), e)
                assert e <= FWD_TOL, f"gates (b={b}, h={h}) {e:.2e}"
                gb = TR.gate_backward(qn, p["W1"][h], p["b1"][h], p["W2"][h], p["b2"][h], up["dgates"][b, h])
                e = rel_err(dq[b, h].float().cpu().numpy(), dq0[b, h] + gb["dq"])
                errs["dq"] = max(errs.get("dq", 0.0), e)
                assert e <= tol, f"dq (b={b}, h={h}) {e:.2e}"
                for k_ in ("dW1", "db1", "dW2", "db2"):
                    want[k_][h] += gb[k_]
            else:
                assert np.array_equal(dq[b, h].float().cpu().numpy(), dq0[b, h])
            if lam:
                e = rel_err(lam_rows[b, h].cpu().numpy(), l_ref)
                errs["lambda"] = max(errs.get("lambda", 0.0), e)
                assert e <= FWD_TOL, f"lambda (b={b}, h={h}) {e:.2e}"
                lb = TR.lambda_backward(qn, p["lam_w"][h], float(p["lam_b"][h]), float(p["lam_c"][h]),
                                        up["dlambda"][b, h])
                want["dlam_w"][h] += lb["dw"]
                want["dlam_b"][h] += lb["db"]
                want["dlam_c"][h] += lb["dc"]
    for k, t in grads.items():
        e = rel_err(t.cpu().numpy(), want[k])
        errs[k] = e
        assert e <= tol, f"{k}: {e:.2e} > {tol}"
    say("   errors:", {k: f"{v:.2e}" for k, v in errs.items()})


def test_token_rules_backward_is_deterministic():
    w = _w("bf16-det", 1, 4, 4096, 128, True, "bf16", seed=91)
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    rules = _rules_dev(W.make_rule_params(w, 64, True))
    up = W.make_rule_grads(w)
    q = to_dev(inp["Q"], cfg.torch_dtype)
    dg, dl = to_dev(up["dgates"], torch.float32), to_dev(up["dlambda"], torch.float32)
    a = E.token_rules_bwd(cfg, rules, q, dg, dl)
    b = E.token_rules_bwd(cfg, rules, q, dg, dl)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k


def test_token_rules_full_size_workload():
    w = W.CAUSAL_16K
    say(f"[rules] {w.name} G=64 lambda")
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=False)
    p = W.make_rule_params(w, 64, True)
    rules = _rules_dev(p)
    q = to_dev(inp["Q"], cfg.torch_dtype)
    gates, lam_rows = E.token_rules_fwd(cfg, rules, q)
    torch.cuda.synchronize()
    for h in (0, 7, 15):
        g_ref, l_ref = _oracle_fwd(inp["Q"][0, h], p, h)
        assert rel_err(gates[0, h].cpu().numpy(), g_ref) <= FWD_TOL
        assert rel_err(lam_rows[0, h].cpu().numpy(), l_ref) <= FWD_TOL


def test_rules_chained_with_the_operator():
    # gates and lambda from the rules feed the operator; the operator's
    # dgates / dlambda feed the rules' backward, whose dq adds to the
    # operator's dQ.  Checked against the same chain through the oracle.
    w = W.Workload("c-bf16-chain-1024", 1, 2, 1024, 128, 64, 128, True, "bf16", recipe="iid",
                   qk_scale=128 ** -0.25, seed=92, centres=16)
    say(f"[rules+operator] {w.name}")
    cfg = cfg_of(w)
    inp = W.make_inputs(w, with_grad=True)
    p = W.make_rule_params(w, 64, True)
    rules = _rules_dev(p)
    dt = cfg.torch_dtype
    q, k, v = (to_dev(inp[n], dt) for n in ("Q", "K", "V"))
    ws, wr = to_dev(inp["W_sort"], torch.float32), to_dev(inp["W_race"], torch.float32)
    do = to_dev(inp["dO"], dt)
    gates, lam_rows = E.token_rules_fwd(cfg, rules, q)
    o, lse, dlr, saved = E.fwd(cfg, q, k, v, ws, wr, gates=gates, lam_rows=lam_rows)
    dq, dk, dv, dg, dl = E.bwd(cfg, q, k, v, wr, do, lse, dlr, saved, gates=gates, want_dgates=True,
                               lam_rows=lam_rows, want_dlambda=True)
    grads = E.token_rules_bwd(cfg, rules, q, dg, dl, dq=dq)
    torch.cuda.synchronize()
    hc = head_cfg_of(cfg)
    tol = TOL["bf16"]
    for h in range(w.H):
        qn = inp["Q"][0, h]
        g_ref, l_ref = _oracle_fwd(qn, p, h)
        args = (qn, inp["K"][0, h], inp["V"][0, h], inp["W_sort"][h], inp["W_race"][h])
        ref = oracle.forward(hc, *args, gates=g_ref, lam_rows=l_ref)
        assert rel_err(o[0, h].float().cpu().numpy(), ref["O"]) <= tol
        rb = oracle.backward(hc, *args, inp["dO"][0, h], gates=g_ref, lam_rows=l_ref)
        gb = TR.gate_backward(qn, p["W1"][h], p["b1"][h], p["W2"][h], p["b2"][h], rb["dgates"])
        lb = TR.lambda_backward(qn, p["lam_w"][h], float(p["lam_b"][h]), float(p["lam_c"][h]), rb["dlambda"])
        checks = {"dQ": (dq[0, h], rb["dQ"] + gb["dq"]), "dK": (dk[0, h], rb["dK"]), "dV": (dv[0, h], rb["dV"]),
                  "dW1": (grads["dW1"][h], gb["dW1"]), "db1": (grads["db1"][h], gb["db1"]),
                  "dW2": (grads["dW2"][h], gb["dW2"]), "db2": (grads["db2"][h], gb["db2"]),
                  "dlam_w": (grads["dlam_w"][h], lb["dw"])}
        errs = {}
        for name, (got, want) in checks.items():
            e = rel_err(got.float().cpu().numpy(), np.asarray(want))
            errs[name] = e
            assert e <= tol, f"{name} (h={h}): {e:.2e}"
        for name, got, want in (("dlam_b", grads["dlam_b"][h], lb["db"]), ("dlam_c", grads["dlam_c"][h], lb["dc"])):
            e = abs(float(got) - want) / max(1.0, abs(want))
            assert e <= tol, f"{name} (h={h}): {e:.2e}"
        say(f"   h={h} errors:", {k_: f"{v_:.2e}" for k_, v_ in errs.items()})
