"""The attention-block step (d_model 1024, 16 heads of 64, N = 32768,
causal, k = r = 128) exactly as the benchmark times it, against the same
chain through the oracle.

GPU chain (paper_2607_20214_amd.block.AttentionBlock, the object the
benchmark steps): QKV = X W_qkv written head-major into one [1, 3H, N, d]
buffer, the operator reading Q, K, V as its head ranges, Y = O W_O,
dO = dY W_O^T, dW_O = O^T dY, the operator backward writing dQ, dK, dV
into the head ranges of one dQKV buffer, dX = dQKV W_qkv^T and
dW_qkv = X^T dQKV.

Oracle chain (Alg. 1 / Alg. 6 with the projections): float64 products
(oracle.gemm) and the float64 operator (oracle.forward / backward), with
the tensors the step stores in bf16 (QKV, O, dO, dQKV) rounded to bf16
(nearest, ties to even) at the same points.

The QKV product of the timed step is compared with the oracle's (every
element within one bf16 step plus 1e-5 max|ref|: float32 and float64
accumulation round to different neighbours only next to a rounding
midpoint, and results near zero carry the float32 sum's absolute error).  Those rare one-step
differences can move a query or key into another hash bucket, so the rest
of the chain is then run again, through the same object and buffers, on the
oracle's QKV: selection bit-exact on all 16 heads; Y and dX on sampled rows
(first and last 64 tokens, 192 random) over all heads; dW_O and dW_qkv
over the columns of two whole heads.  Bar: max|gpu - oracle| / max|oracle|
<= 2e-2 (bf16 storage, float32 accumulation)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20214_amd as E
from gpu_util import cfg_of, elem_stats, say, to_dev
from paper_2607_20214_amd import workloads as W
from paper_2607_20214_amd.block import AttentionBlock

pytestmark = pytest.mark.gpu
TOL = 2e-2
FULL_HEADS = (3, 12)


def bf16_rne(x):
    """float64 -> nearest bfloat16 value (ties to even), as float64."""
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0), e - 8)


class Chain:
    """The GPU step and the oracle chain's inputs, computed once per module."""

    def __init__(self):
        w = W.BLOCK_32K
        self.w = w
        H, N, d, dm = w.H, w.N, w.d, w.d_model
        blk = W.make_block_inputs(w)
        self.X = blk["X"].reshape(N, dm)
        self.dY = blk["dY"].reshape(N, dm)
        self.Wqkv = np.concatenate([blk["W_Q"], blk["W_K"], blk["W_V"]], axis=1)
        self.Wo = blk["W_O"]
        self.ws, self.wr = blk["W_sort"], blk["W_race"]
        self.cfg = cfg_of(w)
        bf = torch.bfloat16
        say(f"[block] GPU step, N={N} d_model={dm} H={H}")
        self.block = AttentionBlock(self.cfg, to_dev(self.X, bf), to_dev(self.dY, bf), to_dev(self.Wqkv, bf),
                                    to_dev(self.Wo, bf), to_dev(self.ws, torch.float32),
                                    to_dev(self.wr, torch.float32))
        self.block.step()
        torch.cuda.synchronize()
        self.qkv_timed = self.block.qkv[0].float().cpu().numpy()
        # oracle QKV (bf16 storage), head-major [3H, N, d]
        self.qkv_ref = oracle.matrix_to_heads(bf16_rne(oracle.gemm(self.X, self.Wqkv)), 3 * H, N)[0]
        # the rest of the chain on the oracle's QKV, same object and buffers
        say("[block] GPU chain on the oracle's QKV")
        self.block.qkv.copy_(torch.from_numpy(self.qkv_ref[None].astype(np.float32)).to(bf))
        self.block.attend_and_backward()
        torch.cuda.synchronize()
        g = self.block
        self.Y = g.Y.cpu().numpy()
        self.dX = g.dX.cpu().numpy()
        self.dW_O = g.dW_O.cpu().numpy()
        self.dW_qkv = g.dW_qkv.cpu().numpy()
        sv = E.saved_views(self.cfg, g.saved)
        self.perm_q = sv["perm_q"].cpu().numpy()[0]
        self.perm_k = sv["perm_k"].cpu().numpy()[0]
        self.dO_ref = oracle.matrix_to_heads(bf16_rne(oracle.gemm(self.dY, self.Wo, False, True)), H, N)[0]
        rng = np.random.default_rng(90)
        rows = np.zeros(N, np.uint8)
        rows[rng.choice(N, 192, replace=False)] = 1
        rows[:64] = 1
        rows[-64:] = 1
        self.mask = rows
        self.rows = np.nonzero(rows)[0]
        self.hc = oracle.head_cfg(w)

    def head(self, h):
        H = self.w.H
        return self.qkv_ref[h], self.qkv_ref[H + h], self.qkv_ref[2 * H + h]


@pytest.fixture(scope="module")
def chain():
    return Chain()


def _check(name, got, ref):
    st = elem_stats(got, ref)
    say(f"   {name}: " + ", ".join(f"{k} {v:.2e}" for k, v in st.items()))
    assert st["rel"] <= TOL, f"{name}: relative error {st['rel']:.3e} > {TOL}"


@pytest.mark.timeout(600)
def test_block_step_qkv_and_selection(chain):
    """The timed step's QKV product, and the selection of every head on the
    oracle's QKV (bit-exact)."""
    got, ref = chain.qkv_timed, chain.qkv_ref
    diff = np.abs(got - ref)
    # one bf16 step (at most 2^-7 |ref|), plus the float32 accumulation error
    # of a 1024-term sum, which exceeds a step only for the few results near 0
    bound = 2.0 ** -7 * np.abs(ref) + 1e-5 * np.abs(ref).max()
    ratio = float((diff / bound).max())
    say(f"   QKV: {int((diff > 0).sum())} of {diff.size} elements differ from the oracle's; "
        f"worst |d| / (2^-7 |ref| + 1e-5 max|ref|) = {ratio:.3f}")
    assert ratio <= 1.0, "QKV: a difference above one bf16 step"
    for h in range(chain.w.H):
        q, k, _ = chain.head(h)
        pq, pk = oracle.select(chain.hc, q, k, chain.ws[h])
        assert np.array_equal(chain.perm_q[h], pq), f"perm_q head {h}"
        assert np.array_equal(chain.perm_k[h], pk), f"perm_k head {h}"


@pytest.mark.timeout(900)
def test_block_step_forward_chain(chain):
    """Y = O W_O on sampled rows (all heads' O), dW_O = O^T dY on the rows of
    two whole heads."""
    w = chain.w
    H, N, d, dm = w.H, w.N, w.d, w.d_model
    O_rows = np.zeros((len(chain.rows), dm))
    for h in range(H):
        q, k, v = chain.head(h)
        full = h in FULL_HEADS
        say(f"[block fwd] oracle head {h}{' (all rows)' if full else ''}")
        ref = oracle.forward(chain.hc, q, k, v, chain.ws[h], chain.wr[h], row_mask=None if full else chain.mask)
        O = bf16_rne(ref["O"])
        O_rows[:, h * d:(h + 1) * d] = O[chain.rows]
        if full:
            _check(f"dW_O rows of head {h}", chain.dW_O[h * d:(h + 1) * d],
                   oracle.gemm(O, chain.dY, True, False))
    _check("Y sampled rows", chain.Y[chain.rows], oracle.gemm(O_rows, chain.Wo))


@pytest.mark.timeout(1200)
def test_block_step_backward_chain(chain):
    """dX = dQKV W_qkv^T on sampled rows (dQ, dK, dV of all heads),
    dW_qkv = X^T dQKV on the Q, K and V columns of two whole heads."""
    w = chain.w
    H, N, d, dm = w.H, w.N, w.d, w.d_model
    dqkv_rows = np.zeros((len(chain.rows), 3 * dm))
    for h in range(H):
        q, k, v = chain.head(h)
        full = h in FULL_HEADS
        say(f"[block bwd] oracle head {h}{' (all rows)' if full else ''}")
        m = None if full else chain.mask
        ref = oracle.backward(chain.hc, q, k, v, chain.ws[h], chain.wr[h], chain.dO_ref[h], q_mask=m, k_mask=m)
        for j, name in enumerate(("dQ", "dK", "dV")):
            g = bf16_rne(ref[name])
            c0 = j * dm + h * d
            dqkv_rows[:, c0:c0 + d] = g[chain.rows]
            if full:
                _check(f"dW_qkv {name} columns of head {h}", chain.dW_qkv[:, c0:c0 + d],
                       oracle.gemm(chain.X, g, True, False))
    _check("dX sampled rows", chain.dX[chain.rows], oracle.gemm(dqkv_rows, chain.Wqkv, False, True))
