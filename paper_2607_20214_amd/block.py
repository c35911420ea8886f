"""One attention-block training step around the ELSAA operator.

Alg. 1 and Alg. 6 project the block input with dense matrices before the
operator (Q = X W_Q, K = X W_K, V = X W_V) and project the operator's
output after it (O_head W_O).  This module wires those products
(``elsaa_gemm`` on the matrix cores) to the operator (``elsaa_fwd`` /
``elsaa_bwd``) with every attention tensor in the operator's head-major
[B, H, N, d_h] layout, so no reshape copy runs between them:

    forward   QKV = X W_qkv        -> one [1, 3H, N, d_h] buffer (Q, K, V are
                                      its contiguous head ranges)
              O   = ELSAA(Q, K, V)
              Y   = O W_O
    backward  dO  = dY W_O^T       (head-major)
              dW_O = O^T dY
              dQ, dK, dV = ELSAA backward, written into one [1, 3H, N, d_h]
                                      buffer dQKV
              dX   = dQKV W_qkv^T
              dW_qkv = X^T dQKV

Every buffer is allocated once, in the constructor; ``step()`` only
enqueues library calls on torch's current stream.  Like the rest of the
package it only marshals arguments.
"""
from __future__ import annotations

import torch

from . import Buffers, Config, bwd, fwd, gemm, gemm_plan, gemm_workspace_bytes


class AttentionBlock:
    """Buffers and launch sequence of one block step (B = 1).

    X, dY: [N, d_model] bf16; W_qkv: [d_model, 3 d_model] bf16 (columns
    W_Q | W_K | W_V, head h of each in columns h d_h .. (h+1) d_h - 1);
    W_O: [d_model, d_model] bf16; w_sort, w_race: the operator's hash
    projections (float32, per head).
    """

    def __init__(self, cfg: Config, X, dY, W_qkv, W_O, w_sort, w_race):
        if cfg.B != 1:
            raise ValueError("the block step keeps Q, K, V as heads of one [1, 3H, N, d_h] buffer (B = 1)")
        if cfg.dtype != "bf16":
            raise ValueError("the block step runs with bf16 storage")
        dev = X.device
        H, N, d = cfg.H, cfg.N, cfg.d_h
        dm = H * d
        for name, t, shp in (("X", X, (N, dm)), ("dY", dY, (N, dm)), ("W_qkv", W_qkv, (dm, 3 * dm)),
                             ("W_O", W_O, (dm, dm))):
            if t.shape != torch.Size(shp) or t.dtype != torch.bfloat16 or not t.is_contiguous():
                raise ValueError(f"{name}: expected contiguous bf16 {shp}, got {t.dtype} {tuple(t.shape)}")
        self.cfg = cfg
        self.X, self.dY, self.W_qkv, self.W_O = X, dY, W_qkv, W_O
        self.w_sort, self.w_race = w_sort, w_race
        bf, f32 = torch.bfloat16, torch.float32
        self.qkv = torch.empty(1, 3 * H, N, d, dtype=bf, device=dev)
        self.dqkv = torch.empty_like(self.qkv)
        self.do = torch.empty(1, H, N, d, dtype=bf, device=dev)
        self.q, self.k, self.v = self.qkv[:, :H], self.qkv[:, H:2 * H], self.qkv[:, 2 * H:]
        self.bufs = Buffers(cfg, dev, backward=True)
        self.bufs.dq, self.bufs.dk, self.bufs.dv = self.dqkv[:, :H], self.dqkv[:, H:2 * H], self.dqkv[:, 2 * H:]
        self.Y = torch.empty(N, dm, dtype=f32, device=dev)
        self.dW_O = torch.empty(dm, dm, dtype=f32, device=dev)
        self.dX = torch.empty(N, dm, dtype=f32, device=dev)
        self.dW_qkv = torch.empty(dm, 3 * dm, dtype=f32, device=dev)
        o = self.bufs.o
        plans = [gemm_plan(X, W_qkv, out=self.qkv), gemm_plan(o, W_O, out=self.Y),
                 gemm_plan(dY, W_O, trans_b=True, out=self.do), gemm_plan(o, dY, trans_a=True, out=self.dW_O),
                 gemm_plan(self.dqkv, W_qkv, trans_b=True, out=self.dX),
                 gemm_plan(X, self.dqkv, trans_a=True, out=self.dW_qkv)]
        ws = max(gemm_workspace_bytes(p) for p in plans)
        self.gws = torch.empty(max(ws, 256), dtype=torch.uint8, device=dev)
        self.lse = self.d_lr = self.saved = None

    def project(self):
        """QKV = X W_qkv, written head-major into the operator's input buffer."""
        gemm(self.X, self.W_qkv, out=self.qkv, workspace=self.gws)

    def attend_and_backward(self):
        """Everything of the step after the QKV product: the operator forward,
        Y, dO, dW_O, the operator backward into dQKV, dX and dW_qkv."""
        cfg, b = self.cfg, self.bufs
        o, self.lse, self.d_lr, self.saved = fwd(cfg, self.q, self.k, self.v, self.w_sort, self.w_race, buffers=b)
        gemm(o, self.W_O, out=self.Y, workspace=self.gws)
        gemm(self.dY, self.W_O, trans_b=True, out=self.do, workspace=self.gws)
        gemm(o, self.dY, trans_a=True, out=self.dW_O, workspace=self.gws)
        bwd(cfg, self.q, self.k, self.v, self.w_race, self.do, self.lse, self.d_lr, self.saved, buffers=b)
        gemm(self.dqkv, self.W_qkv, trans_b=True, out=self.dX, workspace=self.gws)
        gemm(self.X, self.dqkv, trans_a=True, out=self.dW_qkv, workspace=self.gws)

    def step(self):
        """One training step of the block (forward and backward)."""
        self.project()
        self.attend_and_backward()
