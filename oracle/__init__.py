"""CPU reference of the ELSAA operator (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
may import this package.  The GPU library never imports it and shares no
code with it.  ``build()`` compiles ``elsaa_oracle.c`` with gcc
(fp64 arithmetic, no floating-point contraction, OpenMP over rows);
the functions below wrap it with ctypes over float32 numpy inputs and
return float64 results.  See ``elsaa_oracle.c`` for which passage of the
paper each part follows.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "elsaa_oracle.c")
_LIB = os.path.join(_HERE, "libelsaa_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle shared library in-tree and return its path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                        "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter", "-Wno-maybe-uninitialized",
                        _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(C.Structure):
    _fields_ = [("N", C.c_int32), ("d", C.c_int32), ("k", C.c_int32), ("r", C.c_int32),
                ("race_bits", C.c_int32), ("sort_bits", C.c_int32), ("n0", C.c_int32),
                ("causal", C.c_int32), ("beta", C.c_double), ("lam", C.c_double),
                ("eps", C.c_double), ("scale", C.c_double), ("neighbors", C.c_int32),
                ("m_one", C.c_int32)]


@dataclass
class HeadCfg:
    """Settings of one head's operator call (names as in the paper)."""
    N: int
    d: int
    k: int                 # sortLSH block size b
    r: int                 # RACE features L * 2^race_bits
    causal: bool
    race_bits: int = 4     # gamma
    sort_bits: int = 5     # gamma_sort
    n0: Optional[int] = None   # causal base length N_0 (None -> 2k)
    beta: float = 1.0
    lam: float = 1.0
    eps: float = 1e-6
    scale: float = 0.0     # <= 0 -> 1/sqrt(d)
    neighbors: int = 0     # r neighbouring sorted blocks on each side
    m_one: bool = False    # Sort_Lsh_RACE ablation: m_sparse = 1

    def c(self) -> _Cfg:
        return _Cfg(self.N, self.d, self.k, self.r, self.race_bits, self.sort_bits,
                    self.n0 if self.n0 is not None else 2 * self.k, int(self.causal),
                    self.beta, self.lam, self.eps, self.scale, self.neighbors, int(self.m_one))

    @property
    def L(self) -> int:
        return self.r >> self.race_bits


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = C.CDLL(_LIB)
        P = C.c_void_p
        lib.ora_hash.argtypes = [C.c_int, C.c_int, P, C.c_int, P, P]
        lib.ora_num_levels.argtypes = [P]
        lib.ora_perm_length.argtypes = [P]
        lib.ora_perm_length.restype = C.c_int64
        lib.ora_select.argtypes = [P, P, P, P, P, P]
        lib.ora_support_size.argtypes = [P, P, P, P]
        lib.ora_support_size.restype = C.c_int64
        lib.ora_support.argtypes = [P, P, P, P, P, P]
        lib.ora_features.argtypes = [C.c_int, C.c_int, P, C.c_int, C.c_int, C.c_double, P, P]
        lib.ora_forward.argtypes = [P] + [P] * 14
        lib.ora_backward.argtypes = [P] + [P] * 15
        lib.ora_threads.argtypes = [C.c_int]
        _lib = lib
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def threads(n: int = 0) -> int:
    """Set the oracle's OpenMP thread count for later calls (n > 0) and
    return the count in effect (timing runs only)."""
    return _load().ora_threads(int(n))


def hash_keys(X, W, bits: int) -> np.ndarray:
    """sortLSH bucket key (Gray rank of the sign code) of every row of X [n, d]."""
    X, W = _f32(X), _f32(W)
    out = np.empty(X.shape[0], np.uint8)
    _check(_load().ora_hash(X.shape[0], X.shape[1], _ptr(X), bits, _ptr(W), _ptr(out)), "hash")
    return out


def num_levels(cfg: HeadCfg) -> int:
    c = cfg.c()
    return _load().ora_num_levels(C.byref(c))


def perm_length(cfg: HeadCfg) -> int:
    """Entries of one head's sorted lists (N; causal: all levels' lists)."""
    c = cfg.c()
    return _load().ora_perm_length(C.byref(c))


def select(cfg: HeadCfg, Q, K, Wsort):
    """Sorted index lists of one head: non-causal [N]; causal [Lv, N/2] when
    no list is padded, else the levels' lists one after another [P] (zero
    tokens of future halves as -1)."""
    Q, K, Wsort = _f32(Q), _f32(K), _f32(Wsort)
    c = cfg.c()
    if cfg.causal:
        lv = num_levels(cfg)
        if lv < 0:
            raise ValueError("a past half would hold a zero token: no sorted-list layout")
        p = perm_length(cfg)
        shape = (lv, cfg.N // 2) if (cfg.N % 2 == 0 and p == lv * (cfg.N // 2)) else (p,)
    else:
        shape = (cfg.N,)
    pq = np.empty(shape, np.int32)
    pk = np.empty(shape, np.int32)
    _check(_load().ora_select(C.byref(c), _ptr(Q), _ptr(K), _ptr(Wsort), _ptr(pq), _ptr(pk)), "select")
    return pq, pk


def support(cfg: HeadCfg, Q, K, Wsort):
    """CSR (rowptr[N+1], cols) of every query's key support S(i)."""
    Q, K, Wsort = _f32(Q), _f32(K), _f32(Wsort)
    c = cfg.c()
    lib = _load()
    total = lib.ora_support_size(C.byref(c), _ptr(Q), _ptr(K), _ptr(Wsort))
    _check(0 if total >= 0 else total, "support_size")
    rp = np.empty(cfg.N + 1, np.int64)
    cols = np.empty(max(total, 1), np.int32)
    _check(lib.ora_support(C.byref(c), _ptr(Q), _ptr(K), _ptr(Wsort), _ptr(rp), _ptr(cols)), "support")
    return rp, cols[:total]


def features(X, Wrace, race_bits: int, beta: float) -> np.ndarray:
    """RACE soft-hash features phi [n, L*2^race_bits] of Alg. 2 (Wrace [L, g, d])."""
    X, Wrace = _f32(X), _f32(Wrace)
    L = Wrace.shape[0]
    out = np.empty((X.shape[0], L << race_bits), np.float64)
    _check(_load().ora_features(X.shape[0], X.shape[1], _ptr(X), L, race_bits, beta, _ptr(Wrace),
                                _ptr(out)), "features")
    return out


def forward(cfg: HeadCfg, Q, K, V, Wsort, Wrace, gates=None, row_mask=None, lam_rows=None) -> dict:
    """Forward of one head; returns O, lse, d_lr, m, O_s, O_lr (float64).
    lam_rows: per-token lambda_i [N] (None: the scalar cfg.lam)."""
    Q, K, V, Wsort, Wrace = map(_f32, (Q, K, V, Wsort, Wrace))
    g = None if gates is None else _f32(gates)
    lr = None if lam_rows is None else _f32(lam_rows)
    msk = None if row_mask is None else np.ascontiguousarray(row_mask, dtype=np.uint8)
    N, d = cfg.N, cfg.d
    out = {"O": np.zeros((N, d)), "lse": np.zeros(N), "d_lr": np.zeros(N), "m": np.zeros(N),
           "O_s": np.zeros((N, d)), "O_lr": np.zeros((N, d))}
    c = cfg.c()
    _check(_load().ora_forward(C.byref(c), _ptr(Q), _ptr(K), _ptr(V), _ptr(Wsort), _ptr(Wrace),
                               _ptr(g), _ptr(lr), _ptr(msk), _ptr(out["O"]), _ptr(out["lse"]), _ptr(out["d_lr"]),
                               _ptr(out["m"]), _ptr(out["O_s"]), _ptr(out["O_lr"])), "forward")
    return out


def backward(cfg: HeadCfg, Q, K, V, Wsort, Wrace, dO, gates=None, q_mask=None, k_mask=None,
             lam_rows=None) -> dict:
    """Backward of one head; returns dQ, dK, dV, dgates [N,2] and dlambda [N]
    (d/dlambda_i) in float64."""
    Q, K, V, Wsort, Wrace, dO = map(_f32, (Q, K, V, Wsort, Wrace, dO))
    g = None if gates is None else _f32(gates)
    lr = None if lam_rows is None else _f32(lam_rows)
    qm = None if q_mask is None else np.ascontiguousarray(q_mask, dtype=np.uint8)
    km = None if k_mask is None else np.ascontiguousarray(k_mask, dtype=np.uint8)
    N, d = cfg.N, cfg.d
    out = {"dQ": np.zeros((N, d)), "dK": np.zeros((N, d)), "dV": np.zeros((N, d)),
           "dgates": np.zeros((N, 2)), "dlambda": np.zeros(N)}
    c = cfg.c()
    _check(_load().ora_backward(C.byref(c), _ptr(Q), _ptr(K), _ptr(V), _ptr(Wsort), _ptr(Wrace),
                                _ptr(g), _ptr(lr), _ptr(dO), _ptr(qm), _ptr(km), _ptr(out["dQ"]),
                                _ptr(out["dK"]), _ptr(out["dV"]), _ptr(out["dgates"]),
                                _ptr(out["dlambda"])), "backward")
    return out


def head_cfg(w, **over) -> HeadCfg:
    """HeadCfg of a workload description (any object with the workload fields)."""
    kw = dict(N=w.N, d=w.d, k=w.k, r=w.r, causal=bool(w.causal), race_bits=w.race_bits,
              sort_bits=w.sort_bits, n0=getattr(w, "base_len", None))
    kw.update(over)
    return HeadCfg(**kw)


from .projections import gemm, heads_to_matrix, matrix_to_heads  # noqa: E402,F401
