"""ELSAA attention operator on AMD Instinct MI355X (gfx950).

Thin Python binding of the C-ABI library ``libelsaa.so`` (declared in
``include/elsaa.h``).  The functions below only marshal arguments: they
allocate the output, ``saved`` and ``workspace`` buffers with torch on the
tensors' device, pass raw device pointers and torch's current HIP stream,
and raise if the library reports an error.  Every step of the operator runs
in the library's HIP kernels; there is no other code path.  If the library
has not been built, importing works but every call raises.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libelsaa.so")
_lib = None

F32, BF16 = 0, 1
_STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported", -3: "buffer too small", -4: "HIP error"}


class ElsaaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"elsaa error {status} ({_STATUS.get(status, '?')}): {msg}")
        self.status = status


class _Config(C.Structure):
    _fields_ = [("B", C.c_int32), ("H", C.c_int32), ("N", C.c_int32), ("d_h", C.c_int32),
                ("k", C.c_int32), ("r", C.c_int32), ("race_bits", C.c_int32),
                ("sort_bits", C.c_int32), ("n0", C.c_int32), ("causal", C.c_int32),
                ("dtype", C.c_int32), ("beta", C.c_float), ("lam", C.c_float),
                ("eps", C.c_float), ("scale", C.c_float), ("neighbors", C.c_int32),
                ("m_one", C.c_int32)]


class _SavedLayout(C.Structure):
    _fields_ = [("perm_q", C.c_size_t), ("perm_k", C.c_size_t), ("m", C.c_size_t),
                ("o_sparse", C.c_size_t), ("o_lowrank", C.c_size_t), ("u_q", C.c_size_t),
                ("u_k", C.c_size_t), ("race_states", C.c_size_t), ("total", C.c_size_t)]


class _TokenRules(C.Structure):
    _fields_ = [("gate_hidden", C.c_int32), ("W1", C.c_void_p), ("b1", C.c_void_p), ("W2", C.c_void_p),
                ("b2", C.c_void_p), ("lambda_rule", C.c_int32), ("lam_w", C.c_void_p),
                ("lam_b", C.c_void_p), ("lam_c", C.c_void_p), ("lambda_min", C.c_float)]


class _GemmDesc(C.Structure):
    _fields_ = [("M", C.c_int32), ("N", C.c_int32), ("K", C.c_int32), ("trans_a", C.c_int32),
                ("trans_b", C.c_int32), ("lda", C.c_int64), ("ldb", C.c_int64), ("ldc", C.c_int64),
                ("a_heads", C.c_int32), ("b_heads", C.c_int32), ("c_heads", C.c_int32),
                ("seq", C.c_int32), ("c_dtype", C.c_int32)]


@dataclasses.dataclass
class Config:
    """Operator settings (names follow the paper; see include/elsaa.h)."""
    B: int
    H: int
    N: int
    d_h: int
    k: int                  # sortLSH block size b
    r: int                  # RACE features L * 2^race_bits
    causal: bool
    dtype: str = "bf16"     # storage dtype of Q, K, V, O, dO, dQ, dK, dV
    race_bits: int = 4
    sort_bits: int = 5
    n0: int = 0             # <= 0 -> 2k
    beta: float = 1.0
    lam: float = 1.0
    eps: float = 1e-6
    scale: float = 0.0      # <= 0 -> 1/sqrt(d_h)
    neighbors: int = 0      # neighbouring sorted blocks seen on each side
    m_one: bool = False     # m_sparse = 1 (the Sort_Lsh_RACE ablation)

    def c(self) -> _Config:
        return _Config(self.B, self.H, self.N, self.d_h, self.k, self.r, self.race_bits,
                       self.sort_bits, self.n0, int(self.causal),
                       BF16 if self.dtype == "bf16" else F32, self.beta, self.lam, self.eps,
                       self.scale, self.neighbors, int(self.m_one))

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32


def load():
    """Load libelsaa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ElsaaError(-4, f"{LIB_PATH} not built; run paper_2607_20214_amd/build.py")
        lib = C.CDLL(LIB_PATH)
        P, S = C.c_void_p, C.c_size_t
        lib.elsaa_num_levels.argtypes = [P]
        lib.elsaa_perm_length.argtypes = [P]
        lib.elsaa_perm_length.restype = C.c_int64
        lib.elsaa_saved_bytes.argtypes = [P, C.POINTER(C.c_size_t)]
        lib.elsaa_workspace_bytes.argtypes = [P, C.c_int, C.POINTER(C.c_size_t)]
        lib.elsaa_get_saved_layout.argtypes = [P, P]
        lib.elsaa_select.argtypes = [P, P, P, P, P, P, P, S, P]
        lib.elsaa_select_noalloc.argtypes = [P, P, P, P, P, P, P]
        lib.elsaa_fwd.argtypes = [P, P, P, P, P, P, P, P, P, P, P, P, S, P, S, P]
        lib.elsaa_bwd.argtypes = [P, P, P, P, P, P, P, P, P, P, P, P, S, P, P, P, P, P, P, S, P]
        lib.elsaa_gemm_workspace_bytes.argtypes = [P, C.POINTER(C.c_size_t)]
        lib.elsaa_gemm.argtypes = [P, P, P, P, P, S, P]
        lib.elsaa_token_rules_fwd.argtypes = [P, P, P, P, P, P]
        lib.elsaa_token_rules_workspace_bytes.argtypes = [P, P, C.POINTER(C.c_size_t)]
        lib.elsaa_token_rules_bwd.argtypes = [P, P, P, P, P, P] + [P] * 7 + [P, S, P]
        lib.elsaa_profile_enable.argtypes = [C.c_int]
        lib.elsaa_profile_count.argtypes = []
        lib.elsaa_profile_get.argtypes = [C.c_int, C.c_char_p, S, C.POINTER(C.c_double),
                                          C.POINTER(C.c_int64)]
        lib.elsaa_status_string.restype = C.c_char_p
        lib.elsaa_status_string.argtypes = [C.c_int]
        lib.elsaa_last_error.restype = C.c_char_p
        _lib = lib
    return _lib


def _check(rc: int):
    if rc != 0:
        raise ElsaaError(rc, load().elsaa_last_error().decode())


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(dev) -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def profile_enable(on: bool = True):
    """Start (clearing old totals) or stop per-kernel event timing in the library."""
    _check(load().elsaa_profile_enable(int(on)))


def profile_read() -> dict:
    """{kernel name: (total ms, launches)} recorded since profile_enable(True)."""
    lib = load()
    out = {}
    for i in range(lib.elsaa_profile_count()):
        buf = C.create_string_buffer(128)
        ms, n = C.c_double(), C.c_int64()
        _check(lib.elsaa_profile_get(i, buf, 128, C.byref(ms), C.byref(n)))
        out[buf.value.decode()] = (ms.value, n.value)
    return out


def num_levels(cfg: Config) -> int:
    c = cfg.c()
    rc = load().elsaa_num_levels(C.byref(c))
    if rc < 0:
        _check(rc)
    return rc


def saved_bytes(cfg: Config) -> int:
    c, n = cfg.c(), C.c_size_t()
    _check(load().elsaa_saved_bytes(C.byref(c), C.byref(n)))
    return n.value


def workspace_bytes(cfg: Config, backward: bool = False) -> int:
    c, n = cfg.c(), C.c_size_t()
    _check(load().elsaa_workspace_bytes(C.byref(c), int(backward), C.byref(n)))
    return n.value


def saved_layout(cfg: Config) -> dict:
    c, L = cfg.c(), _SavedLayout()
    _check(load().elsaa_get_saved_layout(C.byref(c), C.byref(L)))
    return {f: getattr(L, f) for f, _ in _SavedLayout._fields_}


def perm_length(cfg: Config) -> int:
    """Entries of perm_q / perm_k per (b, h) (see elsaa_perm_length)."""
    c = cfg.c()
    n = load().elsaa_perm_length(C.byref(c))
    if n < 0:
        _check(int(n))
    return n


def _perm_shape(cfg: Config):
    """[B, H, Lv, N/2] for causal lists without padding, [B, H, P] with it,
    [B, H, N] non-causal."""
    if cfg.causal:
        lv, p = num_levels(cfg), perm_length(cfg)
        if lv * (cfg.N // 2) == p and cfg.N % 2 == 0:
            return (cfg.B, cfg.H, lv, cfg.N // 2)
        return (cfg.B, cfg.H, p)
    return (cfg.B, cfg.H, cfg.N)


def saved_views(cfg: Config, saved: torch.Tensor) -> dict:
    """Typed views into ``saved``: perm_q, perm_k, m, o_sparse, o_lowrank."""
    L = saved_layout(cfg)
    B, H, N, d = cfg.B, cfg.H, cfg.N, cfg.d_h
    ps = _perm_shape(cfg)
    npm = 1
    for x in ps:
        npm *= x

    def view(off, count, dtype, shape):
        nbytes = count * (torch.finfo(dtype).bits // 8 if dtype.is_floating_point else torch.iinfo(dtype).bits // 8)
        return saved[off:off + nbytes].view(dtype).view(*shape)

    return {
        "perm_q": view(L["perm_q"], npm, torch.int32, ps),
        "perm_k": view(L["perm_k"], npm, torch.int32, ps),
        "m": view(L["m"], B * H * N, torch.float32, (B, H, N)),
        "o_sparse": view(L["o_sparse"], B * H * N * d, torch.float32, (B, H, N, d)),
        "o_lowrank": view(L["o_lowrank"], B * H * N * d, cfg.torch_dtype, (B, H, N, d)),
    }


def _check_tensor(name, t, shape, dtype, dev):
    if t.shape != torch.Size(shape) or t.dtype != dtype or not t.is_contiguous() or t.device != dev:
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)} on {dev}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def _check_inputs(cfg, q, k, v, w_sort, w_race, gates=None, extra=(), lam_rows=None):
    dev = q.device
    shp = (cfg.B, cfg.H, cfg.N, cfg.d_h)
    for name, t in (("q", q), ("k", k), ("v", v)) + tuple(extra):
        _check_tensor(name, t, shp, cfg.torch_dtype, dev)
    if w_sort is not None:
        _check_tensor("w_sort", w_sort, (cfg.H, cfg.sort_bits, cfg.d_h), torch.float32, dev)
    if w_race is not None:
        _check_tensor("w_race", w_race, (cfg.H, cfg.r >> cfg.race_bits, cfg.race_bits, cfg.d_h),
                      torch.float32, dev)
    if gates is not None:
        _check_tensor("gates", gates, (cfg.B, cfg.H, cfg.N, 2), torch.float32, dev)
    if lam_rows is not None:
        _check_tensor("lam_rows", lam_rows, (cfg.B, cfg.H, cfg.N), torch.float32, dev)
    return dev


class Buffers:
    """Preallocated outputs, saved state and workspaces for repeated calls."""

    def __init__(self, cfg: Config, device, backward: bool = True):
        B, H, N, d = cfg.B, cfg.H, cfg.N, cfg.d_h
        dt = cfg.torch_dtype
        self.o = torch.empty(B, H, N, d, dtype=dt, device=device)
        self.lse = torch.empty(B, H, N, dtype=torch.float32, device=device)
        self.d_lr = torch.empty(B, H, N, dtype=torch.float32, device=device)
        self.saved = torch.empty(saved_bytes(cfg), dtype=torch.uint8, device=device)
        ws = workspace_bytes(cfg, False)
        if backward:
            ws = max(ws, workspace_bytes(cfg, True))
            self.dq = torch.empty(B, H, N, d, dtype=dt, device=device)
            self.dk = torch.empty(B, H, N, d, dtype=dt, device=device)
            self.dv = torch.empty(B, H, N, d, dtype=dt, device=device)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)


def select(cfg: Config, q, k, w_sort, workspace: Optional[torch.Tensor] = None):
    """Sorted index lists (perm_q, perm_k) of the sortLSH selection."""
    dev = _check_inputs(cfg, q, k, k, w_sort, None)
    ps = _perm_shape(cfg)
    pq = torch.empty(ps, dtype=torch.int32, device=dev)
    pk = torch.empty(ps, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(workspace_bytes(cfg), 256), dtype=torch.uint8, device=dev)
    c = cfg.c()
    _check(load().elsaa_select(C.byref(c), _p(q), _p(k), _p(w_sort), _p(pq), _p(pk), _p(workspace),
                               workspace.numel(), _stream(dev)))
    return pq, pk


def select_noalloc(cfg: Config, q, k, w_sort, perm_q: torch.Tensor, perm_k: torch.Tensor):
    """The selection into the caller's perm_q, perm_k through
    elsaa_select_noalloc (no allocation: the library's fixed scratch)."""
    dev = _check_inputs(cfg, q, k, k, w_sort, None)
    ps = _perm_shape(cfg)
    _check_tensor("perm_q", perm_q, ps, torch.int32, dev)
    _check_tensor("perm_k", perm_k, ps, torch.int32, dev)
    c = cfg.c()
    _check(load().elsaa_select_noalloc(C.byref(c), _p(q), _p(k), _p(w_sort), _p(perm_q), _p(perm_k),
                                       _stream(dev)))
    return perm_q, perm_k


def fwd(cfg: Config, q, k, v, w_sort, w_race, gates=None, buffers: Optional[Buffers] = None,
        lam_rows=None):
    """Forward; returns (o, lse, d_lr, saved).  lam_rows: per-token lambda_i
    [B, H, N] float32 (None: the scalar cfg.lam)."""
    dev = _check_inputs(cfg, q, k, v, w_sort, w_race, gates, lam_rows=lam_rows)
    bufs = buffers or Buffers(cfg, dev, backward=False)
    c = cfg.c()
    _check(load().elsaa_fwd(C.byref(c), _p(q), _p(k), _p(v), _p(w_sort), _p(w_race), _p(gates),
                            _p(lam_rows), _p(bufs.o), _p(bufs.lse), _p(bufs.d_lr), _p(bufs.saved),
                            bufs.saved.numel(), _p(bufs.workspace), bufs.workspace.numel(),
                            _stream(dev)))
    return bufs.o, bufs.lse, bufs.d_lr, bufs.saved


def bwd(cfg: Config, q, k, v, w_race, do, lse, d_lr, saved, gates=None, want_dgates=False,
        buffers: Optional[Buffers] = None, lam_rows=None, want_dlambda=False):
    """Backward; returns (dq, dk, dv), followed by dgates [B, H, N, 2] when
    want_dgates and by dlambda [B, H, N] when want_dlambda."""
    dev = _check_inputs(cfg, q, k, v, None, w_race, gates, extra=(("do", do),), lam_rows=lam_rows)
    bufs = buffers
    if bufs is None:
        bufs = Buffers(cfg, dev, backward=True)
    dg = torch.empty(cfg.B, cfg.H, cfg.N, 2, dtype=torch.float32, device=dev) if want_dgates else None
    dl = torch.empty(cfg.B, cfg.H, cfg.N, dtype=torch.float32, device=dev) if want_dlambda else None
    c = cfg.c()
    _check(load().elsaa_bwd(C.byref(c), _p(q), _p(k), _p(v), None, _p(w_race), _p(gates),
                            _p(lam_rows), _p(do), _p(lse), _p(d_lr), _p(saved), saved.numel(),
                            _p(bufs.dq), _p(bufs.dk), _p(bufs.dv), _p(dg), _p(dl),
                            _p(bufs.workspace), bufs.workspace.numel(), _stream(dev)))
    return (bufs.dq, bufs.dk, bufs.dv) + ((dg,) if want_dgates else ()) + ((dl,) if want_dlambda else ())


# ---------------------------------------------------------------------------
# dense projections (elsaa_gemm)
# ---------------------------------------------------------------------------
def _matrix(name, t):
    """(rows, cols, ld, heads, seq) of a stored operand: a 2-D tensor with unit
    column stride (plain) or a contiguous 4-D [B, H, S, dh] tensor (head-major,
    logical rows B*S and columns H*dh)."""
    if t.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError(f"{name}: unsupported dtype {t.dtype}")
    if t.dim() == 2:
        if t.stride(1) != 1:
            raise ValueError(f"{name}: the last dimension must be contiguous")
        return t.shape[0], t.shape[1], t.stride(0), 0, 0
    if t.dim() == 4:
        if not t.is_contiguous():
            raise ValueError(f"{name}: head-major operands must be contiguous [B, H, S, dh]")
        Bb, H, S, dh = t.shape
        return Bb * S, H * dh, 0, H, S
    raise ValueError(f"{name}: expected a 2-D matrix or a 4-D [B, H, S, dh] tensor")


def gemm_plan(a, b, trans_a=False, trans_b=False, out=None):
    """Descriptor of out = op(a) op(b) (see gemm)."""
    ar, ac, lda, ah, aseq = _matrix("a", a)
    br, bc, ldb, bh, bseq = _matrix("b", b)
    M, K = (ac, ar) if trans_a else (ar, ac)
    K2, N = (bc, br) if trans_b else (br, bc)
    if K != K2:
        raise ValueError(f"inner dimensions differ: {K} vs {K2}")
    cr, cc, ldc, ch, cseq = _matrix("out", out) if out is not None else (M, N, N, 0, 0)
    if (cr, cc) != (M, N):
        raise ValueError(f"out: expected a {M} x {N} matrix, got {cr} x {cc}")
    seqs = {s for s in (aseq, bseq, cseq) if s}
    if len(seqs) > 1:
        raise ValueError(f"head-major operands with different sequence lengths {sorted(seqs)}")
    seq = seqs.pop() if seqs else 0
    c_dtype = BF16 if out is None or out.dtype == torch.bfloat16 else F32
    return _GemmDesc(M, N, K, int(trans_a), int(trans_b), lda, ldb, ldc, ah, bh, ch, seq, c_dtype)


def gemm_workspace_bytes(desc: _GemmDesc) -> int:
    n = C.c_size_t()
    _check(load().elsaa_gemm_workspace_bytes(C.byref(desc), C.byref(n)))
    return n.value


def gemm(a, b, trans_a=False, trans_b=False, out=None, out_dtype=torch.bfloat16,
         workspace: Optional[torch.Tensor] = None):
    """out = op(a) @ op(b) on the matrix cores: bfloat16 operands, float32
    accumulation, op(x) = x.T when trans_x.  Operands and `out` are 2-D
    matrices (unit column stride) or contiguous head-major [B, H, S, dh]
    tensors standing for the [B*S, H*dh] matrix.  Without `out`, a plain
    [M, N] tensor of out_dtype is allocated."""
    if a.dtype != torch.bfloat16 or b.dtype != torch.bfloat16:
        raise ValueError("gemm operands must be bfloat16")
    if a.device != b.device:
        raise ValueError("operands on different devices")
    desc = gemm_plan(a, b, trans_a, trans_b, out)
    if out is None:
        out = torch.empty(desc.M, desc.N, dtype=out_dtype, device=a.device)
        desc.ldc = desc.N
        desc.c_dtype = BF16 if out_dtype == torch.bfloat16 else F32
    ws = gemm_workspace_bytes(desc)
    if ws and (workspace is None or workspace.numel() < ws):
        workspace = torch.empty(ws, dtype=torch.uint8, device=a.device)
    _check(load().elsaa_gemm(C.byref(desc), _p(a), _p(b), _p(out), _p(workspace) if ws else None,
                             workspace.numel() if ws else 0, _stream(a.device)))
    return out


# ---------------------------------------------------------------------------
# token-wise rules: gate network and query-dependent lambda
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class TokenRules:
    """Parameters of the gate network (W1 [H, G, d_h], b1 [H, G], W2 [H, 2, G],
    b2 [H, 2]) and of the lambda rule (lam_w [H, d_h], lam_b [H], lam_c [H]),
    float32 tensors on the device; leave a rule's tensors None to switch it off."""
    W1: Optional[torch.Tensor] = None
    b1: Optional[torch.Tensor] = None
    W2: Optional[torch.Tensor] = None
    b2: Optional[torch.Tensor] = None
    lam_w: Optional[torch.Tensor] = None
    lam_b: Optional[torch.Tensor] = None
    lam_c: Optional[torch.Tensor] = None
    lambda_min: float = 1e-6

    @property
    def gate_hidden(self) -> int:
        return 0 if self.W1 is None else self.W1.shape[1]

    @property
    def has_lambda(self) -> bool:
        return self.lam_w is not None

    def c(self, cfg: Config) -> _TokenRules:
        H, d = cfg.H, cfg.d_h
        G = self.gate_hidden
        dev = None
        if G:
            for name, t, shp in (("W1", self.W1, (H, G, d)), ("b1", self.b1, (H, G)),
                                 ("W2", self.W2, (H, 2, G)), ("b2", self.b2, (H, 2))):
                _check_tensor(name, t, shp, torch.float32, t.device if dev is None else dev)
                dev = t.device
        if self.has_lambda:
            for name, t, shp in (("lam_w", self.lam_w, (H, d)), ("lam_b", self.lam_b, (H,)),
                                 ("lam_c", self.lam_c, (H,))):
                _check_tensor(name, t, shp, torch.float32, t.device if dev is None else dev)
                dev = t.device
        return _TokenRules(G, _p(self.W1), _p(self.b1), _p(self.W2), _p(self.b2), int(self.has_lambda),
                           _p(self.lam_w), _p(self.lam_b), _p(self.lam_c), self.lambda_min)


def token_rules_fwd(cfg: Config, rules: TokenRules, q):
    """(gates [B, H, N, 2] or None, lambda_rows [B, H, N] or None) of the rules."""
    dev = _check_inputs(cfg, q, q, q, None, None)
    gates = torch.empty(cfg.B, cfg.H, cfg.N, 2, dtype=torch.float32, device=dev) if rules.gate_hidden else None
    lam = torch.empty(cfg.B, cfg.H, cfg.N, dtype=torch.float32, device=dev) if rules.has_lambda else None
    c, r = cfg.c(), rules.c(cfg)
    _check(load().elsaa_token_rules_fwd(C.byref(c), C.byref(r), _p(q), _p(gates), _p(lam), _stream(dev)))
    return gates, lam


def token_rules_workspace_bytes(cfg: Config, rules: TokenRules) -> int:
    """Bytes of the backward's partial-sum workspace (one record per workgroup)."""
    c, r = cfg.c(), rules.c(cfg)
    n = C.c_size_t()
    _check(load().elsaa_token_rules_workspace_bytes(C.byref(c), C.byref(r), C.byref(n)))
    return n.value


def token_rules_bwd(cfg: Config, rules: TokenRules, q, dgates=None, dlambda=None, dq=None,
                    workspace: Optional[torch.Tensor] = None):
    """Parameter gradients of the rules (dict of tensors shaped like the
    parameters); when dq is given, the gate network's gradient with respect
    to q is added to it in place."""
    dev = _check_inputs(cfg, q, q, q, None, None)
    G = rules.gate_hidden
    if G:
        _check_tensor("dgates", dgates, (cfg.B, cfg.H, cfg.N, 2), torch.float32, dev)
    if rules.has_lambda:
        _check_tensor("dlambda", dlambda, (cfg.B, cfg.H, cfg.N), torch.float32, dev)
    if dq is not None:
        _check_tensor("dq", dq, (cfg.B, cfg.H, cfg.N, cfg.d_h), cfg.torch_dtype, dev)
    H, d = cfg.H, cfg.d_h
    f = lambda *shp: torch.empty(*shp, dtype=torch.float32, device=dev)   # noqa: E731
    out = {}
    if G:
        out.update(dW1=f(H, G, d), db1=f(H, G), dW2=f(H, 2, G), db2=f(H, 2))
    if rules.has_lambda:
        out.update(dlam_w=f(H, d), dlam_b=f(H), dlam_c=f(H))
    c, r = cfg.c(), rules.c(cfg)
    lib = load()
    need = token_rules_workspace_bytes(cfg, rules)
    ws = workspace if workspace is not None and workspace.numel() >= need else \
        torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    g = out.get
    _check(lib.elsaa_token_rules_bwd(C.byref(c), C.byref(r), _p(q), _p(dgates if G else None),
                                     _p(dlambda if rules.has_lambda else None), _p(dq),
                                     _p(g("dW1")), _p(g("db1")), _p(g("dW2")), _p(g("db2")),
                                     _p(g("dlam_w")), _p(g("dlam_b")), _p(g("dlam_c")),
                                     _p(ws), ws.numel(), _stream(dev)))
    return out
