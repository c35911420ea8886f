"""C-ABI library: it loads, exports every declared entry point, and rejects
bad arguments on the host (no GPU needed: validation runs before any HIP call)."""
import ctypes as C
import os
import re

import pytest

import paper_2607_20214_amd as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "elsaa.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(elsaa_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert {"elsaa_fwd", "elsaa_bwd", "elsaa_select"} <= set(names)
    lib = E.load()
    for n in names:
        assert hasattr(lib, n), n


def _cfg(**kw):
    base = dict(B=1, H=2, N=1024, d_h=64, k=64, r=64, causal=True)
    base.update(kw)
    return E.Config(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(N=0), -1), (dict(k=0), -1), (dict(r=40), -1), (dict(sort_bits=9), -1),
    (dict(eps=0.0), -1), (dict(lam=-1.0), -1), (dict(beta=0.0), -1), (dict(dtype="f16"), None),
    (dict(d_h=96), -2), (dict(race_bits=3, r=64), -2), (dict(r=512), -2),
    (dict(N=5, k=1, n0=1), -2),     # a past half would hold one of Alg. 5's zero tokens
])
def test_host_validation_rejects(kw, status):
    if status is None:
        cfg = _cfg(**kw)
        c = cfg.c()
        c.dtype = 7
        rc = E.load().elsaa_num_levels(C.byref(c))
        assert rc == -1
        return
    with pytest.raises(E.ElsaaError) as ei:
        E.num_levels(_cfg(**kw))
    assert ei.value.status == status
    assert E.load().elsaa_last_error().decode()


def test_head_rows_must_fit_32_bit_offsets():
    # N * d_h * element bytes reaches 2^32 for float32 rows at N = 2^23, d_h = 128
    big = dict(N=1 << 23, d_h=128, k=64, r=64, causal=False)
    with pytest.raises(E.ElsaaError) as ei:
        E.num_levels(_cfg(dtype="f32", **big))
    assert ei.value.status == -2
    assert E.num_levels(_cfg(dtype="bf16", **big)) == 0


def test_padded_recursion_levels_and_list_length():
    """Alg. 5 pads odd lists with a zero token: 300 -> 150 -> 75 (+1) -> 38."""
    cfg = _cfg(N=300, k=32)
    assert E.num_levels(cfg) == 3
    assert E.perm_length(cfg) == 150 + 2 * 75 + 4 * 38
    big = _cfg(N=16386, k=128, H=16, d_h=128, r=128)
    assert E.num_levels(big) == 7
    L, total = 16386, 0
    for l in range(7):
        L = (L + 1) // 2
        total += L << l
    assert E.perm_length(big) == total
    assert E.perm_length(_cfg(N=16384, k=128, d_h=128, r=128)) == 6 * 8192


def test_sizes_and_layout():
    cfg = _cfg(N=16384, H=16, d_h=128, k=128, r=128, B=1)
    assert E.num_levels(cfg) == 6
    L = E.saved_layout(cfg)
    P = 6 * 16384 // 2
    assert L["perm_k"] - L["perm_q"] >= 16 * P * 4
    assert L["total"] == E.saved_bytes(cfg)
    assert all(L[k] % 256 == 0 for k in L)
    nc = _cfg(causal=False, N=4096)
    assert E.num_levels(nc) == 0
    assert E.workspace_bytes(nc) > 0


def test_null_pointers_are_rejected_before_any_launch():
    cfg = _cfg()
    c = cfg.c()
    lib = E.load()
    rc = lib.elsaa_fwd(C.byref(c), None, None, None, None, None, None, None, None, None, None, None,
                       0, None, 0, None)
    assert rc == -1
    rc = lib.elsaa_select(C.byref(c), None, None, None, None, None, None, 0, None)
    assert rc == -1
    assert lib.elsaa_status_string(-3) == b"buffer too small"


def test_workspace_too_small_is_rejected():
    cfg = _cfg()
    c = cfg.c()
    lib = E.load()
    fake = C.c_void_p(1 << 20)   # aligned, never dereferenced: the size check fails first
    rc = lib.elsaa_fwd(C.byref(c), fake, fake, fake, fake, fake, None, None, fake, fake, fake, fake,
                       16, fake, 1 << 30, None)
    assert rc == -3


@pytest.mark.parametrize("over", [dict(neighbors=-1), dict(m_one=2)])
def test_variant_fields_are_validated(over):
    cfg = _cfg(**over)
    c = cfg.c()
    fake = C.c_void_p(1 << 20)
    rc = E.load().elsaa_fwd(C.byref(c), fake, fake, fake, fake, fake, None, None, fake, fake, fake,
                            fake, 1 << 40, fake, 1 << 40, None)
    assert rc == -1


def _gdesc(**kw):
    d = E._GemmDesc(M=256, N=256, K=256, trans_a=0, trans_b=0, lda=256, ldb=256, ldc=256,
                    a_heads=0, b_heads=0, c_heads=0, seq=0, c_dtype=E.BF16)
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), -1), (dict(K=-8), -1), (dict(M=100), -2), (dict(trans_a=2), -1), (dict(c_dtype=5), -1),
    (dict(lda=100), -1), (dict(ldb=260), -1), (dict(a_heads=3, seq=256), -1),
    (dict(a_heads=4, seq=100), -1), (dict(a_heads=2, lda=0, seq=256), None),
    (dict(b_heads=64, seq=256), -2), (dict(N=192, b_heads=2, seq=256), -2),
])
def test_gemm_validation(kw, status):
    lib = E.load()
    d = _gdesc(**kw)
    fake = C.c_void_p(1 << 20)   # never dereferenced: validation fails before any launch
    rc = lib.elsaa_gemm(C.byref(d), fake, fake, None if status is None else fake, None, 0, None)
    if status is None:           # the only error left is the NULL output pointer
        assert rc == -1 and b"C is NULL" in lib.elsaa_last_error()
    else:
        assert rc == status, lib.elsaa_last_error()


def test_gemm_split_workspace_and_checks():
    lib = E.load()
    d = _gdesc(M=1024, N=3072, K=32768, lda=1024, ldb=3072, ldc=3072, trans_a=1)
    n = E.gemm_workspace_bytes(d)
    assert n > 0 and n % (1024 * 3072 * 4) == 0      # float32 partials, whole planes
    assert E.gemm_workspace_bytes(_gdesc()) == 0      # 4 tiles, K = 256: no split
    fake = C.c_void_p(1 << 20)
    assert lib.elsaa_gemm(C.byref(d), fake, fake, fake, None, 0, None) == -1
    assert lib.elsaa_gemm(C.byref(d), fake, fake, fake, fake, n - 1, None) == -3
    bad = C.c_void_p((1 << 20) + 8)
    assert lib.elsaa_gemm(C.byref(_gdesc()), bad, fake, fake, None, 0, None) == -1


def _rules(**kw):
    fake = 1 << 20                 # aligned, never dereferenced: validation fails first
    r = E._TokenRules(64, fake, fake, fake, fake, 1, fake, fake, fake, 1e-6)
    for k, v in kw.items():
        setattr(r, k, v)
    return r


@pytest.mark.parametrize("kw,status", [
    (dict(gate_hidden=32), -2), (dict(gate_hidden=0, lambda_rule=0), -1), (dict(lambda_rule=2), -1),
    (dict(W1=None), -1), (dict(lam_c=None), -1), (dict(W1=(1 << 20) + 4), -1),
    (dict(lambda_min=-1.0), -1), (dict(gate_hidden=0, W1=None, b1=None), 0),
])
def test_token_rules_validation(kw, status):
    lib = E.load()
    c = _cfg().c()
    r = _rules(**kw)
    n = C.c_size_t()
    rc = lib.elsaa_token_rules_workspace_bytes(C.byref(c), C.byref(r), C.byref(n))
    assert rc == status
    if status == 0:
        assert n.value > 0
        fake = C.c_void_p(1 << 20)
        # a too-small workspace is caught before any launch
        rc = lib.elsaa_token_rules_bwd(C.byref(c), C.byref(r), fake, None, fake, fake, *([None] * 7),
                                       fake, 16, None)
        assert rc == -3
        # the lambda rule's gradient input is required
        rc = lib.elsaa_token_rules_bwd(C.byref(c), C.byref(r), fake, None, None, fake, *([None] * 7),
                                       fake, 1 << 40, None)
        assert rc == -1


def test_select_noalloc_rejects_on_the_host():
    """The no-allocation selection checks pointers and its fixed scratch
    limit (2 * B*H*N bytes of keys within 32 MiB) before any HIP call."""
    lib = E.load()
    fake = C.c_void_p(1 << 20)
    c = _cfg().c()
    assert lib.elsaa_select_noalloc(C.byref(c), None, fake, fake, fake, fake, None) == -1
    big = _cfg(B=1, H=256, N=65600, causal=False).c()
    assert lib.elsaa_select_noalloc(C.byref(big), fake, fake, fake, fake, fake, None) == -3
    assert "scratch" in lib.elsaa_last_error().decode()
