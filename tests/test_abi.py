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
    (dict(N=300, k=32), -2), (dict(N=96, k=16), -2),
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
    rc = lib.elsaa_fwd(C.byref(c), None, None, None, None, None, None, None, None, None, None, 0,
                       None, 0, None)
    assert rc == -1
    rc = lib.elsaa_select(C.byref(c), None, None, None, None, None, None, 0, None)
    assert rc == -1
    assert lib.elsaa_status_string(-3) == b"buffer too small"


def test_workspace_too_small_is_rejected():
    cfg = _cfg()
    c = cfg.c()
    lib = E.load()
    fake = C.c_void_p(1 << 20)   # aligned, never dereferenced: the size check fails first
    rc = lib.elsaa_fwd(C.byref(c), fake, fake, fake, fake, fake, None, fake, fake, fake, fake, 16,
                       fake, 1 << 30, None)
    assert rc == -3
