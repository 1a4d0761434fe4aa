"""Host-side tests of the C ABI (no GPU needed, nothing is launched).

The library must load, export every entry point include/bkv.h declares, and
reject bad arguments on the host before anything is enqueued.  Only calls
that fail validation are made here, with NULL pointers, so no path can reach
a kernel launch.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
bkv = pytest.importorskip("paper_2609_04971_amd")


def _declared():
    src = open(os.path.join(ROOT, "include", "bkv.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bkv_[a-z_]+)\s*\(", src)))


def test_header_symbols_exported():
    names = _declared()
    assert "bkv_evict" in names and "bkv_score" in names
    lib = ctypes.CDLL(bkv.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in bkv.h but not exported"
    assert sorted(bkv.EXPORTS) == names


def test_version_and_strings():
    assert bkv.abi_version() == 1
    for st in range(7):
        assert bkv.status_string(st)
    assert bkv.status_string(0) == "ok"


def good(**kw):
    d = bkv.dims(B=2, Hq=8, Hkv=2, D=128, N=1000, W=8, C=4, budget=256, n_prefix=2)
    return d.replace(**kw)


@pytest.mark.parametrize("op", range(5))
def test_good_dims_validate(op):
    assert bkv.validate(good(), op) == bkv.OK


@pytest.mark.parametrize("kw,code", [
    (dict(Hq=7), bkv.ERR_SHAPE),             # Hq not a multiple of Hkv
    (dict(Hkv=0), bkv.ERR_SHAPE),
    (dict(D=96), bkv.ERR_SHAPE),
    (dict(N=1001, N_cap=1000), bkv.ERR_SHAPE),
    (dict(N=-1), bkv.ERR_SHAPE),
    (dict(budget=9), bkv.ERR_SHAPE),         # budget < W + n_prefix
    (dict(budget=0, W=0, n_prefix=0), bkv.ERR_SHAPE),
    (dict(C=65), bkv.ERR_SHAPE),
    (dict(W=-1), bkv.ERR_SHAPE),
    (dict(dtype=7), bkv.ERR_DTYPE),
    (dict(B=-1), bkv.ERR_SHAPE),
])
def test_bad_dims(kw, code):
    for op in range(5):
        assert bkv.validate(good(**kw), op) == code


def test_rows_needed_for_scoring_only():
    d = good(C=0, W=0, n_prefix=0)
    assert bkv.validate(d, bkv.OP_SCORE) == bkv.ERR_SHAPE
    assert bkv.validate(d, bkv.OP_EVICT) == bkv.ERR_SHAPE
    assert bkv.validate(d, bkv.OP_TOPK) == bkv.OK
    assert bkv.validate(d, bkv.OP_COMPACT) == bkv.OK
    assert bkv.validate(good(C=0), bkv.OP_BEACON_UPDATE) == bkv.ERR_SHAPE
    assert bkv.validate(good(C=64, W=250), bkv.OP_SCORE) == bkv.ERR_SHAPE  # 64 + 4*250 > 1024 rows


def test_bad_op_and_null_dims():
    lib = bkv.lib()
    assert bkv.validate(good(), 5) == bkv.ERR_INVALID
    assert lib.bkv_validate(None, 0) == bkv.ERR_INVALID
    assert lib.bkv_workspace_bytes(None, 4) == 0


def test_null_pointers_rejected_before_launch():
    lib = bkv.lib()
    d = good()
    r = ctypes.byref(d)
    assert lib.bkv_score(r, None, None, None, None, None, None, 0.0, None, None, None, 0, None) == bkv.ERR_INVALID
    assert lib.bkv_topk(r, None, None, None, 0, None) == bkv.ERR_INVALID
    assert lib.bkv_compact(r, None, None, None, None, 0, None) == bkv.ERR_INVALID
    assert lib.bkv_evict(r, None, None, None, None, None, None, None, 0.0, None, None, None, None, 0,
                         None) == bkv.ERR_INVALID
    assert lib.bkv_beacon_update(r, None, 3, None, None, None, None) == bkv.ERR_INVALID
    assert lib.bkv_beacon_update(r, None, -1, None, None, None, None) == bkv.ERR_SHAPE
    assert lib.bkv_workspace_init(r, None, 0, None) == bkv.ERR_INVALID
    assert lib.bkv_device_status(None, 0, None) == bkv.ERR_INVALID
    bad = good(D=96)
    assert lib.bkv_evict(ctypes.byref(bad), None, None, None, None, None, None, None, 0.0, None, None, None,
                         None, 0, None) == bkv.ERR_SHAPE


def test_empty_work_is_a_no_op():
    lib = bkv.lib()
    for d in (good(B=0), good(N=0)):
        r = ctypes.byref(d)
        assert lib.bkv_score(r, None, None, None, None, None, None, 0.0, None, None, None, 0, None) == bkv.OK
        assert lib.bkv_topk(r, None, None, None, 0, None) == bkv.OK
        assert lib.bkv_compact(r, None, None, None, None, 0, None) == bkv.OK
    assert lib.bkv_beacon_update(ctypes.byref(good()), None, 0, None, None, None, None) == bkv.OK


def test_workspace_sizes():
    d = good()
    assert bkv.workspace_bytes(d, bkv.OP_TOPK) == 0
    assert bkv.workspace_bytes(d, bkv.OP_BEACON_UPDATE) == 0
    c, s, e = (bkv.workspace_bytes(d, op) for op in (bkv.OP_COMPACT, bkv.OP_SCORE, bkv.OP_EVICT))
    assert 0 < c < s < e
    # the control block depends only on B*Hkv and budget, not on N, W or C
    d2 = good(N=5000, N_cap=5000, W=16, C=8)
    assert bkv.workspace_bytes(d2, bkv.OP_COMPACT) == c
    assert bkv.workspace_bytes(d2, bkv.OP_EVICT) > e
    assert bkv.workspace_bytes(good(budget=8192), bkv.OP_COMPACT) > c


def test_missing_library_fails_loudly(monkeypatch):
    # no silent fallback: with the library absent the first use raises
    monkeypatch.setattr(bkv, "_lib", None)
    monkeypatch.setattr(bkv, "LIB_PATH", os.path.join(ROOT, "no-such-dir", "libbkv.so"))
    with pytest.raises(ImportError):
        bkv.validate(good(), bkv.OP_EVICT)


# ---- FPS entry points: rejected on the host, or no-ops -------------------------
_Q = ctypes.c_void_p(0x100000)      # stand-in addresses: only calls that fail
_Q2 = ctypes.c_void_p(0x900000)     # validation (or are no-ops) are made
_PK = ctypes.c_void_p(0x200000)


def _fps(H=2, n=10, m=4, D=128, dt=None, q=_Q, rows=10, picks=_PK):
    dt = bkv.BF16 if dt is None else dt
    return bkv.lib().bkv_fps(H, n, m, D, dt, q, rows, picks, None)


def _gather(H=2, n=10, m=4, D=128, dt=None, src=_Q, rows=10, dst=_Q2, ddt=None, drows=10, picks=None,
            counts=None):
    dt = bkv.BF16 if dt is None else dt
    ddt = dt if ddt is None else ddt
    return bkv.lib().bkv_fps_gather(H, n, m, D, dt, src, rows, dst, ddt, drows, picks, counts, None)


@pytest.mark.parametrize("kw,code", [
    (dict(D=96), bkv.ERR_SHAPE),
    (dict(dt=5), bkv.ERR_DTYPE),
    (dict(n=11), bkv.ERR_SHAPE),                   # more rows than the head holds
    (dict(n=32769, rows=40000), bkv.ERR_SHAPE),   # above the row limit
    (dict(H=-1), bkv.ERR_SHAPE),
    (dict(m=-1), bkv.ERR_SHAPE),
    (dict(q=None), bkv.ERR_INVALID),
    (dict(q=ctypes.c_void_p(0x100004)), bkv.ERR_INVALID),  # not 16-byte aligned
    (dict(picks=None), bkv.ERR_INVALID),
])
def test_fps_rejects(kw, code):
    assert _fps(**kw) == code


def test_fps_empty_is_a_no_op():
    assert _fps(H=0) == bkv.OK
    assert _fps(n=0) == bkv.OK
    assert _fps(m=0) == bkv.OK
    assert _fps(H=0, q=None, picks=None) == bkv.OK
    assert _gather(m=0, dst=None) == bkv.OK


@pytest.mark.parametrize("kw,code", [
    (dict(dt=bkv.F32, ddt=bkv.BF16), bkv.ERR_DTYPE),   # narrowing is not offered
    (dict(ddt=7), bkv.ERR_DTYPE),
    (dict(n=200, rows=200, m=129, drows=200), bkv.ERR_SHAPE),  # more than 128 gathered rows
    (dict(m=4, drows=3), bkv.ERR_SHAPE),                # dst too short for the picks
    (dict(dst=None), bkv.ERR_INVALID),
    (dict(dst=ctypes.c_void_p(0x100000 + 256)), bkv.ERR_INVALID),  # partial overlap with src
    (dict(dst=_Q, drows=12), bkv.ERR_INVALID),          # same base, other layout
    (dict(dst=_Q, ddt=bkv.F32), bkv.ERR_INVALID),       # same base, widened in place
    (dict(D=64, n=33000, rows=33000), bkv.ERR_SHAPE),
])
def test_fps_gather_rejects(kw, code):
    assert _gather(**kw) == code


def test_score_ex_rejects_unknown_flags_and_keeps_rules():
    lib = bkv.lib()
    d = good()
    r = ctypes.byref(d)
    assert lib.bkv_score_ex(r, 4, None, None, None, None, None, None, 0.0, None, None, None, 0, None) == \
        bkv.ERR_INVALID
    assert lib.bkv_evict_ex(r, 8, None, None, None, None, None, None, None, 0.0, None, None, None, None, 0,
                            None) == bkv.ERR_INVALID
    # valid flags, then the same checks as without them
    for f in (1, 2, 3):
        assert lib.bkv_score_ex(r, f, None, None, None, None, None, None, 0.0, None, None, None, 0, None) == \
            bkv.ERR_INVALID
        assert lib.bkv_score_ex(ctypes.byref(good(D=96)), f, None, None, None, None, None, None, 0.0, None, None,
                                None, 0, None) == bkv.ERR_SHAPE
        assert lib.bkv_score_ex(ctypes.byref(good(N=0)), f, None, None, None, None, None, None, 0.0, None, None,
                                None, 0, None) == bkv.OK


def test_compact_fill_rejects_before_launch():
    lib = bkv.lib()
    d = good()
    r = ctypes.byref(d)
    assert lib.bkv_compact_fill(r, None, None, None, None, None, 0, None) == bkv.ERR_INVALID
    big = good(N=70000, N_cap=70000, budget=66000)  # more kept rows per head than the LDS bitmap holds
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: the shape is rejected first
    assert lib.bkv_compact_fill(ctypes.byref(big), fake, fake, fake, fake, None, 0, None) == bkv.ERR_SHAPE
    empty = good(B=0)
    assert lib.bkv_compact_fill(ctypes.byref(empty), None, None, None, None, None, 0, None) == bkv.OK


def test_noalloc_rejects_dims_beyond_its_array():
    # host-only: dims whose workspace exceeds the library's fixed array are
    # refused before anything is enqueued (no device needed)
    lib = bkv.lib()
    big = good(B=64, N=65536, N_cap=65536, budget=8192)
    assert lib.bkv_workspace_bytes(ctypes.byref(big), bkv.OP_EVICT) > (32 << 20)
    st = lib.bkv_evict_noalloc(ctypes.byref(big), 0, None, None, None, None, None, None, None, 0.0, None, None,
                               None, None, None)
    assert st == bkv.ERR_INVALID  # NULL tensors are caught first
    p = ctypes.c_void_p(16)  # any 16-byte aligned value: nothing is dereferenced on the host
    st = lib.bkv_evict_noalloc(ctypes.byref(big), 0, p, p, p, p, p, None, None, 0.0, None, None, None, None, None)
    assert st == bkv.ERR_WORKSPACE
