"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

import paper_2608_18410_amd as rs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rolesub.h")
FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation first


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(rolesub_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(rs.LIB_PATH):
        pytest.fail("librolesub.so is not built; run python -m paper_2608_18410_amd.build")
    return rs.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
    assert set(rs.EXPORTS) == set(names)


def test_status_strings_and_version(lib):
    for code, name in enumerate(["ROLESUB_OK", "ROLESUB_ERR_INVALID_ARG", "ROLESUB_ERR_UNSUPPORTED",
                                 "ROLESUB_ERR_CAPACITY", "ROLESUB_ERR_HIP"]):
        assert rs.status_name(code) == name
    assert lib.rolesub_version() >= 100


def _dims(B=1, T=4, H=2, dh=64, G=8, d=32):
    return rs.Dims(B, T, H, dh, G, d)


def _last():
    return rs.load().rolesub_last_error().decode()


def test_rotate_validation(lib):
    d = _dims(dh=96)
    assert lib.rolesub_rotate_values(ctypes.byref(d), rs.BF16, FAKE, FAKE, FAKE, None) == 2
    assert "head dim" in _last()
    d = _dims()
    assert lib.rolesub_rotate_values(ctypes.byref(d), rs.BF16, None, FAKE, FAKE, None) == 1
    assert lib.rolesub_rotate_values(ctypes.byref(d), 7, FAKE, FAKE, FAKE, None) == 2
    assert lib.rolesub_rotate_values(None, rs.BF16, FAKE, FAKE, FAKE, None) == 1
    # z aliasing v
    assert lib.rolesub_rotate_values(ctypes.byref(d), rs.BF16, FAKE, FAKE, FAKE, None) == 1
    assert "overlaps" in _last()
    # empty problem is a no-op success
    d0 = _dims(T=0)
    assert lib.rolesub_rotate_values(ctypes.byref(d0), rs.BF16, None, None, None, None) == 0


def test_route_noalloc_validation(lib):
    """The no-alloc route call validates like rolesub_route and refuses a
    route workspace beyond its fixed device array before any device call."""
    d = _dims(G=8)
    bad_k = rs.make_budget(rs.TOPK, (9, 1, 8, 8))
    assert lib.rolesub_route_noalloc(ctypes.byref(d), rs.BF16, None, ctypes.byref(bad_k), FAKE, FAKE, FAKE,
                                     None, FAKE, None, None, None) == 1
    assert "rolesub_route_noalloc" in _last() and "k_by_type" in _last()
    ok = rs.make_budget(rs.TOPK, (4, 6, 8, 8))
    assert lib.rolesub_route_noalloc(None, rs.BF16, None, ctypes.byref(ok), FAKE, FAKE, FAKE,
                                     None, FAKE, None, None, None) == 1
    assert lib.rolesub_route_noalloc(ctypes.byref(d), rs.BF16, None, ctypes.byref(ok), FAKE, FAKE, None,
                                     None, FAKE, None, None, None) == 1                 # no router, no scores
    big = _dims(B=600, T=1, G=8, d=4096)
    desc = rs.RouterDesc()
    desc.kind, desc.C, desc.d_e, desc.Hr = rs.MLP2, 8, 128, 128
    for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2"):
        setattr(desc, n, 0x1000)
    assert lib.rolesub_route_workspace_size(ctypes.byref(big), ctypes.byref(desc)) > rs.ROUTE_NOALLOC_MAX_BYTES
    assert lib.rolesub_route_noalloc(ctypes.byref(big), rs.BF16, ctypes.byref(desc), ctypes.byref(ok), FAKE, FAKE,
                                     None, None, FAKE, None, None, None) == 2
    assert "above the" in _last()


def test_route_validation(lib):
    d = _dims(G=8)
    bad_k = rs.make_budget(rs.TOPK, (9, 1, 8, 8))
    assert lib.rolesub_route(ctypes.byref(d), rs.BF16, None, ctypes.byref(bad_k), FAKE, FAKE, FAKE,
                             None, FAKE, None, None, None, 0, None) == 1
    assert "k_by_type" in _last()
    d33 = _dims(G=33)
    ok = rs.make_budget(rs.TOPK, (4, 6, 8, 8))
    assert lib.rolesub_route(ctypes.byref(d33), rs.BF16, None, ctypes.byref(ok), FAKE, FAKE, FAKE,
                             None, FAKE, None, None, None, 0, None) == 2
    thr = rs.make_budget(rs.THRESHOLD, (0, 0, 0, 0), 0.0, 5, 2)
    assert lib.rolesub_route(ctypes.byref(d), rs.BF16, None, ctypes.byref(thr), None, None, FAKE,
                             None, FAKE, None, None, None, 0, None) == 1
    # router missing and no scores
    assert lib.rolesub_route(ctypes.byref(d), rs.BF16, None, ctypes.byref(ok), FAKE, FAKE, None,
                             None, FAKE, None, None, None, 0, None) == 1
    # workspace too small
    desc = rs.RouterDesc()
    desc.kind, desc.C, desc.d_e, desc.Hr = rs.MLP2, 4, 8, 16
    for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2"):
        setattr(desc, n, 0x1000)
    need = lib.rolesub_route_workspace_size(ctypes.byref(d), ctypes.byref(desc))
    assert need > 0
    assert lib.rolesub_route(ctypes.byref(d), rs.BF16, ctypes.byref(desc), ctypes.byref(ok), FAKE, FAKE,
                             None, None, FAKE, None, None, FAKE, need - 1, None) == 1
    assert "workspace" in _last()
    desc.W2 = None
    assert lib.rolesub_route(ctypes.byref(d), rs.BF16, ctypes.byref(desc), ctypes.byref(ok), FAKE, FAKE,
                             None, None, FAKE, None, None, FAKE, need, None) == 1


def test_pack_capacity_check(lib):
    d = _dims(T=10, G=8)
    bu = rs.make_budget(rs.TOPK, (4, 6, 8, 8))
    tc = (ctypes.c_int32 * 4)(6, 3, 1, 0)     # need 6*4 + 3*6 + 1*8 = 50
    assert lib.rolesub_pack_kv(ctypes.byref(d), rs.BF16, ctypes.byref(bu), tc, FAKE, FAKE, FAKE, FAKE,
                               49, None) == 3
    assert "budget" in _last()
    thr = rs.make_budget(rs.THRESHOLD, (0, 0, 0, 0), 0.0, 1, 3)
    assert lib.rolesub_pack_kv(ctypes.byref(d), rs.BF16, ctypes.byref(thr), tc, FAKE, FAKE, FAKE, FAKE,
                               29, None) == 3
    d_bad = _dims(dh=64, G=12)
    assert lib.rolesub_pack_kv(ctypes.byref(d_bad), rs.BF16, None, None, FAKE, FAKE, FAKE, FAKE, 10, None) == 1
    assert lib.rolesub_pack_kv(ctypes.byref(d), rs.BF16, None, None, FAKE, FAKE, FAKE, FAKE, -1, None) == 1


def test_attend_validation(lib):
    d = _dims()
    args = (FAKE, FAKE, FAKE, FAKE, FAKE, 32, FAKE, ctypes.c_float(0.0), FAKE)
    assert lib.rolesub_attend(ctypes.byref(d), rs.BF16, 4, *args, 7, None, 0, None) == 2   # out dtype
    assert lib.rolesub_attend(ctypes.byref(d), rs.F32, 4, *args, rs.BF16, None, 0, None) == 2
    d0 = _dims(T=0)
    assert lib.rolesub_attend(ctypes.byref(d0), rs.BF16, 4, *args, rs.F32, None, 0, None) == 1
    assert "T=0" in _last()
    assert lib.rolesub_attend(ctypes.byref(d), rs.BF16, -1, *args, rs.F32, None, 0, None) == 1
    nan_args = args[:7] + (ctypes.c_float(float("nan")),) + args[8:]
    assert lib.rolesub_attend(ctypes.byref(d), rs.BF16, 4, *nan_args, rs.F32, None, 0, None) == 1
    assert lib.rolesub_attend_workspace_size(ctypes.byref(d), 4) == 0


def _i32x(*vals):
    return (ctypes.c_int32 * len(vals))(*vals)


def test_retain_and_gather_validation(lib):
    ok_len, ok_keep = _i32x(256, 256), _i32x(64, 64)
    assert lib.rolesub_retain_tokens(2, 512, 0, ok_len, ok_keep, FAKE, FAKE, None) == 2
    assert lib.rolesub_retain_tokens(2, 512, 17, ok_len, ok_keep, FAKE, FAKE, None) == 2
    assert lib.rolesub_retain_tokens(2, 500, 2, ok_len, ok_keep, FAKE, FAKE, None) == 1
    assert "sum to 512" in _last()
    assert lib.rolesub_retain_tokens(2, 512, 2, ok_len, _i32x(64, 300), FAKE, FAKE, None) == 1
    assert lib.rolesub_retain_tokens(1, 9000, 1, _i32x(9000), _i32x(5), FAKE, FAKE, None) == 2
    assert lib.rolesub_retain_tokens(2, 512, 2, ok_len, ok_keep, None, FAKE, None) == 1
    assert lib.rolesub_retain_tokens(0, 512, 2, ok_len, ok_keep, None, None, None) == 0   # no samples: no-op
    assert lib.rolesub_gather_tokens(2, 9, 4, 6, FAKE, FAKE, FAKE, None) == 2            # row bytes % 4
    assert lib.rolesub_gather_tokens(2, 9, 4, 16, None, FAKE, FAKE, None) == 1
    assert lib.rolesub_gather_tokens(2, 9, 0, 16, None, None, None, None) == 0


def test_allocate_validation(lib):
    kby = _i32x(4, 6, 8, 8)
    assert lib.rolesub_allocate_groups(1, 4097, 8, kby, FAKE, FAKE, None, FAKE, None, None, None, None) == 2
    assert "4096" in _last()
    assert lib.rolesub_allocate_groups(1, 8, 8, _i32x(9, 1, 1, 1), FAKE, FAKE, None, FAKE, None, None, None,
                                       None) == 1
    assert lib.rolesub_allocate_groups(1, 8, 33, kby, FAKE, FAKE, None, FAKE, None, None, None, None) == 2
    assert lib.rolesub_allocate_groups(1, 8, 8, None, FAKE, FAKE, None, FAKE, None, None, None, None) == 1
    assert lib.rolesub_allocate_groups(1, 8, 8, kby, FAKE, FAKE, None, FAKE, FAKE, None, None, None) == 1
    assert "without scores" in _last()
    assert lib.rolesub_allocate_groups(1, 8, 8, kby, FAKE, FAKE, FAKE, FAKE, None, None, None, None) == 1
    assert lib.rolesub_allocate_groups(1, 8, 8, kby, FAKE, FAKE, None, None, None, None, None, None) == 1
    assert lib.rolesub_allocate_groups(1, 8, 8, kby, None, FAKE, None, FAKE, None, None, None, None) == 1
    assert lib.rolesub_allocate_groups(0, 8, 8, kby, None, None, None, None, None, None, None, None) == 0
    # routing with allocation: router, priority weights and workspace are required
    d = _dims(G=8, d=64)
    desc = rs.RouterDesc()
    desc.kind, desc.C, desc.d_e, desc.Hr = rs.MLP2, 4, 8, 16
    for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2"):
        setattr(desc, n, 0x1000)
    need = lib.rolesub_route_allocate_workspace_size(ctypes.byref(d), ctypes.byref(desc))
    assert need >= lib.rolesub_route_workspace_size(ctypes.byref(d), ctypes.byref(desc))
    args = (FAKE, FAKE, None, None, None, FAKE, None, None)
    assert lib.rolesub_route_allocate(ctypes.byref(d), rs.BF16, ctypes.byref(desc), None, kby, *args,
                                      FAKE, need, None) == 1
    assert "w_pri" in _last()
    assert lib.rolesub_route_allocate(ctypes.byref(d), rs.BF16, ctypes.byref(desc), FAKE, kby, *args,
                                      FAKE, need - 1, None) == 1
    assert "workspace" in _last()
    assert lib.rolesub_route_allocate(ctypes.byref(d), rs.BF16, None, FAKE, kby, *args, FAKE, need, None) == 1


def test_full_width_validation(lib):
    ws = lib.rolesub_full_workspace_size(2, 81, 16)
    assert ws > 2 * 81 * 16 * 4
    d = rs.Dims(2, 81, 32, 128, 16, 0)
    rp = lambda dims, dt=rs.BF16, cap=2 * 81 * 16, ws_bytes=ws, budget=None, tc=None: lib.rolesub_full_rotate_pack(
        ctypes.byref(dims), dt, FAKE, FAKE, FAKE, FAKE, ctypes.c_void_p(0x10000000), cap, budget, tc, FAKE,
        ws_bytes, None)
    assert rp(d, dt=rs.F32) == 2
    assert rp(rs.Dims(2, 81, 64, 64, 16, 0)) == 2                    # head dim 64
    assert rp(rs.Dims(2, 81, 8, 128, 16, 0)) == 2                    # groups of 64 dims
    assert "multiple of 128" in _last()
    assert rp(rs.Dims(1025, 81, 32, 128, 16, 0)) == 2                # batch limit
    assert rp(d, ws_bytes=ws - 1) == 1
    assert rp(d, cap=-1) == 1
    bu = rs.make_budget(rs.TOPK, (4, 16, 16, 16))
    assert rp(d, cap=32 * 4 + 48 * 16, budget=ctypes.byref(bu), tc=_i32x(32, 48, 1, 0)) == 3   # 1 proprio short
    assert rp(rs.Dims(0, 81, 32, 128, 16, 0), ws_bytes=0) == 0
    # values: the head-major output may not overlap the cache
    assert lib.rolesub_full_values(ctypes.byref(d), rs.BF16, FAKE, FAKE, FAKE, FAKE, 2 * 81 * 16, FAKE, FAKE, ws,
                                   None) == 1
    assert "overlaps" in _last()
    assert lib.rolesub_full_values(ctypes.byref(d), rs.BF16, None, FAKE, FAKE, FAKE, 10, FAKE, FAKE, ws, None) == 1
    assert lib.rolesub_full_transpose(100, rs.BF16, FAKE, FAKE, None) == 2
    assert lib.rolesub_full_transpose(128, rs.BF16, FAKE, FAKE, None) == 1
    assert lib.rolesub_full_transpose(128, rs.F32, FAKE, ctypes.c_void_p(0x10000000), None) == 2
    assert lib.rolesub_full_transpose(0, rs.BF16, None, None, None) == 0


def test_attend_values_validation(lib):
    d = rs.Dims(2, 9, 4, 128, 1, 0)
    assert lib.rolesub_attend_values(ctypes.byref(d), rs.F32, 4, FAKE, FAKE, FAKE, ctypes.c_float(0.0), FAKE,
                                     rs.F32, None) == 2
    assert lib.rolesub_attend_values(ctypes.byref(rs.Dims(2, 9, 4, 96, 1, 0)), rs.BF16, 4, FAKE, FAKE, FAKE,
                                     ctypes.c_float(0.0), FAKE, rs.F32, None) == 2
    assert lib.rolesub_attend_values(ctypes.byref(d), rs.BF16, 4, FAKE, None, FAKE, ctypes.c_float(0.0), FAKE,
                                     rs.F32, None) == 1
    assert lib.rolesub_attend_values(ctypes.byref(d), rs.BF16, 0, None, None, None, ctypes.c_float(0.0), None,
                                     rs.F32, None) == 0
    assert lib.rolesub_attend_values(None, rs.BF16, 4, FAKE, FAKE, FAKE, ctypes.c_float(0.0), FAKE, rs.F32, None) == 1
