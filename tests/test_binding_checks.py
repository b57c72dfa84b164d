"""The Python binding checks every tensor's shape and dtype against the sizes it
passes to the library, on the host, before any launch (the C ABI receives
bare pointers and cannot see a buffer's size). CPU tensors only: a call whose
shapes are all consistent gets as far as the device check, which shows that
the shape checks accept it; each planted mismatch must be refused earlier."""
import pytest
import torch

import paper_2608_18410_amd as rs

bf, f32, i32, u8 = torch.bfloat16, torch.float32, torch.int32, torch.uint8
B, T, H, dh, G, Tq, d = 2, 10, 4, 64, 8, 3, 64
ds = dh // G
cap = T * G


def z(*shape, dtype=bf):
    return torch.zeros(shape, dtype=dtype)


def reaches_device_check(fn, *a, **kw):
    with pytest.raises(ValueError, match="device tensors only"):
        fn(*a, **kw)


def refused(fn, *a, match="expected (shape|dtype)", **kw):
    with pytest.raises((ValueError, TypeError), match=match):
        fn(*a, **kw)


def test_rotate_values_shapes():
    reaches_device_check(rs.rotate_values, z(B, T, H, dh), z(H, dh, dh))
    refused(rs.rotate_values, z(B, T, H, dh), z(H + 1, dh, dh))
    refused(rs.rotate_values, z(B, T, H, dh), z(H, dh, dh, dtype=f32))
    refused(rs.rotate_values, z(B, T, H, dh), z(H, dh, dh), out=z(B, T - 1, H, dh))


def test_pack_and_rotate_pack_shapes():
    good = (z(B, T + 1, dtype=i32), z(B, H, cap, ds))
    reaches_device_check(rs.pack_kv, z(B, T, H, dh), z(B, T, dtype=i32), G, cap, out=good)
    refused(rs.pack_kv, z(B, T, H, dh), z(B, T, dtype=u8), G, cap)                    # byte mask
    refused(rs.pack_kv, z(B, T, H, dh), z(B, T + 1, dtype=i32), G, cap)               # mask length
    refused(rs.pack_kv, z(B, T, H, dh), z(B, T, dtype=i32), G, cap,
            out=(z(B, T, dtype=i32), good[1]))                                        # offsets [B,T]
    refused(rs.pack_kv, z(B, T, H, dh), z(B, T, dtype=i32), G, cap,
            out=(good[0], z(B, H, cap - 1, ds)))                                      # fewer slots than cap
    reaches_device_check(rs.rotate_pack, z(B, T, H, dh), z(H, dh, dh), z(B, T, dtype=i32), G, cap, out=good)
    refused(rs.rotate_pack, z(B, T, H, dh), z(H, dh, dh), z(B, T, dtype=i32), G, cap + 5, out=good)
    refused(rs.rotate_pack, z(B, T, H, dh), z(H, dh, dh // 2), z(B, T, dtype=i32), G, cap, out=good)


def _attend_args():
    return dict(q=z(B, Tq, H, dh), k=z(B, T, H, dh), mask=z(B, T, dtype=i32), offsets=z(B, T + 1, dtype=i32),
                Vp=z(B, H, cap, ds), R=z(H, dh, dh))


@pytest.mark.parametrize("name,bad", [
    ("k", z(B, T, H, dh // 2)), ("k", z(B + 1, T, H, dh)), ("mask", z(B, T, dtype=u8)),
    ("mask", z(B, T - 1, dtype=i32)), ("offsets", z(B, T, dtype=i32)), ("Vp", z(B, H, cap, ds + 1)),
    ("Vp", z(B, H - 1, cap, ds)), ("R", z(H, dh, dh - 1)), ("R", z(H, dh, dh, dtype=f32)),
])
def test_attend_shapes(name, bad):
    a = _attend_args()
    reaches_device_check(rs.attend, a["q"], a["k"], a["mask"], a["offsets"], a["Vp"], a["R"], G)
    a[name] = bad
    refused(rs.attend, a["q"], a["k"], a["mask"], a["offsets"], a["Vp"], a["R"], G)


def test_attend_out_and_causal_shapes():
    a = _attend_args()
    refused(rs.attend, a["q"], a["k"], a["mask"], a["offsets"], a["Vp"], a["R"], G, out=z(B, Tq + 1, H, dh))
    c = dict(a, q=z(B, T, H, dh))
    reaches_device_check(rs.attend_causal, c["q"], c["k"], c["mask"], c["offsets"], c["Vp"], c["R"], G)
    refused(rs.attend_causal, a["q"], a["k"], a["mask"], a["offsets"], a["Vp"], a["R"], G)   # Tq != T
    refused(rs.attend_causal, c["q"], c["k"], c["mask"], c["offsets"], c["Vp"], c["R"], G, out=z(B, T, H, 2 * dh))


def _router(C=4, d_e=16, Hr=32, dtype=bf):
    return rs.Router.mlp2(z(C, d, dtype=dtype), z(C, dtype=dtype), z(C, d_e, dtype=dtype),
                          z(Hr, 2 * d + d_e, dtype=dtype), z(Hr, dtype=dtype), z(G, Hr, dtype=dtype),
                          z(G, dtype=dtype))


def test_route_shapes():
    tt = z(B, T, dtype=u8)
    bu = rs.make_budget(rs.TOPK, (2, 3, 8, 8))
    reaches_device_check(rs.route, tt, bu, G, scores_in=z(B, T, G, dtype=f32))
    reaches_device_check(rs.route, tt, bu, G, h=z(B, T, d), router=_router())
    refused(rs.route, z(B, T, dtype=i32), bu, G, scores_in=z(B, T, G, dtype=f32))      # types not bytes
    refused(rs.route, tt, bu, G, scores_in=z(B, T, G + 1, dtype=f32))
    refused(rs.route, tt, bu, G, scores_in=z(B, T, G, dtype=bf))
    refused(rs.route, tt, bu, G, h=z(B, T + 1, d), router=_router())
    refused(rs.route, tt, bu, G, h=z(B, T, d), router=_router(dtype=f32))               # weights in another dtype
    r = _router()
    r.tensors["W2"] = z(G - 1, 32)
    refused(rs.route, tt, bu, G, h=z(B, T, d), router=r)
    refused(rs.route, tt, bu, G, scores_in=z(B, T, G, dtype=f32), out={"mask": z(B, T, dtype=u8)})
    refused(rs.route, tt, bu, G, scores_in=z(B, T, G, dtype=f32), out={"idx": z(B, T, G - 1, dtype=u8)})
    refused(rs.route, tt, bu, G, scores_in=z(B, T, G, dtype=f32), out={"scores": z(B, T, G, dtype=bf)})
    refused(rs.route, tt, bu, G, h=z(B, T, d), router=_router(), workspace=z(64, dtype=f32))


def test_allocation_shapes():
    tt = z(B, T, dtype=u8)
    reaches_device_check(rs.allocate_groups, z(B, T, dtype=f32), tt, (2, 3, 8, 8), G, scores=z(B, T, G, dtype=f32))
    refused(rs.allocate_groups, z(B, T + 1, dtype=f32), tt, (2, 3, 8, 8), G)
    refused(rs.allocate_groups, z(B, T, dtype=bf), tt, (2, 3, 8, 8), G)
    refused(rs.allocate_groups, z(B, T, dtype=f32), tt, (2, 3, 8, 8), G, scores=z(B, T, 2 * G, dtype=f32))
    refused(rs.allocate_groups, z(B, T, dtype=f32), tt, (2, 3, 8, 8), G, out={"k": z(B, T, dtype=i32)})
    reaches_device_check(rs.route_allocate, tt, (2, 3, 8, 8), G, z(B, T, d), _router(), z(4))
    refused(rs.route_allocate, tt, (2, 3, 8, 8), G, z(B, T, d), _router(), z(5))          # one weight per role
    refused(rs.route_allocate, tt, (2, 3, 8, 8), G, z(B, T, d), _router(), z(4),
            out={"priority": z(B, T - 1, dtype=f32)})


def test_retention_shapes():
    reaches_device_check(rs.retain_tokens, z(B, 12, dtype=f32), [6, 6], [2, 3])
    refused(rs.retain_tokens, z(B, 12, dtype=bf), [6, 6], [2, 3])
    refused(rs.retain_tokens, z(B, 12, dtype=f32), [6, 6], [2, 3], out=z(B, 4, dtype=i32))
    refused(rs.retain_tokens, z(B, 12, dtype=f32), [6, 6], [2], match="segments")
    reaches_device_check(rs.gather_tokens, z(B, 12, 7), z(B, 5, dtype=i32))
    refused(rs.gather_tokens, z(B, 12, 7), z(B, 5, dtype=torch.int64))
    refused(rs.gather_tokens, z(B, 12, 7), z(B + 1, 5, dtype=i32))
    refused(rs.gather_tokens, z(B, 12, 7), z(B, 5, dtype=i32), out=z(B, 5, 8))


def test_full_width_shapes():
    S, dv = 4, H * dh
    good = (z(B, T + 1, dtype=i32), z(B, cap, dv // S))
    reaches_device_check(rs.full_transpose, z(dv, dv))
    refused(rs.full_transpose, z(dv, dv - 1))
    reaches_device_check(rs.full_rotate_pack, z(B, T, H, dh), z(dv, dv), z(B, T, dtype=i32), S, cap, out=good)
    refused(rs.full_rotate_pack, z(B, T, H, dh), z(dv, dv // 2), z(B, T, dtype=i32), S, cap, out=good)
    refused(rs.full_rotate_pack, z(B, T, H, dh), z(dv, dv), z(B, T, dtype=i32), S, cap - 1, out=good)
    reaches_device_check(rs.full_values, z(dv, dv), z(B, T, dtype=i32), good[0], good[1], S, H)
    refused(rs.full_values, z(dv, dv), z(B, T + 2, dtype=i32), good[0], good[1], S, H)
    refused(rs.full_values, z(dv, dv), z(B, T, dtype=i32), good[0], good[1], S, H, out=z(B, H, T, dh + 1))
    refused(rs.full_values, z(dv, dv), z(B, T, dtype=i32), good[0], good[1], S, 3, match="heads")
    reaches_device_check(rs.attend_values, z(B, Tq, H, dh), z(B, T, H, dh), z(B, H, T, dh))
    refused(rs.attend_values, z(B, Tq, H, dh), z(B, T, H, dh), z(B, T, H, dh))            # token-major values


def test_micro_batches_and_buffer_rows():
    from paper_2608_18410_amd.pipeline import LayerBuffers, micro_batches
    assert micro_batches(64, 2) == [(0, 32), (32, 64)]
    assert micro_batches(8, 3) == [(0, 2), (2, 5), (5, 8)]
    assert micro_batches(2, 5) == [(0, 1), (1, 2)]      # never more ranges than prefixes
    assert micro_batches(7, 0) == [(0, 7)]
    for B, n in ((64, 2), (177, 7), (5, 5)):
        r = micro_batches(B, n)
        assert r[0][0] == 0 and r[-1][1] == B and all(a[1] == b[0] for a, b in zip(r, r[1:]))
        assert max(b1 - b0 for b0, b1 in r) - min(b1 - b0 for b0, b1 in r) <= 1
    bufs = LayerBuffers.allocate(5, 7, 2, 64, 4, 3, 9, torch.bfloat16, ws_bytes=1024, device="cpu", with_z=False)
    ws = torch.empty(512, dtype=torch.uint8)
    v = bufs.rows(1, 4, ws)
    assert v.mask.shape == (3, 7) and v.offsets.shape == (3, 8) and v.Vp.shape == (3, 2, 9, 16)
    assert v.out.shape == (3, 3, 2, 64) and v.workspace is ws and v.z.numel() == 0
    assert v.mask.data_ptr() == bufs.mask[1].data_ptr() and v.Vp.is_contiguous()
