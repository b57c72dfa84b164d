"""GPU parity of librolesub against the float64 oracle, through the C ABI.

Bars: integer/index/byte outputs (masks, idx, counts, offsets, packed cache)
bit-exact; f32 outputs within 1e-4 and bf16 outputs within 2e-2 maximum
relative error (max |x - ref| / max |ref| over the tensor). The oracle takes
the same seeded inputs and never sees a GPU result; when routing scores come
from the GPU router, masks must match on every token whose decisive margin
exceeds 8x the observed score error (near-margin tokens are reported).
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2608_18410_amd as rs
import synth
from paper_2608_18410_amd.pipeline import LayerBuffers, pack_capacity, run_layer
from tests._gpu_util import (DEV, TOL, decisive_margin, host, host_mask, layer_on_device, max_rel, put,
                             put_mask, put_u8, router_tensors, stack_types, synth_pack_inputs, tdtype)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    rs.load()   # fails loudly if the library is not built


def _say(*a):
    print(*a, flush=True)


# ----------------------------------------------------------------------------
# Group selection from given scores: bit-exact
# ----------------------------------------------------------------------------

def _check_selection(scores, types, budget, G, mode, kbt, tau=0.0, kmin=0, kmax=0):
    B, T = types.shape
    r = rs.route(put_u8(types), budget, G, scores_in=put(scores, torch.float32))
    torch.cuda.synchronize()
    K = O.group_budget(scores, types, mode, kbt, G, tau, kmin, kmax)
    want = O.select_groups(scores, K)
    got = host_mask(r["mask"])
    assert np.array_equal(got, want), f"{int(np.sum(got != want))} masks differ"
    idx, cnt = O.mask_to_idx(want, G)
    assert np.array_equal(host(r["count"]), cnt)
    assert np.array_equal(host(r["idx"]), idx)
    assert np.array_equal(host(r["scores"]).view(np.uint32), scores.view(np.uint32))   # passed through bit for bit


def test_select_threshold_stress_logits():
    w = synth.workload(5)
    B = 4
    scores = np.stack([synth.sample_scores(w, 0, b) for b in range(B)])
    types = stack_types(w, B)
    bu = rs.make_budget(rs.THRESHOLD, (0, 0, 0, 0), 0.0, 1, 32)
    _say("select: threshold stress, 4 x 2048 tokens, G=32")
    _check_selection(scores, types, bu, 32, O.THRESHOLD, (0, 0, 0, 0), 0.0, 1, 32)


def test_select_topk_ties_zero_signs_nan():
    r = np.random.default_rng(7)
    G, B, T = 8, 3, 333
    grid = np.array([-1.0, -0.5, -0.0, 0.0, 0.5, 1.0, np.nan, np.inf, -np.inf], dtype=np.float32)
    scores = grid[r.integers(0, len(grid), size=(B, T, G))]
    scores[1] = r.standard_normal((T, G)).astype(np.float32)
    types = r.integers(0, 4, size=(B, T)).astype(np.uint8)
    kbt = (2, 5, 8, 0)
    _say("select: top-k with ties, signed zeros, NaN, infinities")
    _check_selection(scores, types, rs.make_budget(rs.TOPK, kbt), G, O.TOPK, kbt)


@pytest.mark.parametrize("G,kmin,kmax", [(16, 2, 5), (32, 0, 32), (5, 1, 1)])
def test_select_threshold_clamps(G, kmin, kmax):
    r = np.random.default_rng(G)
    B, T = 2, 517
    scores = (r.integers(-3, 4, size=(B, T, G)) * 0.25).astype(np.float32)
    types = np.zeros((B, T), dtype=np.uint8)
    bu = rs.make_budget(rs.THRESHOLD, (0, 0, 0, 0), 0.0, kmin, kmax)
    _check_selection(scores, types, bu, G, O.THRESHOLD, (0, 0, 0, 0), 0.0, kmin, kmax)


@pytest.mark.parametrize("G,fo,bo", [(16, 1, 3), (32, 2, 1), (16, 0, 0), (5, 1, 2), (5, 0, 0)])
def test_select_unaligned_buffers(G, fo, bo):
    """Scores and idx buffers starting fo floats / bo bytes past a 16-byte
    boundary, with a ragged last workgroup (T = 300)."""
    r = np.random.default_rng(100 + G + fo)
    B, T = 1, 300
    n = B * T * G
    scores = r.standard_normal((B, T, G)).astype(np.float32)
    types = r.integers(0, 4, size=(B, T)).astype(np.uint8)
    kbt = (1, 3, G // 2, G)
    base_in = torch.zeros(n + 4, dtype=torch.float32, device=DEV)
    base_out = torch.zeros(n + 4, dtype=torch.float32, device=DEV)
    base_idx = torch.zeros(n + 16, dtype=torch.uint8, device=DEV)
    s_in = base_in[fo:fo + n].view(B, T, G)
    s_in.copy_(put(scores, torch.float32))
    out = {"scores": base_out[fo:fo + n].view(B, T, G), "idx": base_idx[bo:bo + n].view(B, T, G)}
    res = rs.route(put_u8(types), rs.make_budget(rs.TOPK, kbt), G, scores_in=s_in, out=out)
    torch.cuda.synchronize()
    want = O.select_groups(scores, O.group_budget(scores, types, O.TOPK, kbt, G, 0.0, 0, 0))
    assert np.array_equal(host_mask(res["mask"]), want)
    idx, _ = O.mask_to_idx(want, G)
    assert np.array_equal(host(res["idx"]), idx)
    assert np.array_equal(host(res["scores"]).view(np.uint32), scores.view(np.uint32))
    # nothing written around the views
    assert not host(base_out[:fo]).any() and not host(base_out[fo + n:]).any()
    assert not host(base_idx[:bo]).any() and not host(base_idx[bo + n:]).any()


# ----------------------------------------------------------------------------
# Pack: bit-exact
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cid,B,T,H,dh,G", [
    (1, 1, 80, 4, 64, 8),        # f32, 32-byte groups
    (2, 1, 305, 32, 128, 8),     # bf16, 32-byte groups, 7B layer shape
    (3, 3, 77, 8, 128, 8),       # ragged token count
    (5, 2, 301, 9, 128, 32),     # bf16, 8-byte groups, heads not a multiple of 8
    (5, 2, 70, 4, 64, 32),       # bf16, 4-byte groups
])
def test_pack_bit_exact(cid, B, T, H, dh, G):
    w = synth.workload(cid).replace(n_vis=T, n_lang=0, n_prop=0, H=H, dh=dh, G=G)
    z, m = synth_pack_inputs(w, B)
    dt = tdtype(w)
    cap = T * G
    zd = put(z, dt)
    Vp = torch.full((B, H, cap, dh // G), 7.0, dtype=dt, device=DEV)
    off = torch.empty((B, T + 1), dtype=torch.int32, device=DEV)
    rs.pack_kv(zd, put_mask(m), G, cap, out=(off, Vp))
    torch.cuda.synchronize()
    o_ref, Vp_ref = O.pack(z, m, G, cap)
    assert np.array_equal(host(off), o_ref)
    got = host(Vp)
    for b in range(B):
        n = int(o_ref[b, -1])
        assert np.array_equal(got[b, :, :n], Vp_ref[b, :, :n])
        assert np.all(got[b, :, n:] == 7.0)          # slots past the total untouched


def test_pack_capacity_clips_writes():
    w = synth.workload(2).replace(H=8)
    B, G = 2, 8
    z, m = synth_pack_inputs(w, B)
    budget = w.n_vis * w.k_vis + w.n_lang * w.k_lang + w.n_prop * G
    cap = budget - 50
    Vp = torch.zeros((B, 8, cap, 16), dtype=torch.bfloat16, device=DEV)
    off = torch.empty((B, w.T + 1), dtype=torch.int32, device=DEV)
    rs.pack_kv(put(z, torch.bfloat16), put_mask(m), G, cap, out=(off, Vp))
    torch.cuda.synchronize()
    o_ref, Vp_ref = O.pack(z, m, G, cap)
    assert np.array_equal(host(off), o_ref) and int(o_ref[0, -1]) == budget
    assert np.array_equal(host(Vp), Vp_ref)
    with pytest.raises(rs.RolesubError) as e:
        rs.pack_kv(put(z, torch.bfloat16), put_mask(m), G, cap,
                   budget=rs.make_budget(rs.TOPK, w.k_by_type), type_counts=w.type_counts())
    assert e.value.status == 3


# ----------------------------------------------------------------------------
# Rotation
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cid,B,T,H,dh", [(1, 1, 80, 4, 64), (2, 1, 305, 32, 128), (3, 2, 113, 8, 64),
                                          (3, 3, 1000, 32, 128)])
def test_rotate(cid, B, T, H, dh):
    w = synth.workload(cid).replace(B=B, n_vis=T, n_lang=0, n_prop=0, H=H, dh=dh)
    dt = tdtype(w)
    R = synth.layer_weights(w, 0)["R"]
    v = np.stack([synth.sample_activations(w, 0, b, ("v",))["v"] for b in range(B)])
    z = rs.rotate_values(put(v, dt), put(R, dt))
    torch.cuda.synchronize()
    err = max_rel(host(z), O.rotate(v, R))
    _say(f"rotate {w.dtype} B={B} T={T} H={H} dh={dh}: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]


# ----------------------------------------------------------------------------
# Fused rotation + pack
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cid,B,T,H,dh,G", [
    (1, 1, 80, 4, 64, 8),        # f32 (vector kernel)
    (2, 1, 305, 32, 128, 8),     # bf16, 16-dim groups, 7B layer shape
    (3, 3, 77, 8, 128, 8),       # ragged token count
    (5, 2, 301, 9, 128, 32),     # 4-dim groups, heads not a multiple of 8
    (5, 2, 70, 4, 64, 32),       # 2-dim groups
    (3, 2, 150, 8, 64, 4),       # head dim 64, 16-dim groups
    # the offsets the matrix-core kernel forms for its run of tokens:
    (3, 300, 1, 4, 128, 8),      # one token per sample: 64 samples start inside each run
    (3, 3, 500, 4, 64, 8),       # 64-token runs inside 500-token samples (counts carried from the sample start)
    (3, 2, 512, 4, 64, 8),       # the longest prefix whose offsets the kernel forms itself
    (3, 2, 513, 4, 64, 8),       # one token more: offsets from the scan kernel
    (2, 2, 2000, 32, 128, 8),    # prefixes past 512 tokens: offsets from the scan kernel
    (3, 30, 177, 64, 64, 8),     # runs over two to four samples, ragged last run
])
def test_rotate_pack_fused(cid, B, T, H, dh, G):
    w = synth.workload(cid).replace(B=B, n_vis=T, n_lang=0, n_prop=0, H=H, dh=dh, G=G)
    dt = tdtype(w)
    R = synth.layer_weights(w, 0)["R"]
    v = np.stack([synth.sample_activations(w, 0, b, ("v",))["v"] for b in range(B)])
    m = np.stack([synth.synthetic_masks(w, 0, b, counts=np.random.default_rng(b).integers(0, G + 1, T))
                  for b in range(B)])
    cap = T * G
    vd, Rd, md = put(v, dt), put(R, dt), put_mask(m)
    off_f, Vp_f = rs.rotate_pack(vd, Rd, md, G, cap)
    z = rs.rotate_values(vd, Rd)
    off_u, Vp_u = rs.pack_kv(z, md, G, cap)
    torch.cuda.synchronize()
    o_ref, Vp_ref = O.pack(O.rotate(v, R), m, G, cap)
    assert np.array_equal(host(off_f), o_ref)
    got, unf = host(Vp_f), host(Vp_u)
    for b in range(B):
        n = int(o_ref[b, -1])
        assert np.array_equal(got[b, :, :n], unf[b, :, :n])      # same values as rotate then pack
        if n:
            err = max_rel(got[b, :, :n], Vp_ref[b, :, :n])
            assert err <= TOL[w.dtype], err
    _say(f"rotate_pack {w.dtype} B={B} T={T} H={H} dh={dh} G={G}: ok")


# ----------------------------------------------------------------------------
# Attention over the packed cache
# ----------------------------------------------------------------------------

def _attend_case(w, B, T, Tq, H, dh, G, counts=None, out_dtype=None, seed=0, scale=None):
    w = w.replace(B=B, n_vis=T, n_lang=0, n_prop=0, Tq=Tq, H=H, dh=dh, G=G)
    dt = tdtype(w)
    acts = [synth.sample_activations(w, seed, b, ("q", "k")) for b in range(B)]
    q = np.stack([a["q"] for a in acts])
    k = np.stack([a["k"] for a in acts])
    z = np.stack([synth.synthetic_z(w, seed, b) for b in range(B)])
    m = np.stack([synth.synthetic_masks(w, seed, b, counts=counts) for b in range(B)])
    R = synth.layer_weights(w, seed)["R"]
    cap = T * G
    off, Vp = rs.pack_kv(put(z, dt), put_mask(m), G, cap)
    out = rs.attend(put(q, dt), put(k, dt), put_mask(m), off, Vp, put(R, dt), G, out_dtype=out_dtype,
                    scale=0.0 if scale is None else scale)
    torch.cuda.synchronize()
    o_ref, Vp_ref = O.pack(z, m, G, cap)
    ref = O.attend_packed(q, k, m, o_ref, Vp_ref, R, G, scale=scale)
    return host(out), ref, (q, k, z, m, R)


@pytest.mark.parametrize("cid,B,T,Tq,H,dh,G", [
    (1, 1, 80, 8, 4, 64, 8),           # tiny f32 (vector kernel)
    (2, 1, 305, 56, 32, 128, 8),       # 7B layer shape (matrix cores)
    (3, 3, 113, 56, 32, 128, 8),
    (5, 2, 301, 70, 8, 128, 32),       # G=32 (4-dim groups), 2 query blocks, ragged T
    (3, 2, 97, 20, 8, 64, 8),          # head dim 64 on matrix cores
    (3, 2, 65, 16, 8, 64, 32),         # 2-dim groups
    (1, 2, 33, 3, 4, 128, 4),          # f32, head dim 128
    (3, 301, 70, 20, 4, 128, 8),       # runs of 3 samples per workgroup, last run shorter
    (3, 150, 40, 9, 8, 64, 16),        # one tile per sample: every tile starts and ends one
    (3, 2, 5, 3, 4, 128, 8),           # fewer tokens than one tile, one partial query block
    (5, 2, 31, 17, 8, 128, 32),        # one token short of a tile, 4-dim groups
    (3, 1, 1, 1, 4, 64, 8),            # a single token and a single query
])
def test_attend(cid, B, T, Tq, H, dh, G):
    w = synth.workload(cid)
    counts = np.random.default_rng(T).integers(0, G + 1, size=T)
    got, ref, _ = _attend_case(w, B, T, Tq, H, dh, G, counts=counts)
    err = max_rel(got, ref)
    _say(f"attend {w.dtype} B={B} T={T} Tq={Tq} H={H} dh={dh} G={G}: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]


def _attend_causal_case(w, B, T, H, dh, G, counts=None, out_dtype=None, seed=0, scale=None):
    w = w.replace(B=B, n_vis=T, n_lang=0, n_prop=0, Tq=T, H=H, dh=dh, G=G)
    dt = tdtype(w)
    acts = [synth.sample_activations(w, seed, b, ("q", "k")) for b in range(B)]
    q = np.stack([a["q"] for a in acts])
    k = np.stack([a["k"] for a in acts])
    z = np.stack([synth.synthetic_z(w, seed, b) for b in range(B)])
    m = np.stack([synth.synthetic_masks(w, seed, b, counts=counts) for b in range(B)])
    R = synth.layer_weights(w, seed)["R"]
    cap = T * G
    off, Vp = rs.pack_kv(put(z, dt), put_mask(m), G, cap)
    out = rs.attend_causal(put(q, dt), put(k, dt), put_mask(m), off, Vp, put(R, dt), G, out_dtype=out_dtype,
                           scale=0.0 if scale is None else scale)
    torch.cuda.synchronize()
    o_ref, Vp_ref = O.pack(z, m, G, cap)
    ref = O.attend_packed_causal(q, k, m, o_ref, Vp_ref, R, G, scale=scale)
    return host(out), ref


@pytest.mark.parametrize("cid,B,T,H,dh,G", [
    (1, 1, 80, 4, 64, 8),              # tiny f32 (vector kernel)
    (1, 2, 33, 4, 128, 4),             # f32, head dim 128
    (2, 1, 305, 32, 128, 8),           # 7B layer shape: 5 query blocks, ragged T
    (3, 3, 113, 8, 128, 8),
    (5, 2, 150, 8, 128, 32),           # 4-dim groups
    (3, 2, 97, 8, 64, 8),              # head dim 64
    (3, 2, 65, 4, 64, 32),             # 2-dim groups
    (3, 2, 32, 4, 128, 8),             # one full tile
    (3, 2, 33, 4, 128, 8),             # a tile plus one token
    (3, 3, 1, 4, 128, 8),              # one token: its own routed value
])
def test_attend_causal(cid, B, T, H, dh, G):
    w = synth.workload(cid)
    counts = np.random.default_rng(T + 7).integers(0, G + 1, size=T)
    counts[0] = max(int(counts[0]), 1)
    got, ref = _attend_causal_case(w, B, T, H, dh, G, counts=counts)
    err = max_rel(got, ref)
    _say(f"attend_causal {w.dtype} B={B} T={T} H={H} dh={dh} G={G}: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]


@pytest.mark.parametrize("cid,B,T,Tq,H,dh,G,scale", [
    (2, 2, 177, 56, 8, 128, 8, 0.25),          # matrix cores, a stated positive scale
    (2, 2, 177, 56, 8, 128, 8, -0.0625),       # negative scale: scores of the opposite sign
    (5, 2, 90, 20, 4, 128, 32, -0.3),          # 4-dim groups
    (3, 2, 97, 20, 8, 64, 8, 0.5),             # head dim 64
    (1, 1, 80, 8, 4, 64, 8, -0.2),             # f32 (vector kernel)
])
def test_attend_explicit_scale(cid, B, T, Tq, H, dh, G, scale):
    w = synth.workload(cid)
    counts = np.random.default_rng(T + 3).integers(0, G + 1, size=T)
    got, ref, _ = _attend_case(w, B, T, Tq, H, dh, G, counts=counts, scale=scale)
    err = max_rel(got, ref)
    _say(f"attend scale={scale} {w.dtype} B={B} T={T} Tq={Tq} dh={dh} G={G}: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]
    # the default (1/sqrt(dh)) gives a different result: the scale is really applied
    base, _, _ = _attend_case(w, B, T, Tq, H, dh, G, counts=counts)
    assert max_rel(got, base) > 10 * TOL[w.dtype]


@pytest.mark.parametrize("cid,scale", [(2, -0.125), (2, 0.3), (1, -0.4)])
def test_attend_causal_explicit_scale(cid, scale):
    w = synth.workload(cid)
    counts = np.random.default_rng(11).integers(1, 9, size=70)
    got, ref = _attend_causal_case(w, 2, 70, 4, 128 if cid == 2 else 64, 8, counts=counts, scale=scale)
    err = max_rel(got, ref)
    _say(f"attend_causal scale={scale} {w.dtype}: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]


def test_attend_causal_stack_shape_and_f32_output():
    w = synth.workload(4)
    counts = np.array([4] * 128 + [6] * 48 + [8])
    got, ref = _attend_causal_case(w, 2, 177, 32, 128, 8, counts=counts)
    err = max_rel(got, ref)
    _say(f"attend_causal 7B-stack shape B=2: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]
    got, ref = _attend_causal_case(w, 2, 177, 8, 128, 8, counts=counts, out_dtype=torch.float32)
    assert max_rel(got, ref) <= TOL[w.dtype]


# ----------------------------------------------------------------------------
# Token retention and the retained prefix
# ----------------------------------------------------------------------------

def _retention_scores(seed, B, N):
    r = np.random.default_rng(seed)
    sc = r.standard_normal((B, N)).astype(np.float32)
    sc[:, ::5] = np.round(sc[:, ::5])               # exact ties
    sc[:, 1::7] = 0.0
    sc[:, 3::7] = -0.0                              # -0 equals +0
    sc[:, 2::11] = np.nan                           # NaN ranks after every number
    return sc


@pytest.mark.parametrize("B,seg_len,seg_keep", [
    (64, [256, 256], [64, 64]),                     # 7B stack: 128 of 512 visual tokens, two views
    (16, [256, 256], [4, 4]),                       # the paper's 8 of 512
    (3, [256] * 7 + [256], [16] * 7 + [256]),       # seven views, language kept whole
    (2, [5, 0, 300, 1], [0, 0, 300, 1]),            # keep none / all / empty segment
    (2, [1] * 16, [1, 0] * 8),                      # sixteen segments
    (2, [8192], [1000]),                            # the longest segment
])
def test_retain_tokens_bit_exact(B, seg_len, seg_keep):
    sc = _retention_scores(sum(seg_len) + B, B, sum(seg_len))
    got = host(rs.retain_tokens(torch.from_numpy(sc).to(DEV), seg_len, seg_keep))
    want = O.retain_tokens(sc, seg_len, seg_keep)
    _say(f"retain_tokens B={B} segments={len(seg_len)} kept={sum(seg_keep)}: "
         f"{int(np.sum(got != want))} mismatches")
    assert np.array_equal(got, want)


def test_gather_tokens_rows():
    r = np.random.default_rng(31)
    B, N, d = 4, 512, 4096
    x = synth.round_to(r.standard_normal((B, N, d)), "bf16")
    idx = O.retain_tokens(_retention_scores(32, B, N), [256, 256], [64, 64]).astype(np.int32)
    got = host(rs.gather_tokens(put(x, torch.bfloat16), torch.from_numpy(idx).to(DEV)))
    assert np.array_equal(got, O.gather_tokens(x, idx))
    # 12-byte rows (no 16-byte pieces) and indices outside [0, N) (zero rows)
    y = r.standard_normal((2, 9, 3)).astype(np.float32)
    idx2 = np.array([[0, 8, -1, 4], [9, 3, 3, 100]], dtype=np.int32)
    got2 = host(rs.gather_tokens(torch.from_numpy(y).to(DEV), torch.from_numpy(idx2).to(DEV)))
    for b in range(2):
        for j in range(4):
            t = idx2[b, j]
            assert np.array_equal(got2[b, j], y[b, t] if 0 <= t < 9 else np.zeros(3, np.float32))


# ----------------------------------------------------------------------------
# Role-driven within-type budget allocation (Sec. 3.5): bit-exact
# ----------------------------------------------------------------------------

def _alloc_inputs(w, B, types=None, seed_layer=0):
    pr = np.stack([synth.sample_priorities(w, seed_layer, b) for b in range(B)])
    if types is None:
        types = stack_types(w, B)
    return pr, types


def _check_allocation(pr, types, kby, G, scores=None, label=""):
    want_k = O.allocate_groups(pr, types, kby, G)
    r = rs.allocate_groups(torch.from_numpy(pr).to(DEV), put_u8(types), kby, G,
                           scores=None if scores is None else put(scores, torch.float32))
    torch.cuda.synchronize()
    got_k = host(r["k"])
    _say(f"allocate {label}: B={types.shape[0]} T={types.shape[1]} G={G} K_m={tuple(kby)}: "
         f"{int(np.sum(got_k != want_k))} K mismatches")
    assert np.array_equal(got_k, want_k)
    if scores is not None:
        want = O.select_groups(scores, want_k)
        assert np.array_equal(host_mask(r["mask"]), want)
        idx, cnt = O.mask_to_idx(want, G)
        assert np.array_equal(host(r["count"]), cnt)
        assert np.array_equal(host(r["idx"]), idx)


@pytest.mark.parametrize("cid,B,G,kby", [
    (4, 64, 8, (4, 6, 8, 8)),          # 7B stack: 128 visual, 48 language, 1 proprio token per prefix
    (3, 16, 8, (2, 4, 8, 8)),          # aggressive budgets
    (2, 2, 16, (3, 5, 1, 0)),          # 305 tokens, another G
    (1, 3, 32, (31, 1, 16, 7)),        # G = 32, near-full and near-empty types
    (1, 2, 1, (1, 0, 1, 1)),           # G = 1: no allocation possible
])
def test_allocate_groups_bit_exact(cid, B, G, kby):
    w = synth.workload(cid).replace(B=B)
    pr, types = _alloc_inputs(w, B)
    r = np.random.default_rng(cid)
    scores = r.standard_normal((B, w.T, G)).astype(np.float32)
    scores[:, ::3, : max(1, G // 2)] = 0.5                       # tied groups
    _check_allocation(pr, types, kby, G, scores, f"workload {cid}")
    _check_allocation(pr, types, kby, G, None, f"workload {cid}, K only")


def test_allocate_groups_edge_cases():
    w = synth.workload(1)
    r = np.random.default_rng(41)
    # random types including values outside the four (they keep every group)
    T = 600
    types = r.integers(0, 6, size=(5, T)).astype(np.uint8)
    pr = np.stack([synth.sample_priorities(w.replace(n_vis=T, n_lang=0), 1, b) for b in range(5)])
    pr[1] = 0.0                                                  # all-zero priorities: equal shares
    pr[2] = 2.5                                                  # uniform: the fixed K_m
    pr[3, ::2] = 1e6                                             # half the tokens clipped and capped
    _check_allocation(pr, types, (3, 5, 7, 1), 8, r.standard_normal((5, T, 8)).astype(np.float32), "mixed")
    # the longest prefix, one type
    T = 4096
    types = np.zeros((2, T), dtype=np.uint8)
    pr = np.stack([synth.sample_priorities(w.replace(n_vis=T, n_lang=0), 2, b) for b in range(2)])
    _check_allocation(pr, types, (5, 0, 0, 0), 16, None, "T=4096")
    # one token per sample
    _check_allocation(np.array([[3.0], [np.nan]], np.float32), np.zeros((2, 1), np.uint8), (2, 0, 0, 0), 8,
                      None, "T=1")
    # empty inputs are no-ops; sizes and budgets outside the limits are errors
    e = rs.allocate_groups(torch.empty((0, 5), device=DEV), torch.empty((0, 5), dtype=torch.uint8, device=DEV),
                           (1, 1, 1, 1), 8)
    assert e["k"].shape == (0, 5)
    with pytest.raises(rs.RolesubError, match="above 4096"):
        rs.allocate_groups(torch.zeros((1, 4097), device=DEV), torch.zeros((1, 4097), dtype=torch.uint8,
                                                                          device=DEV), (1, 1, 1, 1), 8)
    with pytest.raises(rs.RolesubError, match="outside 0..G"):
        rs.allocate_groups(torch.zeros((1, 8), device=DEV), torch.zeros((1, 8), dtype=torch.uint8, device=DEV),
                           (9, 1, 1, 1), 8)


def _route_allocate_check(w, B, router, wpri_np, prio_ref, score_ref, label):
    dt = tdtype(w)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)])
    types = stack_types(w, B)
    kby = tuple(w.k_by_type)
    r = rs.route_allocate(put_u8(types), kby, w.G, put(h, dt), router, put(wpri_np, dt))
    torch.cuda.synchronize()
    perr = max_rel(host(r["priority"]), prio_ref(h))
    serr = max_rel(host(r["scores"]), score_ref(h, types))
    # allocation and selection: the stated constraints on the GPU's own priorities and scores
    k = host(r["k"]).astype(np.int64)
    qp = np.floor(np.clip(np.nan_to_num(host(r["priority"]).astype(np.float64), nan=0.0), 0, 256) * 65536)
    for b in range(B):
        for m in range(4):
            i = np.nonzero(types[b] == m)[0]
            km = min(kby[m], w.G)
            assert k[b, i].sum() == km * len(i)
            hi = qp[b, i][:, None] > qp[b, i][None, :]
            assert np.all((k[b, i][:, None] >= k[b, i][None, :]) | ~hi)
    assert np.all((k >= 0) & (k <= w.G))
    mask = host_mask(r["mask"])
    assert np.array_equal(O.popcount(mask), k)
    assert np.array_equal(host(r["count"]), k)
    sc = host(r["scores"])
    bits = (mask[..., None] >> np.arange(w.G, dtype=np.uint32)) & 1
    lo_kept = np.where(bits == 1, sc, np.inf).min(-1)
    hi_drop = np.where(bits == 0, sc, -np.inf).max(-1)
    assert np.all(lo_kept >= hi_drop)
    # bit for bit: the oracle's allocation on the GPU's own float32 priorities
    # (integer arithmetic after an exact quantisation), then its Top-K_i on the
    # GPU's own scores, on every token
    want_k = O.allocate_groups(host(r["priority"]), types, kby, w.G)
    assert np.array_equal(k, want_k), f"{int(np.sum(k != want_k))} budgets differ"
    want = O.select_groups(sc, want_k)
    assert np.array_equal(mask, want)
    idx, cnt = O.mask_to_idx(want, w.G)
    assert np.array_equal(host(r["count"]), cnt) and np.array_equal(host(r["idx"]), idx)
    # end to end: budgets from the oracle's float64 priorities (a last-bit
    # difference in a priority may move one group, so this is reported)
    agree = float(np.mean(k == O.allocate_groups(prio_ref(h).astype(np.float32), types, kby, w.G)))
    _say(f"route_allocate {label}: priority max rel err {perr:.2e}, scores {serr:.2e}; "
         f"K equal to the oracle's from its own priorities on {100 * agree:.1f}% of tokens")
    assert perr <= 1e-4 and serr <= 1e-4


@pytest.mark.parametrize("cid,B", [(4, 8), (2, 1), (1, 2)])
def test_route_allocate(cid, B):
    w = synth.workload(cid).replace(B=B)
    wt = synth.layer_weights(w, 0)
    wpri = synth.priority_weights(w, 0)
    prio = lambda hh: O.role_priority(hh, wt["W_r"], wt["b_r"], wpri)
    ref = lambda hh, tt: O.router_mlp2(hh, tt, wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"],
                                       wt["W2"], wt["b2"])
    _route_allocate_check(w, B, router_tensors(wt, tdtype(w)), wpri, prio, ref, f"mlp2 workload {cid} B={B}")


def test_route_allocate_additive_router():
    w = synth.workload(2).replace(B=2, d=512, G=16, C=6, n_vis=40, n_lang=9, n_prop=1, k_vis=3, k_lang=5,
                                  k_prop=16)
    aw = synth.additive_weights(w, 0)
    wpri = synth.priority_weights(w, 0)
    router = rs.Router.additive(*(put(aw[n], torch.bfloat16) for n in ("W_tok", "b_tok", "W_r", "b_r", "W_role",
                                                                       "W_lang", "b_lang")))
    prio = lambda hh: O.role_priority(hh, aw["W_r"], aw["b_r"], wpri)
    ref = lambda hh, tt: O.router_additive(hh, tt, aw["W_tok"], aw["b_tok"], aw["W_r"], aw["b_r"],
                                           aw["W_role"], aw["W_lang"], aw["b_lang"], 0.1, 0.1)
    _route_allocate_check(w, 2, router, wpri, prio, ref, "additive bf16")


def test_attend_stack_layer_shape():
    # the 7B-stack layer shape with its per-type kept counts (4 of 8 groups for
    # 128 visual tokens, 6 for 48 language tokens, all 8 for the proprio token)
    w = synth.workload(4)
    counts = np.array([4] * 128 + [6] * 48 + [8])
    got, ref, _ = _attend_case(w, 4, 177, 56, 32, 128, 8, counts=counts)
    err = max_rel(got, ref)
    _say(f"attend 7B-stack layer shape, B=4: max rel err {err:.2e}")
    assert err <= TOL[w.dtype]


@pytest.mark.parametrize("B,H", [(2, 16), (70, 8)])
def test_attend_f32_output_from_bf16(B, H):
    w = synth.workload(2)
    got, ref, _ = _attend_case(w, B, 150, 56, H, 128, 8, out_dtype=torch.float32)
    err = max_rel(got, ref)
    _say(f"attend bf16 in, f32 out B={B} H={H}: max rel err {err:.2e}")
    assert err <= 2e-2


def test_attend_no_groups_is_zero_and_all_groups_is_standard_attention():
    w = synth.workload(2)
    T, G = 90, 8
    got0, _, _ = _attend_case(w, 1, T, 56, 8, 128, G, counts=np.zeros(T, dtype=int))
    assert np.all(got0 == 0.0)
    got, _, (q, k, z, m, R) = _attend_case(w, 1, T, 56, 8, 128, G, counts=np.full(T, G))
    v = O.back_rotate(z, R)        # the values whose rotation is z
    s = np.einsum("bqhd,bthd->bhqt", q, k) / np.sqrt(128)
    ref = np.einsum("bhqt,bthd->bqhd", O.softmax(s, -1), v)
    err = max_rel(got, ref)
    _say(f"attend all groups vs standard attention: max rel err {err:.2e}")
    assert err <= 2e-2


# ----------------------------------------------------------------------------
# Router end to end (scores from h)
# ----------------------------------------------------------------------------

def _exact_selection_on_own_scores(w, types, got_scores, got_mask, got_count=None, got_idx=None, K=None):
    """The selection the GPU made, bit for bit on every token: the oracle's
    Top-K_i run on the GPU's own float32 scores (exactly upcast) must give the
    GPU's masks, counts and kept-group lists. K defaults to the budget rule on
    those scores (fixed per-type budgets, or the threshold count)."""
    if K is None:
        K = O.group_budget(got_scores, types, w.mode, w.k_by_type, w.G, w.tau, w.kmin, w.kmax)
    want = O.select_groups(got_scores, K)
    bad = int(np.sum(got_mask != want))
    assert bad == 0, f"{bad} tokens select other groups than the oracle on the GPU's own scores"
    if got_count is not None or got_idx is not None:
        idx, cnt = O.mask_to_idx(want, w.G)
        if got_count is not None:
            assert np.array_equal(got_count, cnt)
        if got_idx is not None:
            assert np.array_equal(got_idx, idx)
    return want

def _route_check(w, h, types, router, wt_or_scores_fn, label):
    dt = tdtype(w)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    r = rs.route(put_u8(types), budget, w.G, h=put(h, dt), router=router)
    torch.cuda.synchronize()
    ref_scores = wt_or_scores_fn(h, types)
    got_scores = host(r["scores"])
    serr = max_rel(got_scores, ref_scores)
    abs_err = float(np.max(np.abs(got_scores - ref_scores)))
    K = O.group_budget(ref_scores, types, w.mode, w.k_by_type, w.G, w.tau, w.kmin, w.kmax)
    want = O.select_groups(ref_scores, K)
    got = host_mask(r["mask"])
    margin = decisive_margin(ref_scores, K, w.tau if w.mode == O.THRESHOLD else None)
    safe = margin > 8 * abs_err
    n_near = int(np.sum(~safe))
    _say(f"route {label}: score max rel err {serr:.2e} (abs {abs_err:.1e}); "
         f"{n_near} near-margin tokens of {safe.size}; mismatches on safe tokens "
         f"{int(np.sum((got != want) & safe))}")
    assert serr <= 1e-4
    # (i) bit-exact on every token against the oracle's selection on the GPU's scores
    _exact_selection_on_own_scores(w, types, got_scores, got, host(r["count"]), host(r["idx"]))
    # (ii) end to end against the oracle's own float64 scores, wherever the margin decides
    assert np.array_equal(got[safe], want[safe])
    assert np.array_equal(host(r["count"])[safe], O.popcount(want)[safe])
    idx_ref, _ = O.mask_to_idx(want, w.G)
    assert np.array_equal(host(r["idx"])[safe], idx_ref[safe])
    return r


@pytest.mark.parametrize("cid,B", [(1, 1), (2, 1), (3, 16), (5, 2), (6, 2)])
def test_route_mlp2(cid, B):
    w = synth.workload(cid).replace(B=B)
    wt = synth.layer_weights(w, 0)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)])
    types = stack_types(w, B)
    ref = lambda hh, tt: O.router_mlp2(hh, tt, wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"],
                                       wt["W2"], wt["b2"])
    _route_check(w, h, types, router_tensors(wt, tdtype(w)), ref, f"mlp2 workload {cid} B={B}")


# bf16 MLP2 shapes that take the other launch paths: partial language terms
# summed by their own kernel (short prefix: a router block spans more than two
# samples; more than 8 column blocks; Hr = 64 on the generic router) and the
# per-row projection (d not a multiple of 512).
@pytest.mark.parametrize("B,d,Hr,n_vis,n_lang", [(3, 1024, 128, 30, 9), (2, 4608, 128, 60, 9),
                                                 (2, 1024, 64, 80, 9), (2, 1088, 128, 80, 9)])
def test_route_mlp2_launch_paths(B, d, Hr, n_vis, n_lang):
    w = synth.workload(2).replace(B=B, d=d, Hr=Hr, n_vis=n_vis, n_lang=n_lang, n_prop=1)
    wt = synth.layer_weights(w, 0)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)])
    types = stack_types(w, B)
    ref = lambda hh, tt: O.router_mlp2(hh, tt, wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"],
                                       wt["W2"], wt["b2"])
    _route_check(w, h, types, router_tensors(wt, torch.bfloat16), ref, f"mlp2 B={B} d={d} Hr={Hr} T={w.T}")


# The split-K router (two workgroups per 96-token tile, T >= 48, d a multiple
# of 128) against the single kernel, which the no-alloc call runs: the same
# bits for every token, including tiles that end inside a sample or past the
# last token, tiles over three samples, 16 and 32 groups, and a second call on
# the same workspace. With the default poll count the two halves of a tile
# share its epilogue; with ROLESUB_SK_POLLS=0 the first to finish leaves the
# tile to the other (unless it has already arrived).
@pytest.mark.parametrize("polls", [None, "0"])
@pytest.mark.parametrize("cid,B,n_vis,G", [(4, 3, 47, 8),      # T = 96: every tile is one whole sample
                                           (4, 2, 48, 8),      # T = 97: tiles straddle samples
                                           (4, 5, 1, 8),       # T = 50: tiles over three samples
                                           (4, 7, 32, 16),     # T = 81: the full-width prefix
                                           (4, 5, 151, 16),    # 16 groups, ragged last tile
                                           (4, 2, 300, 32)])   # 32 groups
def test_route_split_k_matches_single_kernel(cid, B, n_vis, G, polls, monkeypatch):
    if polls is not None:
        monkeypatch.setenv("ROLESUB_SK_POLLS", polls)
    w = synth.workload(cid).replace(B=B, n_vis=n_vis, G=G, k_vis=min(4, G), k_lang=min(6, G), k_prop=min(8, G))
    wt = synth.layer_weights(w, 0)
    h = put(np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)]), torch.bfloat16)
    types = put_u8(stack_types(w, B))
    router = router_tensors(wt, torch.bfloat16)
    budget = rs.make_budget(rs.TOPK, w.k_by_type)
    ws = torch.empty(rs.route_workspace_size(B, w.T, G, w.d, router), dtype=torch.uint8, device=DEV)

    def outs():
        return {"mask": torch.full((B, w.T), -1, dtype=torch.int32, device=DEV),
                "idx": torch.full((B, w.T, G), 7, dtype=torch.uint8, device=DEV),
                "count": torch.full((B, w.T), 9, dtype=torch.uint8, device=DEV),
                "scores": torch.full((B, w.T, G), float("nan"), dtype=torch.float32, device=DEV)}
    _say(f"split-K router vs single kernel: B={B} T={w.T} G={G}")
    a = rs.route(types, budget, G, h=h, router=router, workspace=ws, out=outs())
    a2 = rs.route(types, budget, G, h=h, router=router, workspace=ws, out=outs())
    b = rs.route_noalloc(types, budget, G, h=h, router=router, out=outs())
    torch.cuda.synchronize()
    for r in (a2, b):
        for name in ("mask", "idx", "count"):
            assert torch.equal(r[name], a[name]), name
        assert np.array_equal(host(r["scores"]).view(np.uint32), host(a["scores"]).view(np.uint32))
    assert int(host(a["count"]).sum()) > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_route_additive(dtype):
    w = synth.workload(2).replace(B=2, dtype=dtype, d=512, G=16, C=6, n_vis=40, n_lang=9, n_prop=1,
                                  k_vis=3, k_lang=5, k_prop=16)
    aw = synth.additive_weights(w, 0)
    dt = tdtype(w)
    router = rs.Router.additive(*(put(aw[n], dt) for n in ("W_tok", "b_tok", "W_r", "b_r", "W_role",
                                                          "W_lang", "b_lang")))
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(2)])
    types = stack_types(w, 2)
    ref = lambda hh, tt: O.router_additive(hh, tt, aw["W_tok"], aw["b_tok"], aw["W_r"], aw["b_r"],
                                           aw["W_role"], aw["W_lang"], aw["b_lang"], 0.1, 0.1)
    _route_check(w, h, types, router, ref, f"additive {dtype}")


def _tie_router_weights(w, wt, variant):
    """Router weights built so that the fused ranking meets exact ties: pairs of
    identical W2 rows with equal biases give bitwise-equal group scores (every
    group's sum runs through the same operations), zero rows give zero scores;
    'nonfinite' adds +inf, -inf and NaN biases. G = 32 (threshold budgets):
    most groups pushed below the threshold, so many tokens keep one group by
    the lower clamp and it is chosen among the tied zero groups."""
    wt = dict(wt)
    W2, b2 = wt["W2"].astype(np.float32).copy(), wt["b2"].astype(np.float32).copy()
    if w.G == 8:
        W2[1], b2[1] = W2[0], b2[0]
        W2[3], b2[3] = W2[2], b2[2]
        W2[5], b2[5] = 0.0, -0.0
        W2[6], b2[6] = 0.0, 0.0
        if variant == "nonfinite":
            W2[4], b2[4] = 0.0, np.inf
            b2[6] = -np.inf
            b2[7] = np.nan
    else:
        b2 = synth.round_to(b2.astype(np.float64) - 4.0, "bf16").astype(np.float32)
        W2[0:4] = 0.0
        b2[0:4] = np.array([-0.0, 0.0, -0.0, 0.0], np.float32)
        for a, c in ((4, 5), (8, 9), (12, 13)):
            W2[c], b2[c] = W2[a], b2[a]
    wt["W2"], wt["b2"] = W2, b2
    return wt


def _split_ties(scores, K):
    """Tokens whose K-th and (K+1)-th highest scores are equal (-0 = +0): the
    cut runs through a tie, so only the lower-index rule decides."""
    s = np.where(np.isnan(scores), -np.inf, scores.astype(np.float64))
    s = np.sort(s, axis=-1)[..., ::-1]
    G = s.shape[-1]
    inner = (K > 0) & (K < G)
    kk = np.clip(K, 1, G - 1)
    a = np.take_along_axis(s, (kk - 1)[..., None], -1)[..., 0]
    b = np.take_along_axis(s, kk[..., None], -1)[..., 0]
    return inner & (a == b)


@pytest.mark.parametrize("cid,B,variant", [(3, 4, "ties"), (2, 1, "ties"), (3, 2, "nonfinite"), (5, 2, "ties")])
def test_route_mlp2_forced_ties(cid, B, variant):
    w = synth.workload(cid).replace(B=B)
    wt = _tie_router_weights(w, synth.layer_weights(w, 0), variant)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)])
    types = stack_types(w, B)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    r = rs.route(put_u8(types), budget, w.G, h=put(h, torch.bfloat16), router=router_tensors(wt, torch.bfloat16))
    torch.cuda.synchronize()
    got_scores = host(r["scores"])
    ref = O.router_mlp2(h, types, wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"], wt["W2"], wt["b2"])
    fin = np.isfinite(ref)
    for f in (np.isnan, np.isposinf, np.isneginf):
        assert np.array_equal(f(got_scores), f(ref))
    serr = max_rel(got_scores[fin], ref[fin])
    assert serr <= 1e-4
    K = O.group_budget(got_scores, types, w.mode, w.k_by_type, w.G, w.tau, w.kmin, w.kmax)
    got = host_mask(r["mask"])
    _exact_selection_on_own_scores(w, types, got_scores, got, host(r["count"]), host(r["idx"]), K=K)
    split = _split_ties(got_scores, K)
    if w.G == 8:
        kept = (got[..., None] >> np.arange(8, dtype=np.uint32)) & 1
        zero_split = int(np.sum(kept[..., 5] != kept[..., 6])) if variant == "ties" else 0
        dup_split = int(np.sum((kept[..., 0] != kept[..., 1]) | (kept[..., 2] != kept[..., 3])))
        _say(f"forced ties workload {cid} {variant}: score err {serr:.1e}; {int(split.sum())} tokens cut "
             f"through a tie, duplicated pair split on {dup_split}, zero pair split on {zero_split}")
        assert split.sum() > 0 and dup_split > 0
        if variant == "ties":
            assert zero_split > 0
            # the lower index of a split pair is the kept one
            assert np.all(kept[..., 1] <= kept[..., 0]) and np.all(kept[..., 3] <= kept[..., 2])
            assert np.all(kept[..., 6] <= kept[..., 5])
        else:
            assert np.all(kept[..., 4] == 1)                                   # +inf always kept
            vis = types == O.VIS                                               # K = 2: NaN and -inf never kept
            assert np.all(kept[..., 7][vis] == 0) and np.all(kept[..., 6][vis] == 0)
    else:
        one = K == 1
        n_zero_pick = int(np.sum(one & (host(r["count"]) == 1) & ((got & 0xF) != 0)))
        _say(f"forced ties workload {cid}: score err {serr:.1e}; {int(one.sum())} tokens keep one group, "
             f"{n_zero_pick} of them one of the tied zero groups")
        assert n_zero_pick > 0
        assert np.all((got[one & ((got & 0xF) != 0)] & 0xF) == 1)             # group 0 of the tied zeros


def test_route_sample_without_language_tokens():
    w = synth.workload(3).replace(B=2)
    wt = synth.layer_weights(w, 0)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(2)])
    types = stack_types(w, 2)
    types[1][types[1] == O.LANG] = O.VIS       # sample 1 has no language token: pool is zero
    ref = lambda hh, tt: O.router_mlp2(hh, tt, wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"],
                                       wt["W2"], wt["b2"])
    _route_check(w, h, types, router_tensors(wt, torch.bfloat16), ref, "no-language sample")


# ----------------------------------------------------------------------------
# Whole path: route -> rotate -> pack -> attend
# ----------------------------------------------------------------------------

def _run_gpu_layer(w, layer, acts_dev, types_np, scores_in=None):
    dt = tdtype(w)
    wt = synth.layer_weights(w, layer)
    router = router_tensors(wt, dt)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    ws = rs.route_workspace_size(w.B, w.T, w.G, w.d, router)
    bufs = LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, dt, ws_bytes=ws, device=DEV,
                                 with_z=False)
    run_layer(acts_dev.get("h"), acts_dev["q"], acts_dev["k"], acts_dev["v"], put_u8(types_np),
              put(wt["R"], dt), budget, w.G, bufs, router=router if scores_in is None else None,
              scores_in=scores_in, type_counts=w.type_counts(), fused=True)
    torch.cuda.synchronize()
    return bufs, wt, cap


def _check_sample(w, layer, b, bufs, wt, cap, scores=None):
    a = synth.sample_activations(w, layer, b)
    h, q, k, v = (a[n][None] for n in ("h", "q", "k", "v"))
    if scores is None:
        ref_scores = O.router_mlp2(h, w.types(), wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"],
                                   wt["W2"], wt["b2"])
    else:
        ref_scores = scores[None]
    run = lambda sc: O.pipeline(h, q, k, v, w.types(), wt, w.mode, w.k_by_type, w.G, w.tau, w.kmin, w.kmax,
                                scores=sc, cap=cap)
    ref = run(ref_scores)
    got_mask = host_mask(bufs.mask[b:b + 1])
    got_scores = host(bufs.scores[b:b + 1])
    if scores is not None:
        assert np.array_equal(got_scores.view(np.uint32), ref_scores.astype(np.float32).view(np.uint32))
    # (i) the selection on the GPU's own scores, bit for bit on every token
    _exact_selection_on_own_scores(w, w.types()[None], got_scores, got_mask, host(bufs.count[b:b + 1]),
                                   host(bufs.idx[b:b + 1]))
    # (ii) against the oracle's float64 scores wherever the margin decides
    abs_err = float(np.max(np.abs(got_scores - ref_scores)))
    margin = decisive_margin(ref_scores, ref["K"], w.tau if w.mode == O.THRESHOLD else None)
    safe = margin > 8 * abs_err if scores is None else np.ones_like(margin, dtype=bool)
    assert np.array_equal(got_mask[safe], ref["mask"][safe])
    flips = int(np.sum(got_mask != ref["mask"]))
    if flips:
        # a near-margin token chose differently: the rest of the path is checked
        # on the GPU's selection (exact on its scores, asserted above)
        ref = run(got_scores)
    assert np.array_equal(host(bufs.offsets[b:b + 1]), ref["offsets"])
    n = int(ref["offsets"][0, -1])
    vp_err = max_rel(host(bufs.Vp[b:b + 1, :, :n]), ref["Vp"][:, :, :n]) if n else 0.0
    out_err = max_rel(host(bufs.out[b:b + 1]), ref["out"])
    _say(f"  layer {layer} sample {b}: mask flips {flips} (near-margin {int(np.sum(~safe))}), "
         f"packed cache err {vp_err:.2e}, out err {out_err:.2e}")
    assert vp_err <= TOL[w.dtype] and out_err <= TOL[w.dtype]
    return flips


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_pipeline_small_workloads(cid):
    w = synth.workload(cid)
    _say(f"pipeline workload {cid} ({w.name})")
    acts = layer_on_device(w, 0)
    bufs, wt, cap = _run_gpu_layer(w, 0, acts, stack_types(w))
    for b in range(w.B):
        _check_sample(w, 0, b, bufs, wt, cap)


@pytest.mark.parametrize("layer", [0, 31])
def test_pipeline_stack_full_batch(layer):
    """The 32-layer, batch-64 workload at full size in the bench's launch
    configuration; the oracle checks every prefix of the batch."""
    w = synth.workload(4)
    _say(f"pipeline workload 4 layer {layer}, B={w.B}")
    acts = layer_on_device(w, layer)
    bufs, wt, cap = _run_gpu_layer(w, layer, acts, stack_types(w))
    flips = sum(_check_sample(w, layer, b, bufs, wt, cap) for b in range(w.B))
    _say(f"workload 4 layer {layer}: {flips} near-margin mask flips over {w.B * w.T} tokens")
    cnt = host(bufs.count)
    assert np.all(cnt[:, :w.n_vis] == w.k_vis) and np.all(cnt[:, w.n_vis:w.n_vis + w.n_lang] == w.k_lang)
    assert np.all(host(bufs.offsets)[:, -1] == cap)
    if layer == 0:
        # attention at full size is bitwise repeatable (no workgroup may read
        # metadata or tiles that another wave is still replacing)
        R = put(wt["R"], tdtype(w))
        for rep in range(24):
            again = rs.attend(acts["q"], acts["k"], bufs.mask, bufs.offsets, bufs.Vp, R, w.G)
            torch.cuda.synchronize()
            assert torch.equal(again, bufs.out), f"attend repeat {rep} differs"


def test_pipeline_stress_full_batch_sampled():
    """G=32 threshold workload at full size (B=128, T=2048); sampled oracle checks."""
    w = synth.workload(5)
    _say(f"pipeline workload 5, B={w.B}, T={w.T}")
    acts = layer_on_device(w, 0, need_h=False)
    scores = np.stack([synth.sample_scores(w, 0, b) for b in range(w.B)])
    bufs, wt, cap = _run_gpu_layer(w, 0, acts, stack_types(w), scores_in=put(scores, torch.float32))
    # selection and cache offsets of every prefix, bit for bit
    K = O.group_budget(scores, stack_types(w), O.THRESHOLD, w.k_by_type, w.G, 0.0, 1, 32)
    want = O.select_groups(scores, K)
    assert np.array_equal(host_mask(bufs.mask), want)
    assert np.array_equal(host(bufs.count).astype(np.int64), K)
    off = np.zeros((w.B, w.T + 1), dtype=np.int64)
    off[:, 1:] = np.cumsum(K, axis=1)
    assert np.array_equal(host(bufs.offsets), off)
    # packed cache and attention on sampled prefixes (the oracle takes ~5 s per prefix)
    for b in (0, 19, 38, 57, 77, 96, 115, 127):
        _check_sample(w, 0, b, bufs, wt, cap, scores=scores[b])


# ----------------------------------------------------------------------------
# Full-width routing space (one R over d_v = H*dh, S groups; Sec. 3.2, 4.1)
# ----------------------------------------------------------------------------

def _full_masks(rng, w, B, kinds=None):
    """Masks for the full-width tests: the workload's per-type budgets with
    random kept groups, plus special samples: kinds[b] = 'budget', 'all_full',
    'all_routed' (random K in 0..S-1, K = 0 included) or 'mixed'."""
    S, T = w.G, w.T
    full = (1 << S) - 1
    kinds = kinds or ["budget"] * B
    kk = np.array([w.k_vis] * w.n_vis + [w.k_lang] * w.n_lang + [w.k_prop] * w.n_prop)
    out = np.zeros((B, T), dtype=np.uint32)
    for b in range(B):
        if kinds[b] == "all_full":
            K = np.full(T, S)
        elif kinds[b] == "all_routed":
            K = rng.integers(0, S, size=T)
            K[:3] = 0
        elif kinds[b] == "mixed":
            K = rng.integers(0, S + 1, size=T)
        else:
            K = kk
        for t in range(T):
            gs = rng.choice(S, size=int(K[t]), replace=False)
            out[b, t] = int(np.sum(1 << gs.astype(np.int64))) if len(gs) else 0
    assert np.all(out <= full)
    return out


def _full_case(w, B, seed, kinds=None):
    rng = np.random.default_rng(seed)
    R = synth.full_rotation(w, 0)["R"]
    v = synth.round_to(rng.standard_normal((B, w.T, w.H, w.dh)), "bf16")
    mask = _full_masks(rng, w, B, kinds)
    return R, v, mask


def _dev_bf16(a):
    return put(a, torch.bfloat16)


def test_full_transpose_exact():
    for n in (1024, 4096):
        R = synth.round_to(np.random.default_rng(n).standard_normal((n, n)), "bf16")
        got = host(rs.full_transpose(_dev_bf16(R)))
        assert np.array_equal(got, R.T)


@pytest.mark.parametrize("cid,B,kinds,T", [
    (7, 3, ["budget", "mixed", "all_routed"], None),
    (7, 4, ["all_full", "budget", "mixed", "budget"], 200),      # ragged T, one sample with no routed token
    (6, 2, ["budget", "mixed"], None),                           # d_v = 4096, S = 16 groups of 256
])
def test_full_rotate_pack(cid, B, kinds, T):
    w = synth.workload(cid)
    if T is not None:
        w = w.replace(n_vis=T - w.n_lang - w.n_prop)
    R, v, mask = _full_case(w, B, 50 + cid, kinds)
    S = w.G
    cap = w.T * S
    Rd = _dev_bf16(R)
    off, Vp = rs.full_rotate_pack(_dev_bf16(v), rs.full_transpose(Rd), put_mask(mask), S, cap)
    torch.cuda.synchronize()
    want_off, want_Vp = O.pack_full(v, mask, R, S, cap)
    got_off, got_Vp = host(off), host(Vp)
    assert np.array_equal(got_off, want_off)
    full = (1 << S) - 1
    routed_slot = np.zeros((B, cap), dtype=bool)
    full_slot = np.zeros((B, cap), dtype=bool)
    for b in range(B):
        for t in range(w.T):
            o, n = want_off[b, t], want_off[b, t + 1] - want_off[b, t]
            (full_slot if int(mask[b, t]) == full else routed_slot)[b, o:o + n] = True
    assert np.array_equal(got_Vp[full_slot], want_Vp[full_slot])            # value-space tokens: exact copies
    if routed_slot.any():
        err = max_rel(got_Vp[routed_slot], want_Vp[routed_slot])
        _say(f"full rotate+pack workload {cid} B={B} T={w.T}: routed groups max rel err {err:.2e}")
        assert err <= TOL["bf16"]


@pytest.mark.parametrize("cid,B,kinds", [(7, 3, ["budget", "all_routed", "mixed"]), (6, 2, ["budget", "mixed"])])
def test_full_values(cid, B, kinds):
    w = synth.workload(cid)
    R, v, mask = _full_case(w, B, 60 + cid, kinds)
    S = w.G
    cap = w.T * S
    off, Vp = O.pack_full(v, mask, R, S, cap)
    Vp = synth.round_to(Vp, "bf16")                 # the cache as the GPU stores it
    got = host(rs.full_values(_dev_bf16(R), put_mask(mask), torch.from_numpy(off.astype(np.int32)).to(DEV),
                              _dev_bf16(Vp), S, w.H))
    want = O.values_full(off, Vp, mask, R, S, w.H).transpose(0, 2, 1, 3)   # [B,H,T,dh]
    err = max_rel(got, want)
    _say(f"full values workload {cid} B={B}: max rel err {err:.2e}")
    assert err <= TOL["bf16"]
    full = (1 << S) - 1
    for b in range(B):
        for t in range(w.T):
            if int(mask[b, t]) == full:                                     # value-space tokens: exact
                assert np.array_equal(got[b, :, t], want[b, :, t])
            elif int(mask[b, t]) == 0:
                assert np.all(got[b, :, t] == 0)


@pytest.mark.parametrize("cid,B,kinds", [(7, 3, ["budget", "mixed", "all_routed"]), (6, 4, None)])
def test_full_width_attention_end_to_end(cid, B, kinds):
    from paper_2608_18410_amd.pipeline import FullWidthBuffers, run_full_layer
    w = synth.workload(cid).replace(B=B)
    R, v, mask = _full_case(w, B, 70 + cid, kinds)
    rng = np.random.default_rng(71 + cid)
    q = synth.round_to(rng.standard_normal((B, w.Tq, w.H, w.dh)), "bf16")
    k = synth.round_to(rng.standard_normal((B, w.T, w.H, w.dh)), "bf16")
    S = w.G
    cap = sum(n * min(kk, S) for n, kk in zip(w.type_counts(), w.k_by_type)) if kinds is None else w.T * S
    bufs = FullWidthBuffers.allocate(B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, out_dtype=torch.float32,
                                     device=DEV)
    Rd = _dev_bf16(R)
    budget = rs.make_budget(rs.TOPK, w.k_by_type) if kinds is None else None
    run_full_layer(_dev_bf16(q), _dev_bf16(k), _dev_bf16(v), put_mask(mask), rs.full_transpose(Rd), Rd, S, bufs,
                   budget=budget, type_counts=w.type_counts() if kinds is None else None)
    torch.cuda.synchronize()
    want = O.attend_full_plain(q, k, v, mask, R, S)
    err = max_rel(host(bufs.out), want)
    _say(f"full-width attention workload {cid} B={B}: max rel err {err:.2e} vs the plain form")
    assert err <= TOL["bf16"]


def test_full_width_stack_shape_sampled():
    """The 7B full-width layer at its full batch (64 prefixes, d_v = 4096,
    S = 16) in the launch configuration the bench times; oracle on 3 prefixes."""
    from paper_2608_18410_amd.pipeline import FullWidthBuffers, run_full_layer
    w = synth.workload(6)
    B = w.B
    R, v, mask = _full_case(w, B, 80)
    rng = np.random.default_rng(81)
    q = synth.round_to(rng.standard_normal((B, w.Tq, w.H, w.dh)), "bf16")
    k = synth.round_to(rng.standard_normal((B, w.T, w.H, w.dh)), "bf16")
    S = w.G
    cap = sum(n * min(kk, S) for n, kk in zip(w.type_counts(), w.k_by_type))
    bufs = FullWidthBuffers.allocate(B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, device=DEV)
    Rd = _dev_bf16(R)
    run_full_layer(_dev_bf16(q), _dev_bf16(k), _dev_bf16(v), put_mask(mask), rs.full_transpose(Rd), Rd, S, bufs,
                   budget=rs.make_budget(rs.TOPK, w.k_by_type), type_counts=w.type_counts())
    torch.cuda.synchronize()
    got = host(bufs.out)
    for b in (0, 31, 63):
        want = O.attend_full_plain(q[b:b + 1], k[b:b + 1], v[b:b + 1], mask[b:b + 1], R, S)
        err = max_rel(got[b:b + 1], want)
        _say(f"full-width stack prefix {b}: max rel err {err:.2e}")
        assert err <= TOL["bf16"]


def test_full_width_with_role_driven_budgets_and_repeatable():
    """Role-driven budgets (Sec. 3.5) feeding the full-width path at the
    paper's router shape (C = 6, S = 16): masks from rolesub_route_allocate,
    cache and attention against the oracle on those masks, and bitwise equal
    results on a second run of every call."""
    from paper_2608_18410_amd.pipeline import FullWidthBuffers, run_full_layer
    w = synth.workload(6).replace(B=4, k_vis=4, k_lang=8)      # language routed too
    B, S = w.B, w.G
    wt = synth.layer_weights(w, 0)
    wpri = synth.priority_weights(w, 0)
    h = np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)])
    types = stack_types(w, B)
    r = rs.route_allocate(put_u8(types), w.k_by_type, S, put(h, torch.bfloat16), router_tensors(wt, torch.bfloat16),
                          put(wpri, torch.bfloat16))
    torch.cuda.synchronize()
    mask = host_mask(r["mask"])
    k = host(r["k"]).astype(np.int64)
    for b in range(B):
        for m in range(3):
            sel = types[b] == m
            assert k[b][sel].sum() == min(w.k_by_type[m], S) * sel.sum()
    assert len(np.unique(k[0][types[0] == O.VIS])) > 1          # budgets vary by token
    rng = np.random.default_rng(90)
    R = synth.full_rotation(w, 0)["R"]
    q = synth.round_to(rng.standard_normal((B, w.Tq, w.H, w.dh)), "bf16")
    kk = synth.round_to(rng.standard_normal((B, w.T, w.H, w.dh)), "bf16")
    v = synth.round_to(rng.standard_normal((B, w.T, w.H, w.dh)), "bf16")
    cap = sum(n * min(x, S) for n, x in zip(w.type_counts(), w.k_by_type))
    bufs = FullWidthBuffers.allocate(B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, device=DEV)
    Rd = _dev_bf16(R)
    Rt = rs.full_transpose(Rd)
    args = (_dev_bf16(q), _dev_bf16(kk), _dev_bf16(v), put_mask(mask), Rt, Rd, S, bufs)
    run_full_layer(*args, budget=rs.make_budget(rs.TOPK, w.k_by_type), type_counts=w.type_counts())
    torch.cuda.synchronize()
    first = [t.clone() for t in (bufs.offsets, bufs.Vp, bufs.Vh, bufs.out)]
    want = O.attend_full_plain(q, kk, v, mask, R, S)
    err = max_rel(host(bufs.out), want)
    _say(f"full width with role-driven budgets: max rel err {err:.2e}")
    assert err <= TOL["bf16"]
    for _ in range(3):
        run_full_layer(*args)
    torch.cuda.synchronize()
    for a, b_ in zip(first, (bufs.offsets, bufs.Vp, bufs.Vh, bufs.out)):
        assert torch.equal(a, b_)


@pytest.mark.parametrize("B,T,Tq,H,dh,out_dtype", [(2, 81, 56, 8, 128, torch.bfloat16), (3, 200, 70, 4, 128, torch.float32),
                                                   (2, 37, 9, 4, 64, torch.float32), (2, 1, 5, 2, 128, torch.bfloat16),
                                                   (1, 32, 1, 3, 128, torch.bfloat16)])
def test_attend_values_is_textbook_attention(B, T, Tq, H, dh, out_dtype):
    """Attention over plain head-major values (the full-width path's last step)
    against the oracle with every group kept, where the routed value is v."""
    rng = np.random.default_rng(T + dh)
    q = synth.round_to(rng.standard_normal((B, Tq, H, dh)), "bf16")
    k = synth.round_to(rng.standard_normal((B, T, H, dh)), "bf16")
    v = synth.round_to(rng.standard_normal((B, T, H, dh)), "bf16")
    Vh = _dev_bf16(np.ascontiguousarray(v.transpose(0, 2, 1, 3)))
    got = host(rs.attend_values(_dev_bf16(q), _dev_bf16(k), Vh, out_dtype=out_dtype))
    R = np.eye(H * dh)
    want = O.attend_full_plain(q, k, v, np.full((B, T), 1, np.uint32), R, 1)
    err = max_rel(got, want)
    _say(f"attend_values B={B} T={T} Tq={Tq} H={H} dh={dh}: max rel err {err:.2e}")
    assert err <= TOL["bf16"]          # bf16 inputs; P enters the matrix cores in bf16


def test_full_rotate_pack_never_writes_past_capacity():
    w = synth.workload(7).replace(B=1)
    R, v, mask = _full_case(w, 1, 95, ["mixed"])
    S, ds = w.G, w.ds
    want_off, want_Vp = O.pack_full(v, mask, R, S, w.T * S)
    need = int(want_off[0, -1])
    cap = need // 2
    big = torch.full((1, need + 8, ds), 7.0, dtype=torch.bfloat16, device=DEV)    # sentinel past cap
    Rd = _dev_bf16(R)
    off = torch.empty((1, w.T + 1), dtype=torch.int32, device=DEV)
    rs.full_rotate_pack(_dev_bf16(v), rs.full_transpose(Rd), put_mask(mask), S, cap, out=(off, big[:, :cap]))
    torch.cuda.synchronize()
    got = host(big)
    assert np.array_equal(host(off), want_off)                   # offsets still count every kept group
    assert np.all(got[0, cap:] == 7.0)                           # nothing at or past the capacity
    assert max_rel(got[0, :cap], want_Vp[0, :cap]) <= TOL["bf16"]
