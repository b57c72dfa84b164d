"""Library calls captured in a HIP graph and replayed: every replay must give
the eager pass's bits. The calls keep state across their kernels only in
caller memory (the split-K router's tile tickets, the partial language terms,
the cache offsets the rotate+pack kernel forms), so a replay that found stale
values there would differ. Replays alternate with eager work on other
buffers and with synchronisations, and the outputs are overwritten with
sentinels before each replay, so that every output must be written again.
Also: two layers with their own workspaces on two streams at once give the
bits of the same layers run one after the other."""
import numpy as np
import pytest
import torch

import paper_2608_18410_amd as rs
import synth
from paper_2608_18410_amd.pipeline import (FullWidthBuffers, LayerBuffers, micro_batches, on_streams,
                                          pack_capacity, run_full_layer, run_layer)
from tests._gpu_util import DEV, put, put_mask, put_u8, router_tensors, stack_types

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    rs.load()


def _say(msg):
    print(msg, flush=True)


def _stack_layer(w, seed):
    """Inputs of one 7B-stack layer for w.B prefixes (bf16)."""
    wt = synth.layer_weights(w, seed)
    acts = [synth.sample_activations(w, seed, b, ("h", "q", "k", "v")) for b in range(w.B)]
    get = lambda n: put(np.stack([a[n] for a in acts]), torch.bfloat16)
    return dict(h=get("h"), q=get("q"), k=get("k"), v=get("v"), R=put(wt["R"], torch.bfloat16),
                router=router_tensors(wt, torch.bfloat16), types=put_u8(stack_types(w, w.B)))


def _sentinel(tensors):
    for t in tensors:
        if t.dtype in (torch.float32, torch.bfloat16):
            t.fill_(float("nan"))
        else:
            t.fill_(-1 if t.dtype == torch.int32 else 0xAB)


def _bits(t):
    return t.detach().clone().view(torch.int16 if t.element_size() == 2 else
                                   (torch.int32 if t.element_size() == 4 else torch.uint8))


@pytest.mark.parametrize("noalloc", [False, True])
def test_stack_layer_graph_replays(noalloc):
    # route (split-K MLP2 router, or the allocation-free call) -> rotate+pack
    # (offsets formed in the kernel) -> attend, 8 prefixes of the 7B stack
    w = synth.workload(4).replace(B=8)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    L, other = _stack_layer(w, 0), _stack_layer(w, 1)
    ws = rs.route_workspace_size(w.B, w.T, w.G, w.d, L["router"])
    bufs = LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, torch.bfloat16, device=DEV, with_z=False,
                                 ws_bytes=ws)
    obufs = LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, torch.bfloat16, device=DEV, with_z=False,
                                  ws_bytes=ws)

    def layer(X, b):
        if not noalloc:
            return run_layer(X["h"], X["q"], X["k"], X["v"], X["types"], X["R"], budget, w.G, b, router=X["router"],
                             type_counts=w.type_counts())
        rs.route_noalloc(X["types"], budget, w.G, h=X["h"], router=X["router"],
                         out={"mask": b.mask, "idx": b.idx, "count": b.count, "scores": b.scores})
        rs.rotate_pack(X["v"], X["R"], b.mask, w.G, cap, budget=budget, type_counts=w.type_counts(),
                       out=(b.offsets, b.Vp))
        rs.attend(X["q"], X["k"], b.mask, b.offsets, b.Vp, X["R"], w.G, out=b.out)

    outs = lambda b: (b.mask, b.idx, b.count, b.scores, b.offsets, b.out)
    _say(f"graph replays, 7B-stack layer B={w.B} T={w.T} noalloc={noalloc}")
    layer(L, bufs)
    torch.cuda.synchronize()
    want = [_bits(t) for t in outs(bufs)]
    n_slots = bufs.offsets[:, -1].clone()
    vp_want = [bufs.Vp[b, :, :int(n_slots[b])].clone() for b in range(w.B)]

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer(L, bufs)  # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            layer(L, bufs)
    torch.cuda.synchronize()
    for rep in range(3):
        layer(other, obufs)  # eager work between the replays
        _sentinel(outs(bufs) + (bufs.Vp,))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, a, t in zip(("mask", "idx", "count", "scores", "offsets", "out"), want, outs(bufs)):
            assert torch.equal(a, _bits(t)), (rep, name)
        for b in range(w.B):
            assert torch.equal(vp_want[b].view(torch.int16), bufs.Vp[b, :, :int(n_slots[b])].view(torch.int16)), \
                (rep, "Vp", b)


def test_full_width_layer_graph_replays():
    # full-width rotate+pack -> values -> attention over the values, 4 prefixes
    # of the 7B full-width shape
    w = synth.workload(6).replace(B=4)
    dv, S = w.H * w.dh, w.G
    rng = np.random.default_rng(5)
    g0 = torch.Generator(device=DEV)
    g0.manual_seed(5)
    R = (torch.randn(dv, dv, device=DEV, generator=g0) / dv ** 0.5).bfloat16()
    Rt = rs.full_transpose(R)
    q, k, v = (torch.randn(w.B, n, w.H, w.dh, device=DEV, generator=g0).bfloat16() for n in (w.Tq, w.T, w.T))
    m = np.zeros((w.B, w.T), np.uint32)
    for b in range(w.B):
        for t in range(w.n_vis):
            m[b, t] = int(np.sum(1 << rng.choice(S, w.k_vis, replace=False)))
        m[b, w.n_vis:] = (1 << S) - 1
    mask = put_mask(m)
    cap = sum(n * min(kk, S) for n, kk in zip(w.type_counts(), w.k_by_type))
    bufs = FullWidthBuffers.allocate(w.B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, device=DEV)
    obufs = FullWidthBuffers.allocate(w.B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, device=DEV)
    v2 = torch.randn_like(v, dtype=torch.float32).bfloat16()
    _say(f"graph replays, full-width layer B={w.B} T={w.T}")
    run_full_layer(q, k, v, mask, Rt, R, S, bufs)
    torch.cuda.synchronize()
    outs = lambda b: (b.offsets, b.Vp, b.Vh, b.out)
    want = [_bits(t) for t in outs(bufs)]

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run_full_layer(q, k, v, mask, Rt, R, S, bufs)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            run_full_layer(q, k, v, mask, Rt, R, S, bufs)
    torch.cuda.synchronize()
    for rep in range(3):
        run_full_layer(q, k, v2, mask, Rt, R, S, obufs)
        _sentinel(outs(bufs))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, a, t in zip(("offsets", "Vp", "Vh", "out"), want, outs(bufs)):
            assert torch.equal(a, _bits(t)), (rep, name)


def test_two_layers_on_two_streams_match_sequential():
    # independent calls with their own workspaces may run concurrently: two
    # 7B-stack layers enqueued on two streams (default priority) at once give
    # the bits of the same layers run one after the other
    w = synth.workload(4).replace(B=8)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    Ls = [_stack_layer(w, 0), _stack_layer(w, 1)]
    ws = rs.route_workspace_size(w.B, w.T, w.G, w.d, Ls[0]["router"])
    mk = lambda: LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, torch.bfloat16, device=DEV,
                                       with_z=False, ws_bytes=ws)
    seq, par = [mk(), mk()], [mk(), mk()]
    run = lambda X, b: run_layer(X["h"], X["q"], X["k"], X["v"], X["types"], X["R"], budget, w.G, b,
                                 router=X["router"], type_counts=w.type_counts())
    _say(f"two streams, 7B-stack layers B={w.B}")
    for X, b in zip(Ls, seq):
        run(X, b)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        for b in par:
            _sentinel((b.mask, b.idx, b.count, b.scores, b.offsets, b.out))
        torch.cuda.synchronize()
        for X, b, st in zip(Ls, par, streams):
            st.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(st):
                run(X, b)
        torch.cuda.synchronize()
        for a, b in zip(seq, par):
            for name in ("mask", "idx", "count", "scores", "offsets", "out"):
                assert torch.equal(_bits(getattr(a, name)), _bits(getattr(b, name))), (rep, name)


def test_micro_batches_on_streams_match_whole_batch():
    # a batch split into micro-batches (views of the layer's buffers, one
    # route workspace each), every micro-batch through two layers on its own
    # stream and captured in one graph, gives the bits of whole-batch calls
    w = synth.workload(4).replace(B=8)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    Ls = [_stack_layer(w, 0), _stack_layer(w, 1)]
    mbs = micro_batches(w.B, 3)
    assert [b1 - b0 for b0, b1 in mbs] == [2, 3, 3]
    wsz = [rs.route_workspace_size(b1 - b0, w.T, w.G, w.d, Ls[0]["router"]) for b0, b1 in mbs]
    off = np.concatenate([[0], np.cumsum([(n + 255) // 256 * 256 for n in wsz])]).astype(int)
    whole = [LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, torch.bfloat16, device=DEV, with_z=False,
                                   ws_bytes=rs.route_workspace_size(w.B, w.T, w.G, w.d, Ls[0]["router"]))
             for _ in Ls]
    split = [LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, torch.bfloat16, device=DEV, with_z=False,
                                   ws_bytes=int(off[-1])) for _ in Ls]
    views = [[b.rows(b0, b1, b.workspace[off[i]:off[i] + wsz[i]]) for i, (b0, b1) in enumerate(mbs)] for b in split]
    _say(f"micro-batches {mbs} on streams, 7B-stack layers B={w.B}")
    for X, b in zip(Ls, whole):
        run_layer(X["h"], X["q"], X["k"], X["v"], X["types"], X["R"], budget, w.G, b, router=X["router"],
                  type_counts=w.type_counts())

    def mb(i):
        b0, b1 = mbs[i]
        for X, v in zip(Ls, views):
            run_layer(X["h"][b0:b1], X["q"][b0:b1], X["k"][b0:b1], X["v"][b0:b1], X["types"][b0:b1], X["R"],
                      budget, w.G, v[i], router=X["router"], type_counts=w.type_counts())

    g = torch.cuda.CUDAGraph()
    main = torch.cuda.Stream()
    streams = [torch.cuda.Stream() for _ in mbs]
    main.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(main):
        for i in range(len(mbs)):  # warm-up on the capture stream
            mb(i)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=main):
            on_streams(lambda i, b0, b1: mb(i), mbs, streams)
    torch.cuda.synchronize()
    for rep in range(3):
        for b in split:
            _sentinel((b.mask, b.idx, b.count, b.scores, b.offsets, b.out))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(whole, split):
            for name in ("mask", "idx", "count", "scores", "offsets", "out"):
                assert torch.equal(_bits(getattr(a, name)), _bits(getattr(b, name))), (rep, name)
            for s in range(w.B):
                n = int(a.offsets[s, -1])
                assert torch.equal(a.Vp[s, :, :n].view(torch.int16), b.Vp[s, :, :n].view(torch.int16)), (rep, "Vp", s)
