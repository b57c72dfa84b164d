"""rolesub_route_noalloc (the route call that allocates nothing: its workspace
is a fixed device array inside the library) against rolesub_route, through the
C ABI: identical scores, masks, kept-group lists and counts, on two calls in a
row, the second with a smaller input, then a selection-only call, a size
beyond the array, refused on the host, and the exact sample limit at
d = 4096."""
import numpy as np
import pytest
import torch

import paper_2608_18410_amd as rs
import synth
from tests._gpu_util import DEV, put, put_u8, router_tensors, stack_types

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    rs.load()


def _outs(B, T, G):
    return {"mask": torch.full((B, T), -1, dtype=torch.int32, device=DEV),
            "idx": torch.full((B, T, G), 7, dtype=torch.uint8, device=DEV),
            "count": torch.full((B, T), 9, dtype=torch.uint8, device=DEV),
            "scores": torch.full((B, T, G), float("nan"), dtype=torch.float32, device=DEV)}


def _same(a, b):
    for name in ("mask", "idx", "count"):
        assert torch.equal(a[name], b[name]), name
    sa, sb = a["scores"].cpu().numpy(), b["scores"].cpu().numpy()
    assert np.array_equal(sa.view(np.uint32), sb.view(np.uint32)), "scores differ"


@pytest.mark.parametrize("order", ["large_then_small"])
def test_route_noalloc_matches_route(order):
    # 7B-stack shape at 48 prefixes (bf16 matrix-core router), then the
    # aggressive-budget shape at 3 prefixes: the second call reuses the array
    # the first one filled
    for cid, B in ((4, 48), (3, 3)):
        w = synth.workload(cid).replace(B=B)
        wt = synth.layer_weights(w, 0)
        h = put(np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)]), torch.bfloat16)
        types = put_u8(stack_types(w, B))
        router = router_tensors(wt, torch.bfloat16)
        budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
        print(f"route_noalloc vs route: workload {cid} B={B} T={w.T}", flush=True)
        ref = rs.route(types, budget, w.G, h=h, router=router, out=_outs(B, w.T, w.G))
        got = rs.route_noalloc(types, budget, w.G, h=h, router=router, out=_outs(B, w.T, w.G))
        torch.cuda.synchronize()
        _same(got, ref)
        assert int(got["count"].sum()) > 0


def test_route_noalloc_selection_only_and_limit():
    w = synth.workload(5)
    B = 2
    scores = put(np.stack([synth.sample_scores(w, 0, b) for b in range(B)]), torch.float32)
    types = put_u8(stack_types(w, B))
    budget = rs.make_budget(rs.THRESHOLD, (0, 0, 0, 0), 0.0, 1, 32)
    ref = rs.route(types, budget, w.G, scores_in=scores, out=_outs(B, w.T, w.G))
    got = rs.route_noalloc(types, budget, w.G, scores_in=scores, out=_outs(B, w.T, w.G))
    torch.cuda.synchronize()
    _same(got, ref)
    # a route workspace beyond the array: refused before anything is enqueued
    wb = synth.workload(4).replace(B=600, n_vis=1, n_lang=0, n_prop=0)
    wt = synth.layer_weights(wb, 0)
    router = router_tensors(wt, torch.bfloat16)
    assert rs.route_workspace_size(wb.B, wb.T, wb.G, wb.d, router) > rs.ROUTE_NOALLOC_MAX_BYTES
    h = torch.zeros((wb.B, wb.T, wb.d), dtype=torch.bfloat16, device=DEV)
    out = _outs(wb.B, wb.T, wb.G)
    with pytest.raises(rs.RolesubError, match="above the") as e:
        rs.route_noalloc(put_u8(stack_types(wb)), rs.make_budget(rs.TOPK, wb.k_by_type), wb.G, h=h, router=router,
                         out=out)
    assert e.value.status == 2
    torch.cuda.synchronize()
    assert bool((out["mask"] == -1).all())          # nothing was written


def test_route_noalloc_sample_limit_at_d4096():
    # d = 4096, Hr = 128: the array holds the route workspace of 334 samples
    # (cb, F, pooled states and 16 column blocks of language terms); 335 are
    # refused on the host, 334 give rolesub_route's results
    for B, fits in ((335, False), (334, True)):
        w = synth.workload(4).replace(B=B, n_vis=1, n_lang=0, n_prop=0)
        wt = synth.layer_weights(w, 0)
        router = router_tensors(wt, torch.bfloat16)
        h = put(np.stack([synth.sample_activations(w, 0, b, ("h",))["h"] for b in range(B)]), torch.bfloat16)
        types = put_u8(stack_types(w, B))
        budget = rs.make_budget(rs.TOPK, w.k_by_type)
        print(f"route_noalloc sample limit: B={B}", flush=True)
        out = _outs(B, w.T, w.G)
        if not fits:
            with pytest.raises(rs.RolesubError, match="above the") as e:
                rs.route_noalloc(types, budget, w.G, h=h, router=router, out=out)
            assert e.value.status == 2
            torch.cuda.synchronize()
            assert bool((out["mask"] == -1).all())
            continue
        got = rs.route_noalloc(types, budget, w.G, h=h, router=router, out=out)
        ref = rs.route(types, budget, w.G, h=h, router=router, out=_outs(B, w.T, w.G))
        torch.cuda.synchronize()
        _same(got, ref)
