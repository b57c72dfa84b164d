"""Benchmark of the RoleSub hot path on one MI355X.

A step is one pass of the whole hot path (route -> rotate -> pack -> attend)
over one batch: by default the 32-layer compressed-attention stack at the
OpenVLA-OFT-7B shape (hidden 4096, 32 heads x 128), 64 prefixes of 177 KV
tokens (128 retained visual + 48 language + 1 proprio), 56 action queries,
8 groups of 16 dims, keeping 4/8 visual and 6/8 language groups; every layer
has its own rotations, router weights and activations, all resident in HBM
before timing starts. The whole step (every layer's calls) is captured once in
a HIP graph and replayed (the kernels are the same as the eager calls).

Prints ONE JSON line. `value` counts query tokens per second per layer call,
B * Tq * L / step time. `roofline` is measured live for the attention kernel
with HIP events around back-to-back replays of the 32 attention launches right
after the timed steps; `cpu_baseline` times the float64 oracle on a bounded
sample on the host cores.

--allocation routes with role-driven per-token budgets instead (the router
also emits each token's role priority, then one kernel apportions every type's
group budget over its tokens and selects their groups); the rest of the step
is unchanged. --prefix-attention and --retention time the other rows of the
path at the same shape.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compressed-KV attention query-tokens/sec at 7B shape; achieved HBM GB/s vs peak"
PREFIX_METRIC = "prefix self-attention (causal) over the compressed cache, query-tokens/sec at 7B shape"
ALLOC_METRIC = ("compressed-KV attention query-tokens/sec at 7B shape with role-driven per-token budgets; "
                "achieved HBM GB/s vs peak")
FULL_METRIC = ("full-width routing space (one R over d_v = 4096, S = 16 groups): query-tokens/sec at 7B shape; "
               "achieved MFMA TFLOP/s vs peak")
RETAIN_METRIC = "token retention (top scores per view) + gather of the retained hidden states, tokens/sec"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attend_hbm_traffic.json")


def attend_bytes(w, sum_k: int, out_esize: int, total_k: int | None = None) -> int:
    """Algorithmic HBM bytes of one attention call: q, k, packed values,
    mask + offsets, output, rotations (everything read or written once).
    sum_k: kept groups per sample; total_k (if given): over the whole batch."""
    e = 2 if w.dtype == "bf16" else 4
    tot = w.B * sum_k if total_k is None else total_k
    per = (w.Tq * w.H * w.dh * e + w.T * w.H * w.dh * e + 8 * w.T + w.Tq * w.H * w.dh * out_esize)
    return w.B * per + tot * w.ds * w.H * e + w.H * w.dh * w.dh * e


def stage_bytes(w, sum_k: int, total_k: int | None = None) -> dict:
    """Algorithmic HBM bytes per layer call of each stage as the step runs
    them (rotation and pack fused: v read once, only kept groups written)."""
    e = 2 if w.dtype == "bf16" else 4
    tot = w.B * sum_k if total_k is None else total_k
    route_w = (w.Hr * w.router_in + w.C * w.d + w.G * w.Hr + w.C * w.d_e) * e
    # with given logits the selection reads them instead of running the router
    route_in = 4 * w.B * w.T * w.G if w.scores_in else w.B * w.T * w.d * e + route_w
    return {
        "route": route_in + 4 * w.B * w.T * (w.G + 2),
        "rotate_pack": w.B * w.T * w.H * w.dh * e + w.H * w.dh * w.dh * e
                       + tot * w.ds * w.H * e + 8 * w.B * w.T,
        "attend": attend_bytes(w, sum_k, e, total_k),
    }


def dist(xs) -> dict:
    """median and 10th / 90th percentiles of a list of timings."""
    a = np.asarray(xs, dtype=np.float64)
    return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90)), "n": int(a.size)}


# After the GPU has idled for tens of milliseconds (the eager pass, graph
# capture, creating events), the next 20 or so milliseconds of kernels run
# up to 15 % slower (every kernel of the first five 7B-stack steps, in a
# kernel trace; idle gaps of under 0.1 ms between steps do not do this). So
# the warm-up runs the requested number of steps and then keeps stepping
# until it has lasted WARM_S, and timed work follows it directly.
WARM_S = 0.25


def warm_up(step, n: int) -> int:
    """Runs step() n times, then more until WARM_S seconds of warm-up have
    passed; returns the number of steps run."""
    import torch
    t0 = time.perf_counter()
    runs = 0
    while runs < n or time.perf_counter() - t0 < WARM_S:
        # steps back to back, as in the timed region, in batches of ten
        for _ in range(n - runs if runs < n else 10):
            step()
            runs += 1
        torch.cuda.synchronize()
    return runs


def timed_replays(fn, reps: int, per: int = 1) -> list:
    """HIP events on the current stream around each of `reps` calls of fn,
    after WARM_S of warm-up calls; returns the time per unit (fn does `per`
    units) of each call, in us."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    warm_up(fn, 1)
    ev[0].record()
    for i in range(reps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) * 1e3 / per for i in range(reps)]


def copy_rate(nbytes: int = 1 << 30, reps: int = 20) -> dict:
    """A plain device-to-device copy of nbytes (read + written once), the
    achievable streaming rate on this GPU in the same run."""
    import torch
    src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    us = timed_replays(lambda: dst.copy_(src), reps)
    gbs = [2 * nbytes / (u * 1e-6) / 1e9 for u in us]
    del src, dst
    return {"bytes_read": nbytes, "bytes_written": nbytes, "GBs": dist(gbs), "kernel": "torch copy_ (HIP)"}


def _blas_threads() -> int:
    from threadpoolctl import threadpool_info
    return max([p.get("num_threads", 1) for p in threadpool_info()] + [1])


def _cores() -> dict:
    return {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}


def _source_hash() -> str:
    p = os.path.join(ROOT, "paper_2608_18410_amd", "csrc", "k_attend.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def _traffic(workload_name):
    """HBM traffic per attention launch from committed rocprofv3 counter runs,
    or None when absent, taken on a different kernel source or on another
    workload."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("k_attend_sha256_16") != _source_hash() or not str(t.get("workload", "")).startswith(workload_name):
        return None
    return t.get("bytes_per_launch")


def cpu_baseline(w, budget_s: float = 12.0, allocation: bool = False) -> dict:
    """The float64 oracle (test infrastructure) on whole prefixes, layer 0 first
    and further layers while the time budget lasts."""
    import oracle as O
    import synth
    from threadpoolctl import threadpool_limits

    cores = _cores()
    cap = sum(n * min(k, w.G) for n, k in zip(w.type_counts(), w.k_by_type))
    done, spent, layer = 0, 0.0, 0
    lim = threadpool_limits(limits=cores["affinity"], user_api="blas")
    while spent < budget_s and layer < w.L:
        wt = synth.layer_weights(w, layer)
        wpri = synth.priority_weights(w, layer) if allocation else None
        b = 0
        while spent < budget_s and b < w.B:
            a = synth.sample_activations(w, layer, b)
            t0 = time.perf_counter()
            O.pipeline(a["h"][None], a["q"][None], a["k"][None], a["v"][None], w.types(), wt, w.mode,
                       w.k_by_type, w.G, w.tau, w.kmin, w.kmax, cap=cap, w_pri=wpri)
            spent += time.perf_counter() - t0
            done += 1
            b += 1
        layer += 1
    threads = _blas_threads()
    lim.restore_original_limits()
    single = {} if allocation else cpu_single_thread()
    return {"value": done * w.Tq / spent, "unit": "query-tokens/s", "cores": int(min(threads, cores["affinity"])),
            "kind": "oracle", "nproc": cores["nproc"], "affinity_cores": cores["affinity"], "blas_threads": threads,
            "sample": f"{done} (layer, prefix) pairs, layers 0..{layer - 1} of {w.L} with {w.B} prefixes "
                      f"each (the last layer possibly partial): route->"
                      f"{'allocate->' if allocation else ''}rotate->pack->attend in float64 "
                      f"({spent:.1f} s); BLAS pool {threads} threads, Python loops on one core",
            "single_thread": single}


def cpu_single_thread(budget_s: float = 3.0) -> dict:
    """The oracle's whole layer on the tiny f32 and the one-layer 7B workloads
    with one BLAS thread (query tokens per second)."""
    import oracle as O
    import synth
    from threadpoolctl import threadpool_limits

    out = {}
    with threadpool_limits(limits=1, user_api="blas"):
        for cid in (1, 2):
            w = synth.workload(cid)
            wt = synth.layer_weights(w, 0)
            cap = sum(n * min(k, w.G) for n, k in zip(w.type_counts(), w.k_by_type))
            a = synth.sample_activations(w, 0, 0)
            done, spent = 0, 0.0
            while spent < budget_s or done == 0:
                t0 = time.perf_counter()
                O.pipeline(a["h"][None], a["q"][None], a["k"][None], a["v"][None], w.types(), wt, w.mode,
                           w.k_by_type, w.G, w.tau, w.kmin, w.kmax, cap=cap)
                spent += time.perf_counter() - t0
                done += 1
            out[w.name] = {"value": done * w.Tq / spent, "unit": "query-tokens/s", "calls": done,
                           "seconds": round(spent, 2)}
    return out


def causal_flops(w) -> float:
    """Matrix-core work of one prefix self-attention call: q.k over the causal
    triangle, P.Z over the same pairs (dense head width in the rotated space),
    and the back-rotation of every query."""
    pairs = w.T * (w.T + 1) / 2
    return w.B * w.H * (2 * pairs * 2 * w.dh + 2 * w.T * w.dh * w.dh)


def cpu_baseline_causal(w, masks, budget_s: float = 12.0) -> dict:
    """The float64 oracle's prefix self-attention on whole prefixes of layer 0."""
    import oracle as O
    import synth
    from threadpoolctl import threadpool_info

    wt = synth.layer_weights(w, 0)
    done, spent = 0, 0.0
    while spent < budget_s and done < w.B:
        a = synth.sample_activations(w, 0, done, ("q", "k", "v"))
        m = masks[done][None]
        z = O.rotate(a["v"][None], wt["R"])
        off, Vp = O.pack(z, m, w.G, w.T * w.G)
        t0 = time.perf_counter()
        O.attend_packed_causal(a["q"][None], a["k"][None], m, off, Vp, wt["R"], w.G)
        spent += time.perf_counter() - t0
        done += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": done * w.T / spent, "unit": "query-tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"layer 0, prefixes 0..{done - 1} of {w.B}: causal attention over the packed cache in "
                      f"float64 ({spent:.1f} s, pack excluded); BLAS pool {threads} threads"}


def cpu_baseline_full(w, budget_s: float = 12.0) -> dict:
    """The float64 oracle on whole prefixes of layer 0 at full width: router,
    per-type top-K, full-width cache, attention over the rebuilt values."""
    import oracle as O
    import synth
    from threadpoolctl import threadpool_info

    wt = synth.layer_weights(w, 0)
    R = synth.full_rotation(w, 0)["R"]
    cap = sum(n * min(k, w.G) for n, k in zip(w.type_counts(), w.k_by_type))
    done, spent = 0, 0.0
    while spent < budget_s and done < w.B:
        a = synth.sample_activations(w, 0, done)
        t0 = time.perf_counter()
        sc = O.router_mlp2(a["h"][None], w.types(), wt["W_r"], wt["b_r"], wt["E"], wt["W1"], wt["b1"], wt["W2"],
                           wt["b2"])
        m = O.select_groups(sc, O.group_budget(sc, w.types(), w.mode, w.k_by_type, w.G))
        off, Vp = O.pack_full(a["v"][None], m, R, w.G, cap)
        O.attend_full(a["q"][None], a["k"][None], m, off, Vp, R, w.G)
        spent += time.perf_counter() - t0
        done += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": done * w.Tq / spent, "unit": "query-tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"layer 0, prefixes 0..{done - 1} of {w.B}: route->full-width cache->values->attend in "
                      f"float64 ({spent:.1f} s); BLAS pool {threads} threads"}


def full_width(args, w):
    """The paper's routing space: one R over all 32 x 128 value dims, S = 16
    groups of 256. A step is every layer's route (G = S) -> full-width
    rotate + pack -> routed values -> attention; the transposed R of each layer
    is prepared once before timing (R is frozen)."""
    import concurrent.futures as cf

    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import FullWidthBuffers, LayerBuffers, run_full_layer

    dev = torch.device("cuda:0")
    dt = torch.bfloat16
    S = w.G
    budget = rs.make_budget(rs.TOPK, w.k_by_type)
    cap = sum(n * min(k, S) for n, k in zip(w.type_counts(), w.k_by_type))
    types = torch.from_numpy(np.broadcast_to(w.types(), (w.B, w.T)).copy()).to(dev)
    put = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    layers = []
    t_gen = time.time()
    for l in range(w.L):
        wt = synth.layer_weights(w, l)
        router = rs.Router.mlp2(*(put(wt[n]) for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2")))
        acts = {n: torch.empty(sh, dtype=dt, device=dev) for n, sh in
                (("h", (w.B, w.T, w.d)), ("q", (w.B, w.Tq, w.H, w.dh)), ("k", (w.B, w.T, w.H, w.dh)),
                 ("v", (w.B, w.T, w.H, w.dh)))}
        with cf.ThreadPoolExecutor(16) as ex:
            for b0 in range(0, w.B, 16):
                parts = list(ex.map(lambda b: synth.sample_activations(w, l, b), range(b0, min(w.B, b0 + 16))))
                for i, p_ in enumerate(parts):
                    for n in acts:
                        acts[n][b0 + i].copy_(torch.from_numpy(p_[n]))
        # a Haar rotation of d_v = 4096 per layer, drawn on the device from a
        # seeded generator (QR of a Gaussian with the sign fix); inputs only
        g = torch.Generator(device=dev)
        g.manual_seed(1000 + l)
        qm, rm = torch.linalg.qr(torch.randn(w.dv, w.dv, generator=g, device=dev))
        R = (qm * torch.sign(torch.diagonal(rm))[None, :]).to(dt).contiguous()
        Rt = rs.full_transpose(R)
        del qm, rm
        rb = LayerBuffers.allocate(w.B, w.T, 1, 128, S, 1, 1, dt, device=dev, with_z=False,
                                   ws_bytes=rs.route_workspace_size(w.B, w.T, S, w.d, router))
        fb = FullWidthBuffers.allocate(w.B, w.T, w.H, w.dh, S, w.Tq, cap, dt, device=dev)
        layers.append(dict(acts=acts, router=router, R=R, Rt=Rt, rb=rb, fb=fb))
        print(f"# layer {l} inputs resident ({time.time() - t_gen:.1f} s)", file=sys.stderr, flush=True)
    torch.cuda.synchronize()

    def route(L):
        rb = L["rb"]
        rs.route(types, budget, S, h=L["acts"]["h"], router=L["router"], workspace=rb.workspace,
                 out={"mask": rb.mask, "idx": rb.idx, "count": rb.count, "scores": rb.scores})

    def layer(L):
        route(L)
        a = L["acts"]
        run_full_layer(a["q"], a["k"], a["v"], L["rb"].mask, L["Rt"], L["R"], S, L["fb"], budget=budget,
                       type_counts=w.type_counts())

    def rot(L):
        fb = L["fb"]
        rs.full_rotate_pack(L["acts"]["v"], L["Rt"], L["rb"].mask, S, cap, workspace=fb.workspace,
                            out=(fb.offsets, fb.Vp))

    def vals(L):
        fb = L["fb"]
        rs.full_values(L["R"], L["rb"].mask, fb.offsets, fb.Vp, S, w.H, workspace=fb.workspace, out=fb.Vh)

    def att(L):
        fb, a = L["fb"], L["acts"]
        rs.attend_values(a["q"], a["k"], fb.Vh, out=fb.out)

    for L in layers:
        layer(L)
    torch.cuda.synchronize()
    eager_out = layers[-1]["fb"].out.clone()
    stream = torch.cuda.Stream()
    graphs = {}
    for name, fn in (("step", layer), ("route", route), ("rotate", rot), ("values", vals), ("attend", att)):
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=stream):
            for L in layers:
                fn(L)
        graphs[name] = gr
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_warm = warm_up(graphs["step"].replay, args.warmup)
    e0.record()
    for _ in range(args.steps):
        graphs["step"].replay()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    if not torch.equal(layers[-1]["fb"].out, eager_out):
        raise RuntimeError("graph replay output differs from the eager pass")
    # each call type alone: HIP events around back-to-back replays of the
    # graph holding the 32 layers' calls of that type (same inputs)
    reps = max(2, args.steps // 4)
    per_call = {}
    for name in ("route", "rotate", "values", "attend"):
        warm_up(graphs[name].replay, 1)
        e0.record()
        for _ in range(reps):
            graphs[name].replay()
        e1.record()
        torch.cuda.synchronize()
        per_call[name] = e0.elapsed_time(e1) / (reps * w.L) * 1e3
    if not torch.equal(layers[-1]["fb"].out, eager_out):
        raise RuntimeError("replays changed the output")
    # algorithmic work: every kept group of a routed token costs 2 * d_v * ds
    # flops in the rotation and again in the rebuild of its value
    masks = layers[0]["rb"].mask.cpu().numpy().view(np.uint32)
    full = (1 << S) - 1
    routed_groups = int(sum(bin(int(m)).count("1") for m in masks.reshape(-1) if int(m) != full))
    n_routed = int(np.sum(masks != full))
    flops = 2 * w.dv * w.ds * routed_groups
    dense_flops = 2 * w.dv * w.dv * n_routed
    dom = max(("rotate", "values"), key=lambda n: per_call[n])
    tflops = flops / (per_call[dom] * 1e-6) / 1e12
    line = {
        "metric": FULL_METRIC, "value": w.B * w.Tq * w.L / (ms_step * 1e-3), "unit": "query-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded Gaussian activations/weights, Haar rotations drawn on the device)",
        "config": {"workload": w.name, "layers": w.L, "prefixes": w.B, "kv_tokens": w.T, "visual": w.n_vis,
                   "language": w.n_lang, "proprio": w.n_prop, "queries": w.Tq, "heads": w.H, "head_dim": w.dh,
                   "d_v": w.dv, "groups": S, "group_dim": w.ds, "latent_roles": w.C,
                   "keep": {"vis": w.k_vis, "lang": w.k_lang, "prop": w.k_prop},
                   "value_counts": "query tokens x layers per second (B*Tq*L / step time)", "graphs": True},
        "roofline": {"kernel": f"rolesub_full_{'rotate_pack' if dom == 'rotate' else 'values'} "
                               f"(k_full_prep + k_full_gemm)", "bound": "mfma",
                     "achieved": tflops, "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / BF16_MFMA_PEAK_TFLOPS, "traffic": None,
                     "algorithmic_flops_per_launch": flops, "avg_launch_us": per_call[dom],
                     "dense_flops_per_launch": dense_flops},
        "detail": {"warmup_steps_run": n_warm, "per_layer_us": per_call, "routed_tokens_per_layer": n_routed,
                   "routed_groups_per_layer": routed_groups,
                   "dense_tflops_executed": dense_flops / (per_call[dom] * 1e-6) / 1e12},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_full(w)
    print(json.dumps(line), flush=True)


def _graph(fn):
    """fn's launches captured once into a HIP graph; returns its replay."""
    import torch
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        fn()
    return g.replay


def stress_stages(reps: int = 50) -> dict:
    """The G = 32 stress workload at full size (128 prefixes x 2048 tokens,
    64 queries, 4-dim groups, threshold budgets on given logits): selection,
    rotate + pack and attention, each captured in a graph and replayed
    `reps` times with an event around every replay."""
    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import pack_capacity

    w = synth.workload(5)
    dev, dt = torch.device("cuda:0"), torch.bfloat16
    g = torch.Generator(device=dev)
    g.manual_seed(w.seed)
    q = torch.randn((w.B, w.Tq, w.H, w.dh), generator=g, device=dev, dtype=dt)
    k = torch.randn((w.B, w.T, w.H, w.dh), generator=g, device=dev, dtype=dt)
    v = torch.randn((w.B, w.T, w.H, w.dh), generator=g, device=dev, dtype=dt)
    R = torch.from_numpy(synth.layer_weights(w, 0)["R"]).to(dev).to(dt)
    scores = torch.from_numpy(np.stack([synth.sample_scores(w, 0, b) for b in range(w.B)])).to(dev)
    types = torch.from_numpy(np.broadcast_to(w.types(), (w.B, w.T)).copy()).to(dev)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    sel = {"mask": torch.empty((w.B, w.T), dtype=torch.int32, device=dev),
           "idx": torch.empty((w.B, w.T, w.G), dtype=torch.uint8, device=dev),
           "count": torch.empty((w.B, w.T), dtype=torch.uint8, device=dev),
           "scores": torch.empty((w.B, w.T, w.G), dtype=torch.float32, device=dev)}
    offsets = torch.empty((w.B, w.T + 1), dtype=torch.int32, device=dev)
    Vp = torch.empty((w.B, w.H, cap, w.ds), dtype=dt, device=dev)
    out = torch.empty((w.B, w.Tq, w.H, w.dh), dtype=dt, device=dev)
    f_sel = lambda: rs.route(types, budget, w.G, scores_in=scores, out=sel)
    f_rp = lambda: rs.rotate_pack(v, R, sel["mask"], w.G, cap, out=(offsets, Vp))
    f_att = lambda: rs.attend(q, k, sel["mask"], offsets, Vp, R, w.G, out=out)

    def f_step():
        f_sel()
        f_rp()
        f_att()

    f_step()
    torch.cuda.synchronize()
    total_k = int(offsets[:, -1].sum().item())
    by = stage_bytes(w, total_k // w.B, total_k)
    res = {"workload": w.name, "prefixes": w.B, "kv_tokens": w.T, "queries": w.Tq, "groups": w.G,
           "kept_groups_per_prefix": total_k / w.B, "inputs": "device-seeded Gaussian q, k, v; seeded logits"}
    for name, fn, key in (("select", f_sel, "route"), ("rotate_pack", f_rp, "rotate_pack"),
                          ("attend", f_att, "attend"), ("step", f_step, None)):
        us = timed_replays(_graph(fn), reps)
        mean = float(np.mean(us))
        r = {"us": dist(us), "avg_us": mean}
        nb = sum(by.values()) if key is None else by[key]
        gbs = nb / (mean * 1e-6) / 1e9
        r.update({"algorithmic_bytes": nb, "GBs": gbs, "frac_of_peak": gbs / HBM_PEAK_GBS})
        res[name] = r
    res["attend_query_tokens_per_s"] = w.B * w.Tq / (res["attend"]["avg_us"] * 1e-6)
    del q, k, v, Vp
    torch.cuda.empty_cache()
    return res


def small_layer_calls(cid: int, min_bytes: float = 1.1e9, reps: int = 50) -> dict:
    """One 7B-shape layer call (route -> rotate + pack -> attend) of a small
    workload, per call: cold, cycling through enough distinct copies of every
    input (own activations, router weights and rotations) that together exceed
    the 256 MB memory-side cache, and hot (attention repeated on one copy)."""
    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import LayerBuffers, pack_capacity, run_layer

    w = synth.workload(cid)
    dev, dt = torch.device("cuda:0"), torch.bfloat16
    g = torch.Generator(device=dev)
    g.manual_seed(100 + cid)
    rnd = lambda shape, std=1.0: (torch.randn(shape, generator=g, device=dev, dtype=torch.float32) * std).to(dt)
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    types = torch.from_numpy(np.broadcast_to(w.types(), (w.B, w.T)).copy()).to(dev)
    fin = w.router_in
    per_copy = 2 * (w.B * w.T * (w.d + 2 * w.H * w.dh) + w.B * w.Tq * w.H * w.dh + w.Hr * fin + w.H * w.dh * w.dh)
    n = max(8, int(np.ceil(min_bytes / per_copy)))
    copies = []
    for _ in range(n):
        router = rs.Router.mlp2(rnd((w.C, w.d), w.d ** -0.5), rnd((w.C,), w.d ** -0.5), rnd((w.C, w.d_e)),
                                rnd((w.Hr, fin), fin ** -0.5), rnd((w.Hr,), fin ** -0.5),
                                rnd((w.G, w.Hr), w.Hr ** -0.5), rnd((w.G,), w.Hr ** -0.5))
        bufs = LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, dt, device=dev, with_z=False,
                                     ws_bytes=rs.route_workspace_size(w.B, w.T, w.G, w.d, router))
        copies.append(dict(h=rnd((w.B, w.T, w.d)), q=rnd((w.B, w.Tq, w.H, w.dh)), k=rnd((w.B, w.T, w.H, w.dh)),
                           v=rnd((w.B, w.T, w.H, w.dh)), R=rnd((w.H, w.dh, w.dh), w.dh ** -0.5), router=router,
                           bufs=bufs))

    def layer(c):
        run_layer(c["h"], c["q"], c["k"], c["v"], types, c["R"], budget, w.G, c["bufs"], router=c["router"],
                  type_counts=w.type_counts(), fused=True)

    def att(c):
        b = c["bufs"]
        rs.attend(c["q"], c["k"], b.mask, b.offsets, b.Vp, c["R"], w.G, out=b.out)

    for c in copies:
        layer(c)
    torch.cuda.synchronize()
    total_k = int(copies[0]["bufs"].offsets[:, -1].sum().item())
    by = stage_bytes(w, total_k // w.B, total_k)
    res = {"workload": w.name, "prefixes": w.B, "kv_tokens": w.T, "copies_cycled": n,
           "bytes_cycled": n * per_copy, "inputs": "device-seeded Gaussian activations and weights"}
    for name, fn in (("layer_cold", lambda: [layer(c) for c in copies]),
                     ("attend_cold", lambda: [att(c) for c in copies]),
                     ("attend_hot", lambda: [att(copies[0]) for _ in copies])):
        us = timed_replays(_graph(fn), reps, per=n)
        mean = float(np.mean(us))
        nb = sum(by.values()) if name == "layer_cold" else by["attend"]
        gbs = nb / (mean * 1e-6) / 1e9
        res[name] = {"us_per_call": dist(us), "avg_us": mean, "algorithmic_bytes": nb, "GBs": gbs,
                     "frac_of_peak": gbs / HBM_PEAK_GBS}
    res["note"] = ("latency-bound: a call moves a few MB (tens of MB at batch 16); hot = inputs resident in the "
                   "memory-side cache")
    del copies
    torch.cuda.empty_cache()
    return res


def other_workloads(args) -> dict:
    """The stress workload's stages and the small workloads' per-call times."""
    import synth
    out = {synth.workload(5).name: stress_stages()}
    for cid in (2, 3):
        out[synth.workload(cid).name] = small_layer_calls(cid)
    return {"other_workloads": out}


def full_width_probe(reps: int = 6):
    """The full-width layer calls at the 7B full-width shape (64 prefixes of
    81 tokens: 32 visual keeping 4 of 16 groups, 48 language and 1 proprio in
    value space; d_v = 4096), every call repeated on the same inputs."""
    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import FullWidthBuffers, run_full_layer

    w = synth.workload(6)
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(w.seed)
    rng = np.random.default_rng(w.seed)
    R = (torch.randn(w.dv, w.dv, device=dev, generator=g) / w.dv ** 0.5).bfloat16()
    Rt = rs.full_transpose(R)
    q = torch.randn(w.B, w.Tq, w.H, w.dh, device=dev, generator=g).bfloat16()
    k = torch.randn(w.B, w.T, w.H, w.dh, device=dev, generator=g).bfloat16()
    v = torch.randn(w.B, w.T, w.H, w.dh, device=dev, generator=g).bfloat16()
    S = w.G
    m = np.zeros((w.B, w.T), np.uint32)
    for b in range(w.B):
        for t in range(w.n_vis):
            m[b, t] = int(np.sum(1 << rng.choice(S, w.k_vis, replace=False)))
        m[b, w.n_vis:] = (1 << S) - 1
    mask = torch.from_numpy(m.view(np.int32)).to(dev)
    cap = sum(n * min(kk, S) for n, kk in zip(w.type_counts(), w.k_by_type))
    bufs = FullWidthBuffers.allocate(w.B, w.T, w.H, w.dh, S, w.Tq, cap, torch.bfloat16, device=dev)
    budget = rs.make_budget(rs.TOPK, w.k_by_type)
    for _ in range(reps):
        run_full_layer(q, k, v, mask, Rt, R, S, bufs, budget=budget, type_counts=w.type_counts())
    torch.cuda.synchronize()
    print(json.dumps({"full_width_probe_calls": reps, "workload": w.name}), flush=True)


def prefix_attention(args, w):
    """Prefix self-attention (rolesub_attend_causal) at the 7B-stack layer shape:
    every prefix token is a query and sees the keys before it; masks carry the
    workload's per-type budgets, values are packed by the fused rotate+pack."""
    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import pack_capacity

    dev = torch.device("cuda:0")
    w = w.replace(Tq=w.T)
    dt = torch.bfloat16
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    put = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    masks0 = None
    layers = []
    t_gen = time.time()
    for l in range(w.L):
        wt = synth.layer_weights(w, l)
        acts = {n: torch.empty((w.B, w.T, w.H, w.dh), dtype=dt, device=dev) for n in ("q", "k", "v")}
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(16) as ex:
            for b0 in range(0, w.B, 16):
                parts = list(ex.map(lambda b: synth.sample_activations(w, l, b, ("q", "k", "v")),
                                    range(b0, min(w.B, b0 + 16))))
                for i, p in enumerate(parts):
                    for n in acts:
                        acts[n][b0 + i].copy_(torch.from_numpy(p[n]))
        m = np.stack([synth.synthetic_masks(w, l, b) for b in range(w.B)])
        if l == 0:
            masks0 = m
        mask = torch.from_numpy(m.view(np.int32)).to(dev)
        R = put(wt["R"])
        offsets = torch.empty((w.B, w.T + 1), dtype=torch.int32, device=dev)
        Vp = torch.empty((w.B, w.H, cap, w.ds), dtype=dt, device=dev)
        rs.rotate_pack(acts["v"], R, mask, w.G, cap, out=(offsets, Vp))
        del acts["v"]
        out = torch.empty((w.B, w.T, w.H, w.dh), dtype=dt, device=dev)
        layers.append(dict(q=acts["q"], k=acts["k"], mask=mask, offsets=offsets, Vp=Vp, R=R, out=out))
        print(f"# layer {l} inputs resident ({time.time() - t_gen:.1f} s)", file=sys.stderr, flush=True)
    torch.cuda.synchronize()

    def att(L):
        rs.attend_causal(L["q"], L["k"], L["mask"], L["offsets"], L["Vp"], L["R"], w.G, out=L["out"])

    for L in layers:
        att(L)
    torch.cuda.synchronize()
    eager_out = layers[-1]["out"].clone()
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for L in layers:
            att(L)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_warm = warm_up(g.replay, args.warmup)
    e0.record()
    for _ in range(args.steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    if not torch.equal(layers[-1]["out"], eager_out):
        raise RuntimeError("graph replay output differs from the eager pass")
    call_us = ms_step * 1e3 / w.L
    sum_k = int(layers[0]["offsets"][:, -1].sum().item()) // w.B
    a_bytes = attend_bytes(w, sum_k, 2)
    gbs = a_bytes / (call_us * 1e-6) / 1e9
    tflops = causal_flops(w) / (call_us * 1e-6) / 1e12
    line = {
        "metric": PREFIX_METRIC, "value": w.B * w.T * w.L / (ms_step * 1e-3), "unit": "query-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded Gaussian activations, Haar rotations, per-type group budgets)",
        "config": {"workload": w.name + "-prefix-self-attention", "layers": w.L, "prefixes": w.B,
                   "kv_tokens": w.T, "queries": w.T, "heads": w.H, "head_dim": w.dh, "groups": w.G,
                   "keep": {"vis": w.k_vis, "lang": w.k_lang, "prop": w.k_prop},
                   "value_counts": "prefix query tokens x layers per second", "graphs": True},
        "roofline": {"kernel": "rolesub_attend_causal (k_attend_bf16, causal)", "bound": "hbm",
                     "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                     "traffic": None, "algorithmic_bytes_per_launch": a_bytes, "avg_launch_us": call_us,
                     "mfma": {"achieved": tflops, "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                              "frac": tflops / BF16_MFMA_PEAK_TFLOPS, "flops_per_launch": causal_flops(w)}},
        "detail": {"warmup_steps_run": n_warm},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_causal(w, masks0)
    print(json.dumps(line), flush=True)


def retention(args, w):
    """Token retention at the 7B-stack shape: 64 prefixes whose 512 visual
    tokens come from two 256-patch views; per view the 64 highest-scoring
    tokens are kept (128 retained, the workload's visual count) and their
    hidden states (d = 4096, bf16) are gathered into the compact prefix."""
    import torch

    import paper_2608_18410_amd as rs

    dev = torch.device("cuda:0")
    B, views, per_view, d = w.B, 2, 256, w.d
    keep = [w.n_vis // views] * views
    N, K = views * per_view, sum(keep)
    rng = np.random.default_rng(w.seed)
    n_sets = 6  # distinct inputs cycled so no call finds its data in the memory-side cache
    sets = []
    for _ in range(n_sets):
        sc = torch.from_numpy(rng.standard_normal((B, N)).astype(np.float32)).to(dev)
        h = torch.randn(B, N, d, device=dev, dtype=torch.float32).to(torch.bfloat16)
        sets.append(dict(scores=sc, h=h, idx=torch.empty((B, K), dtype=torch.int32, device=dev),
                         out=torch.empty((B, K, d), dtype=torch.bfloat16, device=dev)))
    torch.cuda.synchronize()

    def call(S):
        rs.retain_tokens(S["scores"], [per_view] * views, keep, out=S["idx"])
        rs.gather_tokens(S["h"], S["idx"], out=S["out"])

    stream = torch.cuda.Stream()
    for S in sets:
        call(S)
    torch.cuda.synchronize()
    ref = sets[0]["out"].clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for S in sets:
            call(S)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_warm = warm_up(g.replay, args.warmup)
    e0.record()
    for _ in range(args.steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    if not torch.equal(sets[0]["out"], ref):
        raise RuntimeError("graph replay output differs from the eager pass")
    call_us = e0.elapsed_time(e1) * 1e3 / (args.steps * n_sets)
    row = d * 2
    moved = B * N * 4 + B * K * 4 * 2 + 2 * B * K * row  # scores, indices (written, read), rows read + written
    gbs = moved / (call_us * 1e-6) / 1e9
    line = {
        "metric": RETAIN_METRIC, "value": B * K / (call_us * 1e-6), "unit": "retained tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": call_us * n_sets / 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32 scores, bf16 rows",
        "data": "synthetic (seeded Gaussian scores and hidden states)",
        "config": {"workload": w.name + "-token-retention", "prefixes": B, "views": views,
                   "tokens_per_view": per_view, "kept_per_view": keep[0], "row": f"hidden {d} x bf16",
                   "value_counts": "retained tokens per second (selection + gather per call)", "graphs": True},
        "roofline": {"kernel": "rolesub_retain_tokens + rolesub_gather_tokens", "bound": "hbm", "achieved": gbs,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": moved, "avg_launch_us": call_us},
        "detail": {"warmup_steps_run": n_warm},
    }
    if not args.no_cpu_baseline:
        import oracle as O
        from threadpoolctl import threadpool_info
        nb = 8  # prefixes per oracle call
        sc = sets[0]["scores"][:nb].cpu().numpy()
        hh = sets[0]["h"][:nb].float().cpu().numpy()
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            idx = O.retain_tokens(sc, [per_view] * views, keep)
            O.gather_tokens(hh, idx)
            reps += 1
        spent = time.perf_counter() - t0
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        line["cpu_baseline"] = {"value": reps * nb * K / spent, "unit": "retained tokens/s", "cores": 1,
                                "kind": "oracle",
                                "sample": f"{reps} oracle calls on {nb} of the {B} prefixes (selection + gather, "
                                          f"{spent:.1f} s); Python loops on one core (BLAS pool {threads} unused)"}
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=4, help="workload id (4: 32-layer 7B stack)")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0: workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other workloads (G = 32 stress, one-layer and batch-16 shapes) after the step")
    ap.add_argument("--eager", action="store_true", help="issue the calls directly, no HIP graphs")
    ap.add_argument("--micro-batches", type=int, default=2,
                    help="split the step's prefixes into this many contiguous micro-batches, each through "
                         "every layer on its own stream (1: the whole batch per call on one stream)")
    ap.add_argument("--prefix-attention", action="store_true",
                    help="time prefix self-attention (rolesub_attend_causal) at the same shape instead")
    ap.add_argument("--full-width", action="store_true",
                    help="the paper's full-width routing space (one R over d_v = 4096, S = 16) instead")
    ap.add_argument("--allocation", action="store_true",
                    help="route with role-driven per-token budgets (rolesub_route_allocate) in the step")
    ap.add_argument("--retention", action="store_true",
                    help="time token retention + gather of the retained hidden states instead")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 4 times (counter calibration) and exit")
    ap.add_argument("--full-width-probe", action="store_true",
                    help="only run the full-width layer calls (rotate + pack, values, attention) 6 times at the "
                         "7B full-width layer shape with a random, non-orthogonal R (for counter collection; "
                         "the counts do not depend on R's values) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path would shard by prefix or by head, with no exchange between GPUs)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_18410_amd as rs
    import synth
    from paper_2608_18410_amd.pipeline import LayerBuffers, micro_batches, on_streams, pack_capacity, run_layer

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        # A plain copy of known size: its FETCH_SIZE / WRITE_SIZE readings
        # calibrate the HBM traffic counters (1 GiB read + 1 GiB written per copy).
        src = torch.ones(2 ** 29, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": src.numel() * 2, "copies": 4}), flush=True)
        return
    rs.load()
    dev = torch.device("cuda:0")
    if args.full_width_probe:
        full_width_probe()
        return
    w = synth.workload(args.workload)
    if args.layers:
        w = w.replace(L=args.layers)
    if args.full_width:
        full_width(args, synth.workload(6).replace(L=args.layers) if args.layers else synth.workload(6))
        return
    if args.prefix_attention:
        prefix_attention(args, w)
        return
    if args.retention:
        retention(args, w)
        return
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    if args.allocation and (w.scores_in or w.mode != rs.TOPK):
        raise SystemExit("--allocation needs a workload with a router and fixed per-type budgets")
    budget = rs.make_budget(w.mode, w.k_by_type, w.tau, w.kmin, w.kmax)
    cap = pack_capacity(w.mode, w.k_by_type, w.type_counts(), w.T, w.G, w.kmax)
    types = torch.from_numpy(np.broadcast_to(w.types(), (w.B, w.T)).copy()).to(dev)
    # Micro-batches: contiguous ranges of prefixes, each taken through every
    # layer on its own stream. Prefixes do not interact, so the calls of one
    # range depend only on that range's earlier calls, and the kernels of the
    # ranges overlap on the GPU, filling each other's ramp-up and tail.
    mbs = micro_batches(w.B, args.micro_batches)

    # ---- inputs resident in HBM
    t_gen = time.time()
    layers = []
    for l in range(w.L):
        wt = synth.layer_weights(w, l)
        put = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
        router = rs.Router.mlp2(*(put(wt[n]) for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2")))
        names = ("q", "k", "v") if w.scores_in else ("h", "q", "k", "v")
        acts = {n: torch.empty(s, dtype=dt, device=dev) for n, s in
                (("h", (w.B, w.T, w.d)), ("q", (w.B, w.Tq, w.H, w.dh)), ("k", (w.B, w.T, w.H, w.dh)),
                 ("v", (w.B, w.T, w.H, w.dh))) if n in names}
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(16) as ex:
            for b0 in range(0, w.B, 16):
                parts = list(ex.map(lambda b: synth.sample_activations(w, l, b, names),
                                    range(b0, min(w.B, b0 + 16))))
                for i, p in enumerate(parts):
                    for n in names:
                        acts[n][b0 + i].copy_(torch.from_numpy(p[n]))
        scores = None
        if w.scores_in:
            scores = torch.from_numpy(np.stack([synth.sample_scores(w, l, b) for b in range(w.B)])).to(dev)
        # one route workspace per micro-batch (calls on one workspace must not
        # overlap), carved from the layer's workspace at 256-byte boundaries
        wsz = [(rs.route_allocate_workspace_size if args.allocation else rs.route_workspace_size)(
            b1 - b0, w.T, w.G, w.d, router) for b0, b1 in mbs]
        ws_off = [0]
        for n in wsz:
            ws_off.append(ws_off[-1] + (n + 255) // 256 * 256)
        bufs = LayerBuffers.allocate(w.B, w.T, w.H, w.dh, w.G, w.Tq, cap, dt, ws_bytes=ws_off[-1], device=dev,
                                     with_z=False)
        mb_bufs = [bufs.rows(b0, b1, bufs.workspace[ws_off[i]:ws_off[i] + max(wsz[i], 1)])
                   for i, (b0, b1) in enumerate(mbs)]
        alloc = None
        if args.allocation:
            alloc = dict(w_pri=put(synth.priority_weights(w, l)),
                         priority=torch.empty((w.B, w.T), dtype=torch.float32, device=dev),
                         k=torch.empty((w.B, w.T), dtype=torch.uint8, device=dev))
        layers.append(dict(acts=acts, router=router if scores is None else None, scores=scores,
                           R=put(wt["R"]), bufs=bufs, mb_bufs=mb_bufs, alloc=alloc))
        print(f"# layer {l} inputs resident ({time.time() - t_gen:.1f} s)", file=sys.stderr, flush=True)
    torch.cuda.synchronize()

    def pre(L, i):
        # route -> rotate + pack for micro-batch i of layer L
        (b0, b1), bf, al = mbs[i], L["mb_bufs"][i], L["alloc"]
        a = {n: t[b0:b1] for n, t in L["acts"].items()}
        if al is not None:
            rs.route_allocate(types[b0:b1], w.k_by_type, w.G, a["h"], L["router"], al["w_pri"],
                              workspace=bf.workspace,
                              out={"mask": bf.mask, "idx": bf.idx, "count": bf.count, "scores": bf.scores,
                                   "priority": al["priority"][b0:b1], "k": al["k"][b0:b1]})
        else:
            rs.route(types[b0:b1], budget, w.G, h=a.get("h"), router=L["router"],
                     scores_in=None if L["scores"] is None else L["scores"][b0:b1], workspace=bf.workspace,
                     out={"mask": bf.mask, "idx": bf.idx, "count": bf.count, "scores": bf.scores})
        rs.rotate_pack(a["v"], L["R"], bf.mask, w.G, cap, out=(bf.offsets, bf.Vp))

    def att(L, i=None):
        # attention for micro-batch i of layer L, or for the whole batch
        if i is None:
            a, bf = L["acts"], L["bufs"]
        else:
            (b0, b1), bf = mbs[i], L["mb_bufs"][i]
            a = {n: t[b0:b1] for n, t in L["acts"].items()}
        rs.attend(a["q"], a["k"], bf.mask, bf.offsets, bf.Vp, L["R"], w.G, out=bf.out)

    def run_mb(i):
        for L in layers:
            pre(L, i)
            att(L, i)

    # ---- one eager pass, micro-batch after micro-batch on one stream (also
    # the reference for the graph replays)
    for i in range(len(mbs)):
        run_mb(i)
    torch.cuda.synchronize()
    eager_out = layers[-1]["bufs"].out.clone()

    if not args.eager:
        # the whole step (every micro-batch through every layer, each
        # micro-batch on its own stream) is one graph; a second graph holds
        # only the layers' whole-batch attention calls, for timing that kernel
        stream = torch.cuda.Stream()
        mb_streams = [torch.cuda.Stream() for _ in mbs]
        g_step, g_att = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_step, stream=stream):
            on_streams(lambda i, b0, b1: run_mb(i), mbs, mb_streams)
        with torch.cuda.graph(g_att, stream=stream):
            for L in layers:
                att(L)
        step = g_step.replay
        att_all = g_att.replay
    else:
        def step():
            for i in range(len(mbs)):
                run_mb(i)

        def att_all():
            for L in layers:
                att(L)

    # K timed steps back to back, an event after each (the mean is the
    # reported step time; the spread comes from the same events). The events
    # exist before the warm-up, which ends with a synchronize, so the timed
    # steps follow it without an idle gap; the replays' output is checked
    # against the eager pass afterwards.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    n_warm = warm_up(step, args.warmup)
    ev[0].record()
    for i in range(args.steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    ms_step = ev[0].elapsed_time(ev[-1]) / args.steps
    if not torch.equal(layers[-1]["bufs"].out, eager_out):
        raise RuntimeError("graph replay output differs from the eager pass")

    # Attention kernel duration: HIP events on the launch stream around each
    # of >= 50 back-to-back replays of the attention calls of every layer
    # (same inputs as the last step), divided by the number of launches; this
    # includes the short dispatch gaps between consecutive kernels of one graph.
    reps = max(50, args.steps)
    att_us = timed_replays(att_all, reps, per=len(layers))
    att_ms = float(np.mean(att_us)) / 1e3
    if not torch.equal(layers[-1]["bufs"].out, eager_out):
        raise RuntimeError("attention replay output differs from the eager pass")

    alloc_us = None
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if args.allocation:
        # the allocation + selection kernel alone: the same call on the step's
        # own priorities and scores (it rewrites identical budgets and masks)
        def alloc_all():
            for L in layers:
                bf, al = L["bufs"], L["alloc"]
                rs.allocate_groups(al["priority"], types, w.k_by_type, w.G, scores=bf.scores,
                                   out={"k": al["k"], "mask": bf.mask, "idx": bf.idx, "count": bf.count})
        if not args.eager:
            g_alloc = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_alloc, stream=stream):
                alloc_all()
            alloc_run = g_alloc.replay
        else:
            alloc_run = alloc_all
        warm_up(alloc_run, 1)
        a0.record()
        for _ in range(reps):
            alloc_run()
        a1.record()
        torch.cuda.synchronize()
        alloc_us = a0.elapsed_time(a1) / (reps * len(layers)) * 1e3

    total_k = int(layers[0]["bufs"].offsets[:, -1].sum().item())
    sum_k = total_k // w.B
    per_stage = stage_bytes(w, sum_k, total_k)
    if args.allocation:
        # over the fixed-budget route: scores read again, priorities written
        # and read, token types and the budgets K_i
        per_stage["allocate"] = w.B * w.T * (4 * w.G + 8 + 1 + 1)
    a_bytes = per_stage["attend"]
    achieved = a_bytes / (att_ms * 1e-3) / 1e9
    value = w.B * w.Tq * w.L / (ms_step * 1e-3)
    extra = {}
    if not args.no_extra and not args.allocation and w.name == synth.workload(4).name:
        extra = other_workloads(args)
    copy = copy_rate()
    copy_gbs = copy["GBs"]["median"]

    line = {
        "metric": ALLOC_METRIC if args.allocation else METRIC,
        "value": value,
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded Gaussian activations/weights, Haar rotations; no trained weights)",
        "config": {"workload": w.name, "layers": w.L, "prefixes": w.B, "kv_tokens": w.T,
                   "visual": w.n_vis, "language": w.n_lang, "proprio": w.n_prop, "queries": w.Tq,
                   "heads": w.H, "head_dim": w.dh, "hidden": w.d, "groups": w.G,
                   "keep": {"vis": w.k_vis, "lang": w.k_lang, "prop": w.k_prop}
                   if w.mode == 0 else {"threshold": w.tau, "kmin": w.kmin, "kmax": w.kmax},
                   "budgets": "role-driven per-token allocation within each type (priority w^T a)"
                   if args.allocation else ("fixed per type" if w.mode == 0 else
                                            "threshold on given logits (selection only)"),
                   "value_counts": "query tokens x layers per second (B*Tq*L / step time)",
                   "graphs": not args.eager,
                   "micro_batches": [b1 - b0 for b0, b1 in mbs],
                   "schedule": "each micro-batch of prefixes through every layer on its own stream"
                   if len(mbs) > 1 else "the whole batch per call on one stream"},
        "roofline": {"kernel": "rolesub_attend (k_attend_bf16), whole-batch launches", "bound": "hbm",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": _traffic(w.name),
                     "algorithmic_bytes_per_launch": a_bytes, "avg_launch_us": att_ms * 1e3,
                     "launch_us": dist(att_us), "copy_GBs_same_run": copy_gbs,
                     "frac_of_copy": achieved / copy_gbs},
        "detail": {"warmup_steps_run": n_warm, "step_ms": dist(step_ms),
                   "copy": copy,
                   "attend_query_tokens_per_s": w.B * w.Tq / (att_ms * 1e-3),
                   "layers_per_s": w.L / (ms_step * 1e-3),
                   "allocate_select_us_per_layer": alloc_us,
                   "stage_algorithmic_bytes": per_stage,
                   "step_algorithmic_GBs": w.L * sum(per_stage.values()) / (ms_step * 1e-3) / 1e9,
                   **extra},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, allocation=args.allocation)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
