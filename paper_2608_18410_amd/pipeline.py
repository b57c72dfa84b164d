"""One layer of the hot path, route -> rotate -> pack -> attend, through the C ABI.

Orchestration only: buffers are allocated once per shape and reused, and the
four library calls are issued in order on one stream. A batch may also be
split into micro-batches (contiguous ranges of prefixes, each with views of
the buffers and its own route workspace) whose calls run on separate streams.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import rolesub as rs


def pack_capacity(mode: int, k_by_type, type_counts, T: int, G: int, kmax: int = 0) -> int:
    """Groups per (sample, head) the packed cache must hold for a budget."""
    if mode == rs.TOPK:
        return int(sum(n * min(k, G) for n, k in zip(type_counts, k_by_type)))
    return int(T * min(kmax, G))


@dataclass
class LayerBuffers:
    mask: torch.Tensor
    idx: torch.Tensor
    count: torch.Tensor
    scores: torch.Tensor
    z: torch.Tensor
    offsets: torch.Tensor
    Vp: torch.Tensor
    out: torch.Tensor
    workspace: torch.Tensor

    @staticmethod
    def allocate(B, T, H, dh, G, Tq, cap, dtype, out_dtype=None, ws_bytes=0, device="cuda", with_z=True):
        u8, i32, f32 = torch.uint8, torch.int32, torch.float32
        return LayerBuffers(
            mask=torch.empty((B, T), dtype=i32, device=device),
            idx=torch.empty((B, T, G), dtype=u8, device=device),
            count=torch.empty((B, T), dtype=u8, device=device),
            scores=torch.empty((B, T, G), dtype=f32, device=device),
            z=torch.empty((B, T, H, dh) if with_z else (0,), dtype=dtype, device=device),
            offsets=torch.empty((B, T + 1), dtype=i32, device=device),
            Vp=torch.empty((B, H, cap, dh // G), dtype=dtype, device=device),
            out=torch.empty((B, Tq, H, dh), dtype=out_dtype or dtype, device=device),
            workspace=torch.empty(max(int(ws_bytes), 256), dtype=u8, device=device),
        )

    def rows(self, b0: int, b1: int, workspace: torch.Tensor) -> "LayerBuffers":
        """The buffers of prefixes b0..b1-1 (views: every per-prefix buffer is
        sliced along its first dimension, so the calls on them write into this
        object's tensors), with their own route workspace."""
        sl = lambda t: t[b0:b1] if t.dim() > 1 else t
        return LayerBuffers(mask=self.mask[b0:b1], idx=self.idx[b0:b1], count=self.count[b0:b1],
                            scores=self.scores[b0:b1], z=sl(self.z), offsets=self.offsets[b0:b1],
                            Vp=self.Vp[b0:b1], out=self.out[b0:b1], workspace=workspace)


def micro_batches(B: int, n: int) -> list:
    """n contiguous, nearly equal ranges (b0, b1) of B prefixes. Prefixes do
    not interact, so the calls of one range may run on their own stream,
    concurrently with the others."""
    n = max(1, min(int(n), B))
    return [((i * B) // n, ((i + 1) * B) // n) for i in range(n)]


def on_streams(issue, ranges, streams) -> None:
    """Calls issue(i, b0, b1) for every range with streams[i] current: each
    stream first waits for the work already queued on the current stream,
    and the current stream then waits for all of them (also inside a HIP
    graph capture, where this makes parallel branches)."""
    cur = torch.cuda.current_stream()
    for s in streams:
        s.wait_stream(cur)
    for i, ((b0, b1), s) in enumerate(zip(ranges, streams)):
        with torch.cuda.stream(s):
            issue(i, b0, b1)
    for s in streams:
        cur.wait_stream(s)


def run_layer(h, q, k, v, types, R, budget: rs.Budget, G: int, bufs: LayerBuffers,
              router: rs.Router | None = None, scores_in=None, type_counts=None, fused=True,
              stream=None):
    """route -> rotate -> pack -> attend. With fused=True rotation and pack run
    as one call (rolesub_rotate_pack) and bufs.z is not written. Returns the
    buffers (filled asynchronously)."""
    rs.route(types, budget, G, h=h, router=router, scores_in=scores_in, workspace=bufs.workspace,
             out={"mask": bufs.mask, "idx": bufs.idx, "count": bufs.count, "scores": bufs.scores},
             stream=stream)
    if fused:
        rs.rotate_pack(v, R, bufs.mask, G, bufs.Vp.shape[2], budget=budget, type_counts=type_counts,
                       out=(bufs.offsets, bufs.Vp), stream=stream)
    else:
        rs.rotate_values(v, R, out=bufs.z, stream=stream)
        rs.pack_kv(bufs.z, bufs.mask, G, bufs.Vp.shape[2], budget=budget, type_counts=type_counts,
                   out=(bufs.offsets, bufs.Vp), stream=stream)
    rs.attend(q, k, bufs.mask, bufs.offsets, bufs.Vp, R, G, out=bufs.out, stream=stream)
    return bufs


@dataclass
class FullWidthBuffers:
    """Buffers of one full-width layer call: the cache (offsets, Vp), the
    head-major routed values Vh and the attention output."""
    offsets: torch.Tensor
    Vp: torch.Tensor
    Vh: torch.Tensor
    out: torch.Tensor
    workspace: torch.Tensor

    @staticmethod
    def allocate(B, T, H, dh, S, Tq, cap, dtype, out_dtype=None, device="cuda"):
        dv = H * dh
        return FullWidthBuffers(
            offsets=torch.empty((B, T + 1), dtype=torch.int32, device=device),
            Vp=torch.empty((B, cap, dv // S), dtype=dtype, device=device),
            Vh=torch.empty((B, H, T, dh), dtype=dtype, device=device),
            out=torch.empty((B, Tq, H, dh), dtype=out_dtype or dtype, device=device),
            workspace=torch.empty(max(rs.full_workspace_size(B, T, S), 256), dtype=torch.uint8, device=device),
        )


def run_full_layer(q, k, v, mask, Rt, R, S: int, bufs: FullWidthBuffers, budget=None, type_counts=None,
                   stream=None):
    """Full-width routing space for one layer, given the group masks:
    rotate + pack (routed tokens' kept groups of R^T v, value-space tokens
    verbatim) -> routed values from the cache -> attention per head."""
    B, T, H, dh = v.shape
    rs.full_rotate_pack(v, Rt, mask, S, bufs.Vp.shape[1], budget=budget, type_counts=type_counts,
                        workspace=bufs.workspace, out=(bufs.offsets, bufs.Vp), stream=stream)
    rs.full_values(R, mask, bufs.offsets, bufs.Vp, S, H, workspace=bufs.workspace, out=bufs.Vh, stream=stream)
    rs.attend_values(q, k, bufs.Vh, out=bufs.out, stream=stream)
    return bufs
