"""ctypes binding of librolesub.

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels. torch tensors supply device memory (data_ptr) and the current
HIP stream. Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librolesub.so")

F32, BF16 = 0, 1
VIS, LANG, PROP, ACT = 0, 1, 2, 3
TOPK, THRESHOLD = 0, 1
MLP2, ADDITIVE = 0, 1

EXPORTS = (
    "rolesub_status_str", "rolesub_last_error", "rolesub_version",
    "rolesub_rotate_values", "rolesub_route_workspace_size", "rolesub_route",
    "rolesub_pack_kv", "rolesub_rotate_pack", "rolesub_attend_workspace_size", "rolesub_attend",
    "rolesub_attend_causal", "rolesub_retain_tokens", "rolesub_gather_tokens",
    "rolesub_allocate_groups", "rolesub_route_allocate_workspace_size", "rolesub_route_allocate",
    "rolesub_full_workspace_size", "rolesub_full_transpose", "rolesub_full_rotate_pack", "rolesub_full_values",
    "rolesub_attend_values", "rolesub_route_noalloc",
)
ROUTE_NOALLOC_MAX_BYTES = 8 << 20


class RolesubError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn} -> {status_name(status)}: {message}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "T", "H", "dh", "G", "d")]


class Budget(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("k_by_type", ctypes.c_int32 * 4), ("tau", ctypes.c_float),
                ("kmin", ctypes.c_int32), ("kmax", ctypes.c_int32)]


class RouterDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("C", ctypes.c_int32), ("d_e", ctypes.c_int32),
                ("Hr", ctypes.c_int32), ("alpha_role", ctypes.c_float), ("alpha_lang", ctypes.c_float)] + \
               [(n, ctypes.c_void_p) for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2",
                                               "W_tok", "b_tok", "W_role", "W_lang", "b_lang")]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load librolesub.so (built in-tree by paper_2608_18410_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"librolesub is not built ({path} is missing); "
                          "run `python -m paper_2608_18410_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.rolesub_status_str.argtypes = [ctypes.c_int]
    lib.rolesub_status_str.restype = ctypes.c_char_p
    lib.rolesub_last_error.argtypes = []
    lib.rolesub_last_error.restype = ctypes.c_char_p
    lib.rolesub_version.argtypes = []
    lib.rolesub_version.restype = I32
    lib.rolesub_rotate_values.argtypes = [P, ctypes.c_int, P, P, P, P]
    lib.rolesub_route_workspace_size.argtypes = [P, P]
    lib.rolesub_route_workspace_size.restype = SZ
    lib.rolesub_route.argtypes = [P, ctypes.c_int, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.rolesub_route_noalloc.argtypes = [P, ctypes.c_int, P, P, P, P, P, P, P, P, P, P]
    lib.rolesub_pack_kv.argtypes = [P, ctypes.c_int, P, P, P, P, P, P, I64, P]
    lib.rolesub_rotate_pack.argtypes = [P, ctypes.c_int, P, P, P, P, P, P, P, I64, P]
    lib.rolesub_attend_workspace_size.argtypes = [P, I32]
    lib.rolesub_attend_workspace_size.restype = SZ
    lib.rolesub_attend.argtypes = [P, ctypes.c_int, I32, P, P, P, P, P, I64, P, ctypes.c_float, P,
                                   ctypes.c_int, P, SZ, P]
    lib.rolesub_attend_causal.argtypes = [P, ctypes.c_int, P, P, P, P, P, I64, P, ctypes.c_float, P,
                                          ctypes.c_int, P, SZ, P]
    lib.rolesub_retain_tokens.argtypes = [I32, I32, I32, P, P, P, P, P]
    lib.rolesub_gather_tokens.argtypes = [I32, I32, I32, I64, P, P, P, P]
    lib.rolesub_allocate_groups.argtypes = [I32, I32, I32, P, P, P, P, P, P, P, P, P]
    lib.rolesub_route_allocate_workspace_size.argtypes = [P, P]
    lib.rolesub_route_allocate.argtypes = [P, ctypes.c_int, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.rolesub_full_workspace_size.argtypes = [I32, I32, I32]
    lib.rolesub_full_workspace_size.restype = SZ
    lib.rolesub_full_transpose.argtypes = [I32, ctypes.c_int, P, P, P]
    lib.rolesub_full_rotate_pack.argtypes = [P, ctypes.c_int, P, P, P, P, P, I64, P, P, P, SZ, P]
    lib.rolesub_full_values.argtypes = [P, ctypes.c_int, P, P, P, P, I64, P, P, SZ, P]
    lib.rolesub_attend_values.argtypes = [P, ctypes.c_int, I32, P, P, P, ctypes.c_float, P, ctypes.c_int, P]
    for fn in ("rolesub_rotate_values", "rolesub_route", "rolesub_route_noalloc", "rolesub_pack_kv",
               "rolesub_rotate_pack", "rolesub_attend"):
        getattr(lib, fn).restype = ctypes.c_int
    _lib = lib
    return lib


def status_name(status: int) -> str:
    return load().rolesub_status_str(status).decode()


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise RolesubError(fn, status, load().rolesub_last_error().decode())


def _code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t, dtype=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch tensor")
    if not t.is_cuda:
        raise ValueError("librolesub takes device tensors only")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _fmt(shape):
    return "[" + ", ".join("*" if x is None else str(int(x)) for x in shape) + "]"


def _need(name, t, shape, dtype=None):
    """Check a tensor argument's shape (None: any extent) and dtype on the host,
    before anything is launched: the library receives bare pointers and would
    otherwise read or write past a wrongly sized buffer."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if t.dim() != len(shape) or any(s is not None and int(s) != int(x) for s, x in zip(shape, t.shape)):
        raise ValueError(f"{name}: expected shape {_fmt(shape)}, got {list(t.shape)}")
    if dtype is not None:
        ok = dtype if isinstance(dtype, tuple) else (dtype,)
        if t.dtype not in ok:
            raise TypeError(f"{name}: expected dtype {' or '.join(str(d) for d in ok)}, got {t.dtype}")


_MASK = (torch.int32, torch.uint32)


def _same_device(*ts):
    devs = {t.device for t in ts if isinstance(t, torch.Tensor)}
    if len(devs) > 1:
        raise ValueError(f"tensors on different devices: {sorted(str(d) for d in devs)}")


def _need_workspace(t):
    if t is not None:
        _need("workspace", t, (None,), torch.uint8)


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def make_budget(mode=TOPK, k_by_type=(0, 0, 0, 0), tau=0.0, kmin=0, kmax=0) -> Budget:
    b = Budget()
    b.mode = mode
    for i, k in enumerate(k_by_type):
        b.k_by_type[i] = int(k)
    b.tau, b.kmin, b.kmax = float(tau), int(kmin), int(kmax)
    return b


@dataclass
class Router:
    """Router weights as device tensors (kept alive while calls are in flight)."""
    kind: int
    C: int
    tensors: dict
    d_e: int = 0
    Hr: int = 0
    alpha_role: float = 0.1
    alpha_lang: float = 0.1

    def desc(self) -> RouterDesc:
        r = RouterDesc()
        r.kind, r.C, r.d_e, r.Hr = self.kind, self.C, self.d_e, self.Hr
        r.alpha_role, r.alpha_lang = self.alpha_role, self.alpha_lang
        for name, t in self.tensors.items():
            setattr(r, name, _ptr(t).value)
        return r

    def check(self, d: int, G: int, dtype) -> None:
        """Weight shapes against the hidden size d and G groups (row-major [out][in])."""
        t, C = self.tensors, self.C
        if self.kind == MLP2:
            shapes = dict(W_r=(C, d), b_r=(C,), E=(C, self.d_e), W1=(self.Hr, 2 * d + self.d_e), b1=(self.Hr,),
                          W2=(G, self.Hr), b2=(G,))
        else:
            shapes = dict(W_tok=(G, d), b_tok=(G,), W_r=(C, d), b_r=(C,), W_role=(G, C), W_lang=(G, d),
                          b_lang=(G,))
        for name, shape in shapes.items():
            if name not in t:
                raise ValueError(f"router: missing {name}")
            _need(f"router.{name}", t[name], shape, dtype)

    @staticmethod
    def mlp2(W_r, b_r, E, W1, b1, W2, b2) -> "Router":
        return Router(MLP2, W_r.shape[0], dict(W_r=W_r, b_r=b_r, E=E, W1=W1, b1=b1, W2=W2, b2=b2),
                      d_e=E.shape[1], Hr=W1.shape[0])

    @staticmethod
    def additive(W_tok, b_tok, W_r, b_r, W_role, W_lang, b_lang, alpha_role=0.1, alpha_lang=0.1):
        return Router(ADDITIVE, W_r.shape[0], dict(W_tok=W_tok, b_tok=b_tok, W_r=W_r, b_r=b_r,
                                                   W_role=W_role, W_lang=W_lang, b_lang=b_lang),
                      alpha_role=alpha_role, alpha_lang=alpha_lang)


# ----------------------------------------------------------------------------
# The four calls
# ----------------------------------------------------------------------------

def rotate_values(v: torch.Tensor, R: torch.Tensor, out: torch.Tensor | None = None, stream=None):
    """z = R_h^T v per head. v [B,T,H,dh], R [H,dh,dh]."""
    _need("v", v, (None, None, None, None))
    B, T, H, dh = v.shape
    _need("R", R, (H, dh, dh), v.dtype)
    _need("out", out, (B, T, H, dh), v.dtype)
    _same_device(v, R, out)
    z = torch.empty_like(v) if out is None else out
    dims = Dims(B, T, H, dh, 1, 0)
    _check("rolesub_rotate_values", load().rolesub_rotate_values(
        ctypes.byref(dims), _code(v), _ptr(v), _ptr(R, v.dtype), _ptr(z, v.dtype), _stream(stream)))
    return z


def route_workspace_size(B, T, G, d, router: Router) -> int:
    dims = Dims(B, T, 1, 64, G, d)
    desc = router.desc()
    return load().rolesub_route_workspace_size(ctypes.byref(dims), ctypes.byref(desc))


def route(token_type: torch.Tensor, budget: Budget, G: int, h: torch.Tensor | None = None,
          router: Router | None = None, scores_in: torch.Tensor | None = None, *,
          want_scores=True, want_idx=True, want_count=True, workspace=None, out=None, stream=None):
    """Routing scores and group selection. Returns dict(mask, idx, count, scores)."""
    _need("token_type", token_type, (None, None), torch.uint8)
    B, T = token_type.shape
    dev = token_type.device
    _need("h", h, (B, T, None), (torch.float32, torch.bfloat16))
    d = 0 if h is None else h.shape[2]
    dtype = torch.float32 if h is None else h.dtype
    _need("scores_in", scores_in, (B, T, G), torch.float32)
    if router is not None and h is not None:
        router.check(d, G, dtype)
    o = out or {}
    for name, shape, dt in (("mask", (B, T), _MASK), ("idx", (B, T, G), torch.uint8),
                            ("count", (B, T), torch.uint8), ("scores", (B, T, G), torch.float32)):
        _need(f"out[{name!r}]", o.get(name), shape, dt)
    _need_workspace(workspace)
    _same_device(token_type, h, scores_in, workspace, *o.values())

    def buf(name, shape, dtype, want=True):
        if not want:
            return None
        return o[name] if name in o else torch.empty(shape, dtype=dtype, device=dev)

    mask = buf("mask", (B, T), torch.int32)
    idx = buf("idx", (B, T, G), torch.uint8, want_idx)
    cnt = buf("count", (B, T), torch.uint8, want_count)
    sco = buf("scores", (B, T, G), torch.float32, want_scores)
    dims = Dims(B, T, 1, 64, G, d)
    desc = router.desc() if router is not None else None
    ws_ptr, ws_bytes = None, 0
    if scores_in is None and router is not None:
        ws_bytes = load().rolesub_route_workspace_size(ctypes.byref(dims), ctypes.byref(desc))
        if workspace is None:
            workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
        ws_ptr, ws_bytes = _ptr(workspace), workspace.numel()
    _check("rolesub_route", load().rolesub_route(
        ctypes.byref(dims), F32 if dtype == torch.float32 else BF16,
        ctypes.byref(desc) if desc is not None else None, ctypes.byref(budget),
        _ptr(h), _ptr(token_type, torch.uint8), _ptr(scores_in, torch.float32), _ptr(sco),
        _ptr(mask), _ptr(idx), _ptr(cnt), ws_ptr, ws_bytes, _stream(stream)))
    return {"mask": mask, "idx": idx, "count": cnt, "scores": sco}


def route_noalloc(token_type: torch.Tensor, budget: Budget, G: int, h: torch.Tensor | None = None,
                  router: Router | None = None, scores_in: torch.Tensor | None = None, *, out, stream=None):
    """rolesub_route with the library's own fixed device scratch as workspace:
    the call allocates nothing. Every output buffer comes from the caller
    (out: dict with mask [B,T] int32 and optionally idx, count, scores)."""
    _need("token_type", token_type, (None, None), torch.uint8)
    B, T = token_type.shape
    _need("h", h, (B, T, None), (torch.float32, torch.bfloat16))
    d = 0 if h is None else h.shape[2]
    dtype = torch.float32 if h is None else h.dtype
    _need("scores_in", scores_in, (B, T, G), torch.float32)
    if router is not None and h is not None:
        router.check(d, G, dtype)
    if "mask" not in out:
        raise ValueError("out['mask'] is required")
    for name, shape, dt in (("mask", (B, T), _MASK), ("idx", (B, T, G), torch.uint8),
                            ("count", (B, T), torch.uint8), ("scores", (B, T, G), torch.float32)):
        _need(f"out[{name!r}]", out.get(name), shape, dt)
    _same_device(token_type, h, scores_in, *out.values())
    dims = Dims(B, T, 1, 64, G, d)
    desc = router.desc() if router is not None else None
    _check("rolesub_route_noalloc", load().rolesub_route_noalloc(
        ctypes.byref(dims), F32 if dtype == torch.float32 else BF16,
        ctypes.byref(desc) if desc is not None else None, ctypes.byref(budget),
        _ptr(h), _ptr(token_type, torch.uint8), _ptr(scores_in, torch.float32), _ptr(out.get("scores")),
        _ptr(out["mask"]), _ptr(out.get("idx")), _ptr(out.get("count")), _stream(stream)))
    return out


def pack_kv(z: torch.Tensor, mask: torch.Tensor, G: int, cap: int, budget: Budget | None = None,
            type_counts=None, out=None, stream=None):
    """Compact group-indexed cache. Returns (offsets [B,T+1] int32, Vp [B,H,cap,ds])."""
    _need("z", z, (None, None, None, None))
    B, T, H, dh = z.shape
    ds = dh // G
    _need("mask", mask, (B, T), _MASK)
    if out is not None:
        _need("offsets", out[0], (B, T + 1), torch.int32)
        _need("Vp", out[1], (B, H, cap, ds), z.dtype)
    _same_device(z, mask, *(out or ()))
    offsets = torch.empty((B, T + 1), dtype=torch.int32, device=z.device) if out is None else out[0]
    Vp = torch.empty((B, H, cap, ds), dtype=z.dtype, device=z.device) if out is None else out[1]
    dims = Dims(B, T, H, dh, G, 0)
    tc = (ctypes.c_int32 * 4)(*type_counts) if type_counts is not None else None
    _check("rolesub_pack_kv", load().rolesub_pack_kv(
        ctypes.byref(dims), _code(z), ctypes.byref(budget) if budget is not None else None, tc,
        _ptr(z), _ptr(mask), _ptr(offsets, torch.int32), _ptr(Vp, z.dtype), int(cap), _stream(stream)))
    return offsets, Vp


def rotate_pack(v: torch.Tensor, R: torch.Tensor, mask: torch.Tensor, G: int, cap: int,
                budget: Budget | None = None, type_counts=None, out=None, stream=None):
    """Rotation and pack in one pass (z is not materialised). Returns (offsets, Vp)."""
    _need("v", v, (None, None, None, None))
    B, T, H, dh = v.shape
    ds = dh // G
    _need("R", R, (H, dh, dh), v.dtype)
    _need("mask", mask, (B, T), _MASK)
    if out is not None:
        _need("offsets", out[0], (B, T + 1), torch.int32)
        _need("Vp", out[1], (B, H, cap, ds), v.dtype)
    _same_device(v, R, mask, *(out or ()))
    offsets = torch.empty((B, T + 1), dtype=torch.int32, device=v.device) if out is None else out[0]
    Vp = torch.empty((B, H, cap, ds), dtype=v.dtype, device=v.device) if out is None else out[1]
    dims = Dims(B, T, H, dh, G, 0)
    tc = (ctypes.c_int32 * 4)(*type_counts) if type_counts is not None else None
    _check("rolesub_rotate_pack", load().rolesub_rotate_pack(
        ctypes.byref(dims), _code(v), ctypes.byref(budget) if budget is not None else None, tc,
        _ptr(v), _ptr(R, v.dtype), _ptr(mask), _ptr(offsets, torch.int32), _ptr(Vp, v.dtype), int(cap),
        _stream(stream)))
    return offsets, Vp


def attend(q, k, mask, offsets, Vp, R, G: int, scale: float = 0.0, out_dtype=None, out=None, stream=None):
    """Attention with full q, k over the packed routed values; returns [B,Tq,H,dh]."""
    _need("q", q, (None, None, None, None))
    B, Tq, H, dh = q.shape
    _need("k", k, (B, None, H, dh), q.dtype)
    T = k.shape[1]
    _need("Vp", Vp, (B, H, None, dh // max(G, 1)), q.dtype)
    cap = Vp.shape[2]
    _need("mask", mask, (B, T), _MASK)
    _need("offsets", offsets, (B, T + 1), torch.int32)
    _need("R", R, (H, dh, dh), q.dtype)
    _need("out", out, (B, Tq, H, dh), (torch.float32, torch.bfloat16))
    _same_device(q, k, mask, offsets, Vp, R, out)
    odt = q.dtype if out_dtype is None else out_dtype
    o = torch.empty((B, Tq, H, dh), dtype=odt, device=q.device) if out is None else out
    dims = Dims(B, T, H, dh, G, 0)
    _check("rolesub_attend", load().rolesub_attend(
        ctypes.byref(dims), _code(q), Tq, _ptr(q), _ptr(k, q.dtype), _ptr(mask), _ptr(offsets, torch.int32),
        _ptr(Vp, q.dtype), int(cap), _ptr(R, q.dtype), float(scale), _ptr(o), _code(o), None, 0,
        _stream(stream)))
    return o


def attend_causal(q, k, mask, offsets, Vp, R, G: int, scale: float = 0.0, out_dtype=None, out=None, stream=None):
    """Prefix self-attention over the packed routed values (query t sees keys
    0..t); q and k are [B,T,H,dh]; returns [B,T,H,dh]."""
    _need("q", q, (None, None, None, None))
    B, T, H, dh = q.shape
    _need("k", k, (B, T, H, dh), q.dtype)
    _need("Vp", Vp, (B, H, None, dh // max(G, 1)), q.dtype)
    cap = Vp.shape[2]
    _need("mask", mask, (B, T), _MASK)
    _need("offsets", offsets, (B, T + 1), torch.int32)
    _need("R", R, (H, dh, dh), q.dtype)
    _need("out", out, (B, T, H, dh), (torch.float32, torch.bfloat16))
    _same_device(q, k, mask, offsets, Vp, R, out)
    odt = q.dtype if out_dtype is None else out_dtype
    o = torch.empty((B, T, H, dh), dtype=odt, device=q.device) if out is None else out
    dims = Dims(B, T, H, dh, G, 0)
    _check("rolesub_attend_causal", load().rolesub_attend_causal(
        ctypes.byref(dims), _code(q), _ptr(q), _ptr(k, q.dtype), _ptr(mask), _ptr(offsets, torch.int32),
        _ptr(Vp, q.dtype), int(cap), _ptr(R, q.dtype), float(scale), _ptr(o), _code(o), None, 0,
        _stream(stream)))
    return o


def retain_tokens(scores, seg_len, seg_keep, out=None, stream=None):
    """Per sample and per segment of consecutive tokens, the indices of the
    seg_keep highest-scoring tokens (int32 [B, sum(seg_keep)])."""
    _need("scores", scores, (None, None), torch.float32)
    B, N = scores.shape
    n = len(seg_len)
    if len(seg_keep) != n:
        raise ValueError(f"seg_keep has {len(seg_keep)} entries for {n} segments")
    _need("out", out, (B, int(sum(seg_keep))), torch.int32)
    _same_device(scores, out)
    lens = (ctypes.c_int32 * n)(*[int(x) for x in seg_len])
    keeps = (ctypes.c_int32 * n)(*[int(x) for x in seg_keep])
    K = int(sum(seg_keep))
    o = torch.empty((B, K), dtype=torch.int32, device=scores.device) if out is None else out
    _check("rolesub_retain_tokens", load().rolesub_retain_tokens(
        B, N, n, lens, keeps, _ptr(scores, torch.float32), _ptr(o, torch.int32), _stream(stream)))
    return o


def gather_tokens(x, idx, out=None, stream=None):
    """Rows x[b, idx[b, j]] of a [B, N, ...] tensor (the retained prefix)."""
    if not isinstance(x, torch.Tensor) or x.dim() < 2:
        raise ValueError("x: expected a [B, N, ...] tensor")
    B, N = x.shape[:2]
    _need("idx", idx, (B, None), torch.int32)
    K = idx.shape[1]
    _need("out", out, (B, K) + tuple(x.shape[2:]), x.dtype)
    _same_device(x, idx, out)
    o = torch.empty((B, K) + tuple(x.shape[2:]), dtype=x.dtype, device=x.device) if out is None else out
    row_bytes = x[0, 0].numel() * x.element_size() if N else 0
    _check("rolesub_gather_tokens", load().rolesub_gather_tokens(
        B, N, K, row_bytes, _ptr(idx, torch.int32), _ptr(x), _ptr(o), _stream(stream)))
    return o


def allocate_groups(priority, token_type, k_by_type, G: int, scores=None, *, want_k=True, want_idx=True,
                    want_count=True, out=None, stream=None):
    """Role-driven within-type group budgets K_i from token priorities, and with
    scores the Top-K_i selection on them. Returns dict(k, mask, idx, count)."""
    _need("token_type", token_type, (None, None), torch.uint8)
    B, T = token_type.shape
    dev = token_type.device
    _need("priority", priority, (B, T), torch.float32)
    _need("scores", scores, (B, T, G), torch.float32)
    o = out or {}
    for name, shape, dt in (("k", (B, T), torch.uint8), ("mask", (B, T), _MASK), ("idx", (B, T, G), torch.uint8),
                            ("count", (B, T), torch.uint8)):
        _need(f"out[{name!r}]", o.get(name), shape, dt)
    _same_device(token_type, priority, scores, *o.values())

    def buf(name, shape, dtype, want=True):
        if not want:
            return None
        return o[name] if name in o else torch.empty(shape, dtype=dtype, device=dev)

    sel = scores is not None
    kk = buf("k", (B, T), torch.uint8, want_k)
    mask = buf("mask", (B, T), torch.int32, sel)
    idx = buf("idx", (B, T, G), torch.uint8, sel and want_idx)
    cnt = buf("count", (B, T), torch.uint8, sel and want_count)
    kby = (ctypes.c_int32 * 4)(*[int(x) for x in k_by_type])
    _check("rolesub_allocate_groups", load().rolesub_allocate_groups(
        B, T, G, kby, _ptr(priority, torch.float32), _ptr(token_type, torch.uint8), _ptr(scores, torch.float32),
        _ptr(kk), _ptr(mask), _ptr(idx), _ptr(cnt), _stream(stream)))
    return {"k": kk, "mask": mask, "idx": idx, "count": cnt}


def route_allocate_workspace_size(B, T, G, d, router: Router) -> int:
    dims = Dims(B, T, 1, 64, G, d)
    desc = router.desc()
    return load().rolesub_route_allocate_workspace_size(ctypes.byref(dims), ctypes.byref(desc))


def route_allocate(token_type, k_by_type, G: int, h, router: Router, w_pri, *, want_priority=True,
                   want_scores=True, want_k=True, want_idx=True, want_count=True, workspace=None, out=None,
                   stream=None):
    """Routing with role-driven budgets: scores, priorities p = w_pri^T a, the
    allocated K_i and the Top-K_i selection. Returns dict(mask, idx, count, k,
    scores, priority)."""
    _need("token_type", token_type, (None, None), torch.uint8)
    B, T = token_type.shape
    dev = token_type.device
    _need("h", h, (B, T, None), (torch.float32, torch.bfloat16))
    d = h.shape[2]
    router.check(d, G, h.dtype)
    _need("w_pri", w_pri, (router.C,), h.dtype)
    o = out or {}
    for name, shape, dt in (("mask", (B, T), _MASK), ("idx", (B, T, G), torch.uint8), ("count", (B, T), torch.uint8),
                            ("k", (B, T), torch.uint8), ("scores", (B, T, G), torch.float32),
                            ("priority", (B, T), torch.float32)):
        _need(f"out[{name!r}]", o.get(name), shape, dt)
    _need_workspace(workspace)
    _same_device(token_type, h, w_pri, workspace, *o.values())

    def buf(name, shape, dtype, want=True):
        if not want:
            return None
        return o[name] if name in o else torch.empty(shape, dtype=dtype, device=dev)

    mask = buf("mask", (B, T), torch.int32)
    idx = buf("idx", (B, T, G), torch.uint8, want_idx)
    cnt = buf("count", (B, T), torch.uint8, want_count)
    kk = buf("k", (B, T), torch.uint8, want_k)
    sco = buf("scores", (B, T, G), torch.float32, want_scores)
    pri = buf("priority", (B, T), torch.float32, want_priority)
    dims = Dims(B, T, 1, 64, G, d)
    desc = router.desc()
    ws_bytes = load().rolesub_route_allocate_workspace_size(ctypes.byref(dims), ctypes.byref(desc))
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    kby = (ctypes.c_int32 * 4)(*[int(x) for x in k_by_type])
    _check("rolesub_route_allocate", load().rolesub_route_allocate(
        ctypes.byref(dims), F32 if h.dtype == torch.float32 else BF16, ctypes.byref(desc), _ptr(w_pri, h.dtype),
        kby, _ptr(h), _ptr(token_type, torch.uint8), _ptr(pri), _ptr(sco), _ptr(kk), _ptr(mask), _ptr(idx),
        _ptr(cnt), _ptr(workspace), workspace.numel(), _stream(stream)))
    return {"mask": mask, "idx": idx, "count": cnt, "k": kk, "scores": sco, "priority": pri}


# ----------------------------------------------------------------------------
# Full-width routing space (one R over all H*dh value dims, S groups)
# ----------------------------------------------------------------------------

def full_workspace_size(B, T, S) -> int:
    return load().rolesub_full_workspace_size(B, T, S)


def full_transpose(R, out=None, stream=None):
    """R^T of a frozen [d_v, d_v] rotation (the layout full_rotate_pack takes)."""
    _need("R", R, (None, None))
    n = R.shape[0]
    _need("R", R, (n, n))
    _need("out", out, (n, n), R.dtype)
    _same_device(R, out)
    Rt = torch.empty_like(R) if out is None else out
    _check("rolesub_full_transpose", load().rolesub_full_transpose(n, _code(R), _ptr(R), _ptr(Rt, R.dtype),
                                                                   _stream(stream)))
    return Rt


def full_rotate_pack(v, Rt, mask, S: int, cap: int, budget: Budget | None = None, type_counts=None,
                     workspace=None, out=None, stream=None):
    """Full-width cache: (offsets [B,T+1] int32, Vp [B,cap,d_v/S])."""
    _need("v", v, (None, None, None, None))
    B, T, H, dh = v.shape
    dv = H * dh
    _need("Rt", Rt, (dv, dv), v.dtype)
    _need("mask", mask, (B, T), _MASK)
    if out is not None:
        _need("offsets", out[0], (B, T + 1), torch.int32)
        _need("Vp", out[1], (B, cap, dv // max(S, 1)), v.dtype)
    _need_workspace(workspace)
    _same_device(v, Rt, mask, workspace, *(out or ()))
    if out is None:
        out = (torch.empty((B, T + 1), dtype=torch.int32, device=v.device),
               torch.empty((B, cap, dv // S), dtype=v.dtype, device=v.device))
    offsets, Vp = out
    if workspace is None:
        workspace = torch.empty(max(full_workspace_size(B, T, S), 1), dtype=torch.uint8, device=v.device)
    tc = (ctypes.c_int32 * 4)(*[int(x) for x in type_counts]) if type_counts is not None else None
    dims = Dims(B, T, H, dh, S, 0)
    _check("rolesub_full_rotate_pack", load().rolesub_full_rotate_pack(
        ctypes.byref(dims), _code(v), _ptr(Rt, v.dtype), _ptr(v), _ptr(mask), _ptr(offsets, torch.int32),
        _ptr(Vp, v.dtype), cap, ctypes.byref(budget) if budget is not None else None, tc, _ptr(workspace),
        workspace.numel(), _stream(stream)))
    return offsets, Vp


def full_values(R, mask, offsets, Vp, S: int, H: int, workspace=None, out=None, stream=None):
    """Routed values [B,H,T,dh] (head-major) from the full-width cache."""
    _need("Vp", Vp, (None, None, None))
    B, cap, ds = Vp.shape
    _need("offsets", offsets, (B, None), torch.int32)
    T = offsets.shape[1] - 1
    if H < 1 or (ds * S) % H:
        raise ValueError(f"d_v = {ds * S} does not split into {H} heads")
    dh = ds * S // H
    _need("R", R, (ds * S, ds * S), Vp.dtype)
    _need("mask", mask, (B, T), _MASK)
    _need("out", out, (B, H, T, dh), Vp.dtype)
    _need_workspace(workspace)
    _same_device(Vp, offsets, R, mask, out, workspace)
    Vh = torch.empty((B, H, T, dh), dtype=Vp.dtype, device=Vp.device) if out is None else out
    if workspace is None:
        workspace = torch.empty(max(full_workspace_size(B, T, S), 1), dtype=torch.uint8, device=Vp.device)
    dims = Dims(B, T, H, dh, S, 0)
    _check("rolesub_full_values", load().rolesub_full_values(
        ctypes.byref(dims), _code(Vp), _ptr(R, Vp.dtype), _ptr(mask), _ptr(offsets, torch.int32), _ptr(Vp),
        cap, _ptr(Vh, Vp.dtype), _ptr(workspace), workspace.numel(), _stream(stream)))
    return Vh


def attend_values(q, k, V, scale: float = 0.0, out_dtype=None, out=None, stream=None):
    """Attention over plain head-major values V [B,H,T,dh] (the full-width
    routing space's rebuilt values). Returns [B,Tq,H,dh]."""
    _need("q", q, (None, None, None, None))
    B, Tq, H, dh = q.shape
    _need("k", k, (B, None, H, dh), q.dtype)
    T = k.shape[1]
    _need("V", V, (B, H, T, dh), q.dtype)
    _need("out", out, (B, Tq, H, dh), (torch.float32, torch.bfloat16))
    _same_device(q, k, V, out)
    od = out.dtype if out is not None else (out_dtype or q.dtype)
    o = torch.empty((B, Tq, H, dh), dtype=od, device=q.device) if out is None else out
    dims = Dims(B, T, H, dh, 1, 0)
    _check("rolesub_attend_values", load().rolesub_attend_values(
        ctypes.byref(dims), _code(q), Tq, _ptr(q), _ptr(k, q.dtype), _ptr(V, q.dtype), ctypes.c_float(scale),
        _ptr(o), _code(o), _stream(stream)))
    return o
