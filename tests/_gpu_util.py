"""Shared helpers of the GPU parity tests (not collected: no test_ prefix)."""
import numpy as np
import torch

import synth

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None
TOL = {"f32": 1e-4, "bf16": 2e-2}


def tdtype(w):
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def put(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype)


def put_u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(DEV)


def put_mask(m):
    return torch.from_numpy(np.ascontiguousarray(m, dtype=np.uint32).view(np.int32)).to(DEV)


def host(t):
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.numpy()


def host_mask(t):
    return t.detach().cpu().numpy().view(np.uint32)


def max_rel(x, ref):
    """max |x - ref| / max |ref| over the tensor."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(x - ref)) / max(float(np.max(np.abs(ref))), 1e-300))


def router_tensors(wt, dtype):
    import paper_2608_18410_amd as rs
    return rs.Router.mlp2(*(put(wt[n], dtype) for n in ("W_r", "b_r", "E", "W1", "b1", "W2", "b2")))


def decisive_margin(scores, K, tau=None):
    """Per token: the gap that decides its selection (f64).

    TOPK: gamma_(K) - gamma_(K+1) of the sorted scores (inf when K is 0 or G).
    THRESHOLD: the smallest |gamma_s - tau|."""
    s = np.sort(np.asarray(scores, dtype=np.float64), axis=-1)[..., ::-1]
    G = s.shape[-1]
    if tau is not None:
        return np.min(np.abs(np.asarray(scores, dtype=np.float64) - tau), axis=-1)
    K = np.asarray(K)
    out = np.full(K.shape, np.inf)
    inner = (K > 0) & (K < G)
    kk = np.clip(K, 1, G - 1)
    a = np.take_along_axis(s, (kk - 1)[..., None], -1)[..., 0]
    b = np.take_along_axis(s, kk[..., None], -1)[..., 0]
    out[inner] = (a - b)[inner]
    return out


def stack_types(w, B=None):
    B = w.B if B is None else B
    return np.broadcast_to(w.types(), (B, w.T)).copy()


def synth_pack_inputs(w, B, layer=0):
    z = np.stack([synth.synthetic_z(w, layer, b) for b in range(B)])
    m = np.stack([synth.synthetic_masks(w, layer, b) for b in range(B)])
    return z, m


def layer_on_device(w, layer, need_h=True, chunk=16):
    """Generate one layer's activations sample by sample straight into device tensors."""
    import concurrent.futures as cf
    dt = tdtype(w)
    out = {"q": torch.empty((w.B, w.Tq, w.H, w.dh), dtype=dt, device=DEV),
           "k": torch.empty((w.B, w.T, w.H, w.dh), dtype=dt, device=DEV),
           "v": torch.empty((w.B, w.T, w.H, w.dh), dtype=dt, device=DEV)}
    if need_h:
        out["h"] = torch.empty((w.B, w.T, w.d), dtype=dt, device=DEV)
    with cf.ThreadPoolExecutor(16) as ex:
        for b0 in range(0, w.B, chunk):
            names = tuple(out)
            parts = list(ex.map(lambda b: synth.sample_activations(w, layer, b, names),
                                range(b0, min(w.B, b0 + chunk))))
            for i, p in enumerate(parts):
                for name in out:
                    out[name][b0 + i].copy_(torch.from_numpy(p[name]))
    return out
