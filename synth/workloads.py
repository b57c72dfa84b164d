"""Seeded synthetic workloads for the RoleSub hot path.

The paper evaluates on OpenVLA-OFT-7B (Llama-2-7B backbone: hidden 4096,
32 heads x 128) with a multimodal prefix of 512 visual tokens from two camera
views, language, proprioceptive and action-context tokens, and an 8-step
action chunk decoded in parallel (Sec. 4.1, "Model" and "Token-level
reduction"). Trained weights and LIBERO data are not available, so these
generators stand in for them with seeded Gaussian draws of the same shapes.

Every value is drawn as float32 and then rounded once (round-to-nearest-even)
to the workload's storage type, so the arrays returned here are exactly
representable in that type. The float64 oracle upcasts them exactly; the GPU
path converts them to bf16/f32 device tensors exactly. No arithmetic of the
method lives here.

Streams: every tensor has its own PCG64 stream keyed by
``SeedSequence(seed, spawn_key=(layer, kind, sample, tensor))`` so any single
(layer, sample) can be regenerated alone.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

VIS, LANG, PROP, ACT = 0, 1, 2, 3
TOPK, THRESHOLD = 0, 1

__all__ = [
    "VIS", "LANG", "PROP", "ACT", "TOPK", "THRESHOLD", "Workload", "WORKLOADS",
    "workload", "bf16_round", "round_to", "layer_weights", "additive_weights",
    "sample_activations", "layer_activations", "sample_scores", "synthetic_z",
    "synthetic_masks", "haar_orthogonal", "priority_weights", "sample_priorities", "full_rotation",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    B: int          # independent prefixes
    L: int          # layers
    H: int          # heads
    dh: int         # head dim
    d: int          # hidden size
    G: int          # value groups per head (S in the paper)
    n_vis: int
    n_lang: int
    n_prop: int
    Tq: int         # action-query tokens
    dtype: str      # "f32" or "bf16"
    mode: int       # TOPK or THRESHOLD
    k_vis: int
    k_lang: int
    k_prop: int
    C: int          # latent roles
    d_e: int        # role-vector width
    Hr: int         # router hidden width
    seed: int
    kmin: int = 0
    kmax: int = 0
    tau: float = 0.0
    scores_in: bool = False          # selection from synthetic logits
    near_frac: float = 0.0           # fraction of tokens with near-threshold logits
    full_width: bool = False         # one R over all H*dh value dims, G groups of H*dh/G

    @property
    def T(self) -> int:
        return self.n_vis + self.n_lang + self.n_prop

    @property
    def ds(self) -> int:
        return (self.H * self.dh if self.full_width else self.dh) // self.G

    @property
    def dv(self) -> int:
        return self.H * self.dh

    @property
    def k_by_type(self) -> tuple:
        return (self.k_vis, self.k_lang, self.k_prop, self.G)

    @property
    def router_in(self) -> int:
        return 2 * self.d + self.d_e

    def types(self) -> np.ndarray:
        """Token types in prefix order [vis | lang | prop]."""
        return np.array([VIS] * self.n_vis + [LANG] * self.n_lang + [PROP] * self.n_prop,
                        dtype=np.uint8)

    def type_counts(self) -> tuple:
        return (self.n_vis, self.n_lang, self.n_prop, 0)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads. 7B shape = Llama-2-7B attention (32 heads x 128, hidden 4096).
WORKLOADS = {
    1: Workload(1, "tiny-f32", B=1, L=1, H=4, dh=64, d=256, G=8, n_vis=64, n_lang=16, n_prop=0,
                Tq=8, dtype="f32", mode=TOPK, k_vis=4, k_lang=6, k_prop=8, C=4, d_e=64, Hr=128,
                seed=0),
    2: Workload(2, "7b-layer", B=1, L=1, H=32, dh=128, d=4096, G=8, n_vis=256, n_lang=48, n_prop=1,
                Tq=56, dtype="bf16", mode=TOPK, k_vis=4, k_lang=6, k_prop=8, C=8, d_e=128, Hr=128,
                seed=2),
    3: Workload(3, "7b-aggressive-b16", B=16, L=1, H=32, dh=128, d=4096, G=8, n_vis=64, n_lang=48,
                n_prop=1, Tq=56, dtype="bf16", mode=TOPK, k_vis=2, k_lang=4, k_prop=8, C=8, d_e=128,
                Hr=128, seed=3),
    4: Workload(4, "7b-stack32-b64", B=64, L=32, H=32, dh=128, d=4096, G=8, n_vis=128, n_lang=48,
                n_prop=1, Tq=56, dtype="bf16", mode=TOPK, k_vis=4, k_lang=6, k_prop=8, C=8,
                d_e=128, Hr=128, seed=4),
    5: Workload(5, "stress-g32-b128", B=128, L=1, H=32, dh=128, d=4096, G=32, n_vis=1792,
                n_lang=256, n_prop=0, Tq=64, dtype="bf16", mode=THRESHOLD, k_vis=32, k_lang=32,
                k_prop=32, C=8, d_e=128, Hr=128, seed=5, kmin=1, kmax=32, tau=0.0,
                scores_in=True, near_frac=0.3),
    # The paper's own routing space (Sec. 4.1): one R over d_v = 4096, S = 16 groups of 256,
    # C = 6 latent roles; 32 retained visual tokens (1/16 of 512) keep K_vis = 4 groups,
    # language and proprio values uncompressed.
    6: Workload(6, "7b-fullwidth-stack32-b64", B=64, L=32, H=32, dh=128, d=4096, G=16, n_vis=32,
                n_lang=48, n_prop=1, Tq=56, dtype="bf16", mode=TOPK, k_vis=4, k_lang=16, k_prop=16,
                C=6, d_e=128, Hr=128, seed=6, full_width=True),
    # A smaller full-width case for whole-tensor parity: d_v = 1024, S = 8 groups of 128.
    7: Workload(7, "fullwidth-small", B=3, L=1, H=8, dh=128, d=1024, G=8, n_vis=40, n_lang=20,
                n_prop=1, Tq=16, dtype="bf16", mode=TOPK, k_vis=2, k_lang=8, k_prop=8, C=6,
                d_e=128, Hr=128, seed=7, full_width=True),
}


def workload(cid: int) -> Workload:
    return WORKLOADS[cid]


# ----------------------------------------------------------------------------
# Rounding (storage types only; no method arithmetic)
# ----------------------------------------------------------------------------

def bf16_round(x) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    u = a.view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    out = ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = np.where(nan, np.float32(np.nan), out)
    return out


def round_to(x, dtype: str) -> np.ndarray:
    x32 = np.asarray(x, dtype=np.float32)
    return bf16_round(x32) if dtype == "bf16" else x32


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def _normal(seed, key, shape, std=1.0) -> np.ndarray:
    g = _rng(seed, *key)
    x = g.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x = (x.astype(np.float64) * std).astype(np.float32)
    return x


def haar_orthogonal(rng: np.random.Generator, n: int) -> np.ndarray:
    """Haar-distributed orthogonal matrix (float64): QR of a Gaussian with the
    sign of R's diagonal folded into Q (Mezzadri, 2007)."""
    a = rng.standard_normal((n, n))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


# weight tensor ids inside a layer (kind 0)
_W_R, _W_BR, _W_E, _W_W1, _W_B1, _W_W2, _W_B2, _W_TOK, _W_BTOK, _W_ROLE, _W_LANG, _W_BLANG = range(12)
_W_ROT = 100
_W_PRI = 101
_W_ROT_FULL = 102
# activation tensor ids inside a (layer, sample) (kind 1)
_A_H, _A_Q, _A_K, _A_V, _A_S, _A_PERM, _A_J, _A_Z, _A_MASK, _A_PRI, _A_PRI_KIND = range(11)


def layer_weights(w: Workload, layer: int) -> dict:
    """Router, role and rotation weights of one layer.

    Weights and biases are N(0, fan_in^-1/2); the role vectors E are N(0, 1);
    each head's R_h is an independent Haar sample (Sec. 4.1 initialises R from a
    random Stiefel matrix). 'R_master' keeps the float64 orthonormal matrices.
    """
    s = w.seed
    fin = w.router_in
    out = {
        "W_r": _normal(s, (layer, 0, 0, _W_R), (w.C, w.d), w.d ** -0.5),
        "b_r": _normal(s, (layer, 0, 0, _W_BR), (w.C,), w.d ** -0.5),
        "E": _normal(s, (layer, 0, 0, _W_E), (w.C, w.d_e), 1.0),
        "W1": _normal(s, (layer, 0, 0, _W_W1), (w.Hr, fin), fin ** -0.5),
        "b1": _normal(s, (layer, 0, 0, _W_B1), (w.Hr,), fin ** -0.5),
        "W2": _normal(s, (layer, 0, 0, _W_W2), (w.G, w.Hr), w.Hr ** -0.5),
        "b2": _normal(s, (layer, 0, 0, _W_B2), (w.G,), w.Hr ** -0.5),
    }
    masters = np.stack([haar_orthogonal(_rng(s, layer, 0, hh, _W_ROT), w.dh) for hh in range(w.H)])
    out["R_master"] = masters
    out["R"] = masters.astype(np.float32)
    out = {k: (v if k == "R_master" else round_to(v, w.dtype)) for k, v in out.items()}
    return out


def additive_weights(w: Workload, layer: int) -> dict:
    """Weights of the paper-literal additive router (token head f_v and language
    head f_lang linear d->G with bias, W_role G x C without bias)."""
    s = w.seed
    out = {
        "W_tok": _normal(s, (layer, 0, 0, _W_TOK), (w.G, w.d), w.d ** -0.5),
        "b_tok": _normal(s, (layer, 0, 0, _W_BTOK), (w.G,), w.d ** -0.5),
        "W_role": _normal(s, (layer, 0, 0, _W_ROLE), (w.G, w.C), w.C ** -0.5),
        "W_lang": _normal(s, (layer, 0, 0, _W_LANG), (w.G, w.d), w.d ** -0.5),
        "b_lang": _normal(s, (layer, 0, 0, _W_BLANG), (w.G,), w.d ** -0.5),
        "W_r": _normal(s, (layer, 0, 0, _W_R), (w.C, w.d), w.d ** -0.5),
        "b_r": _normal(s, (layer, 0, 0, _W_BR), (w.C,), w.d ** -0.5),
    }
    return {k: round_to(v, w.dtype) for k, v in out.items()}


def sample_activations(w: Workload, layer: int, b: int, names=("h", "q", "k", "v")) -> dict:
    """Hidden states h [T,d] and q [Tq,H,dh], k/v [T,H,dh] of one prefix, all N(0,1)."""
    s, T = w.seed, w.T
    spec = {"h": (_A_H, (T, w.d)), "q": (_A_Q, (w.Tq, w.H, w.dh)),
            "k": (_A_K, (T, w.H, w.dh)), "v": (_A_V, (T, w.H, w.dh))}
    return {n: round_to(_normal(s, (layer, 1, b, spec[n][0]), spec[n][1]), w.dtype) for n in names}


def sample_scores(w: Workload, layer: int, b: int) -> np.ndarray:
    """Synthetic router logits [T,G] float32 for threshold-mode stress.

    A seeded permutation picks round(near_frac*T) tokens whose logits are
    j * 2^-10 with j uniform on {-2..2}: exact zeros (dropped by the strict
    threshold) and exact ties. The first tenth of those draw j from {-2..0}
    only, so no group passes the threshold and the lower clamp keeps one group
    chosen among ties. The other tokens draw N(0,1) per group."""
    s, T, G = w.seed, w.T, w.G
    x = _normal(s, (layer, 1, b, _A_S), (T, G))
    n_near = int(round(w.near_frac * T))
    perm = _rng(s, layer, 1, b, _A_PERM).permutation(T)[:n_near]
    j = _rng(s, layer, 1, b, _A_J).integers(-2, 3, size=(n_near, G))
    n_none = n_near // 10
    j[:n_none] = -np.abs(j[:n_none])
    x[perm] = (j.astype(np.float32) * np.float32(2.0 ** -10))
    return x


def _threads() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def layer_activations(w: Workload, layer: int, samples=None) -> dict:
    """Stack sample_activations over samples (default: all B), drawn in threads."""
    idx = list(range(w.B)) if samples is None else list(samples)
    with _cf.ThreadPoolExecutor(_threads()) as ex:
        parts = list(ex.map(lambda b: sample_activations(w, layer, b), idx))
    return {k: np.stack([p[k] for p in parts]) for k in parts[0]}


def synthetic_z(w: Workload, layer: int, b: int) -> np.ndarray:
    """A stand-alone rotated-value tensor [T,H,dh] for testing the pack step alone."""
    return round_to(_normal(w.seed, (layer, 1, b, _A_Z), (w.T, w.H, w.dh)), w.dtype)


def synthetic_masks(w: Workload, layer: int, b: int, counts=None) -> np.ndarray:
    """Random group masks [T] uint32 for testing pack/attend alone.

    counts: per-token number of kept groups (default: the workload's budget by
    type; threshold workloads draw uniformly from [kmin, kmax])."""
    g = _rng(w.seed, layer, 1, b, _A_MASK)
    if counts is None:
        if w.mode == TOPK:
            kt = np.array(w.k_by_type)
            counts = np.minimum(kt[w.types()], w.G)
        else:
            counts = g.integers(w.kmin, w.kmax + 1, size=w.T)
    masks = np.zeros(w.T, dtype=np.uint32)
    for t, c in enumerate(counts):
        chosen = g.permutation(w.G)[: int(c)]
        m = 0
        for s_ in chosen:
            m |= 1 << int(s_)
        masks[t] = m
    return masks


def priority_weights(w: Workload, layer: int) -> np.ndarray:
    """One priority weight per latent role [C]: 1 + N(0, 1), so that most roles
    raise a token's priority and some lower it (rounded to the workload dtype)."""
    return round_to(1.0 + _normal(w.seed, (layer, 0, 0, _W_PRI), (w.C,), 1.0), w.dtype)


def sample_priorities(w: Workload, layer: int, b: int) -> np.ndarray:
    """Synthetic token priorities [T] float32 for testing the allocation alone.

    Most tokens draw an exponential priority with mean 1; a seeded tenth each
    are exact zeros, negative, exact copies of another token's priority (ties),
    values above the 256 clip, NaN, and multiples of 2^-16 (integer weights
    whose proportional shares often tie)."""
    g = _rng(w.seed, layer, 1, b, _A_PRI)
    T = w.T
    x = g.exponential(1.0, size=T).astype(np.float32)
    kind = _rng(w.seed, layer, 1, b, _A_PRI_KIND).integers(0, 10, size=T)
    x[kind == 0] = 0.0
    x[kind == 1] = -x[kind == 1]
    if T > 1:
        src = g.integers(0, T, size=T)
        x[kind == 2] = x[src[kind == 2]]
    x[kind == 3] = 300.0 + x[kind == 3]
    x[kind == 4] = np.nan
    x[kind == 5] = (g.integers(1, 8, size=int(np.sum(kind == 5))) * 2.0 ** -16).astype(np.float32)
    return x


def full_rotation(w: Workload, layer: int) -> dict:
    """The layer's full-width rotation over d_v = H*dh value dims (Haar, Sec. 4.1
    initialises R from a random Stiefel matrix): 'R_master' float64 and 'R'
    rounded to the workload dtype, both [d_v, d_v] with R[k, j] the k-th value
    coordinate of rotated coordinate j."""
    m = haar_orthogonal(_rng(w.seed, layer, 0, 0, _W_ROT_FULL), w.dv)
    return {"R_master": m, "R": round_to(m, w.dtype)}
