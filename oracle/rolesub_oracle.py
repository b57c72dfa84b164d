"""Float64 CPU oracle of RoleSub's inference hot path.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg; never by the product path.

Written from the paper (Role-Conditioned Sub-Token Routing, Sec. 3):
plain, slow, obviously checkable numpy float64. Each function names the
passage it follows. Inputs arrive as arrays whose values are exactly
representable in the workload's storage type; everything here is computed in
float64 except where a discrete decision is taken (group selection), which is
taken on the scores exactly as given.

Readings of points the paper leaves open (listed with reasons in the design
notes of the repository):
  * one orthonormal R_h per head, groups are equal slices of each head's
    rotated value, one mask per token shared by all heads;
  * z = R^T v (row form z_j = sum_k R[k, j] v_k) and back-rotation o = R u;
  * router "MLP2": [h | e | mean_lang(h)] -> Hr -> exact-erf GELU -> G, with
    e = a E the role-mixed vector and a = softmax(W_r h + b_r);
  * router "additive": the paper's routing-score equation with linear heads;
  * top-K ties go to the lower group index, -0 equals +0, NaN ranks lowest;
  * threshold budgets keep count(gamma > tau) groups clamped to [kmin, kmax];
  * attention: scale 1/sqrt(dh), no mask, keys unchanged, routed values;
  * prefix self-attention: the prefix tokens are the queries, query t sees
    keys 0..t (causal), keys unchanged, routed values;
  * token retention: per view (a run of consecutive tokens) the highest
    token scores are kept with the same order as group selection; a budget
    that does not divide evenly gives the first views one more token;
  * role-driven budget allocation: priorities are an input, quantised to
    integers, and each type's budget is apportioned by largest remainders
    with a cap of G groups per token (details at allocate_groups);
  * full-width routing space (the paper's own operating point): one R over
    all H*dh value dimensions, S groups of H*dh/S consecutive rotated
    dimensions; a token keeping all S groups is cached in value space (its
    routed value is v itself), a routed token caches its kept groups of z.

Parity: every function here is pinned by CPU tests against closed forms, the
paper's printed KV fractions, brute-force enumeration and textbook special
cases; none is "parity unpinned".
"""
from __future__ import annotations

from fractions import Fraction
import math

import numpy as np
from scipy.special import erf as _erf

VIS, LANG, PROP, ACT = 0, 1, 2, 3
TOPK, THRESHOLD = 0, 1

__all__ = [
    "VIS", "LANG", "PROP", "ACT", "TOPK", "THRESHOLD",
    "rotate", "back_rotate", "latent_role", "language_pool", "gelu",
    "router_mlp2", "router_additive", "group_budget", "select_groups",
    "attend_packed_causal", "attend_plain_causal",
    "retained_count", "split_evenly", "retain_tokens", "gather_tokens",
    "role_priority", "quantize_priority", "allocate_groups",
    "rotate_full", "routed_values_full", "pack_full", "values_full", "attend_full", "attend_full_plain",
    "mask_to_idx", "popcount", "pack", "unpack", "expand_mask", "routed_values",
    "attend_packed", "attend_plain", "softmax", "pipeline",
    "kv_fraction", "packed_groups",
]


def _f64(x):
    return np.asarray(x, dtype=np.float64)


# ----------------------------------------------------------------------------
# Sec. 3.2, orthogonal value-space decomposition
# ----------------------------------------------------------------------------

def rotate(v, R):
    """z = R^T v for every token and head (Sec. 3.2, value into routing space).

    v: [..., H, dh]; R: [H, dh, dh] with R[h] the orthonormal matrix of head h.
    Returns z with the same shape as v; z[..., h, j] = sum_k R[h, k, j] v[..., h, k].
    """
    v, R = _f64(v), _f64(R)
    return np.einsum("hkj,...hk->...hj", R, v)


def back_rotate(u, R):
    """o = R u per head (Sec. 3.2, routed representation back to value space)."""
    u, R = _f64(u), _f64(R)
    return np.einsum("hkj,...hj->...hk", R, u)


def expand_mask(mask, G, dh):
    """Diagonal of M_i = diag(m_{i,1} I_ds, ..., m_{i,S} I_ds) (Sec. 3.2).

    mask: integer bitmask array (bit s set = group s kept). Returns a float64
    array [..., dh] of 0/1 entries."""
    ds = dh // G
    mask = np.asarray(mask, dtype=np.uint64)
    bits = (mask[..., None] >> np.arange(G, dtype=np.uint64)) & np.uint64(1)
    return np.repeat(bits.astype(np.float64), ds, axis=-1)


def routed_values(v, mask, R, G):
    """v~ = R M R^T v with explicit dh x dh matrices per token and head (Sec. 3.2).

    v: [B,T,H,dh]; mask [B,T]; R [H,dh,dh]. Plain but slow: builds each
    projection matrix R_h M_i R_h^T."""
    v, R = _f64(v), _f64(R)
    B, T, H, dh = v.shape
    mdiag = expand_mask(mask, G, dh)
    out = np.zeros_like(v)
    for b in range(B):
        for t in range(T):
            M = np.diag(mdiag[b, t])
            for h in range(H):
                P = R[h] @ M @ R[h].T
                out[b, t, h] = P @ v[b, t, h]
    return out


# ----------------------------------------------------------------------------
# Sec. 3.3 latent role, Sec. 3.4 role-conditioned value routing
# ----------------------------------------------------------------------------

def softmax(x, axis=-1):
    x = _f64(x)
    m = np.max(x, axis=axis, keepdims=True)
    e = np.exp(x - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def latent_role(h, W_r, b_r):
    """a = softmax(f_role(h)) with f_role linear (Eq. latentrole, Sec. 3.3)."""
    return softmax(_f64(h) @ _f64(W_r).T + _f64(b_r), axis=-1)


def language_pool(h, types):
    """Pool of the retained language tokens' hidden states (Sec. 3.4).

    h: [B,T,d]; types: [T] or [B,T]. Arithmetic mean per sample; the zero
    vector when a sample has no language token."""
    h = _f64(h)
    types = np.broadcast_to(np.asarray(types), h.shape[:2])
    out = np.zeros((h.shape[0], h.shape[2]))
    for b in range(h.shape[0]):
        sel = types[b] == LANG
        if sel.any():
            out[b] = h[b][sel].mean(axis=0)
    return out


def gelu(x, activation="gelu"):
    """Exact GELU, x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)); 'identity' passes x."""
    x = _f64(x)
    if activation == "identity":
        return x
    return 0.5 * x * (1.0 + _erf(x / np.sqrt(2.0)))


def router_mlp2(h, types, W_r, b_r, E, W1, b1, W2, b2, activation="gelu"):
    """Group scores from [token state | role-mixed vector | pooled language].

    Sec. 3.4 conditions the scores on the token's hidden state, its latent role
    (Eq. latentrole) and the pooled language context. This learned form feeds
    the concatenation [h | e | h_lang] with e = a E through one hidden layer:
    gamma = W2 act(W1 [h|e|h_lang] + b1) + b2.
    h: [B,T,d]; returns [B,T,G] float64."""
    h = _f64(h)
    B, T, d = h.shape
    a = latent_role(h, W_r, b_r)                     # [B,T,C]
    e = a @ _f64(E)                                  # [B,T,d_e]
    hl = language_pool(h, types)                     # [B,d]
    x = np.concatenate([h, e, np.broadcast_to(hl[:, None, :], (B, T, d))], axis=-1)
    pre = x @ _f64(W1).T + _f64(b1)
    return gelu(pre, activation) @ _f64(W2).T + _f64(b2)


def router_additive(h, types, W_tok, b_tok, W_r, b_r, W_role, W_lang, b_lang,
                    alpha_role=0.1, alpha_lang=0.1):
    """Eq. routingscore: gamma = f_v(h) + alpha_role W_role a + alpha_lang f_lang(h_lang).

    f_v and f_lang are linear heads d -> G with bias; W_role is G x C (Sec. 3.4).
    alpha_role = alpha_lang = 0.1 in the paper's setup (Sec. 4.1)."""
    h = _f64(h)
    g_tok = h @ _f64(W_tok).T + _f64(b_tok)
    a = latent_role(h, W_r, b_r)
    g_role = a @ _f64(W_role).T
    g_lang = language_pool(h, types) @ _f64(W_lang).T + _f64(b_lang)   # [B,G]
    return g_tok + alpha_role * g_role + alpha_lang * g_lang[:, None, :]


# ----------------------------------------------------------------------------
# Sec. 3.4 Top-K_i selection, Sec. 3.5 token-type budgets
# ----------------------------------------------------------------------------

def group_budget(scores, types, mode, k_by_type, G, tau=0.0, kmin=0, kmax=0):
    """K_i for every token (Sec. 3.5).

    TOPK: K_i = min(K_type(i), G) (a fixed per-type budget K_m, Sec. 3.5).
    THRESHOLD: K_i = clamp(#{s : gamma_s > tau}, kmin, kmax), then capped at G."""
    scores = np.asarray(scores)
    types = np.broadcast_to(np.asarray(types), scores.shape[:-1])
    if mode == TOPK:
        k = np.asarray(k_by_type)[types.astype(np.int64)]
        return np.minimum(k, G).astype(np.int64)
    cnt = np.sum(scores > tau, axis=-1)
    return np.minimum(np.clip(cnt, kmin, kmax), G).astype(np.int64)


def select_groups(scores, K):
    """Keep the K_i groups with the highest routing scores (Sec. 3.4).

    Order: larger score first; equal scores (with -0 equal to +0) by lower
    group index; NaN after every number. Returns the bitmask [...] uint32.
    The decision is taken on the scores exactly as given (no rounding)."""
    scores = np.asarray(scores)
    G = scores.shape[-1]
    flat = scores.reshape(-1, G)
    kf = np.broadcast_to(np.asarray(K), scores.shape[:-1]).reshape(-1)
    isnan = np.isnan(flat)
    val = np.where(isnan, 0.0, flat.astype(np.float64))
    idx = np.broadcast_to(np.arange(G), flat.shape)
    # lexsort: last key is primary -> NaN flag, then descending value, then index
    order = np.lexsort((idx, -val, isnan), axis=-1)
    masks = np.zeros(flat.shape[0], dtype=np.uint64)
    for n in range(flat.shape[0]):
        for s in order[n, : int(kf[n])]:
            masks[n] |= np.uint64(1) << np.uint64(int(s))
    return masks.astype(np.uint32).reshape(scores.shape[:-1])


def popcount(mask):
    mask = np.asarray(mask, dtype=np.uint64)
    return np.array([bin(int(m)).count("1") for m in mask.reshape(-1)],
                    dtype=np.int64).reshape(mask.shape)


def mask_to_idx(mask, G):
    """Kept group ids in ascending order, padded with 0xFF; and the counts."""
    mask = np.asarray(mask, dtype=np.uint64)
    idx = np.full(mask.shape + (G,), 0xFF, dtype=np.uint8)
    cnt = np.zeros(mask.shape, dtype=np.uint8)
    for pos in np.ndindex(mask.shape):
        kept = [s for s in range(G) if (int(mask[pos]) >> s) & 1]
        idx[pos][: len(kept)] = kept
        cnt[pos] = len(kept)
    return idx, cnt


# ----------------------------------------------------------------------------
# Compact group-indexed value cache (masked representation z~ = M z, Sec. 3.2)
# ----------------------------------------------------------------------------

def pack(z, mask, G, cap):
    """Store only the kept groups of M_i z_i.

    offsets[b, i] = number of groups kept by tokens 0..i-1 of sample b, and
    offsets[b, T] is the sample's total. Vp[b, h, offsets[b,i] + r] holds the
    r-th kept group (ascending group id) of token i, head h. Groups whose slot
    would be >= cap are not stored (the offsets still count them).
    z: [B,T,H,dh]; returns (offsets int64 [B,T+1], Vp float64 [B,H,cap,ds])."""
    z = _f64(z)
    B, T, H, dh = z.shape
    ds = dh // G
    pc = popcount(np.asarray(mask, dtype=np.uint64) & np.uint64((1 << G) - 1))
    offsets = np.zeros((B, T + 1), dtype=np.int64)
    offsets[:, 1:] = np.cumsum(pc, axis=1)
    Vp = np.zeros((B, H, cap, ds))
    for b in range(B):
        for t in range(T):
            m = int(mask[b, t])
            r = 0
            for s in range(G):
                if (m >> s) & 1:
                    slot = offsets[b, t] + r
                    if slot < cap:
                        Vp[b, :, slot, :] = z[b, t, :, s * ds:(s + 1) * ds]
                    r += 1
    return offsets, Vp


def unpack(offsets, Vp, mask, G, T):
    """Rebuild M_i z_i [B,T,H,dh] from the compact cache (dropped groups are 0)."""
    Vp = _f64(Vp)
    B, H, cap, ds = Vp.shape
    out = np.zeros((B, T, H, G * ds))
    for b in range(B):
        for t in range(T):
            m = int(mask[b, t])
            r = 0
            for s in range(G):
                if (m >> s) & 1:
                    slot = int(offsets[b, t]) + r
                    if slot < cap:
                        out[b, t, :, s * ds:(s + 1) * ds] = Vp[b, :, slot, :]
                    r += 1
    return out


def packed_groups(offsets):
    """Total groups stored per sample."""
    return np.asarray(offsets)[:, -1]


def kv_fraction(n_tokens_by_kind, kept_groups, G):
    """Retained KV relative to dense KV (Sec. 4.2 and the language-KV equation).

    Keys stay full width and values keep K_i / S of their width, so token i
    costs (1 + K_i/S)/2 of a dense token. n_tokens_by_kind: total tokens in
    the dense prefix; kept_groups: array of K_i for the tokens kept (a token not
    routed has K_i = S)."""
    kept_groups = np.asarray(kept_groups, dtype=np.float64)
    return float(np.sum((1.0 + kept_groups / G) / 2.0) / n_tokens_by_kind)


# ----------------------------------------------------------------------------
# Attention with unchanged queries/keys over routed values (Sec. 3, Sec. 3.2)
# ----------------------------------------------------------------------------

def _scale(dh, scale):
    return 1.0 / np.sqrt(dh) if (scale is None or scale == 0.0) else float(scale)


def attend_packed(q, k, mask, offsets, Vp, R, G, scale=None):
    """Method form: softmax(q k^T * scale) over all tokens, P.V accumulated in the
    rotated space over each token's kept groups only, then o = R_h u.

    q [B,Tq,H,dh], k [B,T,H,dh], mask [B,T], offsets [B,T+1], Vp [B,H,cap,ds],
    R [H,dh,dh]. Returns [B,Tq,H,dh] float64."""
    q, k = _f64(q), _f64(k)
    B, Tq, H, dh = q.shape
    T = k.shape[1]
    zt = unpack(offsets, Vp, mask, G, T)                          # M z in rotated coords
    s = np.einsum("bqhd,bthd->bhqt", q, k) * _scale(dh, scale)
    p = softmax(s, axis=-1)
    u = np.einsum("bhqt,bthd->bqhd", p, zt)
    return back_rotate(u, R)


def _causal_scores(q, k, scale):
    q, k = _f64(q), _f64(k)
    B, T, H, dh = q.shape
    s = np.einsum("bqhd,bthd->bhqt", q, k) * _scale(dh, scale)
    future = np.triu(np.ones((T, T), dtype=bool), k=1)            # key index > query index
    s[:, :, future] = -np.inf
    return s


def attend_packed_causal(q, k, mask, offsets, Vp, R, G, scale=None):
    """Prefix self-attention over the routed cache (Sec. 3, Sec. 3.2): the T prefix
    tokens are the queries and query t attends keys 0..t; softmax over those
    keys, P.V in the rotated space over each token's kept groups, o = R_h u.

    q, k [B,T,H,dh], mask [B,T], offsets [B,T+1], Vp [B,H,cap,ds], R [H,dh,dh].
    Returns [B,T,H,dh] float64."""
    T = _f64(k).shape[1]
    zt = unpack(offsets, Vp, mask, G, T)
    p = softmax(_causal_scores(q, k, scale), axis=-1)
    u = np.einsum("bhqt,bthd->bqhd", p, zt)
    return back_rotate(u, R)


def attend_plain_causal(q, k, v, mask, R, G, scale=None):
    """Plain form of the prefix self-attention: causal textbook attention whose
    values are the explicit routed values v~_i = R M_i R^T v_i (Sec. 3.2)."""
    vt = routed_values(v, mask, R, G)
    p = softmax(_causal_scores(q, k, scale), axis=-1)
    return np.einsum("bhqt,bthd->bqhd", p, vt)


def attend_plain(q, k, v, mask, R, G, scale=None):
    """Plain form: textbook softmax attention whose values are the routed values
    v~_i = R M_i R^T v_i built as explicit matrices (Sec. 3.2)."""
    q, k = _f64(q), _f64(k)
    B, Tq, H, dh = q.shape
    vt = routed_values(v, mask, R, G)
    s = np.einsum("bqhd,bthd->bhqt", q, k) * _scale(dh, scale)
    p = softmax(s, axis=-1)
    return np.einsum("bhqt,bthd->bqhd", p, vt)


# ----------------------------------------------------------------------------
# Full-width routing space (Sec. 3.2 with d_v = H * dh; Sec. 4.1 configuration)
# ----------------------------------------------------------------------------

def rotate_full(v, R):
    """z = R^T v over the whole value vector (Sec. 3.2): v [B,T,H,dh] is read as
    [B,T,d_v] with d_v = H*dh; R [d_v, d_v]; z_j = sum_k R[k, j] v_k."""
    v = _f64(v)
    B, T = v.shape[:2]
    return v.reshape(B, T, -1) @ _f64(R)


def routed_values_full(v, mask, R, S):
    """v~ = R M R^T v over the whole value vector with M = diag(m_1 I, ..., m_S I)
    (Sec. 3.2). v [B,T,H,dh], mask [B,T] (bit s = group s kept), R [d_v, d_v].
    Returns [B,T,H,dh] float64."""
    v = _f64(v)
    B, T, H, dh = v.shape
    R = _f64(R)
    m = expand_mask(mask, S, H * dh)                 # [B,T,d_v]
    z = v.reshape(B, T, -1) @ R
    return ((z * m) @ R.T).reshape(B, T, H, dh)


def pack_full(v, mask, R, S, cap):
    """Compact cache of the full-width routed values: offsets [B,T+1] in group
    units as pack(); Vp [B, cap, d_v/S]. A token that keeps all S groups is
    stored as its value vector cut into S pieces (v~ = v exactly, since
    R R^T = I); any other token stores its kept groups of z = R^T v in
    ascending group order."""
    v = _f64(v)
    B, T, H, dh = v.shape
    dv = H * dh
    ds = dv // S
    full = (1 << S) - 1
    z = rotate_full(v, R)
    vf = v.reshape(B, T, dv)
    pc = popcount(np.asarray(mask, dtype=np.uint64) & np.uint64(full))
    offsets = np.zeros((B, T + 1), dtype=np.int64)
    offsets[:, 1:] = np.cumsum(pc, axis=1)
    Vp = np.zeros((B, cap, ds))
    for b in range(B):
        for t in range(T):
            mt = int(mask[b, t]) & full
            src = vf[b, t] if mt == full else z[b, t]
            r = 0
            for g in range(S):
                if (mt >> g) & 1:
                    slot = offsets[b, t] + r
                    if slot < cap:
                        Vp[b, slot] = src[g * ds:(g + 1) * ds]
                    r += 1
    return offsets, Vp


def values_full(offsets, Vp, mask, R, S, H):
    """Routed values [B,T,H,dh] from the full-width cache: v for tokens keeping
    all S groups, R z~ for the others (dropped groups are zero)."""
    Vp, R = _f64(Vp), _f64(R)
    B, cap, ds = Vp.shape
    T = np.asarray(offsets).shape[1] - 1
    dv = ds * S
    full = (1 << S) - 1
    out = np.zeros((B, T, dv))
    for b in range(B):
        for t in range(T):
            mt = int(mask[b, t]) & full
            zt = np.zeros(dv)
            r = 0
            for g in range(S):
                if (mt >> g) & 1:
                    zt[g * ds:(g + 1) * ds] = Vp[b, int(offsets[b, t]) + r]
                    r += 1
            out[b, t] = zt if mt == full else R @ zt
    return out.reshape(B, T, H, dv // H)


def attend_full(q, k, mask, offsets, Vp, R, S, scale=None):
    """Method form at full width: textbook attention per head with unchanged
    q, k (Sec. 3) over the routed values rebuilt from the cache."""
    q, k = _f64(q), _f64(k)
    H, dh = q.shape[2], q.shape[3]
    vt = values_full(offsets, Vp, mask, R, S, H)
    s_ = np.einsum("bqhd,bthd->bhqt", q, k) * _scale(dh, scale)
    return np.einsum("bhqt,bthd->bqhd", softmax(s_, axis=-1), vt)


def attend_full_plain(q, k, v, mask, R, S, scale=None):
    """Plain form at full width: textbook attention over v~ = R M R^T v."""
    q, k = _f64(q), _f64(k)
    dh = q.shape[3]
    vt = routed_values_full(v, mask, R, S)
    s_ = np.einsum("bqhd,bthd->bhqt", q, k) * _scale(dh, scale)
    return np.einsum("bhqt,bthd->bqhd", softmax(s_, axis=-1), vt)


# ----------------------------------------------------------------------------
# Whole path
# ----------------------------------------------------------------------------

def pipeline(h, q, k, v, types, weights, mode, k_by_type, G, tau=0.0, kmin=0, kmax=0,
             scores=None, cap=None, w_pri=None):
    """route -> rotate -> pack -> attend for one layer.

    weights: dict with R and the MLP2 router weights (W_r, b_r, E, W1, b1, W2, b2).
    scores: optional given logits (selection only). w_pri: optional priority
    weights per latent role; with them (fixed budgets only) the per-token
    budgets come from the role-driven allocation of Sec. 3.5 on float32
    priorities. Returns a dict of every intermediate."""
    T = np.asarray(k).shape[1]
    if scores is None:
        scores = router_mlp2(h, types, weights["W_r"], weights["b_r"], weights["E"],
                             weights["W1"], weights["b1"], weights["W2"], weights["b2"])
    if w_pri is not None:
        assert mode == TOPK, "role-driven allocation distributes fixed per-type budgets"
        pri = role_priority(h, weights["W_r"], weights["b_r"], w_pri).astype(np.float32)
        K = allocate_groups(pri, types, k_by_type, G)
    else:
        K = group_budget(scores, types, mode, k_by_type, G, tau, kmin, kmax)
    mask = select_groups(scores, K)
    z = rotate(v, weights["R"])
    if cap is None:
        cap = T * G
    offsets, Vp = pack(z, mask, G, cap)
    out = attend_packed(q, k, mask, offsets, Vp, weights["R"], G)
    return {"scores": scores, "K": K, "mask": mask, "z": z, "offsets": offsets,
            "Vp": Vp, "out": out}


# ----------------------------------------------------------------------------
# Token-level retention ahead of the routed path (Sec. 3.1; Sec. 4.1)
# ----------------------------------------------------------------------------

def retained_count(r, n):
    """ceil(r * n): tokens of a type kept at retention ratio r (Sec. 3.1),
    exact for the float r as given."""
    return int(math.ceil(Fraction(r) * int(n)))


def split_evenly(total, n_parts):
    """The retained budget divided evenly between views (Sec. 4.1); when it does
    not divide, the first views take one more token."""
    q, rem = divmod(int(total), int(n_parts))
    return [q + (1 if v < rem else 0) for v in range(int(n_parts))]


def retain_tokens(scores, seg_len, seg_keep):
    """Per sample and per segment (a run of consecutive tokens, e.g. one camera
    view), keep the seg_keep highest-scoring tokens (Sec. 3.1): a larger score
    first, equal scores (-0 equal to +0) by lower index, NaN after every
    number. scores [B, N] with N = sum(seg_len). Returns [B, sum(seg_keep)]
    int64 token indices, ascending within each segment, segments in order."""
    scores = np.asarray(scores)
    B, N = scores.shape
    assert sum(seg_len) == N and all(0 <= k <= n for n, k in zip(seg_len, seg_keep))
    out = np.zeros((B, sum(seg_keep)), dtype=np.int64)
    for b in range(B):
        pos = o = 0
        for n, k in zip(seg_len, seg_keep):
            sc = scores[b, pos:pos + n]
            isnan = np.isnan(sc)
            val = np.where(isnan, 0.0, sc.astype(np.float64))
            order = np.lexsort((np.arange(n), -val, isnan))
            out[b, o:o + k] = pos + np.sort(order[:k])
            pos += n
            o += k
    return out


def gather_tokens(x, idx):
    """Rows of the retained tokens, x[b, idx[b, j]] for x [B, N, ...]."""
    x = np.asarray(x)
    return np.stack([x[b, idx[b]] for b in range(x.shape[0])])


# ----------------------------------------------------------------------------
# Role-driven within-type budget allocation (Sec. 3.5, the allocator B)
# ----------------------------------------------------------------------------

def role_priority(h, W_r, b_r, w_pri):
    """Token-level priority from the latent role representation (Sec. 3.5):
    p_i = w^T a_i with a_i = softmax(W_r h_i + b_r) (Eq. latentrole) and one
    priority weight per latent role. Returns [B,T] float64."""
    return latent_role(h, W_r, b_r) @ _f64(w_pri)


def quantize_priority(p):
    """Integer priority weights: floor(min(max(p, 0), 256) * 2^16) for float32
    priorities p (NaN counts as 0). Exact: scaling by a power of two and the
    floor introduce no rounding, so any implementation gets the same integers."""
    p = np.asarray(p, dtype=np.float32).astype(np.float64)
    p = np.where(np.isnan(p), 0.0, np.clip(p, 0.0, 256.0))
    return np.floor(p * 65536.0).astype(np.int64)


def _apportion(q, budget, G):
    """Largest-remainder apportionment of `budget` units over weights q (int64,
    tokens in index order) with at most G units each. A token whose quota
    budget*q_i/Q exceeds G is capped at G and the rest is apportioned again
    among the others; all-zero weights count as equal. Leftover units go to
    the largest remainders, lower index first on ties."""
    n = len(q)
    K = np.zeros(n, dtype=np.int64)
    active = list(range(n))
    while active:
        w = np.array([q[i] for i in active], dtype=object)
        if sum(w) == 0:
            w = np.ones(len(active), dtype=object)
        Q = int(sum(w))
        over = [a for a, wi in zip(active, w) if budget * int(wi) > G * Q]
        if over:
            for a in over:
                K[a] = G
            budget -= G * len(over)
            active = [a for a in active if a not in over]
            continue
        floors = [budget * int(wi) // Q for wi in w]
        rems = [budget * int(wi) % Q for wi in w]
        left = budget - sum(floors)
        order = sorted(range(len(active)), key=lambda j: (-rems[j], active[j]))
        for j, a in enumerate(active):
            K[a] = floors[j]
        for j in order[:left]:
            K[active[j]] += 1
        break
    return K


def allocate_groups(priority, types, k_by_type, G):
    """Per-token group budgets K_i (Sec. 3.5): within each sample and token type
    m the B_m = K_m * |I_m| groups are distributed by role-derived priority,
    with 0 <= K_i <= G and sum K_i = B_m. Types with K_m >= G keep all G
    groups (no allocation), K_m = 0 keeps none; a token whose type is not one
    of the four keeps all G groups (as with fixed budgets). priority [B, T]
    float32, types [T] or [B, T], k_by_type[4]. Returns K [B, T] int64."""
    priority = np.asarray(priority)
    B, T = priority.shape
    types = np.broadcast_to(np.asarray(types), (B, T))
    q = quantize_priority(priority)
    K = np.where(types > ACT, G, 0).astype(np.int64)
    for b in range(B):
        for m in range(4):
            toks = np.nonzero(types[b] == m)[0]
            if len(toks) == 0:
                continue
            km = min(int(k_by_type[m]), G)
            if km >= G or km == 0:
                K[b, toks] = km
                continue
            K[b, toks] = _apportion([int(x) for x in q[b, toks]], km * len(toks), G)
    return K
