"""CPU pins of the float64 oracle against facts fixed by the paper and by mathematics.

Each check is independent of the oracle's own formulas: closed forms, the
paper's printed KV fractions (tests/golden), brute-force subset enumeration,
library routines (scipy softmax / normal CDF) and textbook special cases.
"""
import itertools
import json
import math
import os
from decimal import ROUND_HALF_UP, Decimal
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import softmax as sp_softmax
from scipy.stats import norm

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


def _haar(n, seed):
    return synth.haar_orthogonal(np.random.default_rng(seed), n)


# ----------------------------------------------------------------------------
# Rotation (Sec. 3.2)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_generated_R_is_orthonormal(cid):
    w = synth.workload(cid)
    Rm = synth.layer_weights(w, 0)["R_master"]
    for h in range(w.H):
        assert np.max(np.abs(Rm[h].T @ Rm[h] - np.eye(w.dh))) <= 1e-12


def test_rotate_plane_rotation_closed_form():
    # R is a rotation by theta; z = R^T v rotates v by -theta.
    th = 0.7
    c, s = math.cos(th), math.sin(th)
    R = np.array([[[c, -s], [s, c]]])
    z1 = O.rotate(np.array([[1.0, 0.0]]), R)[0]
    z2 = O.rotate(np.array([[0.0, 1.0]]), R)[0]
    assert np.allclose(z1, [c, -s], atol=1e-15)
    assert np.allclose(z2, [s, c], atol=1e-15)


def test_rotate_permutation_closed_form():
    dh, H = 64, 3
    perms = [RNG.permutation(dh) for _ in range(H)]
    R = np.zeros((H, dh, dh))
    for h, p in enumerate(perms):
        R[h, p, np.arange(dh)] = 1.0        # column j of R_h is e_{p[j]}
    v = RNG.standard_normal((5, H, dh))
    z = O.rotate(v, R)
    for h, p in enumerate(perms):
        assert np.array_equal(z[:, h, :], v[:, h, p])       # z_j = v_{p[j]}


def test_rotate_identity_is_plain_routing():
    # R = I is the plain sub-token routing control (Sec. 4.2).
    v = RNG.standard_normal((2, 7, 4, 64))
    R = np.broadcast_to(np.eye(64), (4, 64, 64))
    assert np.array_equal(O.rotate(v, R), v)


def test_rotate_parseval_and_round_trip():
    R = np.stack([_haar(128, s) for s in range(3)])
    v = RNG.standard_normal((4, 9, 3, 128))
    z = O.rotate(v, R)
    assert np.allclose(np.linalg.norm(z, axis=-1), np.linalg.norm(v, axis=-1), rtol=1e-13)
    # lossless change of basis: R R^T v = v (Sec. 3.2)
    assert np.max(np.abs(O.back_rotate(z, R) - v)) < 1e-12


# ----------------------------------------------------------------------------
# Latent role (Eq. latentrole), language pool, GELU
# ----------------------------------------------------------------------------

def test_latent_role_closed_form():
    p = np.array([0.1, 0.2, 0.3, 0.4])
    d = 16
    a = O.latent_role(RNG.standard_normal((3, 5, d)), np.zeros((4, d)), np.log(p))
    assert np.allclose(a, np.broadcast_to(p, a.shape), atol=1e-15)


def test_latent_role_matches_library_softmax():
    h = RNG.standard_normal((2, 6, 32))
    W = RNG.standard_normal((8, 32))
    b = RNG.standard_normal(8)
    ref = sp_softmax(h @ W.T + b, axis=-1)
    a = O.latent_role(h, W, b)
    assert np.allclose(a, ref, atol=1e-15)
    assert np.allclose(a.sum(-1), 1.0)


def test_language_pool_closed_form():
    d = 8
    h = np.zeros((3, 6, d))
    types = np.array([[0, 1, 1, 1, 2, 0], [0, 0, 0, 0, 0, 2], [1, 0, 0, 0, 0, 0]])
    for j, t in enumerate([1, 2, 3]):
        h[0, t] = j + 1.0                   # language rows hold 1, 2, 3
    h[0, 0] = 100.0                         # a visual row, must be ignored
    h[2, 0] = 5.0
    pooled = O.language_pool(h, types)
    assert np.allclose(pooled[0], 2.0)       # mean of 1, 2, 3
    assert np.array_equal(pooled[1], np.zeros(d))   # no language token
    assert np.allclose(pooled[2], 5.0)       # a single language token


def test_gelu_identities():
    x = np.linspace(-6, 6, 101)
    g = O.gelu(x)
    assert O.gelu(np.array([0.0]))[0] == 0.0
    assert np.allclose(g - O.gelu(-x), x, atol=1e-14)          # x Phi(x) - (-x) Phi(-x) = x
    assert np.allclose(g, x * norm.cdf(x), atol=1e-14)          # library normal CDF
    assert abs(O.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15


# ----------------------------------------------------------------------------
# Router (Sec. 3.4): each conditioning path in isolation, and the additive form
# ----------------------------------------------------------------------------

def _router_zero(d, C, d_e, Hr, G):
    return dict(W_r=np.zeros((C, d)), b_r=np.zeros(C), E=np.zeros((C, d_e)),
                W1=np.zeros((Hr, 2 * d + d_e)), b1=np.zeros(Hr), W2=np.zeros((G, Hr)),
                b2=np.zeros(G))


def test_router_token_path_only():
    d, C, d_e, G = 8, 3, 5, 8
    w = _router_zero(d, C, d_e, d, G)
    w["W1"][:, :d] = np.eye(d)              # hidden = h
    w["W2"] = np.eye(G)
    h = RNG.standard_normal((2, 4, d))
    types = np.array([0, 1, 1, 0])
    g = O.router_mlp2(h, types, **w)
    assert np.allclose(g, h * norm.cdf(h), atol=1e-14)


def test_router_role_path_only():
    d, C, G = 6, 4, 4
    w = _router_zero(d, C, C, C, G)
    w["W_r"] = RNG.standard_normal((C, d))
    w["b_r"] = RNG.standard_normal(C)
    w["E"] = np.eye(C)                       # e = a
    w["W1"][:, d:d + C] = np.eye(C)          # hidden = e
    w["W2"] = np.eye(G)
    w["b2"] = np.arange(G, dtype=float)
    h = RNG.standard_normal((1, 5, d))
    a = sp_softmax(h @ w["W_r"].T + w["b_r"], axis=-1)
    g = O.router_mlp2(h, np.zeros(5, dtype=int), **w)
    assert np.allclose(g, a * norm.cdf(a) + np.arange(G), atol=1e-14)


def test_router_language_path_only():
    d, C, d_e, G = 8, 2, 3, 8
    w = _router_zero(d, C, d_e, d, G)
    w["W1"][:, d + d_e:] = np.eye(d)         # hidden = pooled language state
    w["W2"] = np.eye(G)
    h = RNG.standard_normal((2, 5, d))
    types = np.array([[1, 1, 0, 0, 2], [0, 0, 1, 0, 0]])
    means = np.stack([h[0, :2].mean(0), h[1, 2]])
    g = O.router_mlp2(h, types, **w)
    for b in range(2):
        assert np.allclose(g[b], np.broadcast_to(means[b] * norm.cdf(means[b]), (5, d)), atol=1e-14)


def test_additive_router_is_folded_linear_mlp2():
    d, C, G = 32, 6, 16
    ar, al = 0.1, 0.1
    W_tok, b_tok = RNG.standard_normal((G, d)), RNG.standard_normal(G)
    W_r, b_r = RNG.standard_normal((C, d)), RNG.standard_normal(C)
    W_role = RNG.standard_normal((G, C))
    W_lang, b_lang = RNG.standard_normal((G, d)), RNG.standard_normal(G)
    h = RNG.standard_normal((2, 7, d))
    types = np.array([0, 0, 1, 1, 1, 2, 0])
    g_add = O.router_additive(h, types, W_tok, b_tok, W_r, b_r, W_role, W_lang, b_lang, ar, al)
    W1 = np.concatenate([W_tok, ar * W_role, al * W_lang], axis=1)
    g_mlp = O.router_mlp2(h, types, W_r, b_r, np.eye(C), W1, b_tok + al * b_lang, np.eye(G),
                          np.zeros(G), activation="identity")
    assert np.allclose(g_add, g_mlp, atol=1e-12)


def test_additive_router_shapes_match_paper_parameter_count():
    # Sec. 4.1: routing heads add about 4.20M parameters over 32 layers
    # (d = 4096, S = 16 groups, C = 6 roles).
    w = synth.workload(2).replace(G=16, C=6)
    aw = synth.additive_weights(w.replace(d=64), 0)     # small d to run; shapes scale
    per_layer = lambda d: (16 * d + 16) * 2 + 16 * 6
    assert sum(aw[k].size for k in ("W_tok", "b_tok", "W_lang", "b_lang", "W_role")) == per_layer(64)
    assert round(32 * per_layer(4096) / 1e6, 2) == 4.20
    h = RNG.standard_normal((1, 3, 64))
    g = O.router_additive(h, np.array([0, 1, 2]), aw["W_tok"], aw["b_tok"], aw["W_r"], aw["b_r"],
                          aw["W_role"], aw["W_lang"], aw["b_lang"])
    assert g.shape == (1, 3, 16)


# ----------------------------------------------------------------------------
# Group selection (Sec. 3.4 Top-K_i, Sec. 3.5 budgets)
# ----------------------------------------------------------------------------

def brute_force_select(row, K):
    """Size-K subset with the largest exact score sum; ties to the
    lexicographically smallest sorted tuple of group ids."""
    best, best_key = (), None
    for sub in itertools.combinations(range(len(row)), K):
        key = (sum(Fraction(float(row[s])) for s in sub), tuple(-s for s in sub))
        if best_key is None or key > best_key:
            best, best_key = sub, key
    return sum(1 << s for s in best)


@pytest.mark.parametrize("G", [4, 8])
def test_select_matches_brute_force_with_ties(G):
    # scores on a coarse grid force many exact ties; include -0.0 and +0.0
    grid = np.array([-1.0, -0.5, -0.0, 0.0, 0.5, 1.0], dtype=np.float32)
    scores = grid[RNG.integers(0, len(grid), size=(300, G))]
    for K in range(G + 1):
        masks = O.select_groups(scores, np.full(300, K))
        for n in range(300):
            assert int(masks[n]) == brute_force_select(scores[n], K), (n, K, scores[n])


def test_select_matches_brute_force_random_f32():
    scores = RNG.standard_normal((200, 8)).astype(np.float32)
    for K in (1, 2, 4, 6):
        masks = O.select_groups(scores, np.full(200, K))
        for n in range(200):
            assert int(masks[n]) == brute_force_select(scores[n], K)


def test_select_nan_ranks_lowest_and_zero_signs_tie():
    s = np.array([np.nan, 1.0, 0.0, -0.0, -np.inf], dtype=np.float32)
    assert int(O.select_groups(s, 1)) == 0b00010
    assert int(O.select_groups(s, 2)) == 0b00110           # +0 and -0 tie: lower index wins
    assert int(O.select_groups(s, 3)) == 0b01110
    assert int(O.select_groups(s, 4)) == 0b11110           # -inf beats NaN
    assert int(O.select_groups(s, 5)) == 0b11111
    assert int(O.select_groups(s, 0)) == 0


def test_select_popcount_equals_budget():
    w = synth.workload(1)
    scores = RNG.standard_normal((1, w.T, w.G))
    K = O.group_budget(scores, w.types(), O.TOPK, w.k_by_type, w.G)
    m = O.select_groups(scores, K)
    assert np.array_equal(O.popcount(m), K)
    assert np.array_equal(K[0], np.where(w.types() == O.VIS, 4, 6))
    idx, cnt = O.mask_to_idx(m, w.G)
    for t in range(w.T):
        kept = [s for s in range(w.G) if (int(m[0, t]) >> s) & 1]
        assert list(idx[0, t, :cnt[0, t]]) == kept and np.all(idx[0, t, cnt[0, t]:] == 0xFF)


def test_threshold_budget_count_rule():
    w = synth.workload(5)
    s = synth.sample_scores(w, 0, 0)
    K = O.group_budget(s, w.types(), O.THRESHOLD, w.k_by_type, w.G, 0.0, 1, 32)
    cnt = np.array([sum(1 for x in row if x > 0) for row in s])
    assert np.array_equal(K, np.clip(cnt, 1, 32))
    assert (cnt == 0).any() and (K >= 1).all()         # the clamp is exercised
    m = O.select_groups(s, K)
    for t in np.nonzero(cnt >= 1)[0][:200]:
        assert int(m[t]) == sum(1 << g for g in range(w.G) if s[t, g] > 0)   # exactly the positives
    for t in np.nonzero(cnt == 0)[0][:50]:
        assert int(m[t]) == brute_force_select(s[t], 1)        # top-1, lowest index on ties


# ----------------------------------------------------------------------------
# Pack: the compact group-indexed cache stores exactly M z (Sec. 3.2)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("cid", [1, 5])
def test_pack_unpack_is_masked_z(cid):
    w = synth.workload(cid)
    T = min(w.T, 96)
    w = w.replace(n_vis=T, n_lang=0, n_prop=0, H=min(w.H, 4))
    z = synth.synthetic_z(w, 0, 0)[None]
    m = synth.synthetic_masks(w, 0, 0)[None]
    off, Vp = O.pack(z, m, w.G, T * w.G)
    mz = z * O.expand_mask(m, w.G, w.dh)[:, :, None, :]
    assert np.array_equal(O.unpack(off, Vp, m, w.G, T), mz)
    pc = O.popcount(m)
    assert off[0, 0] == 0 and np.all(np.diff(off[0]) == pc[0]) and off[0, -1] == pc.sum()
    # r-th slot of a token holds its r-th kept group in ascending order
    t = int(np.argmax(pc[0]))
    kept = [s for s in range(w.G) if (int(m[0, t]) >> s) & 1]
    for r, s in enumerate(kept):
        assert np.array_equal(Vp[0, :, off[0, t] + r], z[0, t, :, s * w.ds:(s + 1) * w.ds])


def test_pack_size_equals_budget_and_capacity_clips():
    w = synth.workload(2).replace(H=2)
    z = synth.synthetic_z(w, 0, 0)[None]
    m = synth.synthetic_masks(w, 0, 0)[None]
    budget = w.n_vis * w.k_vis + w.n_lang * w.k_lang + w.n_prop * w.G
    off, Vp = O.pack(z, m, w.G, budget)
    assert off[0, -1] == budget
    assert Vp.size == w.H * w.ds * budget         # packed elements = H * ds * sum K_i
    cap = budget - 37
    off2, Vp2 = O.pack(z, m, w.G, cap)
    assert np.array_equal(off2, off) and np.array_equal(Vp2, Vp[:, :, :cap])


def _table_prefix_fraction(n_dense, routed, K, unrouted, S=16):
    """Pack a synthetic prefix and account its KV from the packed offsets."""
    w = synth.workload(1).replace(H=1, dh=S * 2, G=S, n_vis=routed, n_lang=0, n_prop=0)
    z = synth.synthetic_z(w, 0, 0)[None]
    m = synth.synthetic_masks(w, 0, 0, counts=K)[None]
    off, _ = O.pack(z, m, S, routed * S)
    kept = np.diff(off[0])
    return O.kv_fraction(n_dense, np.concatenate([kept, np.full(unrouted, S)]), S)


def _printed(x, nd):
    """Round the way the paper prints percentages (half away from zero)."""
    return float(Decimal(repr(x)).quantize(Decimal(1).scaleb(-nd), rounding=ROUND_HALF_UP))


def test_kv_fractions_reproduce_paper_tables():
    g = json.load(open(os.path.join(GOLDEN, "kv_fractions.json")))
    S = g["S"]
    for n, K, pct in g["table1_visual_kv"]["rows"]:
        f = _table_prefix_fraction(g["dense_visual_tokens"], n, np.full(n, K), 0, S)
        assert _printed(100 * f, 2) == pct, (n, K, 100 * f)
    for K, vpct, kvpct in g["table3_language"]["rows"]:
        f = _table_prefix_fraction(48, 48, np.full(48, K), 0, S)
        assert _printed(100 * K / S, 2) == vpct and _printed(100 * f, 2) == kvpct
    pr = g["table4_combined"]["prefix_reading"]
    for n, comb, visonly in g["table4_combined"]["rows"]:
        nl, no = pr["language"], pr["uncompressed_other"]
        Ks = np.concatenate([np.full(n, 1), np.full(nl, 1)])
        f_c = _table_prefix_fraction(pr["dense_tokens"], n + nl, Ks, no, S)
        f_v = _table_prefix_fraction(pr["dense_tokens"], n, np.full(n, 1), nl + no, S)
        assert _printed(100 * f_c, 1) == comb and _printed(100 * f_v, 1) == visonly


# ----------------------------------------------------------------------------
# Attention over the routed values
# ----------------------------------------------------------------------------

def _attn_case(B=2, T=11, Tq=5, H=3, dh=64, G=8, seed=0):
    r = np.random.default_rng(seed)
    q = r.standard_normal((B, Tq, H, dh))
    k = r.standard_normal((B, T, H, dh))
    v = r.standard_normal((B, T, H, dh))
    R = np.stack([_haar(dh, seed * 100 + h) for h in range(H)])
    return q, k, v, R


def _textbook(q, k, v, scale=None):
    dh = q.shape[-1]
    s = np.einsum("bqhd,bthd->bhqt", q, k) * (1 / math.sqrt(dh) if scale is None else scale)
    return np.einsum("bhqt,bthd->bqhd", sp_softmax(s, axis=-1), v)


def test_attend_all_groups_is_textbook_attention():
    q, k, v, R = _attn_case()
    G = 8
    m = np.full((2, 11), (1 << G) - 1, dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, G, 11 * G)
    out = O.attend_packed(q, k, m, off, Vp, R, G)
    assert np.max(np.abs(out - _textbook(q, k, v))) < 1e-12


def test_attend_single_group_full_width_is_textbook():
    q, k, v, R = _attn_case(dh=64)
    m = np.ones((2, 11), dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, 1, 11)
    assert np.max(np.abs(O.attend_packed(q, k, m, off, Vp, R, 1) - _textbook(q, k, v))) < 1e-12


def test_attend_one_token_returns_routed_value():
    q, k, v, R = _attn_case(T=1)
    G, dh = 8, 64
    m = np.array([[0b10110010], [0b00000001]], dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, G, G)
    out = O.attend_packed(q, k, m, off, Vp, R, G)
    for b in range(2):
        M = np.diag(np.repeat([(int(m[b, 0]) >> s) & 1 for s in range(G)], dh // G).astype(float))
        for h in range(3):
            vt = R[h] @ M @ R[h].T @ v[b, 0, h]
            assert np.allclose(out[b, :, h], np.broadcast_to(vt, (5, dh)), atol=1e-12)


def test_attend_no_groups_gives_zero():
    q, k, v, R = _attn_case()
    m = np.zeros((2, 11), dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, 8, 8)
    assert np.max(np.abs(O.attend_packed(q, k, m, off, Vp, R, 8))) == 0.0


def test_attend_scale_closed_form():
    # two tokens whose logits differ by ln 3 after the 1/sqrt(dh) scale -> p = (3/4, 1/4)
    dh, G = 64, 8
    q = np.zeros((1, 1, 1, dh)); q[0, 0, 0, 0] = 1.0
    k = np.zeros((1, 2, 1, dh)); k[0, 0, 0, 0] = math.sqrt(dh) * math.log(3.0)
    v = np.random.default_rng(3).standard_normal((1, 2, 1, dh))
    R = np.eye(dh)[None]
    m = np.array([[0b00001111, 0b11110000]], dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, G, 2 * G)
    out = O.attend_packed(q, k, m, off, Vp, R, G)[0, 0, 0]
    want = 0.75 * np.where(np.arange(dh) < 32, v[0, 0, 0], 0) + 0.25 * np.where(np.arange(dh) >= 32, v[0, 1, 0], 0)
    assert np.allclose(out, want, atol=1e-14)


def test_attend_method_form_equals_plain_form():
    q, k, v, R = _attn_case(B=2, T=13, Tq=4, H=2, dh=64, G=8, seed=5)
    G = 8
    m = np.stack([synth.synthetic_masks(synth.workload(1).replace(n_vis=13, n_lang=0), 0, b,
                                        counts=np.random.default_rng(b).integers(0, G + 1, 13))
                  for b in range(2)])
    off, Vp = O.pack(O.rotate(v, R), m, G, 13 * G)
    a = O.attend_packed(q, k, m, off, Vp, R, G)
    b = O.attend_plain(q, k, v, m, R, G)
    assert np.max(np.abs(a - b)) < 1e-12


# ----------------------------------------------------------------------------
# Prefix self-attention (causal) over the routed values
# ----------------------------------------------------------------------------

def _causal_case(seed=11, B=2, T=9, H=2, dh=64, G=8):
    q, k, v, R = _attn_case(B=B, T=T, Tq=T, H=H, dh=dh, G=G, seed=seed)
    m = np.random.default_rng(seed).integers(0, 1 << G, size=(B, T)).astype(np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, G, T * G)
    return q, k, v, R, m, off, Vp


def test_attend_causal_row_t_is_attention_over_the_first_t_plus_1_tokens():
    q, k, v, R, m, off, Vp = _causal_case()
    G, T = 8, 9
    out = O.attend_packed_causal(q, k, m, off, Vp, R, G)
    for t in range(T):
        # the prefix 0..t packs to the same slots (offsets are prefix sums)
        ref = O.attend_packed(q[:, t:t + 1], k[:, :t + 1], m[:, :t + 1], off[:, :t + 2], Vp, R, G)
        assert np.max(np.abs(out[:, t:t + 1] - ref)) < 1e-12


def test_attend_causal_first_query_returns_its_routed_value():
    q, k, v, R, m, off, Vp = _causal_case(seed=12)
    G, dh = 8, 64
    out = O.attend_packed_causal(q, k, m, off, Vp, R, G)
    for b in range(2):
        M = np.diag(np.repeat([(int(m[b, 0]) >> s) & 1 for s in range(G)], dh // G).astype(float))
        for h in range(2):
            assert np.allclose(out[b, 0, h], R[h] @ M @ R[h].T @ v[b, 0, h], atol=1e-12)


def test_attend_causal_all_groups_is_textbook_causal_attention():
    q, k, v, R = _attn_case(B=2, T=10, Tq=10, H=2, dh=64, seed=13)
    G = 8
    m = np.full((2, 10), (1 << G) - 1, dtype=np.uint32)
    off, Vp = O.pack(O.rotate(v, R), m, G, 10 * G)
    out = O.attend_packed_causal(q, k, m, off, Vp, R, G)
    for b in range(2):
        for h in range(2):
            for t in range(10):
                s = k[b, :t + 1, h] @ q[b, t, h] / math.sqrt(64)
                p = np.exp(s - s.max())
                p /= p.sum()
                assert np.allclose(out[b, t, h], p @ v[b, :t + 1, h], atol=1e-12)


def test_attend_causal_method_form_equals_plain_form():
    q, k, v, R, m, off, Vp = _causal_case(seed=14, T=12)
    a = O.attend_packed_causal(q, k, m, off, Vp, R, 8)
    b = O.attend_plain_causal(q, k, v, m, R, 8)
    assert np.max(np.abs(a - b)) < 1e-12


# ----------------------------------------------------------------------------
# Token-level retention
# ----------------------------------------------------------------------------

def test_retained_counts_are_the_printed_ones():
    g = json.load(open(os.path.join(GOLDEN, "retention_counts.json")))
    for r, kept in g["rows"]:
        assert O.retained_count(r, g["dense_visual_tokens"]) == kept
        per_view = O.split_evenly(kept, g["views"])
        assert per_view == [kept // 2, kept // 2] and sum(per_view) == kept
    assert O.retained_count(1.0, 177) == 177 and O.retained_count(0.5, 3) == 2   # ceiling
    assert O.split_evenly(7, 3) == [3, 2, 2]


def _scores_with_ties(rng, B, N):
    sc = rng.standard_normal((B, N)).astype(np.float32)
    sc[:, ::5] = np.round(sc[:, ::5])               # exact ties
    sc[:, 1::7] = 0.0
    sc[:, 3::7] = -0.0                              # -0 equals +0
    sc[:, 2::11] = np.nan                           # NaN ranks after every number
    return sc


def test_retention_equals_group_selection_on_short_segments():
    # a segment of <= 32 tokens is exactly a group-selection problem, whose
    # oracle is pinned by brute force above
    rng = np.random.default_rng(21)
    seg_len, seg_keep = [7, 32, 1, 20], [3, 12, 1, 0]
    sc = _scores_with_ties(rng, 5, sum(seg_len))
    got = O.retain_tokens(sc, seg_len, seg_keep)
    for b in range(5):
        pos = o = 0
        for n, k in zip(seg_len, seg_keep):
            m = int(O.select_groups(sc[b, pos:pos + n][None], np.array([k]))[0])
            want = [pos + s for s in range(n) if (m >> s) & 1]
            assert list(got[b, o:o + k]) == want
            pos += n
            o += k


def test_retention_keeps_the_highest_scores():
    rng = np.random.default_rng(22)
    seg_len, seg_keep = [256, 256], [16, 16]
    sc = _scores_with_ties(rng, 3, 512)
    got = O.retain_tokens(sc, seg_len, seg_keep)
    for b in range(3):
        for v in range(2):
            kept = got[b, 16 * v:16 * v + 16]
            assert np.all(np.diff(kept) > 0) and np.all((kept >= 256 * v) & (kept < 256 * (v + 1)))
            seg = sc[b, 256 * v:256 * (v + 1)]
            key = lambda i: (np.isnan(seg[i]), -np.nan_to_num(seg[i], nan=0.0), i)
            kept_keys = [key(i - 256 * v) for i in kept]
            dropped = [key(i) for i in range(256) if 256 * v + i not in set(kept.tolist())]
            assert max(kept_keys) < min(dropped)


def test_gather_tokens_takes_the_listed_rows():
    rng = np.random.default_rng(23)
    x = rng.standard_normal((2, 9, 3, 4))
    idx = np.array([[0, 4, 8], [1, 2, 3]])
    g = O.gather_tokens(x, idx)
    for b in range(2):
        for j in range(3):
            assert np.array_equal(g[b, j], x[b, idx[b, j]])


def test_routed_value_is_a_projection():
    _, _, v, R = _attn_case(T=20, seed=9)
    G = 8
    m = RNG.integers(0, 1 << G, size=(2, 20)).astype(np.uint32)
    vt = O.routed_values(v, m, R, G)
    z = O.rotate(v, R)
    mz = z * O.expand_mask(m, G, 64)[:, :, None, :]
    assert np.all(np.linalg.norm(vt, axis=-1) <= np.linalg.norm(v, axis=-1) + 1e-12)
    assert np.allclose(np.linalg.norm(vt, axis=-1) ** 2, np.sum(mz ** 2, axis=-1), rtol=1e-12)
    assert np.allclose(O.routed_values(vt, m, R, G), vt, atol=1e-12)      # idempotent


# ----------------------------------------------------------------------------
# Whole path on the tiny workload
# ----------------------------------------------------------------------------

def test_pipeline_tiny_invariants():
    w = synth.workload(1)
    wt = synth.layer_weights(w, 0)
    a = synth.layer_activations(w, 0)
    r = O.pipeline(a["h"], a["q"], a["k"], a["v"], w.types(), wt, w.mode, w.k_by_type, w.G)
    assert np.array_equal(O.popcount(r["mask"])[0], np.where(w.types() == O.VIS, 4, 6))
    assert r["offsets"][0, -1] == 64 * 4 + 16 * 6
    assert r["out"].shape == (1, w.Tq, w.H, w.dh) and np.all(np.isfinite(r["out"]))
    plain = O.attend_plain(a["q"], a["k"], a["v"], r["mask"], wt["R"], w.G)
    assert np.max(np.abs(plain - r["out"])) < 1e-12


# ----------------------------------------------------------------------------
# Role-driven within-type budget allocation (Sec. 3.5)
# ----------------------------------------------------------------------------

def test_role_priority_special_cases():
    rng = np.random.default_rng(30)
    h = rng.standard_normal((2, 5, 8))
    w = np.array([0.5, 2.0, -1.0])
    # one role: a = 1, the priority is its weight
    p1 = O.role_priority(h, np.zeros((1, 8)), np.zeros(1), w[:1])
    assert np.allclose(p1, 0.5, rtol=0, atol=1e-15)
    # equal logits: a is uniform, the priority is the mean weight
    pu = O.role_priority(h, np.zeros((3, 8)), np.zeros(3), w)
    assert np.allclose(pu, w.mean(), rtol=0, atol=1e-15)
    # one dominant logit: the priority is that role's weight
    pd = O.role_priority(h, np.zeros((3, 8)), np.array([0.0, 800.0, 0.0]), w)
    assert np.allclose(pd, 2.0, rtol=0, atol=1e-12)


def test_quantize_priority_exact_values():
    x = np.array([1.0, 2.0 ** -16, 1.5 * 2.0 ** -16, 0.0, -0.0, -3.0, np.nan, 256.0, 1e9, np.inf,
                  0.1, 3.75], dtype=np.float32)
    want = [65536, 1, 1, 0, 0, 0, 0, 1 << 24, 1 << 24, 1 << 24,
            int(np.floor(float(np.float32(0.1)) * 65536)), 245760]
    assert O.quantize_priority(x).tolist() == want
    assert want[10] == 6553


def _alloc_case(rng, B, T, G):
    pr = rng.standard_normal((B, T)).astype(np.float32) * 2 + 1
    pr[rng.random((B, T)) < 0.15] = 0.0
    pr[rng.random((B, T)) < 0.05] = np.nan
    pr[:, 1::7] = pr[:, 0:1]                     # ties
    types = rng.integers(0, 4, size=(B, T)).astype(np.uint8)
    return pr, types


@pytest.mark.parametrize("G", [4, 8, 16])
def test_allocation_meets_the_stated_constraints(G):
    rng = np.random.default_rng(31 + G)
    pr, types = _alloc_case(rng, 3, 40, G)
    for kby in ([1, 2, 3, 0], [G // 2, G, 1, G - 1], [0, 0, 0, 0]):
        K = O.allocate_groups(pr, types, kby, G)
        assert np.all((K >= 0) & (K <= G))
        for b in range(3):
            for m in range(4):
                sel = types[b] == m
                assert K[b][sel].sum() == min(kby[m], G) * sel.sum()


def test_allocation_uniform_priorities_give_the_fixed_budget():
    types = np.array([0] * 7 + [1] * 5 + [2, 3])
    kby = [3, 5, 8, 2]
    for val in (0.0, 1.25, 300.0):
        K = O.allocate_groups(np.full((2, 14), val, np.float32), types, kby, 8)
        assert np.array_equal(K, np.broadcast_to(np.array(kby)[types], (2, 14)))


def test_allocation_is_monotone_in_priority():
    rng = np.random.default_rng(32)
    pr, types = _alloc_case(rng, 4, 60, 8)
    K = O.allocate_groups(pr, types, [2, 3, 5, 1], 8)
    q = O.quantize_priority(pr)
    for b in range(4):
        for m in range(4):
            i = np.nonzero(types[b] == m)[0]
            qi, ki = q[b, i], K[b, i]
            hi = qi[:, None] > qi[None, :]
            assert np.all((ki[:, None] >= ki[None, :]) | ~hi)


def test_allocation_worked_examples():
    # one dominant token: 16 groups over weights 100:1:1:1 give it 15.5 > G = 8,
    # so it keeps 8 and the other 8 go 8/3 each: floors 2, 2, 2, then the equal
    # remainders go to the lower indices
    assert O.allocate_groups(np.array([[100.0, 1, 1, 1]], np.float32), [0] * 4, [4, 0, 0, 0], 8).tolist() == \
        [[8, 3, 3, 2]]
    # a cap that only appears after the first one: 24 groups over 100:60:10:10:10:10
    # cap token 0 (12 > 8); 16 over 60:10:10:10:10 caps token 1 (9.6 > 8);
    # 8 over four equal weights gives 2 each
    assert O.allocate_groups(np.array([[100.0, 60, 10, 10, 10, 10]], np.float32), [1] * 6, [0, 4, 0, 0],
                             8).tolist() == [[8, 8, 2, 2, 2, 2]]
    # zero priorities share what the capped token leaves, equally
    assert O.allocate_groups(np.array([[1.0, 0, 0]], np.float32), [0] * 3, [4, 0, 0, 0], 8).tolist() == \
        [[8, 2, 2]]
    # proportional with remainders: 10 groups over 3:2:1 -> quotas 5, 3.33, 1.67
    assert O.allocate_groups(np.array([[3.0, 2.0, 1.0, 7.0]], np.float32), [2, 2, 2, 0], [8, 8, 10 // 3, 8],
                             8).tolist() == [[5, 3, 1, 8]]


def _water_filled_quotas(q, budget, G):
    """Continuous allocation x_i = min(G, lam * q_i) with sum x = budget (a
    water level lam found by trying every capped prefix), equal shares when the
    uncapped weights are all zero. Exact rationals."""
    n = len(q)
    order = sorted(range(n), key=lambda i: -q[i])
    for c in range(n + 1):
        capped, rest = order[:c], order[c:]
        left = budget - G * c
        if left < 0:
            break
        Qr = sum(q[i] for i in rest)
        x = [Fraction(0)] * n
        for i in capped:
            x[i] = Fraction(G)
        if Qr == 0:
            if not rest:
                if left == 0:
                    return x
                continue
            share = Fraction(left, len(rest))
            if share <= G:
                for i in rest:
                    x[i] = share
                return x
            continue
        lam = Fraction(left, Qr)
        if all(lam * q[i] <= G for i in rest) and all(lam * q[i] >= G for i in capped):
            for i in rest:
                x[i] = lam * q[i]
            return x
    raise AssertionError("no water level")


def test_allocation_is_the_nearest_integer_split_of_the_water_filled_quotas():
    """Brute force: among all integer K with 0 <= K_i <= G and sum = B_m, the
    allocation minimises sum (K_i - x_i)^2 for the continuous capped quotas x,
    and among equal minimisers gives the extra groups to the lower indices."""
    import itertools
    rng = np.random.default_rng(33)
    cases = 0
    for _ in range(300):
        n = int(rng.integers(1, 6))
        G = int(rng.integers(2, 5))
        km = int(rng.integers(1, G))
        kind = rng.integers(0, 3)
        if kind == 0:
            pr = rng.integers(0, 6, size=n).astype(np.float32)       # small integers: ties, zeros
        elif kind == 1:
            pr = (rng.random(n) * 5).astype(np.float32)
        else:
            pr = np.where(rng.random(n) < 0.5, 0.0, rng.integers(1, 50, size=n)).astype(np.float32)
        q = [int(x) for x in O.quantize_priority(pr)]
        budget = km * n
        try:
            x = _water_filled_quotas(q, budget, G)
        except AssertionError:
            continue
        best, arg = None, []
        for K in itertools.product(range(G + 1), repeat=n):
            if sum(K) != budget:
                continue
            dev = sum((Fraction(k) - xi) ** 2 for k, xi in zip(K, x))
            if best is None or dev < best:
                best, arg = dev, [K]
            elif dev == best:
                arg.append(K)
        want = max(arg)       # lexicographically largest: lower index first
        got = O.allocate_groups(pr[None, :], [0] * n, [km, 0, 0, 0], G)[0].tolist()
        assert got == list(want), (pr, G, km, got, want)
        cases += 1
    assert cases > 200


def test_allocation_groups_are_per_sample_and_type():
    rng = np.random.default_rng(34)
    pr, types = _alloc_case(rng, 3, 30, 8)
    kby = [3, 2, 5, 6]
    K = O.allocate_groups(pr, types, kby, 8)
    for b in range(3):
        for m in range(4):
            i = np.nonzero(types[b] == m)[0]
            alone = O.allocate_groups(pr[b, i][None], np.full(len(i), m), kby, 8)[0]
            assert np.array_equal(K[b, i], alone)
    # a token of no listed type keeps every group
    t2 = types.copy()
    t2[0, 3] = 7
    assert O.allocate_groups(pr, t2, kby, 8)[0, 3] == 8


def test_pipeline_with_allocation_keeps_the_type_budgets():
    w = synth.workload(1)
    wt = synth.layer_weights(w, 0)
    a = synth.layer_activations(w, 0)
    wpri = synth.priority_weights(w, 0)
    r = O.pipeline(a["h"], a["q"], a["k"], a["v"], w.types(), wt, w.mode, w.k_by_type, w.G, w_pri=wpri)
    pri = O.role_priority(a["h"], wt["W_r"], wt["b_r"], wpri).astype(np.float32)
    assert np.array_equal(r["K"], O.allocate_groups(pri, w.types(), w.k_by_type, w.G))
    assert np.array_equal(O.popcount(r["mask"]), r["K"])
    assert r["offsets"][0, -1] == 64 * 4 + 16 * 6        # same total as the fixed budgets
    assert len(np.unique(r["K"][0][w.types() == O.VIS])) > 1   # budgets do vary by token


# ----------------------------------------------------------------------------
# Full-width routing space (Sec. 3.2 with one R over all heads; Sec. 4.1)
# ----------------------------------------------------------------------------

def _block_rotation_full(R_heads, S):
    """The full-width R that reproduces per-head routing with S groups: R_full =
    blockdiag(R_h) with columns permuted so that full-width group s (d_v/S
    consecutive dims) holds slice s of every head's rotated value."""
    H, dh, _ = R_heads.shape
    ds = dh // S
    dv = H * dh
    Rf = np.zeros((dv, dv))
    for h in range(H):
        for j in range(dh):
            s, r = divmod(j, ds)
            c = s * (H * ds) + h * ds + r
            Rf[h * dh:(h + 1) * dh, c] = R_heads[h][:, j]
    return Rf


def test_full_width_with_block_rotation_equals_per_head_routing():
    rng = np.random.default_rng(40)
    H, dh, S, B, T, Tq = 4, 16, 4, 2, 9, 3
    R_heads = np.stack([synth.haar_orthogonal(rng, dh) for _ in range(H)])
    Rf = _block_rotation_full(R_heads, S)
    assert np.allclose(Rf.T @ Rf, np.eye(H * dh), atol=1e-12)
    q = rng.standard_normal((B, Tq, H, dh))
    k = rng.standard_normal((B, T, H, dh))
    v = rng.standard_normal((B, T, H, dh))
    mask = rng.integers(0, 1 << S, size=(B, T)).astype(np.uint32)
    mask[0, 0] = (1 << S) - 1
    assert np.allclose(O.routed_values_full(v, mask, Rf, S), O.routed_values(v, mask, R_heads, S), atol=1e-12)
    ref = O.attend_plain(q, k, v, mask, R_heads, S)
    assert np.allclose(O.attend_full_plain(q, k, v, mask, Rf, S), ref, atol=1e-12)
    off, Vp = O.pack_full(v, mask, Rf, S, T * S)
    assert np.allclose(O.attend_full(q, k, mask, off, Vp, Rf, S), ref, atol=1e-12)


def test_full_width_plane_rotation_closed_form():
    th = 0.3
    c, s_ = np.cos(th), np.sin(th)
    R = np.array([[c, -s_], [s_, c]])
    v = np.array([1.0, 0.0]).reshape(1, 1, 1, 2)
    # z = R^T v = (c, -s); keeping group 0 leaves (c, 0); back: R (c, 0) = c (c, s)
    got = O.routed_values_full(v, np.array([[1]], np.uint32), R, 2)
    assert np.allclose(got.reshape(2), [c * c, c * s_], atol=1e-15)
    got1 = O.routed_values_full(v, np.array([[2]], np.uint32), R, 2)
    assert np.allclose(got1.reshape(2), [s_ * s_, -c * s_], atol=1e-15)   # the other group: the rest of v
    assert np.allclose(got.reshape(2) + got1.reshape(2), [1.0, 0.0], atol=1e-15)


def test_full_width_cache_special_cases():
    rng = np.random.default_rng(41)
    H, dh, S, B, T = 2, 8, 4, 2, 6
    Rf = synth.haar_orthogonal(rng, H * dh)
    v = rng.standard_normal((B, T, H, dh))
    full = (1 << S) - 1
    mask = np.array([[full, 0, 5, full, 1, 8], [3, full, full, 0, 15, 6]], np.uint32)
    z = O.rotate_full(v, Rf)
    assert np.allclose(z @ Rf.T, v.reshape(B, T, -1), atol=1e-12)                 # R R^T = I
    assert np.allclose(np.sum(z ** 2, -1), np.sum(v.reshape(B, T, -1) ** 2, -1))  # Parseval
    off, Vp = O.pack_full(v, mask, Rf, S, T * S)
    assert off[0, -1] == 4 + 0 + 2 + 4 + 1 + 1
    # a token keeping every group is cached as its value vector, exactly
    assert np.array_equal(Vp[0, 0:4].reshape(-1), v[0, 0].reshape(-1))
    # a routed token caches its kept groups of z, ascending
    assert np.array_equal(Vp[0, 4:6], np.stack([z[0, 2, 0:4], z[0, 2, 8:12]]))
    vt = O.values_full(off, Vp, mask, Rf, S, H)
    assert np.array_equal(vt[0, 0], v[0, 0]) and np.all(vt[0, 1] == 0) and np.all(vt[1, 3] == 0)
    assert np.allclose(vt, O.routed_values_full(v, mask, Rf, S), atol=1e-12)
    # all groups kept everywhere: textbook attention
    q = rng.standard_normal((B, 3, H, dh))
    k = rng.standard_normal((B, T, H, dh))
    allm = np.full((B, T), full, np.uint32)
    sc = np.einsum("bqhd,bthd->bhqt", q, k) / np.sqrt(dh)
    want = np.einsum("bhqt,bthd->bqhd", sp_softmax(sc, axis=-1), v)
    assert np.allclose(O.attend_full_plain(q, k, v, allm, Rf, S), want, atol=1e-12)
