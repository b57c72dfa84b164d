/*
 * librolesub: the inference hot path of Role-Conditioned Sub-Token Routing
 * (RoleSub) on AMD Instinct MI355X (gfx950).
 *
 * The four calls follow the paper's statement of the method (Sec. 3):
 *   rolesub_rotate_values  z = R^T v per head              (Sec. 3.2)
 *   rolesub_route          latent role + routing score + Top-K_i groups
 *                                                           (Eq. latentrole,
 *                                                            Eq. routingscore,
 *                                                            Sec. 3.4, 3.5)
 *   rolesub_pack_kv        compact cache of the kept groups of M z (Sec. 3.2)
 *   rolesub_rotate_pack    the two above in one pass, z never stored
 *   rolesub_attend         attention with unchanged queries and keys over the
 *                          routed values v~ = R M R^T v     (Sec. 3, 3.2)
 *
 * Conventions shared by every call
 *   - Layouts are dense, row-major, innermost dimension last, no padding.
 *   - Every tensor argument is a DEVICE pointer into memory the caller owns;
 *     the library never allocates, frees or keeps device memory and holds no
 *     state between calls. Descriptor structs are HOST pointers read during
 *     the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). All
 *     work is enqueued asynchronously on it; the call returns before the GPU
 *     finishes. Inputs must stay valid and unmodified until then.
 *   - Validation happens on the host before anything is enqueued. On any
 *     non-OK status nothing was enqueued and the outputs are untouched, except
 *     ROLESUB_ERR_HIP, where a launch failed (the message says which).
 *     rolesub_last_error() returns a thread-local description of the most
 *     recent failure on the calling thread.
 *   - Element type: ROLESUB_F32 (float) or ROLESUB_BF16 (bfloat16). One dtype
 *     covers all floating-point tensors of a call except scores (always f32).
 *     Inside kernels accumulation and softmax are f32; bf16 outputs are
 *     rounded to nearest even.
 *   - Supported shapes: dh in {64, 128}; G divides dh; 1 <= G <= 32.
 *     The bf16 path uses matrix-core kernels for dh = 128 and vector kernels
 *     otherwise.
 *
 * Routing space reading: every head h has its own orthonormal R_h (dh x dh);
 * group s of a token is the s-th slice of width ds = dh/G of each head's
 * rotated value, and one group mask per token is shared by all heads. This is
 * the paper's single R with R = blockdiag(R_h) up to a fixed permutation of
 * coordinates, so the paper's losslessness property (all groups kept gives
 * back v) holds unchanged.
 */
#ifndef ROLESUB_H
#define ROLESUB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rolesub_status {
  ROLESUB_OK = 0,
  ROLESUB_ERR_INVALID_ARG = 1,  /* null pointer, negative size, K > G, ... */
  ROLESUB_ERR_UNSUPPORTED = 2,  /* valid but not implemented: dh, G, dtype  */
  ROLESUB_ERR_CAPACITY = 3,     /* packed-cache capacity below the budget   */
  ROLESUB_ERR_HIP = 4           /* a HIP launch or runtime call failed      */
} rolesub_status;

typedef enum rolesub_dtype { ROLESUB_F32 = 0, ROLESUB_BF16 = 1 } rolesub_dtype;

/* Token types of the multimodal sequence X = [X^vis, X^lang, X^prop, X^act]
 * (Sec. 3). */
enum { ROLESUB_VIS = 0, ROLESUB_LANG = 1, ROLESUB_PROP = 2, ROLESUB_ACT = 3 };

/* B independent prefixes of T key/value tokens; H heads of width dh; G value
 * groups per head (S in the paper); d hidden size of the router input. */
typedef struct rolesub_dims {
  int32_t B, T, H, dh, G, d;
} rolesub_dims;

/* Group budget per token (Sec. 3.5).
 * TOPK:      K_i = k_by_type[type_i]           (0 <= k <= G; k = G keeps all)
 * THRESHOLD: K_i = clamp(#{s : gamma_s > tau}, kmin, kmax)  (0<=kmin<=kmax<=G)
 * Then the K_i groups with the largest scores are kept; equal scores go to
 * the lower group index, -0 equals +0 and NaN ranks below every number. */
enum { ROLESUB_BUDGET_TOPK = 0, ROLESUB_BUDGET_THRESHOLD = 1 };
typedef struct rolesub_budget {
  int32_t mode;
  int32_t k_by_type[4];   /* indexed by ROLESUB_VIS .. ROLESUB_ACT */
  float tau;
  int32_t kmin, kmax;
} rolesub_budget;

/* Router weights (Sec. 3.3, 3.4). All matrices row-major [out][in] in the
 * call's dtype; biases [out] in the call's dtype; device pointers.
 *
 * ROLESUB_ROUTER_MLP2 (learned scoring functions):
 *   a     = softmax(W_r h + b_r)                 W_r [C][d], b_r [C]
 *   e     = sum_c a_c E_c                        E [C][d_e]
 *   hl    = mean of the sample's LANG rows of h (zero if it has none)
 *   gamma = W2 gelu(W1 [h | e | hl] + b1) + b2   W1 [Hr][2d+d_e], b1 [Hr],
 *                                                W2 [G][Hr], b2 [G]
 *   gelu is the exact form x * Phi(x).
 * ROLESUB_ROUTER_ADDITIVE (Eq. routingscore with linear heads):
 *   gamma = W_tok h + b_tok + alpha_role W_role a + alpha_lang (W_lang hl + b_lang)
 *   W_tok [G][d], b_tok [G], W_role [G][C], W_lang [G][d], b_lang [G];
 *   a as above (W_r, b_r). */
enum { ROLESUB_ROUTER_MLP2 = 0, ROLESUB_ROUTER_ADDITIVE = 1 };
typedef struct rolesub_router {
  int32_t kind;
  int32_t C, d_e, Hr;
  float alpha_role, alpha_lang;
  const void *W_r, *b_r;
  const void *E, *W1, *b1, *W2, *b2;                  /* MLP2     */
  const void *W_tok, *b_tok, *W_role, *W_lang, *b_lang; /* ADDITIVE */
} rolesub_router;

const char* rolesub_status_str(rolesub_status s);
const char* rolesub_last_error(void);
/* Library version as major*10000 + minor*100 + patch. */
int32_t rolesub_version(void);

/* ---------------------------------------------------------------------------
 * rolesub_rotate_values: value into the orthogonal routing space (Sec. 3.2).
 *   z[b,t,h,j] = sum_k R[h,k,j] * v[b,t,h,k]      (z = R_h^T v)
 * v, z: [B,T,H,dh]; R: [H,dh,dh] (R[h] is R_h, orthonormal by contract, not
 * checked). z must not overlap v. dims->G and dims->d are not used.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_rotate_values(const rolesub_dims* dims, rolesub_dtype dtype,
                                     const void* v, const void* R, void* z, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_route: routing scores and group selection (Eq. latentrole,
 * Eq. routingscore, Sec. 3.4 Top-K_i, Sec. 3.5 budgets).
 *   h          [B,T,d] hidden states (dtype)
 *   token_type [B,T]   uint8, ROLESUB_VIS..ROLESUB_ACT
 *   scores_in  [B,T,G] f32 or NULL. Non-NULL: the router is skipped and the
 *              selection runs on these scores (router may then be NULL and h
 *              is not read).
 *   scores_out [B,T,G] f32 or NULL: the scores the selection used.
 *   mask       [B,T]   uint32: bit s set = group s kept.
 *   idx        [B,T,G] uint8 or NULL: kept group ids ascending, then 0xFF.
 *   count      [B,T]   uint8 or NULL: K_i actually kept.
 *   workspace  device scratch of at least rolesub_route_workspace_size()
 *              bytes (may be NULL if that size is 0). Nothing in it needs
 *              clearing; calls sharing one workspace must not overlap.
 * The environment variable ROLESUB_SK_POLLS (0..1000, default 32), read at
 * each call, bounds how long the first workgroup of a split-K router tile
 * waits for the second to share the tile's epilogue; the outputs are the
 * same bits for every value.
 * ------------------------------------------------------------------------ */
size_t rolesub_route_workspace_size(const rolesub_dims* dims, const rolesub_router* router);
rolesub_status rolesub_route(const rolesub_dims* dims, rolesub_dtype dtype,
                             const rolesub_router* router, const rolesub_budget* budget,
                             const void* h, const uint8_t* token_type, const float* scores_in,
                             float* scores_out, uint32_t* mask, uint8_t* idx, uint8_t* count,
                             void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_route_noalloc: rolesub_route without a workspace argument, for
 * callers that cannot allocate device memory (code under stream capture,
 * serving loops that forbid allocation). Same arguments as rolesub_route and
 * the same results, bit for bit (the bf16 MLP2 router runs as its single
 * kernel here, which sums the same terms in the same order as the split-K
 * form rolesub_route uses); the route workspace is a file-scope device array of
 * ROLESUB_ROUTE_NOALLOC_MAX_BYTES that each device holds until the process
 * ends (its address is looked up once per device, with that device current).
 * Nothing is allocated or freed, by the library or any routine it calls.
 *   - Calls whose route workspace exceeds the maximum return
 *     ROLESUB_ERR_UNSUPPORTED before anything is enqueued (with d = 4096 and
 *     Hr = 128: more than 334 samples). That workspace is
 *     rolesub_route_workspace_size() less the split-K partial products and
 *     tile counters, which the single kernel does not use.
 *   - stream must belong to the current device (else ROLESUB_ERR_INVALID_ARG).
 *   - Every call on one device shares that device's array and overwrites it
 *     (every byte the kernels read is written earlier in the same call, so
 *     nothing needs clearing): calls that may overlap on one device, e.g. on
 *     two streams without ordering between them, race and must not be issued.
 *   - With scores_in the array is not used.
 * ------------------------------------------------------------------------ */
#define ROLESUB_ROUTE_NOALLOC_MAX_BYTES (8u << 20)
rolesub_status rolesub_route_noalloc(const rolesub_dims* dims, rolesub_dtype dtype,
                                     const rolesub_router* router, const rolesub_budget* budget,
                                     const void* h, const uint8_t* token_type, const float* scores_in,
                                     float* scores_out, uint32_t* mask, uint8_t* idx, uint8_t* count,
                                     void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_pack_kv: the compact group-indexed value cache, i.e. the kept
 * groups of z~ = M z (Sec. 3.2).
 *   offsets[b,i] = sum_{j<i} popcount(mask[b,j] & (2^G-1)); offsets[b,T] = total
 *   Vp[b,h,offsets[b,i]+r,:] = z[b,i,h, g_r*ds : (g_r+1)*ds]
 * where g_r is the r-th set bit of mask[b,i] in ascending order.
 *   z       [B,T,H,dh] (dtype), mask [B,T] uint32 (bits >= G ignored)
 *   offsets [B,T+1] int32 (written)
 *   Vp      [B,H,cap_groups,ds] (dtype, written; slots past offsets[b,T]
 *           are not touched)
 * Capacity: if budget and type_counts (host array [4], tokens of each type per
 * sample) are both non-NULL, the call fails with ROLESUB_ERR_CAPACITY unless
 * cap_groups >= sum_t type_counts[t]*min(k_by_type[t],G) (TOPK) or
 * T*min(kmax,G) (THRESHOLD). Independently the kernel never writes a slot
 * >= cap_groups; offsets still count every kept group, so offsets[b,T] >
 * cap_groups reveals a mask that exceeded the capacity.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_pack_kv(const rolesub_dims* dims, rolesub_dtype dtype,
                               const rolesub_budget* budget, const int32_t* type_counts,
                               const void* z, const uint32_t* mask, int32_t* offsets, void* Vp,
                               int64_t cap_groups, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_rotate_pack: rolesub_rotate_values followed by rolesub_pack_kv in
 * one pass (Sec. 3.2: z = R^T v, then the kept groups of M z), without
 * materialising z. Arguments, layouts, capacity rules and outputs (offsets,
 * Vp) are those of the two calls: v and R as for rolesub_rotate_values; mask,
 * offsets, Vp, cap_groups, budget and type_counts as for rolesub_pack_kv.
 * Vp holds the same bits the two calls would produce.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_rotate_pack(const rolesub_dims* dims, rolesub_dtype dtype,
                                   const rolesub_budget* budget, const int32_t* type_counts,
                                   const void* v, const void* R, const uint32_t* mask,
                                   int32_t* offsets, void* Vp, int64_t cap_groups, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_attend: attention with full queries and keys over the routed
 * values (Sec. 3: queries and keys unchanged; Sec. 3.2: v~ = R M R^T v).
 *   s[q,i] = scale * <q_q, k_i> over all T tokens (no causal mask)
 *   P      = softmax_i(s)
 *   u_q    = sum_i P[q,i] * (M_i z_i)      accumulated from the packed groups
 *   out_q  = R_h u_q
 *   q   [B,Tq,H,dh], k [B,T,H,dh] (dtype); mask [B,T]; offsets [B,T+1] and
 *   Vp [B,H,cap_groups,ds] as written by rolesub_pack_kv; R [H,dh,dh].
 *   scale: 0 means 1/sqrt(dh).
 *   out [B,Tq,H,dh] in out_dtype (f32 or the call's dtype).
 * Packed slots >= cap_groups read as zero. workspace: at least
 * rolesub_attend_workspace_size() bytes (0 for the current kernels).
 * ------------------------------------------------------------------------ */
size_t rolesub_attend_workspace_size(const rolesub_dims* dims, int32_t Tq);
rolesub_status rolesub_attend(const rolesub_dims* dims, rolesub_dtype dtype, int32_t Tq,
                              const void* q, const void* k, const uint32_t* mask,
                              const int32_t* offsets, const void* Vp, int64_t cap_groups,
                              const void* R, float scale, void* out, rolesub_dtype out_dtype,
                              void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_attend_causal: prefix self-attention over the routed values. In the
 * single forward pass the T prefix tokens are also queries (Sec. 3: queries
 * and keys unchanged; Sec. 3.2: routed values); query t sees keys 0..t:
 *   s[t,i] = scale * <q_t, k_i> for i <= t
 *   P      = softmax_{i <= t}(s)
 *   u_t    = sum_{i <= t} P[t,i] * (M_i z_i)
 *   out_t  = R_h u_t
 *   q, k [B,T,H,dh] (dtype; q holds the prefix tokens' queries); mask,
 *   offsets, Vp, cap_groups, R, scale, workspace and errors as for
 *   rolesub_attend; out [B,T,H,dh] in out_dtype (f32 or the call's dtype).
 * T = 0 or B = 0 does nothing and returns OK.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_attend_causal(const rolesub_dims* dims, rolesub_dtype dtype, const void* q,
                                     const void* k, const uint32_t* mask, const int32_t* offsets,
                                     const void* Vp, int64_t cap_groups, const void* R, float scale,
                                     void* out, rolesub_dtype out_dtype, void* workspace,
                                     size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_retain_tokens: token-level retention ahead of the routed path
 * (Sec. 3.1: the ceil(r_m |I_m|) highest-scoring tokens of a type are kept;
 * Sec. 4.1: the visual budget is divided evenly between the camera views).
 * Each sample's N tokens form n_seg segments of consecutive tokens (e.g. one
 * per view); segment s has seg_len[s] tokens, of which the seg_keep[s] with
 * the highest scores are kept: a larger score first, equal scores (-0 equal
 * to +0) by lower index, NaN after every number.
 *   scores   [B,N] f32 (device)
 *   keep_idx [B,K] int32 (device), K = sum(seg_keep): the kept token indices,
 *            ascending within each segment, segments in order
 *   seg_len, seg_keep: n_seg host integers; sum(seg_len) == N;
 *            1 <= n_seg <= 16, seg_len[s] <= 8192
 * B = 0 or K = 0 does nothing and returns OK.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_retain_tokens(int32_t B, int32_t N, int32_t n_seg, const int32_t* seg_len,
                                     const int32_t* seg_keep, const float* scores, int32_t* keep_idx,
                                     void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_gather_tokens: rows of the retained tokens (the compact prefix the
 * routed path runs on): dst[b,j,:] = src[b, keep_idx[b,j], :].
 *   src [B,N,row_bytes], dst [B,K,row_bytes] (device, any element type);
 *   keep_idx [B,K] int32 (device); row_bytes a multiple of 4 (16 is fastest).
 * An index outside [0, N) gives a zero row. One sample's rows must be
 * below 2 GiB. B, K or row_bytes = 0 does nothing and returns OK.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_gather_tokens(int32_t B, int32_t N, int32_t K, int64_t row_bytes, const int32_t* keep_idx,
                                     const void* src, void* dst, void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_attend_values: attention with unchanged queries and keys (Sec. 3)
 * over plain per-head values, for the full-width routing space whose routed
 * values rolesub_full_values rebuilds:
 *   out[b,q,h,:] = sum_t softmax_t(scale * q[b,q,h,:] . k[b,t,h,:]) V[b,h,t,:]
 * q [B,Tq,H,dh], k [B,T,H,dh], V [B,H,T,dh] (head-major), out [B,Tq,H,dh];
 * bf16 inputs, dh 64 or 128, out_dtype f32 or bf16; scale 0 means 1/sqrt(dh).
 * dims->G and dims->d are not used. B = 0 or Tq = 0 does nothing.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_attend_values(const rolesub_dims* dims, rolesub_dtype dtype, int32_t Tq, const void* q,
                                     const void* k, const void* V, float scale, void* out, rolesub_dtype out_dtype,
                                     void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_allocate_groups: role-driven within-type budget allocation
 * (Sec. 3.5, the allocator B), optionally followed by the Top-K_i group
 * selection (Sec. 3.4) with the allocated budgets.
 * Within each sample and token type m (ROLESUB_VIS..ROLESUB_ACT) the
 * B_m = K_m * n_m groups of the type's n_m tokens are distributed by the
 * tokens' role-derived priorities, with 0 <= K_i <= G and sum K_i = B_m:
 *   weights    w_i = floor(min(max(p_i, 0), 256) * 2^16), NaN as 0 (exact);
 *   shares     B_m * w_i / sum w; a token whose share exceeds G gets G and
 *              the rest of the budget is shared again among the others;
 *              all-zero weights count as equal;
 *   rounding   the floors of the shares, then one more group to each of the
 *              largest remainders (equal remainders: lower token index).
 * K_m = 0 gives 0 and K_m = G gives G to every token of the type; a token of
 * any other type value gets G.
 *   k_by_type  4 host integers K_m, 0 <= K_m <= G
 *   priority   [B,T] f32 (device), token_type [B,T] uint8 (device)
 *   scores     [B,T,G] f32 (device) or NULL. Non-NULL: each token keeps its
 *              K_i highest-scoring groups, order as rolesub_route, written
 *              to mask (required), idx and count (optional, as
 *              rolesub_route). NULL: mask, idx and count must be NULL.
 *   k_out      [B,T] uint8 (device) or NULL: the K_i; required when scores
 *              is NULL.
 * 1 <= G <= 32, T <= 4096. B*T = 0 does nothing and returns OK.
 * ------------------------------------------------------------------------ */
rolesub_status rolesub_allocate_groups(int32_t B, int32_t T, int32_t G, const int32_t* k_by_type,
                                       const float* priority, const uint8_t* token_type, const float* scores,
                                       uint8_t* k_out, uint32_t* mask, uint8_t* idx, uint8_t* count,
                                       void* stream);

/* ---------------------------------------------------------------------------
 * rolesub_route_allocate: routing with role-driven budgets (Eq. latentrole,
 * Eq. routingscore, Sec. 3.5 allocator, Sec. 3.4 Top-K_i) in one call:
 * the router's scores gamma and the token priority p_i = w_pri^T a_i from
 * the latent role representation a_i, then rolesub_allocate_groups on them.
 *   router, h, token_type, dims  as rolesub_route
 *   w_pri        [C] priority weight per latent role (call dtype, device)
 *   k_by_type    4 host integers K_m, 0 <= K_m <= G
 *   priority_out [B,T] f32 or NULL, scores_out [B,T,G] f32 or NULL
 *   k_out [B,T] uint8 or NULL; mask [B,T] uint32 (required); idx, count as
 *   rolesub_route
 *   workspace    at least rolesub_route_allocate_workspace_size() bytes
 *                (device scratch, always required)
 * T <= 4096. The kept-group total per sample equals that of the fixed
 * budgets, so pack capacities sized for k_by_type hold.
 * ------------------------------------------------------------------------ */
size_t rolesub_route_allocate_workspace_size(const rolesub_dims* dims, const rolesub_router* router);
rolesub_status rolesub_route_allocate(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_router* router,
                                      const void* w_pri, const int32_t* k_by_type, const void* h,
                                      const uint8_t* token_type, float* priority_out, float* scores_out,
                                      uint8_t* k_out, uint32_t* mask, uint8_t* idx, uint8_t* count,
                                      void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Full-width routing space (Sec. 3.2 with a single R over the whole value
 * vector, d_v = H*dh; Sec. 4.1 uses d_v = 4096, S = 16 groups of 256).
 * dims->G is S; group s is rotated dims [s*ds, (s+1)*ds), ds = d_v/S. One
 * mask per token (bit s = group s kept), as rolesub_route writes with G = S.
 * Cache: offsets [B,T+1] as rolesub_pack_kv; Vp [B,cap_groups,ds] (sample-
 * major, one slot = one group of ds values). A token that keeps all S groups
 * has R M R^T v = v and is stored in value space: its S consecutive slots
 * hold v itself. Any other token stores its kept groups of z = R^T v in
 * ascending group order. Requirements: bf16; dh = 128; 1 <= S <= 32 with ds a
 * multiple of 128; B <= 1024, T <= 4096; values, cache and R each below 2 GiB.
 * workspace: at least rolesub_full_workspace_size(B, T, S) bytes of device
 * scratch (per-sample routed-token lists), not kept between calls.
 * ------------------------------------------------------------------------ */
size_t rolesub_full_workspace_size(int32_t B, int32_t T, int32_t S);

/* Rt[j][k] = R[k][j] for an n x n bf16 matrix (n a multiple of 64): the
 * operand layout rolesub_full_rotate_pack takes. R is frozen per layer, so
 * this runs once per layer, not per call. */
rolesub_status rolesub_full_transpose(int32_t n, rolesub_dtype dtype, const void* R, void* Rt, void* stream);

/* z = R^T v for the routed tokens, their kept groups and the value-space
 * tokens into the cache (Sec. 3.2).
 *   Rt   [d_v, d_v] = R^T (rolesub_full_transpose of R; R[k][j] is value
 *        coordinate k of rotated coordinate j)
 *   v    [B,T,H,dh] (= [B,T,d_v]); mask [B,T] uint32
 *   offsets [B,T+1] int32 written; Vp [B,cap_groups,ds] written (slots at or
 *        past cap_groups are never written; offsets still count them)
 *   budget, type_counts: optional capacity check as rolesub_pack_kv. */
rolesub_status rolesub_full_rotate_pack(const rolesub_dims* dims, rolesub_dtype dtype, const void* Rt,
                                        const void* v, const uint32_t* mask, int32_t* offsets, void* Vp,
                                        int64_t cap_groups, const rolesub_budget* budget,
                                        const int32_t* type_counts, void* workspace, size_t ws_bytes,
                                        void* stream);

/* Routed values from the cache, head-major for attention (Sec. 3.2):
 *   Vh[b,h,t,:] = (R z~_t)[h*dh : (h+1)*dh] for routed tokens (dropped groups
 *   are zero, so a token keeping none gets 0), and v_t's slice for tokens
 *   stored in value space.
 *   R [d_v, d_v]; mask, offsets, Vp as written by rolesub_full_rotate_pack;
 *   Vh [B,H,T,dh] written; rolesub_attend_values then gives the paper's
 *   attention over these values. */
rolesub_status rolesub_full_values(const rolesub_dims* dims, rolesub_dtype dtype, const void* R,
                                   const uint32_t* mask, const int32_t* offsets, const void* Vp, int64_t cap_groups,
                                   void* Vh, void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ROLESUB_H */
