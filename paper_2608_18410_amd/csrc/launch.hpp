// Internal launcher interface between the C-ABI layer and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rolesub {

struct RouteParams {
  int B, T, d, G, C, d_e, Hr, kind;
  float alpha_role, alpha_lang;
  const void* h;
  const uint8_t* types;
  const void *W_r, *b_r, *E, *W1, *b1, *W2, *b2;
  const void *W_tok, *b_tok, *W_role, *W_lang, *b_lang;
  float* cb;  // [B][Hr or G] per-sample language term (workspace)
  float* F;   // [Hr or G][C] folded role term (workspace)
  float* hbar;  // [B][d] pooled language state (workspace)
  float* pcb;   // [ncb][B][Hr] partial language terms per column block (bf16 MLP2; workspace)
  float* rpart;  // split-K router: both halves' partial products per 96-token tile, or null (workspace)
  int* rcnt;     // split-K router: finished halves per tile, zeroed by the pool kernel (workspace)
  int sk_polls;  // split-K router: polls the first half of a tile makes for the second (0: never shares)
  int mode;
  int k_by_type[4];
  float tau;
  int kmin, kmax;
  const float* scores_in;
  float* scores_out;
  const void* w_pri;  // [C] role priority weights (call dtype), with priority
  float* priority;    // [B][T] p = w^T a, or null
  uint32_t* mask;     // null: scores (and priority) only, no selection
  uint8_t* idx;
  uint8_t* count;
};

// Sizes of the route workspace pieces (floats).
inline size_t route_cb_floats(int B, int Hr, int G, int kind) {
  return static_cast<size_t>(B) * (kind == 0 ? Hr : G);
}
inline size_t route_F_floats(int Hr, int G, int C, int kind) {
  return static_cast<size_t>(kind == 0 ? Hr : G) * C;
}
inline size_t route_hbar_floats(int B, int d) { return static_cast<size_t>(B) * d; }
// column blocks of 256 (the smallest block the pool kernel uses, f32) bound
// the number of partial language terms for any dtype
inline size_t route_pcb_floats(int B, int d, int Hr, int kind) {
  return kind == 0 ? static_cast<size_t>((d + 255) / 256) * B * Hr : 0;
}

// Split-K form of the bf16 MLP2 router (Hr = 128): 96-token tiles, each
// computed by two workgroups over half of the hidden size.
constexpr int kRouteSkTok = 96;
// shortest prefix the split form takes: a tile then touches at most three samples
constexpr int kRouteSkMinT = kRouteSkTok / 2;
inline size_t route_sk_tiles(int B, int T) { return (static_cast<size_t>(B) * T + kRouteSkTok - 1) / kRouteSkTok; }
// floats of both halves' partials (144 products per token) and ints of the tile counters
inline size_t route_sk_part_floats(int B, int T, int Hr, int kind) {
  return kind == 0 && Hr == 128 ? route_sk_tiles(B, T) * 2 * kRouteSkTok * 144 : 0;
}
inline size_t route_sk_cnt_ints(int B, int T, int Hr, int kind) {
  return kind == 0 && Hr == 128 ? route_sk_tiles(B, T) : 0;
}

hipError_t launch_route(const RouteParams& p, bool bf16, hipStream_t s);
// LDS bytes the generic (one token per workgroup) router needs.
size_t route_generic_shm(int d, int G, int C, int Hr, int kind);
hipError_t launch_select(const RouteParams& p, hipStream_t s);

// Role-driven within-type group allocation (and optional selection).
constexpr int kAllocMaxT = 4096;  // tokens per sample
struct AllocParams {
  int B, T, G;
  int k_by_type[4];
  const float* priority;   // [B][T]
  const uint8_t* types;    // [B][T]
  const float* scores;     // [B][T][G] or null (no selection)
  uint8_t* k_out;          // [B][T] or null
  uint32_t* mask;          // [B][T], with scores
  uint8_t* idx;            // [B][T][G] or null
  uint8_t* count;          // [B][T] or null
};
hipError_t launch_allocate(const AllocParams& p, hipStream_t s);

// Full-width routing space: one R over d_v = H*dh value dims, S groups of ds.
constexpr int kFullMaxT = 4096, kFullMaxB = 1024;
struct FullParams {
  int B, T, H, dv, S, ds;
  int64_t cap;
  const uint32_t* mask;  // [B][T]
  int32_t* offsets;      // [B][T+1]: written by the rotate step, read by the values step
  int32_t* counts;       // [B] routed tokens per sample (workspace)
  int32_t* rlist;        // [B][T] routed token indices (workspace)
  int32_t* counts_g;     // [B][S] routed tokens keeping group g (workspace)
  int32_t* starts_g;     // [B][S] start of group g's list in pairs[b] (workspace)
  int32_t* pairs;        // [B][T*S] per sample: the routed tokens keeping group 0, then 1, ... (workspace)
  const void* v;         // [B][T][dv] (rotate)
  const void* Rm;        // [dv][dv]: R^T (rotate) or R (values)
  void* Vp;              // [B][cap][ds] cache: written (rotate) or read (values)
  void* Vh;              // [B][H][T][dh] routed values (values)
};
// mode 0: rotate + pack; mode 1: values from the cache
hipError_t launch_full(const FullParams& p, int mode, hipStream_t s);
hipError_t launch_transpose(const void* R, void* Rt, int n, hipStream_t s);

struct RotateParams {
  int ntok, T, H, G, tok_per_wg;
  const void* v;
  const void* R;
  void* z;                  // rotate only
  const uint32_t* mask;     // fused rotate + pack
  int32_t* offsets;         // written by the matrix-core kernel (head 0's workgroups) unless off_ready
  int off_ready;            // offsets already hold the scan (long prefixes)
  int dyn_tiles;            // all workgroups resident at once: tiles handed out on demand
  void* Vp;
  int64_t cap;
};
hipError_t launch_rotate(bool bf16, int ntok, int H, int dh, const void* v, const void* R, void* z,
                         hipStream_t s);
// Fused rotation + pack; also writes the offsets (the exclusive scan of the
// kept counts per sample).
hipError_t launch_rotate_pack(bool bf16, int B, int T, int H, int dh, int G, const void* v, const void* R,
                              const uint32_t* mask, int32_t* offsets, void* Vp, int64_t cap,
                              hipStream_t s);
hipError_t launch_pack_offsets(int B, int T, int G, const uint32_t* mask, int32_t* offsets, hipStream_t s);

hipError_t launch_pack(bool bf16, int B, int T, int H, int dh, int G, const void* z,
                       const uint32_t* mask, int32_t* offsets, void* Vp, int64_t cap,
                       hipStream_t s);

struct AttendParams {
  int B, T, H, dh, G, Tq;
  const void *q, *k;
  const uint32_t* mask;
  const int32_t* offsets;
  const void* Vp;
  int64_t cap;
  const void* R;
  float scale;
  void* out;
  int out_f32;
  int causal;  // prefix self-attention: Tq == T and query t sees keys 0..t
  int dense;   // plain per-head values Vp = [B][H][T][dh]: no masks, offsets or rotation
};
hipError_t launch_attend(const AttendParams& p, bool bf16, hipStream_t s);

// Token retention (Sec. 3.1): per sample, per segment of consecutive tokens,
// the seg_keep highest scores. Segments are at most kRetainMaxSeg tokens.
constexpr int kRetainMaxSegments = 16, kRetainMaxSeg = 8192;
struct RetainParams {
  int B, N, K, n_seg;
  int seg_start[kRetainMaxSegments], seg_len[kRetainMaxSegments], seg_keep[kRetainMaxSegments],
      seg_out[kRetainMaxSegments];
  const float* scores;  // [B][N]
  int32_t* keep_idx;    // [B][K]
};
hipError_t launch_retain(const RetainParams& p, hipStream_t s);

struct GatherParams {
  int B, N, K;
  int64_t row_bytes;
  const int32_t* idx;  // [B][K]
  const void* src;     // [B][N][row_bytes]
  void* dst;           // [B][K][row_bytes]
};
hipError_t launch_gather_rows(const GatherParams& p, hipStream_t s);

}  // namespace rolesub
