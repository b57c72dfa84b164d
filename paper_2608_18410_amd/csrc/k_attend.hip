// Attention with unchanged queries and keys over the routed values
// (Sec. 3: q, k unchanged; Sec. 3.2: v~ = R M R^T v).
//
//   s[q,i] = scale <q, k_i>,  P = softmax_i(s) over all tokens,
//   u_q    = sum_i P[q,i] (M_i z_i)      -- only the kept groups are read
//   out_q  = R_h u_q                     -- once per query, after the sum
//
// Back-rotation is linear, so applying R_h after the weighted sum equals
// summing the back-rotated routed values v~_i.
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

__device__ __forceinline__ uint32_t group_mask(int G) { return G >= 32 ? 0xFFFFFFFFu : ((1u << G) - 1u); }

// Scheduling of N LDS fragment reads feeding N MFMAs: the reads run two MFMAs
// ahead (left to itself the compiler reuses one register set and waits on
// every read).
template <int N>
__device__ __forceinline__ void sched_reads_ahead() {
  constexpr int kDsRead = 0x100, kMfma = 0x008;
  __builtin_amdgcn_sched_group_barrier(kDsRead, N < 2 ? N : 2, 0);
#pragma unroll
  for (int i = 0; i + 2 < N; ++i) {
    __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(kMfma, N < 2 ? N : 2, 0);
}

// ---------------------------------------------------------------------------
// bf16 matrix-core kernel. One workgroup = one (sample, head) and up to 64
// queries; wave w owns queries 16w..16w+15. R_h is brought into LDS by DMA at
// the start. KV tokens stream in tiles of TK (32 at head dim 128, 64 at head
// dim 64):
//   * K tile (TK x DH) -> LDS, shared by the four waves;
//   * the tile's packed groups -> a zero-filled, transposed LDS tile
//     Zt[row][token] (token pairs packed in one dword), its rows the dims in
//     the permuted order that store_v describes;
//   * S^T = K Q^T on MFMA (queries are the B operand held in registers), so
//     each lane owns one query column and TK/4 token rows;
//   * online softmax per query: in-lane, then 2 cross-lane steps, against a
//     reference that lags the running maximum by at most kSlack;
//   * O^T += Z~^T P^T on MFMA. The lane's own softmax values form the P^T
//     fragment directly once the A fragment lists its tokens in the same
//     order (tokens 4q..4q+3 and 16+4q..16+4q+3 of each 32 tokens).
// Loads are software-pipelined two tiles deep: while tile i is computed from
// LDS, the K rows and packed groups of tiles i+1 and i+2 are in flight into
// registers, and the masks and cache offsets that address tile i+2's packed
// groups arrived with tile i's operands.
// After the last tile, O^T = R_h U^T is one more MFMA chain (U in bf16, R_h
// fragments from LDS), and each wave stages its 16 output rows in LDS and
// writes them as whole 16-byte units.
// VM: how the 8-dim chunks of the value tile map to packed groups:
//   kWide  groups of >= 8 dims (one 16-byte load per token and chunk)
//   kDs4   4-dim groups (two 8-byte loads), kDs2  2-dim groups (four 4-byte loads)
//   kDense plain per-head values [B][H][T][dh] (the full-width routing space
//          rebuilds them): token t is slot t, no masks, offsets or R_h, and
//          the output is the normalised accumulator itself
constexpr int kWide = 0, kDs4 = 1, kDs2 = 2, kDense = 3;

template <bool B>
struct Flag {
  static constexpr bool value = B;
};

// Three waves per SIMD (three workgroups per CU): the register budget is
// capped at 168 so that occupancy, not just the pipeline, hides latency.
template <int DH, int VM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void k_attend_bf16(AttendParams p) {
  // 32-token tiles at DH = 128 (shorter per-tile chains, 140 registers); 64 at
  // DH = 64 so that every thread has a value item per tile
  constexpr int TK = DH == 128 ? 32 : 64, MT = DH / 16, KS = DH / 32, KLD = DH + 8, ZLD = TK / 2 + 2;
  constexpr int NM2 = TK / 16, NHF = TK / 32;  // 16-token score blocks, 32-token P.V steps
  constexpr int NKP = TK * DH / 8 / 256;          // 16-byte K pieces per thread per tile
  constexpr int NVI = (TK / 2) * (DH / 8) / 256;  // (token pair, 8-dim chunk) items per thread
  // R_h has its own LDS region, filled by buffer->LDS DMA at the start so its
  // load overlaps the key loop; rows are unpadded with 16-byte chunks
  // XOR-swizzled by row. The Z~^T tile's row stride of TK/2 + 2 dwords keeps
  // both its 4-byte writes and its 8-byte fragment reads free of bank
  // conflicts (a stride of TK/2 + 4 made both two-way). The output staging
  // reuses R_h and the tile buffers after the back-rotation. About 51 KB of
  // LDS at DH = 128: three workgroups per CU.
  constexpr int RBY = DH * 2, RCH = RBY / 16;  // bytes and 16-byte chunks per R_h row
  constexpr int RB = DH * RBY, KB = TK * KLD * 2, ZB = DH * ZLD * 4, SB = 4 * 16 * DH * 4;
  constexpr int SMEM = RB + KB + ZB > SB ? RB + KB + ZB : SB;
  static_assert(NKP >= 1 && NVI >= 1 && NHF >= 1, "tile shape");
  static_assert(RB % (4 * 1024) == 0, "R_h splits into whole 1 KB DMA blocks per wave");
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  char* Rs = smem;
  bf16* Ks = reinterpret_cast<bf16*>(smem + RB);
  uint32_t* Zt = reinterpret_cast<uint32_t*>(smem + RB + KB);
  __shared__ uint32_t s_mask[2][TK];
  __shared__ int32_t s_off[2][TK];
  int h, b;
  // 1D grid of (sample, head) items x query blocks. When B*H is a multiple of
  // 8 the query blocks of one item are consecutive workgroups of one XCD, so
  // the blocks after the first find the item's keys and values in that L2.
  int qb;
  {
    const int nqb = (p.Tq + 63) / 64, lin = blockIdx.x;
    int item;
    if ((p.B * p.H) % 8 == 0) {
      const int xcd = lin & 7, slot = lin >> 3;
      item = (slot / nqb) * 8 + xcd;
      qb = slot % nqb;
    } else {
      item = lin / nqb;
      qb = lin % nqb;
    }
    xcd_split(item, p.H, h, b);
  }
  constexpr bool DENSE = VM == kDense;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int T = p.T, H = p.H, G = DENSE ? 1 : p.G, ds = DH / G;
  const uint32_t gm = group_mask(G);
  const int qq = qb * 64 + 16 * w + l16;
  const int q_first = qb * 64 + 16 * __builtin_amdgcn_readfirstlane(w);  // this wave's first query
  const bool qvalid = qq < p.Tq;

  // R_h: wave w brings 1 KB blocks w*NRD .. w*NRD+NRD-1; lane i of a block
  // lands at byte 16i, which holds global chunk (16i % RBY)/16 ^ (row % RCH)
  if constexpr (!DENSE) {
    constexpr int NRD = RB / 1024 / 4;
    const rsrc_t r_R = make_rsrc(static_cast<const bf16*>(p.R) + static_cast<size_t>(h) * DH * DH, RB);
    const uint32_t rbase = lds_addr(Rs);
    const int wu = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
    for (int u = 0; u < NRD; ++u) {
      const int j = wu * NRD + u;
      const int byte = 1024 * j + 16 * lane, row = byte / RBY, cp = (byte % RBY) / 16;
      dma16(r_R, static_cast<uint32_t>(row * RBY + 16 * (cp ^ (row % RCH))), rbase + 1024u * j);
    }
  }
  bf16x8 qf[KS];
  {
    const rsrc_t r_q = make_rsrc(static_cast<const bf16*>(p.q) + (static_cast<size_t>(b) * p.Tq * H + h) * DH,
                                 clamp_bytes((static_cast<size_t>(p.Tq - 1) * H + 1) * DH * 2));
    const uint32_t qo = static_cast<uint32_t>(qq) * H * DH * 2 + 16u * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = __builtin_bit_cast(bf16x8, bload16(r_q, qvalid ? qo + 64u * ks : kOOB));
  }
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  // softmax in base 2 with a positive factor: a negative scale is applied by
  // negating the queries (exact in bf16), once they have arrived
  const float sl2 = fabsf(p.scale) * 1.4426950408889634f;
  constexpr float kSlack = 8.f;  // the softmax reference lags the running maximum by at most this (log2)

  // Buffer resources: a masked or out-of-range element loads as zero with no
  // memory access, so every load below is unconditional.
  const rsrc_t r_off = make_rsrc(p.offsets + static_cast<size_t>(b) * (T + 1), (T + 1) * 4u);
  const rsrc_t r_mask = make_rsrc(p.mask + static_cast<size_t>(b) * T, T * 4u);
  const rsrc_t r_v = make_rsrc(static_cast<const bf16*>(p.Vp) + (static_cast<size_t>(b) * H + h) * p.cap * ds,
                               clamp_bytes(static_cast<size_t>(p.cap) * ds * 2));
  const uint32_t kstride = static_cast<uint32_t>(H) * DH * 2;  // bytes between tokens
  const rsrc_t r_k = make_rsrc(static_cast<const bf16*>(p.k) + (static_cast<size_t>(b) * T * H + h) * DH,
                               clamp_bytes(static_cast<size_t>(T - 1) * kstride + DH * 2));

  // mask/offset of token t0+tid of a tile (threads 0..TK-1)
  auto load_meta = [&](int t0, uint32_t& m, int32_t& o) {
    const int t = t0 + tid;
    const bool ok = tid < TK && t < T;
    if constexpr (DENSE) {
      m = ok ? 1u : 0u;
      o = t;
    } else {
      m = bload4(r_mask, oob_unless(ok, 4u * t));  // masked to G bits when stored (no wait here)
      o = static_cast<int32_t>(bload4(r_off, oob_unless(ok, 4u * t)));
    }
  };
  // two register sets (A, B) for tile operands in flight
  u32x4 kA[NKP], kB[NKP];
  auto load_k = [&](u32x4 (&kreg)[NKP], int t0) {
#pragma unroll
    for (int r = 0; r < NKP; ++r) {
      const int pc = tid + 256 * r;
      const int row = pc / (DH / 8), c8 = pc % (DH / 8);
      const int t = t0 + row;
      kreg[r] = bload16(r_k, oob_unless(t < T, t * kstride + 16u * c8));
    }
  };
  // Item it = (token pair pp, 8-dim chunk cc). Bits 0 and 1 of cc are swapped
  // against the lane order so that the two chunks written by one 32-lane
  // half-wave land 8 tile rows apart (distinct banks, see store_tile).
  auto item_of = [](int it, int& pp, int& cc) {
    pp = it % (TK / 2);
    const int gi = it / (TK / 2);
    cc = (gi & ~3) | ((gi & 1) << 1) | ((gi >> 1) & 1);
  };
  // packed groups of 2 tokens x 8 dims for each item, addressed through the LDS masks/offsets
  u32x4 vA[NVI][2], vB[NVI][2];
  const int64_t cap = p.cap;
  // slots are < 2^31 (the cache per (sample, head) is < 2 GiB); the select is
  // pinned so that no load ends up behind a branch
  const int cap32 = static_cast<int>(cap);
  auto slot_off = [&](uint32_t m, int o, int g, bool tok_ok, int elem) -> uint32_t {
    const int sl = o + __popc(m & ((1u << g) - 1u));
    const bool ok = tok_ok & (((m >> g) & 1u) != 0u) & (sl < cap32);
    return oob_unless(ok, static_cast<uint32_t>((sl * ds + elem) * 2));
  };
  auto load_v = [&](u32x4 (&vreg)[NVI][2], int t0, int slot) {
#pragma unroll
    for (int r = 0; r < NVI; ++r) {
      int pp, cc;
      item_of(tid + 256 * r, pp, cc);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int tl = 2 * pp + e;
        const bool tok_ok = t0 + tl < T;
        const uint32_t m = s_mask[slot][tl];
        const int o = s_off[slot][tl];
        if constexpr (VM == kWide || DENSE) {
          const int g = (8 * cc) / ds;
          vreg[r][e] = bload16(r_v, slot_off(m, o, g, tok_ok, 8 * cc - g * ds));
        } else if constexpr (VM == kDs4) {
          const u32x2 x0 = bload8(r_v, slot_off(m, o, 2 * cc, tok_ok, 0));
          const u32x2 x1 = bload8(r_v, slot_off(m, o, 2 * cc + 1, tok_ok, 0));
          vreg[r][e] = u32x4{x0[0], x0[1], x1[0], x1[1]};
        } else {
          vreg[r][e] = u32x4{bload4(r_v, slot_off(m, o, 4 * cc, tok_ok, 0)),
                             bload4(r_v, slot_off(m, o, 4 * cc + 1, tok_ok, 0)),
                             bload4(r_v, slot_off(m, o, 4 * cc + 2, tok_ok, 0)),
                             bload4(r_v, slot_off(m, o, 4 * cc + 3, tok_ok, 0))};
        }
      }
    }
  };
  auto store_k = [&](const u32x4 (&kreg)[NKP]) {
#pragma unroll
    for (int r = 0; r < NKP; ++r) {
      const int pc = tid + 256 * r;
      const int row = pc / (DH / 8), c8 = pc % (DH / 8);
      *reinterpret_cast<u32x4*>(Ks + row * KLD + 8 * c8) = kreg[r];
    }
  };
  auto store_v = [&](const u32x4 (&vreg)[NVI][2]) {
#pragma unroll
    for (int r = 0; r < NVI; ++r) {
      int pp, cc;
      item_of(tid + 256 * r, pp, cc);
      // dim 32a + 8b + c sits in tile row 32a + 4b + (c % 4) + 16 (c / 4), so
      // that the P.V accumulator of lane quarter g4 holds dims 32ks + 8g4 ..
      // + 7 for each ks (one 16-byte R_h chunk in the back-rotation)
      uint32_t* zc = Zt + (32 * (cc >> 2) + 4 * (cc & 3)) * ZLD + pp;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = 2 * (j & 1) + 16 * (j >> 1);  // dims 2j, 2j + 1 of the chunk
        zc[row * ZLD] = (vreg[r][0][j] & 0xFFFFu) | (vreg[r][1][j] << 16);
        zc[(row + 1) * ZLD] = (vreg[r][0][j] >> 16) | (vreg[r][1][j] & 0xFFFF0000u);
      }
    }
  };
  auto store_tile = [&](const u32x4 (&kreg)[NKP], const u32x4 (&vreg)[NVI][2]) {
    store_k(kreg);
    store_v(vreg);
  };

  // ---- pipeline: the operands of tiles i+1 and i+2 are in flight while
  // tile i is computed. Tile i+2's packed groups are addressed through its
  // masks and offsets, which were requested together with tile i's operands,
  // so each iteration waits only for what was issued two iterations earlier.
  // Register sets alternate A, B, A, ... (the loop body runs twice per pass;
  // a second half past the last tile computes a fully masked tile).
  // Prologue: tile 0's keys (they need no metadata), the metadata of tiles 0
  // and 1 into LDS, then the rest of tiles 0 and 1 and the metadata of tiles
  // 2 and 3: the loop is entered with the loads of its back edge outstanding,
  // in the same order.
  uint32_t mA, mB;
  int32_t oA, oB;
  load_k(kA, 0);
  {
    uint32_t m0, m1;
    int32_t o0, o1;
    load_meta(0, m0, o0);
    load_meta(TK, m1, o1);
    if (tid < TK) {
      s_mask[0][tid] = m0 & gm;
      s_off[0][tid] = o0;
      s_mask[1][tid] = m1 & gm;
      s_off[1][tid] = o1;
    }
  }
  __syncthreads();
  if (p.scale < 0.f) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, qf[ks]) ^ u32x4{0x80008000u, 0x80008000u,
                                                                                   0x80008000u, 0x80008000u});
  }
  load_v(vA, 0, 0);
  load_meta(2 * TK, mA, oA);
  load_k(kB, TK);
  load_v(vB, TK, 1);
  load_meta(3 * TK, mB, oB);
  // every wave has read slots 0 and 1 (tiles 0 and 1) before the first step
  // overwrites slot 0 with tile 2's metadata
  __syncthreads();

  // SPLIT (the first tile only): its packed groups were requested one
  // metadata round trip after its keys, so the keys go to LDS first and the
  // scores and softmax are computed while the groups are still in flight;
  // the groups are stored (and the next loads into their registers issued)
  // just before P.V, behind one more barrier.
  auto step = [&](auto split, int t0, int slot, u32x4 (&kreg)[NKP], u32x4 (&vreg)[NVI][2], uint32_t& mreg,
                  int32_t& oreg) {
    constexpr bool SPLIT = decltype(split)::value;
    if constexpr (SPLIT) store_k(kreg);
    else store_tile(kreg, vreg);
    if (tid < TK) {  // masks/offsets of tile t0 + 2*TK into this tile's slot
      s_mask[slot][tid] = mreg & gm;
      s_off[slot][tid] = oreg;
    }
    __syncthreads();
    // operands two tiles ahead; past the end every load is out of range (no
    // memory access), so there is no branch here: a branch around the loads
    // makes the compiler wait on every outstanding load at its join
    load_k(kreg, t0 + 2 * TK);
    if constexpr (!SPLIT) load_v(vreg, t0 + 2 * TK, slot);
    load_meta(t0 + 4 * TK, mreg, oreg);

    // ---- S^T = K Q^T (rows: tile tokens 16*m2 + 4*g4 + i; column: this lane's query)
    f32x4 s[NM2];
    {
      // fragment i = (ks, m2) with m2 fastest: the NM2 accumulation chains alternate
      bf16x8 kf[NM2 * KS];
#pragma unroll
      for (int i = 0; i < NM2 * KS; ++i)
        kf[i] = *reinterpret_cast<const bf16x8*>(Ks + (16 * (i % NM2) + l16) * KLD + 32 * (i / NM2) + 8 * g4);
#pragma unroll
      for (int m2 = 0; m2 < NM2; ++m2) s[m2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < NM2 * KS; ++i) s[i % NM2] = mfma_16x16x32(kf[i], qf[i / NM2], s[i % NM2]);
      sched_reads_ahead<NM2 * KS>();
    }
    // ---- online softmax (base 2) with a lazily moved reference: scores are
    // taken relative to m_run, which moves only when a tile's maximum exceeds
    // it by more than kSlack (then acc and l_run are rescaled, for the whole
    // wave at once). Softmax does not depend on the reference, P stays below
    // 2^kSlack, and most tiles skip the rescale. Scores past T (only in the
    // last tile) are masked to -inf.
    float mx = -INFINITY;
    // full tile: inside T and, for prefix self-attention, entirely before this
    // wave's first query
    if (t0 + TK <= T && (!p.causal || t0 + TK - 1 <= q_first)) {
#pragma unroll
      for (int m2 = 0; m2 < NM2; ++m2)
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[m2][i]);
    } else {
#pragma unroll
      for (int m2 = 0; m2 < NM2; ++m2)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 16 * m2 + 4 * g4 + i;
          s[m2][i] = (t < T) & (!p.causal | (t <= qq)) ? s[m2][i] : -INFINITY;
          mx = fmaxf(mx, s[m2][i]);
        }
    }
    mx = max_xor32(max_xor16(mx));
    const float m_cand = fmaxf(m_run, mx * sl2);  // sl2 >= 0
    if (__builtin_amdgcn_ballot_w64(m_cand > m_run + kSlack) != 0) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_cand);  // 0 on the first tile
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] *= alpha;
      l_run *= alpha;
      m_run = m_cand;
    }
    float psum = 0.f;
    bf16x8 pb[NHF];
#pragma unroll
    for (int m2 = 0; m2 < NM2; ++m2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pr = __builtin_amdgcn_exp2f(fmaf(s[m2][i], sl2, -m_run));
        psum += pr;
        pb[m2 >> 1][4 * (m2 & 1) + i] = static_cast<bf16>(pr);
      }
    l_run += psum;
    if constexpr (SPLIT) {
      store_v(vreg);
      load_v(vreg, t0 + 2 * TK, slot);
      __syncthreads();
    }
    // ---- O^T += Z~^T P^T, one MFMA per 32 tokens
    {
      u32x4 zf[MT * NHF];
#pragma unroll
      for (int i = 0; i < MT * NHF; ++i) {
        const uint32_t* zr = Zt + (16 * (i / NHF) + l16) * ZLD + 2 * g4 + 16 * (i % NHF);
        const u32x2 lo = *reinterpret_cast<const u32x2*>(zr);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(zr + 8);
        zf[i] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      }
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int hf = 0; hf < NHF; ++hf)
          acc[m] = mfma_16x16x32(__builtin_bit_cast(bf16x8, zf[m * NHF + hf]), pb[hf], acc[m]);
      sched_reads_ahead<MT * NHF>();
    }
    __syncthreads();
  };
  // prefix self-attention: keys past this block's last query are all masked
  const int t_stop = p.causal ? min(T, qb * 64 + 64) : T;
  // t_stop >= 1 (T >= 1): the first pair always runs, with no branch around it
  step(Flag<true>{}, 0, 0, kA, vA, mA, oA);
  step(Flag<false>{}, TK, 1, kB, vB, mB, oB);
  for (int t0 = 2 * TK; t0 < t_stop; t0 += 2 * TK) {
    step(Flag<false>{}, t0, 0, kA, vA, mA, oA);
    step(Flag<false>{}, t0 + TK, 1, kB, vB, mB, oB);
  }

  // ---- R_h has landed (its DMA was issued before every other load; the loop
  // ended on a barrier, and this wait plus one more barrier covers all waves)
  wait_vmcnt<0>();
  __syncthreads();
  // ---- normalise and rotate back: O^T = R_h U^T
  const float lsum = add_xor32(add_xor16(l_run));
  const float inv = 1.f / lsum;
  bf16x8 ub[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ub[ks][i] = static_cast<bf16>(acc[2 * ks][i] * inv);
      ub[ks][4 + i] = static_cast<bf16>(acc[2 * ks + 1][i] * inv);
    }
  f32x4 o[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    o[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (DENSE) {
      // no rotation: the normalised accumulator, dims 32(m/2) + 8 g4 +
      // 4(m%2) + i (the tile row order), placed accordingly when staged
      o[m] = acc[m] * inv;
      continue;
    }
    // A fragment: R_h row 16m + l16 at the dims of ub[ks], 32ks + 8g4 .. + 7:
    // one 16-byte chunk, 4ks + g4
    const int row = 16 * m + l16;
    const char* rr = Rs + row * RBY;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 av = *reinterpret_cast<const u32x4*>(rr + 16 * ((4 * ks + g4) ^ (row % RCH)));
      o[m] = mfma_16x16x32(__builtin_bit_cast(bf16x8, av), ub[ks], o[m]);
    }
  }
  // ---- output: each wave stages its 16 query rows in LDS (over R_h, once
  // every wave is done with it) in row order, 16-byte chunks XOR-swizzled by
  // row, and writes them with consecutive lanes on consecutive 16-byte units
  // (scattered 8-byte stores from the MFMA layout waste write bandwidth).
  // Rows past Tq fall outside the output resource and are dropped.
  __syncthreads();
  const int q0 = qb * 64 + 16 * w;  // this wave's first query
  const uint32_t esz = p.out_f32 ? 4u : 2u;
  const uint32_t ostride = static_cast<uint32_t>(H) * DH * esz;  // bytes between queries
  const rsrc_t r_o = make_rsrc(static_cast<char*>(p.out) + ((static_cast<size_t>(b) * p.Tq) * H + h) * DH * esz,
                               clamp_bytes((static_cast<size_t>(p.Tq - 1) * H + 1) * DH * esz));
  char* stg = smem + w * (16 * DH * 4);  // 16 rows of up to 4-byte elements
  if (p.out_f32) {
    constexpr int NC = DH / 4;  // 16-byte chunks per f32 row
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      // 16-byte chunk of o[m]: dims 16m + 4g4 .. (rotated) or the tile row order (dense)
      const int c = DENSE ? 8 * (m >> 1) + 2 * g4 + (m & 1) : 4 * m + g4;
      *reinterpret_cast<f32x4*>(stg + l16 * (DH * 4) + 16 * (c ^ l16)) = o[m];
    }
#pragma unroll
    for (int i = 0; i < 16 * NC / 64; ++i) {
      const int u = 64 * i + lane, r = u / NC, c = u % NC;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + r * (DH * 4) + 16 * (c ^ r));
      __builtin_amdgcn_raw_buffer_store_b128(v, r_o, oob_unless(q0 + r < p.Tq, (q0 + r) * ostride + 16u * c), 0, 0);
    }
  } else {
    constexpr int NC = DH / 8;  // 16-byte chunks per bf16 row
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      bf16x4 ov;
      ov[0] = static_cast<bf16>(o[m][0]);
      ov[1] = static_cast<bf16>(o[m][1]);
      ov[2] = static_cast<bf16>(o[m][2]);
      ov[3] = static_cast<bf16>(o[m][3]);
      // 16-byte chunk and 8-byte half of o[m] (see the f32 case)
      const int c = DENSE ? 4 * (m >> 1) + g4 : 2 * m + (g4 >> 1), hf = DENSE ? (m & 1) : (g4 & 1);
      *reinterpret_cast<bf16x4*>(stg + l16 * (DH * 2) + 16 * (c ^ (l16 % NC)) + 8 * hf) = ov;
    }
#pragma unroll
    for (int i = 0; i < 16 * NC / 64; ++i) {
      const int u = 64 * i + lane, r = u / NC, c = u % NC;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + r * (DH * 2) + 16 * (c ^ (r % NC)));
      __builtin_amdgcn_raw_buffer_store_b128(v, r_o, oob_unless(q0 + r < p.Tq, (q0 + r) * ostride + 16u * c), 0, 0);
    }
  }
}

// ---------------------------------------------------------------------------
// Vector-ALU kernel for f32 (and any head width). One workgroup per
// (sample, head, query); thread j owns output dimension j.
template <class E>
__global__ __launch_bounds__(128) void k_attend_generic(AttendParams p) {
  __shared__ float red[2];
  __shared__ float us[128];
  const int dh = p.dh, j = threadIdx.x, lane = j & 63, w = j >> 6;
  const size_t id = blockIdx.x;
  const int qi = static_cast<int>(id % p.Tq);
  const int h = static_cast<int>((id / p.Tq) % p.H);
  const int b = static_cast<int>(id / (static_cast<size_t>(p.Tq) * p.H));
  const int T = p.T, H = p.H, G = p.G, ds = dh / G;
  const int g = j / ds, e = j % ds;
  const uint32_t gm = group_mask(G);
  const E* qv = static_cast<const E*>(p.q) + ((static_cast<size_t>(b) * p.Tq + qi) * H + h) * dh;
  const E* kv = static_cast<const E*>(p.k);
  const E* Vp = static_cast<const E*>(p.Vp);
  const float qj = tof(qv[j]);
  float m = -INFINITY, l = 0.f, u = 0.f;
  const int nw = (dh + 63) / 64;
  const int t_stop = p.causal ? min(T, qi + 1) : T;
  for (int t = 0; t < t_stop; ++t) {
    float part = qj * tof(kv[((static_cast<size_t>(b) * T + t) * H + h) * dh + j]);
    part = wave_sum(part);
    if (nw > 1) {
      if (lane == 0) red[w] = part;
      __syncthreads();
      part = red[0] + red[1];
      __syncthreads();
    }
    const float sc = part * p.scale;
    const float mn = fmaxf(m, sc);
    const float al = expf(m - mn), pr = expf(sc - mn);
    l = l * al + pr;
    const uint32_t mk = p.mask[static_cast<size_t>(b) * T + t] & gm;
    float zv = 0.f;
    if ((mk >> g) & 1u) {
      const int64_t slot = p.offsets[static_cast<size_t>(b) * (T + 1) + t] + __popc(mk & ((1u << g) - 1u));
      if (slot < p.cap) zv = tof(Vp[((static_cast<size_t>(b) * H + h) * p.cap + slot) * ds + e]);
    }
    u = u * al + pr * zv;
    m = mn;
  }
  us[j] = u / l;
  __syncthreads();
  const E* Rh = static_cast<const E*>(p.R) + static_cast<size_t>(h) * dh * dh;
  float o = 0.f;
  for (int jj = 0; jj < dh; ++jj) o += tof(Rh[j * dh + jj]) * us[jj];
  const size_t oi = ((static_cast<size_t>(b) * p.Tq + qi) * H + h) * dh + j;
  if (p.out_f32)
    static_cast<float*>(p.out)[oi] = o;
  else
    static_cast<E*>(p.out)[oi] = fromf<E>(o);
}

}  // namespace

hipError_t launch_attend(const AttendParams& p, bool bf16, hipStream_t s) {
  if (p.B == 0 || p.Tq == 0 || p.H == 0) return hipSuccess;
  if (bf16 && (p.dh == 128 || p.dh == 64)) {
    const dim3 grid(static_cast<unsigned>(p.B * p.H * ((p.Tq + 63) / 64)));
    const int ds = p.dh / p.G;
    const int vm = ds >= 8 ? kWide : (ds == 4 ? kDs4 : kDs2);
    auto k = p.dense ? (p.dh == 128 ? k_attend_bf16<128, kDense> : k_attend_bf16<64, kDense>)
             : p.dh == 128 ? (vm == kWide ? k_attend_bf16<128, kWide> : vm == kDs4 ? k_attend_bf16<128, kDs4>
                                                                                  : k_attend_bf16<128, kDs2>)
                           : (vm == kWide ? k_attend_bf16<64, kWide> : vm == kDs4 ? k_attend_bf16<64, kDs4>
                                                                                 : k_attend_bf16<64, kDs2>);
    hipLaunchKernelGGL(k, grid, dim3(256), 0, s, p);
  } else {
    const dim3 grid(static_cast<unsigned>(static_cast<size_t>(p.B) * p.H * p.Tq));
    if (bf16)
      hipLaunchKernelGGL(k_attend_generic<rolesub::bf16>, grid, dim3(p.dh), 0, s, p);
    else
      hipLaunchKernelGGL(k_attend_generic<float>, grid, dim3(p.dh), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace rolesub
