// Full-width routing space (Sec. 3.2 with one R over the whole value vector,
// d_v = H*dh; Sec. 4.1 runs d_v = 4096 with S = 16 groups of 256).
//
// Tokens that keep all S groups have R M R^T v = v, so the cache holds their
// value vector (S consecutive slots = d_v contiguous values). Routed tokens
// (any other mask) go through two dense contractions on the bf16 matrix cores:
//   rotate:  z  = R^T v  for every routed token, only the kept groups stored;
//   values:  v~ = R z~   for every routed token, written head-major
//            [B][H][T][dh] for the attention kernel.
// Both are one gather-GEMM C[m][n] = sum_k A[m][k] * Bt[n][k] over the routed
// tokens of all samples (m), with Bt = R^T (rotate; the caller supplies the
// transpose of the frozen R) or Bt = R (values), so that both operands are
// read along k. A routed-token list per sample and the cache offsets come from
// a small preparation kernel.
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

constexpr int kBM0 = 64, kBM1 = 128, kBN = 128, kBK = 64;  // row tiles: rotate, values
constexpr int kLd = kBK + 8;  // LDS row stride (elements): 144 bytes, conflict-free 16-byte fragment reads
constexpr int kPrepChunks = 16;

__device__ __forceinline__ uint32_t full_bits(int S) { return S >= 32 ? 0xFFFFFFFFu : ((1u << S) - 1u); }

// Inclusive scan over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

// Per sample: the routed-token list (and its length), the cache offsets
// (PACK), and the value-space copies of the tokens that keep every group:
// into the cache (PACK: v -> Vp) or from it into the head-major values
// (!PACK: Vp -> Vh, at the given offsets). kPrepChunks workgroups per sample
// share the copies; the first one writes the list, count and offsets, and
// (PACK) workgroup c builds the per-group lists of groups c, c + kPrepChunks.
template <bool PACK>
__global__ __launch_bounds__(256) void k_full_prep(FullParams p) {
  // offsets, the value-space token list and (PACK) the masks of the sample,
  // sized by T at launch (prep_shm)
  extern __shared__ __attribute__((aligned(16))) char prep_smem[];
  int* s_off = reinterpret_cast<int*>(prep_smem);
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(prep_smem + 4 * (p.T + 1));
  uint16_t* s_full = reinterpret_cast<uint16_t*>(prep_smem + 4 * (p.T + 1) + (PACK ? 4 * p.T : 0));
  __shared__ int wtot[4], wfull[4];
  __shared__ int wcnt[4][32];
  const int b = blockIdx.x / kPrepChunks, chunk = blockIdx.x % kPrepChunks;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int T = p.T, S = p.S;
  const uint32_t full = full_bits(S);
  const uint32_t* mk = p.mask + static_cast<size_t>(b) * T;
  int run_pc = 0, run_rt = 0, run_full = 0;
  for (int c0 = 0; c0 < T; c0 += 256) {
    const int t = c0 + tid;
    const bool valid = t < T;
    const uint32_t m = valid ? (mk[t] & full) : 0u;
    const bool routed = valid && m != full, isfull = valid && m == full;
    // packed scan: kept-group count (low 16 bits, at most 256 * 32 per
    // chunk) and routed flag (high bits); full tokens by ballot
    const int x = (valid ? __popc(m) : 0) | (routed ? (1 << 16) : 0);
    const int inc = wave_incl_scan(x);
    const uint64_t bal = __ballot(isfull);
    if (lane == 63) wtot[w] = inc;
    if (lane == 0) wfull[w] = __popcll(bal);
    __syncthreads();
    int before = 0, before_full = 0;
    for (int v = 0; v < w; ++v) {
      before += wtot[v];
      before_full += wfull[v];
    }
    const int ex = before + inc - x;
    const int ex_pc = ex & 0xFFFF, ex_rt = ex >> 16;
    const int ex_full = before_full + __popcll(bal & ((1ull << lane) - 1ull));
    if (valid) s_off[t] = run_pc + ex_pc;
    if (PACK && valid) s_mask[t] = m;
    if (chunk == 0 && routed) p.rlist[static_cast<size_t>(b) * T + run_rt + ex_rt] = t;
    if (isfull) s_full[run_full + ex_full] = static_cast<uint16_t>(t);
    const int tot = wtot[0] + wtot[1] + wtot[2] + wtot[3];
    run_pc += tot & 0xFFFF;
    run_rt += tot >> 16;
    run_full += wfull[0] + wfull[1] + wfull[2] + wfull[3];
    __syncthreads();
  }
  if (chunk == 0) {
    if (tid == 0) p.counts[b] = run_rt;
    if (PACK) {
      int32_t* off = p.offsets + static_cast<size_t>(b) * (T + 1);
      for (int t = tid; t < T; t += 256) off[t] = s_off[t];
      if (tid == 0) off[T] = run_pc;
    }
  }
  if (PACK) {
    // Per group: the routed tokens that keep it, in token order, after the
    // earlier groups' lists. Every workgroup of the sample counts every
    // group's tokens (one ballot per group per 256 tokens) and then lists
    // the tokens of its own groups (chunk, chunk + kPrepChunks).
    int32_t* pr = p.pairs + static_cast<size_t>(b) * T * S;
    int run_g[32];
#pragma unroll
    for (int gg = 0; gg < 32; ++gg) run_g[gg] = 0;
    for (int c0 = 0; c0 < T; c0 += 256) {
      const int t = c0 + tid;
      const uint32_t m = t < T ? s_mask[t] : full;
      const uint32_t kept = m != full ? m : 0u;
#pragma unroll
      for (int gg = 0; gg < 32; ++gg) {
        if (gg < S) {
          const uint64_t bal = __ballot((kept >> gg) & 1u);
          if (lane == 0) wcnt[w][gg] = __popcll(bal);
        }
      }
      __syncthreads();
#pragma unroll
      for (int gg = 0; gg < 32; ++gg)
        if (gg < S) run_g[gg] += wcnt[0][gg] + wcnt[1][gg] + wcnt[2][gg] + wcnt[3][gg];
      __syncthreads();
    }
    for (int g = chunk; g < S; g += kPrepChunks) {
      int start = 0;
#pragma unroll
      for (int gg = 0; gg < 32; ++gg) start += gg < g ? run_g[gg] : 0;
      int n_g = 0;
#pragma unroll
      for (int gg = 0; gg < 32; ++gg) n_g = gg == g ? run_g[gg] : n_g;
      if (tid == 0) {
        p.counts_g[static_cast<size_t>(b) * S + g] = n_g;
        p.starts_g[static_cast<size_t>(b) * S + g] = start;
      }
      int run = start;
      for (int c0 = 0; c0 < T; c0 += 256) {
        const int t = c0 + tid;
        const uint32_t m = t < T ? s_mask[t] : full;
        const bool keeps = m != full && ((m >> g) & 1u);
        const uint64_t bal = __ballot(keeps);
        if (lane == 0) wtot[w] = __popcll(bal);
        __syncthreads();
        int o = run + __popcll(bal & ((1ull << lane) - 1ull));
        for (int v = 0; v < w; ++v) o += wtot[v];
        if (keeps) pr[o] = t;
        run += wtot[0] + wtot[1] + wtot[2] + wtot[3];
        __syncthreads();
      }
    }
  }
  // value-space copies of the full tokens: d_v/8 16-byte pieces each, work
  // items (token, piece) spread over the chunks' threads, 8 loads in flight.
  const int pieces = p.dv / 8, dh = p.dv / p.H;
  const int cc = chunk, ncc = kPrepChunks;
  const int n_items = run_full * pieces;
  const rsrc_t r_cache = make_rsrc(static_cast<const bf16*>(p.Vp) + static_cast<size_t>(b) * p.cap * p.ds,
                                   clamp_bytes(static_cast<size_t>(p.cap) * p.ds * 2));
  const rsrc_t r_v = make_rsrc(static_cast<const bf16*>(p.v) + static_cast<size_t>(b) * T * p.dv,
                               clamp_bytes(static_cast<size_t>(T) * p.dv * 2));
  const int32_t* goff = p.offsets + static_cast<size_t>(b) * (T + 1);
  for (int i0 = (cc * 256 + tid); i0 < n_items; i0 += 8 * 256 * ncc) {
    u32x4 val[8];
    int tok[8], pc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 * ncc;
      const bool ok = i < n_items;
      tok[u] = ok ? s_full[i / pieces] : 0;
      pc[u] = i % pieces;
      uint32_t src;
      if (PACK) {
        src = oob_unless(ok, static_cast<uint32_t>((tok[u] * p.dv + 8 * pc[u]) * 2));
        val[u] = bload16(r_v, src);
      } else {
        // the piece lies in slot o + 8 pc / ds of the token's S consecutive slots
        const int o = ok ? goff[tok[u]] : 0;
        const bool in_cap = o + (8 * pc[u]) / p.ds < p.cap;
        src = oob_unless(ok && in_cap, static_cast<uint32_t>((static_cast<size_t>(o) * p.ds + 8 * pc[u]) * 2));
        val[u] = bload16(r_cache, src);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 * ncc;
      if (i >= n_items) continue;
      if (PACK) {
        const int o = s_off[tok[u]];
        if (o + (8 * pc[u]) / p.ds < p.cap) {
          bf16* dst = static_cast<bf16*>(p.Vp) + (static_cast<size_t>(b) * p.cap + o) * p.ds + 8 * pc[u];
          *reinterpret_cast<u32x4*>(dst) = val[u];
        }
      } else {
        const int e = 8 * pc[u], h = e / dh;
        bf16* dst = static_cast<bf16*>(p.Vh) + ((static_cast<size_t>(b) * p.H + h) * T + tok[u]) * dh + (e - h * dh);
        *reinterpret_cast<u32x4*>(dst) = val[u];
      }
    }
  }
}

// C[m][n] = sum_k A[m][k] * Bt[n][k] on 16x16x32 bf16 MFMA; 128 x 128 tile per
// workgroup, four waves of 64 x 64, k in steps of 64 (two MFMA k-steps per
// barrier) through a double-buffered LDS tile, the next step's operands in
// flight in registers.
// 128-row tiles: about 78 KB of LDS and 224 registers, two workgroups per CU;
// 64-row tiles: 59 KB, two per CU.
//   MODE 0 (rotate): rows are the routed tokens of all samples that keep the
//   workgroup's group g (per-sample lists from the preparation kernel), so only
//   kept groups are computed; A = v, Bt = the rows of R^T for group g's output
//   dims; results to the cache.
//   MODE 1 (values): rows are the routed tokens of all samples; A = their cached
//   groups of z~ (zero where dropped; steps of groups that no row of the tile
//   keeps are skipped), Bt = R; results head-major.
// Rows map to (sample, token) through the prefix of the per-sample counts.
// Groups (MODE 0) or column tiles (MODE 1) are pinned to XCDs so that each XCD
// reads only its share of R into its L2.
template <int MODE, int TBM, int NS>
__global__ __launch_bounds__(256, 2) void k_full_gemm(FullParams p) {
  // A and B tiles (double-buffered) in one region, reused for the output tile
  constexpr int kTileA = TBM * kLd, kTileB = kBN * kLd;
  constexpr int NA = TBM / 32, NB = kBN / 32, MI = TBM / 32;  // A, B pieces per thread, 16-row blocks per wave
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * kTileA + 2 * kTileB];
  // tile i of A at smem + i * kTileA, of B at smem + 2 * kTileA + i * kTileB
  __shared__ int pre[kFullMaxB + 1];
  __shared__ int r_b[TBM], r_t[TBM], r_off[TBM];
  __shared__ uint32_t r_mask[TBM];
  __shared__ uint32_t s_or;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int B = p.B, T = p.T, dv = p.dv, S = p.S, ds = p.ds;
  // which tile: (group g, column sub-tile, row tile) or (column tile, row tile)
  const int lin = blockIdx.x;
  int g = 0, n0 = 0, mt = 0;
  if (MODE == 0) {
    const int nsub = ds / kBN;
    int rest;
    if ((S & 7) == 0) {
      const int xcd = lin & 7, slot = lin >> 3, per = S >> 3;
      g = xcd + 8 * (slot % per);
      rest = slot / per;
    } else {
      g = lin % S;
      rest = lin / S;
    }
    n0 = g * ds + (rest % nsub) * kBN;
    mt = rest / nsub;
  } else {
    const int ntn = dv / kBN;
    int nt;
    if ((ntn & 7) == 0) {
      const int xcd = lin & 7, slot = lin >> 3, per = ntn >> 3;
      nt = xcd + 8 * (slot % per);
      mt = slot / per;
    } else {
      nt = lin % ntn;
      mt = lin / ntn;
    }
    n0 = nt * kBN;
  }
  const int m0 = mt * TBM;

  // prefix over samples of the row counts (one wave, 64 samples per step)
  if (w == 0) {
    int run = 0;
    for (int c0 = 0; c0 < B; c0 += 64) {
      const int x = c0 + lane < B ? (MODE == 0 ? p.counts_g[static_cast<size_t>(c0 + lane) * S + g]
                                               : p.counts[c0 + lane]) : 0;
      const int inc = wave_incl_scan(x);
      if (c0 + lane < B) pre[c0 + lane] = run + inc - x;
      run += __shfl(inc, 63, kWave);
    }
    if (lane == 0) pre[B] = run;
  }
  if (tid == 0) s_or = 0;
  __syncthreads();
  const int total = pre[B];
  if (m0 >= total) return;  // the same in every thread
  if (tid < TBM) {
    const int r = m0 + tid;
    int bb = -1, tt = 0, oo = 0;
    uint32_t mm = 0;
    if (r < total) {
      int lo = 0, hi = B - 1;  // largest bb with pre[bb] <= r
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= r) lo = mid; else hi = mid - 1;
      }
      bb = lo;
      const int j = r - pre[bb];
      tt = MODE == 0 ? p.pairs[static_cast<size_t>(bb) * T * S + p.starts_g[static_cast<size_t>(bb) * S + g] + j]
                     : p.rlist[static_cast<size_t>(bb) * T + j];
      mm = p.mask[static_cast<size_t>(bb) * T + tt] & full_bits(S);
      oo = p.offsets[static_cast<size_t>(bb) * (T + 1) + tt];
      if (MODE == 1) atomicOr(&s_or, mm);
    }
    r_b[tid] = bb;
    r_t[tid] = tt;
    r_mask[tid] = mm;
    r_off[tid] = oo;
  }
  __syncthreads();
  const uint32_t tile_or = MODE == 1 ? s_or : full_bits(S);

  // operand sources
  const rsrc_t r_A = MODE == 0
      ? make_rsrc(p.v, clamp_bytes(static_cast<size_t>(B) * T * dv * 2))
      : make_rsrc(p.Vp, clamp_bytes(static_cast<size_t>(B) * p.cap * ds * 2));
  const rsrc_t r_B = make_rsrc(p.Rm, clamp_bytes(static_cast<size_t>(dv) * dv * 2));
  // this thread's NA A pieces and NB B pieces per step: piece q = tid + 256 u,
  // row q / 8, 16-byte chunk q % 8
  constexpr int NP = NA > NB ? NA : NB;
  int arow[NP], ach[NP];
#pragma unroll
  for (int u = 0; u < NP; ++u) {
    arow[u] = (tid + 256 * u) >> 3;
    ach[u] = (tid + 256 * u) & 7;
  }
  // this thread's A rows, read once: MODE 0 the byte offset of the token's
  // value row, MODE 1 the byte offset of the sample's cache and the token's
  // mask and first slot
  uint32_t a_base[NA], a_mask[NA];
  int a_slot0[NA];
  bool a_ok[NA];
#pragma unroll
  for (int u = 0; u < NA; ++u) {
    const int row = arow[u];
    const int bb = r_b[row];
    a_ok[u] = bb >= 0;
    a_mask[u] = r_mask[row];
    a_slot0[u] = r_off[row];
    a_base[u] = MODE == 0 ? static_cast<uint32_t>(((static_cast<size_t>(bb < 0 ? 0 : bb) * T + r_t[row]) * dv + 8 * ach[u]) * 2)
                          : static_cast<uint32_t>((static_cast<size_t>(bb < 0 ? 0 : bb) * p.cap * ds + 8 * ach[u]) * 2);
  }
  auto a_off = [&](int u, int k0) -> uint32_t {
    if (MODE == 0) {
      return oob_unless(a_ok[u], a_base[u] + static_cast<uint32_t>(k0) * 2u);
    } else {
      const int g = k0 / ds;
      const int slot = a_slot0[u] + __popc(a_mask[u] & ((1u << g) - 1u));
      const bool ok = a_ok[u] && ((a_mask[u] >> g) & 1u) && slot < p.cap;
      return oob_unless(ok, a_base[u] + static_cast<uint32_t>((slot * ds + (k0 - g * ds)) * 2));
    }
  };
  auto b_off = [&](int u, int k0) -> uint32_t {
    const size_t e = static_cast<size_t>(n0 + arow[u]) * dv + k0 + 8 * ach[u];
    return static_cast<uint32_t>(e * 2);
  };
  // k steps: every step of every group in tile_or (MODE 0: all groups);
  // branch-free, and k >= dv stays at dv (loads past the end read zeros)
  auto next_k = [&](int k0) -> int {
    const int k1 = k0 + kBK;
    const int gb = k1 / ds;
    const uint32_t rest = gb < 32 ? (tile_or >> gb) : 0u;
    const int kg = rest ? (gb + static_cast<int>(__builtin_ctz(rest))) * ds : dv;
    const int kn = (k1 % ds != 0) ? k1 : kg;
    return k0 >= dv ? dv : (kn < dv ? kn : dv);
  };
  const int k_first = tile_or == 0 ? dv : static_cast<int>(__builtin_ctz(tile_or)) * ds;
  // active steps: a multiple of 2 (ds is a multiple of 128: at least 2 steps
  // per group), which NS divides. Steps of 64 columns (two MFMA k-steps per
  // barrier) took the values product from 110-121 to 100-109 us (prep
  // included) with two operand sets; more sets were slower for both products
  // (the rotation: 107 us with four sets of 64 columns, 104 with eight of 32,
  // against 72-77).
  const int nsteps = MODE == 0 ? dv / kBK : __popc(tile_or) * (ds / kBK);

  // the loop body covers NS steps and picks the LDS buffer by step parity:
  // NS must be even and divide the step count
  static_assert(NS == 2 || NS == 4, "operand sets: even and a divisor of 4");
  f32x4 acc[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int wm = w >> 1, wn = w & 1;
  // NS register sets: step s's operands arrive in set s % NS, issued NS - 1
  // steps before they are written to LDS
  u32x4 ra[NS][NA], rbv[NS][NB];
  // MODE 1 computes the offsets unconditionally: with a branch around its
  // (longer) address computation the compiler reuses an in-flight load's
  // registers and waits for every load (values 117.6 -> 110.4 us). The
  // rotation's short computation is faster with the select (71.7 vs 82.2 us;
  // both measured in one process).
  auto load_set = [&](u32x4 (&a)[NA], u32x4 (&bb)[NB], int k0) {
    const bool real = k0 < dv;
    if constexpr (MODE == 1) {
      const int kk = real ? k0 : 0;
#pragma unroll
      for (int u = 0; u < NA; ++u) a[u] = bload16(r_A, oob_unless(real, a_off(u, kk)));
#pragma unroll
      for (int u = 0; u < NB; ++u) bb[u] = bload16(r_B, oob_unless(real, b_off(u, kk)));
    } else {
#pragma unroll
      for (int u = 0; u < NA; ++u) a[u] = bload16(r_A, real ? a_off(u, k0) : kOOB);
#pragma unroll
      for (int u = 0; u < NB; ++u) bb[u] = bload16(r_B, real ? b_off(u, k0) : kOOB);
    }
  };
  auto store_set = [&](const u32x4 (&a)[NA], const u32x4 (&bb)[NB], int buf) {
#pragma unroll
    for (int u = 0; u < NA; ++u)
      *reinterpret_cast<u32x4*>(&(smem + buf * kTileA)[arow[u] * kLd + 8 * ach[u]]) = a[u];
#pragma unroll
    for (int u = 0; u < NB; ++u)
      *reinterpret_cast<u32x4*>(&(smem + 2 * kTileA + buf * kTileB)[arow[u] * kLd + 8 * ach[u]]) = bb[u];
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      bf16x8 af[MI], bfr[4];
#pragma unroll
      for (int i = 0; i < MI; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(
            &(smem + buf * kTileA)[((TBM / 2) * wm + 16 * i + l16) * kLd + 32 * ks + 8 * g4]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        bfr[i] = *reinterpret_cast<const bf16x8*>(
            &(smem + 2 * kTileA + buf * kTileB)[(64 * wn + 16 * i + l16) * kLd + 32 * ks + 8 * g4]);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_16x16x32(af[i], bfr[j], acc[i][j]);
    }
  };
  // prologue: steps 0..NS-1 issued in the same order the loop keeps
  int kq = k_first;
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) {
    load_set(ra[j], rbv[j], kq);
    kq = next_k(kq);
  }
  store_set(ra[0], rbv[0], 0);
  load_set(ra[NS - 1], rbv[NS - 1], kq);
  kq = next_k(kq);
  __syncthreads();
  for (int s = 0; s < nsteps; s += NS) {
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      // set j is free (step s+j is in LDS): step s+j+NS into it
      load_set(ra[j], rbv[j], kq);
      kq = next_k(kq);
      compute(j & 1);
      store_set(ra[(j + 1) % NS], rbv[(j + 1) % NS], (j + 1) & 1);
      __syncthreads();
    }
  }

  // stage the bf16 tile in LDS (row stride kBN + 8), then 16-byte stores
  constexpr int kCs = kBN + 8;
  static_assert(TBM * kCs <= 2 * kTileA + 2 * kTileB, "C tile fits the A and B buffers");
  bf16* Cs = smem;
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Cs[((TBM / 2) * wm + 16 * i + 4 * g4 + e) * kCs + 64 * wn + 16 * j + l16] = static_cast<bf16>(acc[i][j][e]);
  __syncthreads();
#pragma unroll
  for (int u = 0; u < TBM * kBN / 8 / 256; ++u) {
    const int q = tid + 256 * u, row = q / (kBN / 8), c = q % (kBN / 8);
    const int bb = r_b[row];
    if (bb < 0) continue;
    const u32x4 val = *reinterpret_cast<const u32x4*>(&Cs[row * kCs + 8 * c]);
    const int n = n0 + 8 * c;
    if (MODE == 0) {
      const uint32_t mm = r_mask[row];
      const int slot = r_off[row] + __popc(mm & ((1u << g) - 1u));
      if (slot < p.cap) {
        bf16* dst = static_cast<bf16*>(p.Vp) + (static_cast<size_t>(bb) * p.cap + slot) * ds + (n - g * ds);
        *reinterpret_cast<u32x4*>(dst) = val;
      }
    } else {
      const int dh = dv / p.H, h = n / dh;
      bf16* dst = static_cast<bf16*>(p.Vh) + ((static_cast<size_t>(bb) * p.H + h) * T + r_t[row]) * dh + (n - h * dh);
      *reinterpret_cast<u32x4*>(dst) = val;
    }
  }
}

// Rt[j][k] = R[k][j] for an n x n bf16 matrix, 64 x 64 tiles through LDS.
__global__ __launch_bounds__(256) void k_transpose_bf16(const bf16* __restrict__ R, bf16* __restrict__ Rt, int n) {
  __shared__ bf16 tile[64][66];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int bx = blockIdx.x % (n / 64), by = blockIdx.x / (n / 64);
  for (int r = ty; r < 64; r += 4) tile[r][tx] = R[static_cast<size_t>(by * 64 + r) * n + bx * 64 + tx];
  __syncthreads();
  for (int r = ty; r < 64; r += 4) Rt[static_cast<size_t>(bx * 64 + r) * n + by * 64 + tx] = tile[tx][r];
}

}  // namespace

hipError_t launch_full(const FullParams& p, int mode, hipStream_t s) {
  if (p.B == 0 || p.T == 0) return hipSuccess;
  const dim3 gprep(static_cast<unsigned>(p.B) * kPrepChunks);
  const size_t shm_pack = 4 * static_cast<size_t>(p.T + 1) + 4 * static_cast<size_t>(p.T) + 2 * static_cast<size_t>(p.T);
  const size_t shm_vals = 4 * static_cast<size_t>(p.T + 1) + 2 * static_cast<size_t>(p.T);
  // row tiles: at most every token of every sample is a row (upper bound;
  // tiles past the actual count return at once). The rotation has fewer rows
  // per group than the values step has in all, so it takes 64-row tiles.
  const size_t rows = static_cast<size_t>(p.B) * p.T;
  if (mode == 0) {
    hipLaunchKernelGGL(k_full_prep<true>, gprep, dim3(256), shm_pack, s, p);
    const unsigned ncol = static_cast<unsigned>(p.S * (p.ds / kBN));
    const unsigned nmt = static_cast<unsigned>((rows + kBM0 - 1) / kBM0);
    hipLaunchKernelGGL((k_full_gemm<0, kBM0, 2>), dim3(ncol * nmt), dim3(256), 0, s, p);
  } else {
    hipLaunchKernelGGL(k_full_prep<false>, gprep, dim3(256), shm_vals, s, p);
    const unsigned ntn = static_cast<unsigned>(p.dv / kBN);
    const unsigned nmt = static_cast<unsigned>((rows + kBM1 - 1) / kBM1);
    hipLaunchKernelGGL((k_full_gemm<1, kBM1, 2>), dim3(ntn * nmt), dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_transpose(const void* R, void* Rt, int n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_transpose_bf16, dim3(static_cast<unsigned>((n / 64) * (n / 64))), dim3(256), 0, s,
                     static_cast<const bf16*>(R), static_cast<bf16*>(Rt), n);
  return hipGetLastError();
}

}  // namespace rolesub
