// Value rotation into the orthogonal routing space, z = R_h^T v (Sec. 3.2).
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

// bf16 matrix-core rotation. Each workgroup owns one head h and a contiguous
// run of tokens (flattened over samples); each wave takes 16-token tiles. The
// product is computed transposed, Z^T = R_h^T V^T, so the streamed operand
// (the values, 16 B per lane straight from HBM) is the MFMA B fragment and
// every lane ends up with 4 consecutive outputs of its token. R_h^T lives in
// LDS (staged once per workgroup, 16-byte chunks XOR-swizzled by row so that
// fragment reads are conflict-free) and its fragments are read per tile,
// which keeps the register count low. Workgroups of one head are placed on
// one XCD so R_h stays in its L2.
//
// A tile's results are not stored from the MFMA layout (8 bytes per lane,
// scattered over 16 tokens): such partial-line writes run at about two thirds
// of the bandwidth of contiguous ones. They are first written to a per-wave
// LDS tile in output order and then copied out with consecutive lanes on
// consecutive 16-byte units.
//
// OUT = kZ writes z (16 rows of dh values). The pack modes write only the
// kept groups into the compact cache (the kept groups of M z, Sec. 3.2) at
// the slots given by the offsets, so z never reaches memory; the tile then
// holds the tile's slots in cache order and a slot -> token table. The copy
// unit is 16 bytes (kPack16, ds >= 8), 8 bytes (kPack8, ds = 4) or 4 bytes
// (kPack4, ds = 2), never wider than a slot. For prefixes of at most
// kRotMaxRun tokens the pack modes also form the cache offsets of their run
// of tokens from the masks (an exclusive scan of the kept counts within each
// sample), while R_h is being staged, and the workgroups of head 0 write
// them out; for longer prefixes (a run's sample may start thousands of
// tokens earlier) they read offsets the scan kernel wrote (off_ready).
enum RotOut { kZ = 0, kPack16 = 1, kPack8 = 2, kPack4 = 3 };
constexpr int kRotMaxRun = 512;  // tokens per workgroup at most (two per thread)

template <int DH>
__device__ __forceinline__ int rt_chunk_swz(int j) {
  // 16-byte chunk permutation of R^T row j: rows of 256 B (dh = 128) use j mod
  // 16; rows of 128 B (dh = 64) share a bank line in pairs, so j/2 mod 8
  return DH == 128 ? (j & 15) : ((j >> 1) & 7);
}

template <int DH, int OUT>
__global__ __launch_bounds__(256) void k_rotate_bf16(RotateParams p) {
  constexpr bool PACK = OUT != kZ;
  constexpr int MT = DH / 16, KS = DH / 32;
  constexpr int U = OUT == kPack4 ? 4 : (OUT == kPack8 ? 8 : 16);  // copy-out unit, bytes
  constexpr int NSLOT = PACK ? 16 * 32 : 1;  // slots of one tile: 16 tokens x G <= 32
  __shared__ __attribute__((aligned(16))) bf16 Rt[DH * DH];  // Rt[j][k] = R[k][j], swizzled
  __shared__ __attribute__((aligned(16))) bf16 Ost[4][16 * DH];  // per-wave output tile
  __shared__ uint8_t Otok[4][NSLOT];                           // slot -> token of the tile
  __shared__ int32_t Obase[4][PACK ? 16 : 1], Opre[4][PACK ? 16 : 1];
  // PACK: exclusive scan of the kept counts over the run (< 2^16: at most
  // 511 tokens of at most 32 groups); 16-bit entries keep three workgroups
  // per CU within the LDS
  __shared__ uint16_t Sexc[PACK ? kRotMaxRun : 1];
  const int H = p.H, ntok = p.ntok;
  int h, chunk;
  xcd_split(blockIdx.x, H, h, chunk);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int t_begin = chunk * p.tok_per_wg;
  const int t_end = min(t_begin + p.tok_per_wg, ntok);
  const uint32_t gm = p.G >= 32 ? 0xFFFFFFFFu : ((1u << p.G) - 1u);
  const bf16* Rh = static_cast<const bf16*>(p.R) + static_cast<size_t>(h) * DH * DH;
  // this workgroup's tokens of head h; rows past t_end load as zero
  const uint32_t tstride = static_cast<uint32_t>(H) * DH * 2;
  const rsrc_t r_v = make_rsrc(static_cast<const bf16*>(p.v) + (static_cast<size_t>(t_begin) * H + h) * DH,
                               static_cast<uint32_t>(t_end - t_begin - 1) * tstride + DH * 2);
  // PACK: group masks and cache offsets of the run's tokens
  const rsrc_t r_m = make_rsrc(p.mask + t_begin, static_cast<uint32_t>(t_end - t_begin) * 4u);
  // rotate only: this run's rows of z
  const rsrc_t r_z = make_rsrc(static_cast<bf16*>(p.z) + (static_cast<size_t>(t_begin) * H + h) * DH,
                               PACK ? 0u : static_cast<uint32_t>(t_end - t_begin - 1) * tstride + DH * 2);
  // off_ready: offsets are [B][T+1], token (b, t) at b*(T+1)+t
  const rsrc_t r_o = make_rsrc(p.offsets, PACK && p.off_ready ? static_cast<uint32_t>(ntok + ntok / p.T) * 4u : 0u);
  const int ds = DH / p.G;
  // G divides dh (a power of two), so ds is one too: shifts, no divisions
  const int lds = __builtin_ctz(ds);
  const int cap32 = static_cast<int>(p.cap);  // < 2^31: the cache per (sample, head) is < 2 GiB

  struct Tile {
    bf16x8 v[KS];
    uint32_t mask;
    int32_t off;  // off_ready: the token's cache offset
  };
  // Loads are unconditional (rows past the run read as zeros through the
  // buffer bounds): a branch around them makes later waits cover every
  // outstanding memory operation.
  auto load = [&](Tile& x, int tt) {
    const int tok = tt + l16;
    const bool ok = tok < t_end;
    const uint32_t o = static_cast<uint32_t>(tok - t_begin) * tstride + 16u * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) x.v[ks] = __builtin_bit_cast(bf16x8, bload16(r_v, oob_unless(ok, o + 64u * ks)));
    x.mask = 0;
    x.off = 0;
    if constexpr (PACK) {
      x.mask = bload4(r_m, oob_unless(ok, 4u * (tok - t_begin)));
      x.off = static_cast<int32_t>(bload4(r_o, oob_unless(ok && p.off_ready, 4u * (tok + tok / p.T))));
    }
  };
  // one tile in flight ahead of the one being processed (A and B alternate);
  // the first is requested before R_h is staged, so that its round trip
  // overlaps the staging. Tiles w and w + 4 of the run go to wave w. When
  // every workgroup is resident at once (dyn_tiles) the others are handed
  // out in order from an LDS counter to whichever wave asks next, so that
  // waves slowed by their memory requests take fewer and the workgroup ends
  // with its last tile; otherwise (later workgroups fill the CUs that free
  // up) wave w takes every fourth tile.
  __shared__ int s_next;
  const int ntile = (t_end - t_begin + 15) >> 4;
  if (tid == 0) s_next = 8;
  int snext = w + 4;
  auto grab = [&]() {
    if (!p.dyn_tiles) return snext += 4;
    int i = 0;
    if (lane == 0) i = atomicAdd(&s_next, 1);
    return __builtin_amdgcn_readfirstlane(__shfl(i, 0, kWave));
  };
  Tile A, B;
  int ia = w, ib = w + 4;
  load(A, t_begin + 16 * ia);

  uint32_t mk0 = 0, mk1 = 0;
  int cpre = 0, run_pre = 0;  // run_pre: kept count of t_begin's sample before the run
  {
    // Transposed staging. An item is (row pair p, 8-column chunk jc): rows 2p
    // and 2p+1 of R_h are read 16 bytes each and written as 8 dwords
    // Rt[jc*8+e][2p..2p+1]; consecutive lanes take consecutive p, so each
    // store instruction fills distinct dwords of one LDS row.
    constexpr int NPAIR = DH / 2, NCH = DH / 8, NI = NPAIR * NCH / 256;
    uint32_t* Rt32 = reinterpret_cast<uint32_t*>(Rt);
    u32x4 lo[NI], hi[NI];
#pragma unroll
    for (int r = 0; r < NI; ++r) {
      const int it = tid + 256 * r;
      const int pr = it % NPAIR, jc = it / NPAIR;
      lo[r] = *reinterpret_cast<const u32x4*>(Rh + (2 * pr) * DH + 8 * jc);
      hi[r] = *reinterpret_cast<const u32x4*>(Rh + (2 * pr + 1) * DH + 8 * jc);
    }
    // PACK: the masks of this thread's two tokens of the run (2 tid, 2 tid + 1)
    // and the kept count of the earlier tokens of t_begin's sample (fewer
    // than T <= kRotMaxRun, two per thread), requested while R_h is in
    // flight. The loads are unconditional, bounded by their buffers: a load
    // under a branch is waited for at once, and that wait also drains R_h
    // and the first tile, one more full round trip per load.
    if (PACK && !p.off_ready) {
      // two 4-byte loads (the pinned offset keeps them from being merged
      // into one 8-byte load, whose bounds check would drop a run's last
      // token when the run is odd)
      mk0 = bload4(r_m, 8u * tid) & gm;
      mk1 = bload4(r_m, oob_unless(true, 8u * tid + 4u)) & gm;
      const int s0 = (t_begin / p.T) * p.T;
      const rsrc_t r_pm = make_rsrc(p.mask + s0, static_cast<uint32_t>(t_begin - s0) * 4u);
      cpre = __popc(bload4(r_pm, 4u * tid) & gm) + __popc(bload4(r_pm, 4u * tid + 1024u) & gm);
    }
#pragma unroll
    for (int r = 0; r < NI; ++r) {
      const int it = tid + 256 * r;
      const int pr = it % NPAIR, jc = it / NPAIR;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int j = 8 * jc + 2 * q + e;  // row of R^T = column of R
          const uint32_t d = e == 0 ? ((lo[r][q] & 0xFFFFu) | (hi[r][q] << 16))
                                    : ((lo[r][q] >> 16) | (hi[r][q] & 0xFFFF0000u));
          Rt32[j * (DH / 2) + (((pr >> 2) ^ rt_chunk_swz<DH>(j)) << 2) + (pr & 3)] = d;
        }
      }
    }
  }
  if (PACK && !p.off_ready) {
    // Offsets of the run's tokens. With E(t) the exclusive scan of the kept
    // counts over the run (from t_begin) and run_pre the kept count of t_begin's
    // sample before t_begin, a token whose sample starts at or before
    // t_begin has offset run_pre + E(t), one whose sample starts at ss inside
    // the run E(t) - E(ss).
    int* Sred = reinterpret_cast<int*>(Ost[0]);  // the output tiles are not in use yet
    const int c0 = __popc(mk0), c1 = __popc(mk1);
    int x = c0 + c1;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, kWave);
      if (lane >= o) x += y;
    }
    int r = cpre;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) r += __shfl_xor(r, o, kWave);
    if (lane == 63) Sred[w] = x;
    if (lane == 0) Sred[4 + w] = r;
    __syncthreads();
    int e0 = x - c0 - c1;
    for (int i = 0; i < w; ++i) e0 += Sred[i];
    run_pre = Sred[4] + Sred[5] + Sred[6] + Sred[7];
    const int T = p.T, ta = t_begin + 2 * tid;
    const bool in0 = ta < t_end, in1 = ta + 1 < t_end;
    if (in0) Sexc[2 * tid] = static_cast<uint16_t>(e0);
    if (in1) Sexc[2 * tid + 1] = static_cast<uint16_t>(e0 + c0);
    __syncthreads();
    // offsets are [B][T+1]: token t at t + t/T, each sample's total after its
    // last token; one workgroup per run writes them
    if (h == 0) {
      auto fin = [&](int t, int e) {
        const int ss = (t / T) * T;
        return ss <= t_begin ? run_pre + e : e - Sexc[ss - t_begin];
      };
      const int o0 = in0 ? fin(ta, e0) : 0, o1 = in1 ? fin(ta + 1, e0 + c0) : 0;
      if (in0) {
        p.offsets[ta + ta / T] = o0;
        if (ta % T == T - 1) p.offsets[ta + ta / T + 1] = o0 + c0;
      }
      if (in1) {
        p.offsets[ta + 1 + (ta + 1) / T] = o1;
        if ((ta + 1) % T == T - 1) p.offsets[ta + 1 + (ta + 1) / T + 1] = o1 + c1;
      }
    }
  }
  __syncthreads();

  bf16* ost = Ost[w];
  char* ostb = reinterpret_cast<char*>(ost);
  auto process = [&](const Tile& x, int tt) {
    // keep the R^T fragments in LDS: without this the compiler hoists the
    // loop-invariant LDS reads into ~128 registers and occupancy collapses
    asm volatile("" ::: "memory");
    f32x4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int j = 16 * m + l16;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(Rt + j * DH + 8 * ((4 * ks + g4) ^ rt_chunk_swz<DH>(j)));
        acc[m] = mfma_16x16x32(a, x.v[ks], acc[m]);
      }
    }
    if constexpr (!PACK) {
      // tile row r = token tt + r; 16-byte chunk c of row r at c ^ (r mod NC)
      constexpr int NC = DH / 8;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        bf16x4 o;
        o[0] = static_cast<bf16>(acc[m][0]);
        o[1] = static_cast<bf16>(acc[m][1]);
        o[2] = static_cast<bf16>(acc[m][2]);
        o[3] = static_cast<bf16>(acc[m][3]);
        const int c = 2 * m + (g4 >> 1);
        *reinterpret_cast<bf16x4*>(ost + l16 * DH + 8 * (c ^ (l16 % NC)) + 4 * (g4 & 1)) = o;
      }
#pragma unroll
      for (int i = 0; i < 16 * NC / 64; ++i) {
        const int u = 64 * i + lane, r = u / NC, c = u % NC;
        const u32x4 d = *reinterpret_cast<const u32x4*>(ost + r * DH + 8 * (c ^ (r % NC)));
        const uint32_t off = static_cast<uint32_t>(tt + r - t_begin) * tstride + 16u * c;
        __builtin_amdgcn_raw_buffer_store_b128(d, r_z, oob_unless(tt + r < t_end, off), 0, 0);
      }
    } else {
      const int tok = tt + l16;
      // the token's offset from the run's scan (see the prologue)
      int off = x.off;
      if (!p.off_ready) {
        const int ss = (tok / p.T) * p.T;
        const int e = Sexc[min(tok - t_begin, kRotMaxRun - 1)];
        const int es = Sexc[min(max(ss - t_begin, 0), kRotMaxRun - 1)];
        off = tok < t_end ? (ss <= t_begin ? run_pre + e : e - es) : 0;
      }
      const uint32_t cmask = x.mask & gm;  // zero for rows past the run
      // groups of this token that fit the cache, and its first local slot
      const int cnt = min(__popc(cmask), max(cap32 - off, 0));
      int incl = cnt;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const int y = __shfl_up(incl, o, 16);
        if (l16 >= o) incl += y;
      }
      const int pre = incl - cnt;
      const int nslot = __shfl(incl, 15, 16);
      // the tile's tokens span samples b0.. ; slots are addressed relative to
      // (b0, h) so that offsets stay small however large the cache is
      const int b0 = __builtin_amdgcn_readfirstlane(tt / p.T);
      const int b1 = __builtin_amdgcn_readfirstlane(min(tt + 15, t_end - 1) / p.T);
      const size_t hstride = static_cast<size_t>(p.cap) * ds;  // elements per (sample, head)
      const rsrc_t r_vp = make_rsrc(static_cast<bf16*>(p.Vp) + (static_cast<size_t>(b0) * H + h) * hstride,
                                    clamp_bytes((static_cast<size_t>(b1 - b0) * H + 1) * hstride * 2));
      if (g4 == 0) {
        Obase[w][l16] = static_cast<int32_t>(static_cast<uint32_t>((tok / p.T - b0) * H) *
                                                 static_cast<uint32_t>(hstride) +
                                             (static_cast<uint32_t>(off) << lds));
        Opre[w][l16] = pre;
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int dim = 16 * m + 4 * g4;  // this lane's 4 outputs: dims dim..dim+3
        if constexpr (OUT != kPack4) {
          const int g = dim >> lds;
          const int rank = __popc(cmask & ((1u << g) - 1u));
          if (((cmask >> g) & 1u) && rank < cnt) {
            bf16x4 o;
            o[0] = static_cast<bf16>(acc[m][0]);
            o[1] = static_cast<bf16>(acc[m][1]);
            o[2] = static_cast<bf16>(acc[m][2]);
            o[3] = static_cast<bf16>(acc[m][3]);
            const int ls = pre + rank;
            *reinterpret_cast<bf16x4*>(ost + (ls << lds) + (dim & (ds - 1))) = o;
            if ((dim & (ds - 1)) == 0) Otok[w][ls] = static_cast<uint8_t>(l16);
          }
        } else {
          // 2-dim groups: the lane's outputs cover groups dim/2 and dim/2+1
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int g = dim / 2 + u;
            const int rank = __popc(cmask & ((1u << g) - 1u));
            if (((cmask >> g) & 1u) && rank < cnt) {
              const int ls = pre + rank;
              *reinterpret_cast<uint32_t*>(ost + 2 * ls) = pack_bf16x2(acc[m][2 * u], acc[m][2 * u + 1]);
              Otok[w][ls] = static_cast<uint8_t>(l16);
            }
          }
        }
      }
      // copy-out: unit q covers bytes [q U, q U + U) of the tile's slots. A
      // fixed number of store instructions (units past the tile's slots go
      // out of range) keeps the count of outstanding stores known, so the
      // next tile's wait does not also drain these stores.
      constexpr int NQ = 16 * DH * 2 / U;  // units of a fully kept tile
      const int lsu = lds + 1 - __builtin_ctz(U);  // log2(units per slot)
      const int nunit = nslot << lsu;
      // unrolled by 4 only: fully unrolled, the 8 rounds of 8-byte units (G = 32)
      // kept every round's address live and cost a wave per SIMD (188
      // registers against 146)
#pragma unroll 4
      for (int q0 = 0; q0 < NQ; q0 += 64) {
        const int q = q0 + lane;
        const int ls = min(q >> lsu, NSLOT - 1);
        const int t = Otok[w][ls] & 15;  // stale entries past the tile's slots stay in range
        const uint32_t go = static_cast<uint32_t>(Obase[w][t]) +
                            (static_cast<uint32_t>(ls - Opre[w][t]) << lds) +
                            static_cast<uint32_t>((q & ((1 << lsu) - 1)) * (U / 2));
        const uint32_t off = oob_unless(q < nunit, 2u * go);
        if constexpr (U == 16)
          __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(ostb + 16 * q), r_vp, off, 0, 0);
        else if constexpr (U == 8)
          __builtin_amdgcn_raw_buffer_store_b64(*reinterpret_cast<const u32x2*>(ostb + 8 * q), r_vp, off, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b32(*reinterpret_cast<const uint32_t*>(ostb + 4 * q), r_vp, off, 0, 0);
      }
    }
  };
  // Every wave's tiles come in increasing order: the first past the run
  // ends its loop (its loads read nothing). A wave asks for a tile one step
  // before it requests its data, so the counter's round trip overlaps a
  // tile's work; the index it holds when it stops is past the run as well.
  if (ia < ntile) {
    int nx = grab();
    load(B, t_begin + 16 * ib);
    for (;;) {
      process(A, t_begin + 16 * ia);
      if (ib >= ntile) break;
      ia = nx;
      nx = grab();
      load(A, t_begin + 16 * ia);
      process(B, t_begin + 16 * ib);
      if (ia >= ntile) break;
      ib = nx;
      nx = grab();
      load(B, t_begin + 16 * ib);
    }
  }
}

// Vector-ALU rotation for f32 (and any head width): one thread per output.
template <class T>
__global__ __launch_bounds__(256) void k_rotate_generic(const T* __restrict__ v, const T* __restrict__ R,
                                                        T* __restrict__ z, int ntok, int H, int dh) {
  const int per = 256 / dh;
  if (static_cast<int>(threadIdx.x) >= per * dh) return;
  const size_t th = static_cast<size_t>(blockIdx.x) * per + threadIdx.x / dh;
  if (th >= static_cast<size_t>(ntok) * H) return;
  const int j = threadIdx.x % dh;
  const int h = static_cast<int>(th % H);
  const T* vr = v + th * dh;
  const T* Rh = R + static_cast<size_t>(h) * dh * dh;
  float acc = 0.f;
  for (int k = 0; k < dh; ++k) acc += tof(Rh[k * dh + j]) * tof(vr[k]);
  z[th * dh + j] = fromf<T>(acc);
}

// Vector-ALU fused rotation + pack: one thread per output element; the
// element is stored only if its group is kept.
template <class T>
__global__ __launch_bounds__(256) void k_rotate_pack_generic(RotateParams p, int dh) {
  const int per = 256 / dh;
  if (static_cast<int>(threadIdx.x) >= per * dh) return;
  const size_t th = static_cast<size_t>(blockIdx.x) * per + threadIdx.x / dh;
  if (th >= static_cast<size_t>(p.ntok) * p.H) return;
  const int j = threadIdx.x % dh;
  const int h = static_cast<int>(th % p.H);
  const size_t tok = th / p.H;
  const int b = static_cast<int>(tok / p.T);
  const int ds = dh / p.G, g = j / ds;
  const uint32_t gm = p.G >= 32 ? 0xFFFFFFFFu : ((1u << p.G) - 1u);
  const uint32_t m = p.mask[tok] & gm;
  const int64_t slot = p.offsets[tok + b] + __popc(m & ((1u << g) - 1u));
  if (!((m >> g) & 1u) || slot >= p.cap) return;
  const T* vr = static_cast<const T*>(p.v) + th * dh;
  const T* Rh = static_cast<const T*>(p.R) + static_cast<size_t>(h) * dh * dh;
  float acc = 0.f;
  for (int k = 0; k < dh; ++k) acc += tof(Rh[k * dh + j]) * tof(vr[k]);
  static_cast<T*>(p.Vp)[((static_cast<size_t>(b) * p.H + h) * p.cap + slot) * ds + (j - g * ds)] = fromf<T>(acc);
}

}  // namespace

namespace {
// workgroups of the matrix-core rotation resident at once: three per CU at
// dh = 128, four at dh = 64
long rotate_slots(int dh) {
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
    ncu = 256;
  return static_cast<long>(dh == 128 ? 3 : 4) * ncu;
}

int rotate_tokens_per_wg(int ntok, int H, int dh) {
  // A workgroup stages R_h (32 KB at dh = 128, as much as 128 tokens of
  // values) and then streams its run of tokens; the workgroups resident at
  // once form a round, and a second, partly filled round costs nearly a
  // whole one. Runs (multiples of 16 tokens, 64 to 512) are chosen to
  // minimise rounds x (run + 128), the longer run on ties; past four rounds
  // of 512-token runs, 512.
  const long slots = rotate_slots(dh);
  if (static_cast<long>((ntok + kRotMaxRun - 1) / kRotMaxRun) * H > 4 * slots) return kRotMaxRun;
  int best = kRotMaxRun;
  long best_cost = -1;
  for (int tpw = kRotMaxRun; tpw >= 64; tpw -= 16) {
    const long wgs = static_cast<long>((ntok + tpw - 1) / tpw) * H;
    const long cost = (wgs + slots - 1) / slots * (tpw + 128);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = tpw;
    }
  }
  return best;
}
}  // namespace

hipError_t launch_rotate(bool bf16, int ntok, int H, int dh, const void* v, const void* R, void* z,
                         hipStream_t s) {
  if (ntok == 0 || H == 0) return hipSuccess;
  if (bf16 && (dh == 128 || dh == 64)) {
    RotateParams p = {};
    p.ntok = ntok;
    p.H = H;
    p.v = v;
    p.R = R;
    p.z = z;
    p.G = 1;
    p.tok_per_wg = rotate_tokens_per_wg(ntok, H, dh);
    const dim3 grid(static_cast<unsigned>(((ntok + p.tok_per_wg - 1) / p.tok_per_wg) * H));
    p.dyn_tiles = static_cast<long>(grid.x) <= rotate_slots(dh) ? 1 : 0;
    if (dh == 128)
      hipLaunchKernelGGL((k_rotate_bf16<128, kZ>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((k_rotate_bf16<64, kZ>), grid, dim3(256), 0, s, p);
  } else {
    const int per = 256 / dh;
    const size_t n = static_cast<size_t>(ntok) * H;
    const dim3 grid(static_cast<unsigned>((n + per - 1) / per));
    if (bf16)
      hipLaunchKernelGGL(k_rotate_generic<rolesub::bf16>, grid, dim3(256), 0, s,
                         static_cast<const rolesub::bf16*>(v), static_cast<const rolesub::bf16*>(R),
                         static_cast<rolesub::bf16*>(z), ntok, H, dh);
    else
      hipLaunchKernelGGL(k_rotate_generic<float>, grid, dim3(256), 0, s, static_cast<const float*>(v),
                         static_cast<const float*>(R), static_cast<float*>(z), ntok, H, dh);
  }
  return hipGetLastError();
}

hipError_t launch_rotate_pack(bool bf16, int B, int T, int H, int dh, int G, const void* v, const void* R,
                              const uint32_t* mask, int32_t* offsets, void* Vp, int64_t cap,
                              hipStream_t s) {
  const int ntok = B * T;
  if (B == 0) return hipSuccess;
  const bool mfma = bf16 && (dh == 128 || dh == 64) && dh / G >= 2;
  // the matrix-core kernel forms the offsets itself for prefixes of at most
  // kRotMaxRun tokens; otherwise (or when it does not run) they come first
  // from their own kernel
  const bool off_ready = !mfma || T > kRotMaxRun;
  if (off_ready || ntok == 0 || H == 0 || cap == 0) {
    const hipError_t e = launch_pack_offsets(B, T, G, mask, offsets, s);
    if (e != hipSuccess) return e;
  }
  if (ntok == 0 || H == 0 || cap == 0) return hipSuccess;
  RotateParams p = {};
  p.ntok = ntok;
  p.T = T;
  p.H = H;
  p.G = G;
  p.v = v;
  p.R = R;
  p.mask = mask;
  p.offsets = offsets;
  p.Vp = Vp;
  p.cap = cap;
  p.off_ready = off_ready ? 1 : 0;
  if (mfma) {
    p.tok_per_wg = rotate_tokens_per_wg(ntok, H, dh);
    const dim3 grid(static_cast<unsigned>(((ntok + p.tok_per_wg - 1) / p.tok_per_wg) * H));
    p.dyn_tiles = static_cast<long>(grid.x) <= rotate_slots(dh) ? 1 : 0;
    // G <= 32, so 2-dim groups occur only at dh = 64
    const int ds = dh / G;
    if (dh == 128 && ds >= 8)
      hipLaunchKernelGGL((k_rotate_bf16<128, kPack16>), grid, dim3(256), 0, s, p);
    else if (dh == 128)
      hipLaunchKernelGGL((k_rotate_bf16<128, kPack8>), grid, dim3(256), 0, s, p);
    else if (ds >= 8)
      hipLaunchKernelGGL((k_rotate_bf16<64, kPack16>), grid, dim3(256), 0, s, p);
    else if (ds == 4)
      hipLaunchKernelGGL((k_rotate_bf16<64, kPack8>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((k_rotate_bf16<64, kPack4>), grid, dim3(256), 0, s, p);
  } else {
    const int per = 256 / dh;
    const size_t n = static_cast<size_t>(ntok) * H;
    const dim3 grid(static_cast<unsigned>((n + per - 1) / per));
    if (bf16)
      hipLaunchKernelGGL(k_rotate_pack_generic<rolesub::bf16>, grid, dim3(256), 0, s, p, dh);
    else
      hipLaunchKernelGGL(k_rotate_pack_generic<float>, grid, dim3(256), 0, s, p, dh);
  }
  return hipGetLastError();
}

}  // namespace rolesub
