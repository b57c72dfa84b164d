// Value rotation into the orthogonal routing space, z = R_h^T v (Sec. 3.2).
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

// bf16 matrix-core rotation. Each workgroup owns one head h and a contiguous
// run of tokens (flattened over samples). The product is computed transposed,
// Z^T = R_h^T V^T, so the streamed operand (the values, 16 B per lane straight
// from HBM) is the MFMA B fragment and every lane ends up with 4 consecutive
// outputs of its token. R_h^T lives in LDS (staged once per workgroup) and
// its fragments are read from there per tile, which keeps the register count
// low: occupancy, not software pipelining, hides the memory latency.
// Workgroups of one head are placed on one XCD so R_h stays in its L2.
//
// PACK = false writes z. PACK = true writes only the kept groups into the
// compact cache (the kept groups of M z, Sec. 3.2) at the slots given by the
// offsets, so z never reaches memory.
template <int DH, bool PACK>
__global__ __launch_bounds__(256) void k_rotate_bf16(RotateParams p) {
  constexpr int MT = DH / 16, KS = DH / 32, LD = DH + 8;
  __shared__ __attribute__((aligned(16))) bf16 Rt[DH * LD];  // Rt[j][k] = R[k][j]
  const int H = p.H, ntok = p.ntok;
  int h, chunk;
  xcd_split(blockIdx.x, H, h, chunk);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const bf16* Rh = static_cast<const bf16*>(p.R) + static_cast<size_t>(h) * DH * DH;
  {
    // Transposed staging. An item is (row pair p, 8-column chunk jc): rows 2p
    // and 2p+1 of R_h are read 16 bytes each and written as 8 dwords
    // Rt[jc*8+e][2p..2p+1]; consecutive lanes take consecutive p, so each
    // store instruction fills consecutive dwords of one LDS row.
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
#pragma unroll
    for (int r = 0; r < NI; ++r) {
      const int it = tid + 256 * r;
      const int pr = it % NPAIR, jc = it / NPAIR;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        Rt32[(8 * jc + 2 * q) * (LD / 2) + pr] = (lo[r][q] & 0xFFFFu) | (hi[r][q] << 16);
        Rt32[(8 * jc + 2 * q + 1) * (LD / 2) + pr] = (lo[r][q] >> 16) | (hi[r][q] & 0xFFFF0000u);
      }
    }
  }
  __syncthreads();

  const int t_begin = chunk * p.tok_per_wg;
  const int t_end = min(t_begin + p.tok_per_wg, ntok);
  // this workgroup's tokens of head h; rows past t_end load as zero
  const uint32_t tstride = static_cast<uint32_t>(H) * DH * 2;
  const rsrc_t r_v = make_rsrc(static_cast<const bf16*>(p.v) + (static_cast<size_t>(t_begin) * H + h) * DH,
                               static_cast<uint32_t>(t_end - t_begin - 1) * tstride + DH * 2);
  // PACK: group masks and cache offsets of the run's tokens
  const rsrc_t r_m = make_rsrc(p.mask + t_begin, static_cast<uint32_t>(t_end - t_begin) * 4u);
  const uint32_t gm = p.G >= 32 ? 0xFFFFFFFFu : ((1u << p.G) - 1u);
  const int ds = DH / p.G;

  bf16x8 nxt[KS];
  uint32_t nmask = 0;
  int32_t noff = 0;
  auto load = [&](int tt) {
    const int tok = tt + l16;
    const bool ok = tok < t_end;
    const uint32_t o = static_cast<uint32_t>(tok - t_begin) * tstride + 16u * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) nxt[ks] = __builtin_bit_cast(bf16x8, bload16(r_v, ok ? o + 64u * ks : kOOB));
    if constexpr (PACK) {
      nmask = bload4(r_m, ok ? 4u * (tok - t_begin) : kOOB);
      // offsets are [B][T+1]: token (b, t) sits at b*(T+1)+t
      const int tk = ok ? tok : t_begin;
      const int b = tk / p.T;
      noff = p.offsets[static_cast<size_t>(tk) + b];
    }
  };
  int t0 = t_begin + 16 * w;
  if (t0 < t_end) load(t0);
  for (; t0 < t_end; t0 += 64) {
    bf16x8 cur[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) cur[ks] = nxt[ks];
    const uint32_t cmask = nmask & gm;
    const int32_t coff = noff;
    if (t0 + 64 < t_end) load(t0 + 64);
    // keep the R^T fragments in LDS: without this the compiler hoists the
    // loop-invariant LDS reads into ~128 registers and occupancy collapses
    asm volatile("" ::: "memory");
    f32x4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(Rt + (16 * m + l16) * LD + 32 * ks + 8 * g4);
        acc[m] = mfma_16x16x32(a, cur[ks], acc[m]);
      }
    }
    const int tok = t0 + l16;
    if (tok < t_end) {
      if constexpr (!PACK) {
        bf16* zr = static_cast<bf16*>(p.z) + (static_cast<size_t>(tok) * H + h) * DH + 4 * g4;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          bf16x4 o;
          o[0] = static_cast<bf16>(acc[m][0]);
          o[1] = static_cast<bf16>(acc[m][1]);
          o[2] = static_cast<bf16>(acc[m][2]);
          o[3] = static_cast<bf16>(acc[m][3]);
          *reinterpret_cast<bf16x4*>(zr + 16 * m) = o;
        }
      } else {
        const int b = tok / p.T;
        bf16* vb = static_cast<bf16*>(p.Vp) + (static_cast<size_t>(b) * H + h) * p.cap * ds;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int dim = 16 * m + 4 * g4;  // this lane's 4 outputs: dims dim..dim+3
          if (ds >= 4) {
            const int g = dim / ds;
            const int64_t slot = coff + __popc(cmask & ((1u << g) - 1u));
            if (((cmask >> g) & 1u) && slot < p.cap) {
              bf16x4 o;
              o[0] = static_cast<bf16>(acc[m][0]);
              o[1] = static_cast<bf16>(acc[m][1]);
              o[2] = static_cast<bf16>(acc[m][2]);
              o[3] = static_cast<bf16>(acc[m][3]);
              *reinterpret_cast<bf16x4*>(vb + slot * ds + (dim - g * ds)) = o;
            }
          } else {
            // 2-dim groups: the lane's outputs cover groups dim/2 and dim/2+1
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const int g = dim / 2 + u;
              const int64_t slot = coff + __popc(cmask & ((1u << g) - 1u));
              if (((cmask >> g) & 1u) && slot < p.cap)
                *reinterpret_cast<uint32_t*>(vb + slot * 2) = pack_bf16x2(acc[m][2 * u], acc[m][2 * u + 1]);
            }
          }
        }
      }
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
int rotate_tokens_per_wg(int ntok, int H) {
  // enough workgroups to fill 256 CUs several times over, but long enough
  // token runs to amortise staging R_h
  int tpw = 256;
  while (tpw > 64 && static_cast<long>((ntok + tpw - 1) / tpw) * H < 4096) tpw >>= 1;
  return tpw;
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
    p.tok_per_wg = rotate_tokens_per_wg(ntok, H);
    const dim3 grid(static_cast<unsigned>(((ntok + p.tok_per_wg - 1) / p.tok_per_wg) * H));
    if (dh == 128)
      hipLaunchKernelGGL((k_rotate_bf16<128, false>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((k_rotate_bf16<64, false>), grid, dim3(256), 0, s, p);
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
                              const uint32_t* mask, const int32_t* offsets, void* Vp, int64_t cap,
                              hipStream_t s) {
  const int ntok = B * T;
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
  if (bf16 && (dh == 128 || dh == 64) && dh / G >= 2) {
    p.tok_per_wg = rotate_tokens_per_wg(ntok, H);
    const dim3 grid(static_cast<unsigned>(((ntok + p.tok_per_wg - 1) / p.tok_per_wg) * H));
    if (dh == 128)
      hipLaunchKernelGGL((k_rotate_bf16<128, true>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((k_rotate_bf16<64, true>), grid, dim3(256), 0, s, p);
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
