// Value rotation into the orthogonal routing space, z = R_h^T v (Sec. 3.2).
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

// bf16 matrix-core rotation. Each workgroup owns one head h and a contiguous
// run of tokens. The product is computed transposed, Z^T = R_h^T V^T, so the
// streamed operand (the values, 16 B per lane straight from HBM) is the MFMA
// B fragment and every lane stores 4 consecutive outputs (8 B) of its token.
// R_h^T is staged once through LDS and then held in registers as A fragments
// (DH/16 x DH/32 fragments), so the token loop reads only v and writes only z.
// Workgroups of one head are placed on one XCD so R_h stays in its L2.
template <int DH>
__global__ __launch_bounds__(256) void k_rotate_bf16(const bf16* __restrict__ v,
                                                     const bf16* __restrict__ R,
                                                     bf16* __restrict__ z, int ntok, int H,
                                                     int tok_per_wg) {
  constexpr int MT = DH / 16, KS = DH / 32, LD = DH + 8;
  __shared__ __attribute__((aligned(16))) bf16 Rt[DH * LD];  // Rt[j][k] = R[k][j]
  int h, chunk;
  xcd_split(blockIdx.x, H, h, chunk);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const bf16* Rh = R + static_cast<size_t>(h) * DH * DH;
  {
    constexpr int NP = DH * DH / 8 / 256;  // 16-byte pieces of R_h per thread
    bf16x8 val[NP];
#pragma unroll
    for (int r = 0; r < NP; ++r) {
      const int pc = tid + 256 * r;
      val[r] = *reinterpret_cast<const bf16x8*>(Rh + (pc / (DH / 8)) * DH + (pc % (DH / 8)) * 8);
    }
#pragma unroll
    for (int r = 0; r < NP; ++r) {
      const int pc = tid + 256 * r;
      const int k = pc / (DH / 8), j0 = (pc % (DH / 8)) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) Rt[(j0 + e) * LD + k] = val[r][e];
    }
  }
  __syncthreads();
  bf16x8 af[MT][KS];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      af[m][ks] = *reinterpret_cast<const bf16x8*>(Rt + (16 * m + l16) * LD + 32 * ks + 8 * g4);

  const int t_begin = chunk * tok_per_wg;
  const int t_end = min(t_begin + tok_per_wg, ntok);
  // this workgroup's tokens of head h; rows past t_end load as zero
  const uint32_t tstride = static_cast<uint32_t>(H) * DH * 2;
  const rsrc_t r_v = make_rsrc(v + (static_cast<size_t>(t_begin) * H + h) * DH,
                               static_cast<uint32_t>(t_end - t_begin - 1) * tstride + DH * 2);
  int t0 = t_begin + 16 * w;
  bf16x8 nxt[KS];
  auto load = [&](int tt) {
    const int tok = tt + l16;
    const uint32_t o = static_cast<uint32_t>(tok - t_begin) * tstride + 16u * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) nxt[ks] = __builtin_bit_cast(bf16x8, bload16(r_v, tok < t_end ? o + 64u * ks : kOOB));
  };
  if (t0 < t_end) load(t0);
  for (; t0 < t_end; t0 += 64) {
    bf16x8 cur[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) cur[ks] = nxt[ks];
    if (t0 + 64 < t_end) load(t0 + 64);
    f32x4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc[m] = mfma_16x16x32(af[m][ks], cur[ks], acc[m]);
    }
    const int tok = t0 + l16;
    if (tok < t_end) {
      bf16* zr = z + (static_cast<size_t>(tok) * H + h) * DH + 4 * g4;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        bf16x4 o;
        o[0] = static_cast<bf16>(acc[m][0]);
        o[1] = static_cast<bf16>(acc[m][1]);
        o[2] = static_cast<bf16>(acc[m][2]);
        o[3] = static_cast<bf16>(acc[m][3]);
        *reinterpret_cast<bf16x4*>(zr + 16 * m) = o;
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

}  // namespace

hipError_t launch_rotate(bool bf16, int ntok, int H, int dh, const void* v, const void* R, void* z,
                         hipStream_t s) {
  if (ntok == 0 || H == 0) return hipSuccess;
  if (bf16 && (dh == 128 || dh == 64)) {
    // enough workgroups to fill 256 CUs several times over, but long enough
    // token runs to amortise staging R_h
    int tpw = 256;
    while (tpw > 64 && static_cast<long>((ntok + tpw - 1) / tpw) * H < 2048) tpw >>= 1;
    const int chunks = (ntok + tpw - 1) / tpw;
    const dim3 grid(static_cast<unsigned>(chunks * H));
    if (dh == 128)
      hipLaunchKernelGGL(k_rotate_bf16<128>, grid, dim3(256), 0, s, static_cast<const rolesub::bf16*>(v),
                         static_cast<const rolesub::bf16*>(R), static_cast<rolesub::bf16*>(z), ntok, H, tpw);
    else
      hipLaunchKernelGGL(k_rotate_bf16<64>, grid, dim3(256), 0, s, static_cast<const rolesub::bf16*>(v),
                         static_cast<const rolesub::bf16*>(R), static_cast<rolesub::bf16*>(z), ntok, H, tpw);
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

}  // namespace rolesub
