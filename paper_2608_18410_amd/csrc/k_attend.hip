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

// ---------------------------------------------------------------------------
// bf16 matrix-core kernel. One workgroup = one (sample, head) and up to 64
// queries; wave w owns queries 16w..16w+15. KV tokens stream in tiles of 32:
//   * K tile (32 x DH) -> LDS, shared by the four waves;
//   * the tile's packed groups -> a zero-filled, transposed LDS tile
//     Zt[dim][token] (token pairs packed in one dword);
//   * S^T = K Q^T on MFMA (queries are the B operand held in registers), so
//     each lane owns one query column and 8 token rows;
//   * online softmax per query: 8 values in-lane, then 2 cross-lane steps;
//   * O^T += Z~^T P^T on MFMA. The lane's own softmax values form the P^T
//     fragment directly once the A fragment lists its tokens in the same
//     order (tokens 4q..4q+3 and 16+4q..16+4q+3 of the tile).
// After the last tile, O^T = R_h U^T (one more MFMA chain, U in bf16) and
// each lane stores 4 consecutive outputs of its query.
template <int DH>
__global__ __launch_bounds__(256) void k_attend_bf16(AttendParams p) {
  constexpr int TK = 32, MT = DH / 16, KS = DH / 32, KLD = DH + 8, ZLD = TK / 2 + 2;
  __shared__ __attribute__((aligned(16))) bf16 Ks[TK * KLD];
  __shared__ __attribute__((aligned(16))) uint32_t Zt[DH * ZLD];
  int h, b;
  xcd_split(blockIdx.x, p.H, h, b);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int T = p.T, H = p.H, G = p.G, ds = DH / G;
  const uint32_t gm = group_mask(G);
  const bf16* q = static_cast<const bf16*>(p.q);
  const bf16* k = static_cast<const bf16*>(p.k);
  const int qq = blockIdx.y * 64 + 16 * w + l16;
  const bool qvalid = qq < p.Tq;
  const bf16x8 zero8 = {};

  bf16x8 qf[KS];
  {
    const bf16* qr = q + ((static_cast<size_t>(b) * p.Tq + (qvalid ? qq : 0)) * H + h) * DH + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = qvalid ? *reinterpret_cast<const bf16x8*>(qr + 32 * ks) : zero8;
  }
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = p.scale * 1.4426950408889634f;  // softmax in base 2

  const int pp = tid & 15, cc = tid >> 4;  // Zt fill: token pair, 8-dim chunk
  const int32_t* ob = p.offsets + static_cast<size_t>(b) * (T + 1);
  const uint32_t* mb = p.mask + static_cast<size_t>(b) * T;
  const bf16* Vh = static_cast<const bf16*>(p.Vp) + (static_cast<size_t>(b) * H + h) * p.cap * ds;
  const bf16* kb = k + (static_cast<size_t>(b) * T * H + h) * DH;

  for (int t0 = 0; t0 < T; t0 += TK) {
    // ---- K tile
#pragma unroll
    for (int r = 0; r < TK * DH / 8 / 256; ++r) {
      const int pc = tid + 256 * r;
      const int row = pc / (DH / 8), c8 = pc % (DH / 8);
      const int t = t0 + row;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (t < T) val = *reinterpret_cast<const u32x4*>(kb + static_cast<size_t>(t) * H * DH + 8 * c8);
      *reinterpret_cast<u32x4*>(Ks + row * KLD + 8 * c8) = val;
    }
    // ---- routed value tile, transposed, dropped groups = 0
    if (cc < DH / 8) {
      uint32_t ev[2][4];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        ev[e][0] = ev[e][1] = ev[e][2] = ev[e][3] = 0u;
        const int t = t0 + 2 * pp + e;
        if (t < T) {
          const uint32_t m = mb[t] & gm;
          const int o = ob[t];
          if (ds >= 8) {
            const int g = (8 * cc) / ds;
            if ((m >> g) & 1u) {
              const int64_t slot = o + __popc(m & ((1u << g) - 1u));
              if (slot < p.cap) {
                const u32x4 val = *reinterpret_cast<const u32x4*>(Vh + slot * ds + (8 * cc - g * ds));
                ev[e][0] = val[0]; ev[e][1] = val[1]; ev[e][2] = val[2]; ev[e][3] = val[3];
              }
            }
          } else if (ds == 4) {
            // the 8-dim chunk spans two groups of 4
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const int g = 2 * cc + u;
              if ((m >> g) & 1u) {
                const int64_t slot = o + __popc(m & ((1u << g) - 1u));
                if (slot < p.cap) {
                  const u32x2 val = *reinterpret_cast<const u32x2*>(Vh + slot * 4);
                  ev[e][2 * u] = val[0];
                  ev[e][2 * u + 1] = val[1];
                }
              }
            }
          } else {
            // ds == 2: the chunk spans four groups of 2
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int g = 4 * cc + u;
              if ((m >> g) & 1u) {
                const int64_t slot = o + __popc(m & ((1u << g) - 1u));
                if (slot < p.cap) ev[e][u] = *reinterpret_cast<const uint32_t*>(Vh + slot * 2);
              }
            }
          }
        }
      }
      uint32_t* zc = Zt + 8 * cc * ZLD + pp;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        zc[(2 * j) * ZLD] = (ev[0][j] & 0xFFFFu) | (ev[1][j] << 16);
        zc[(2 * j + 1) * ZLD] = (ev[0][j] >> 16) | (ev[1][j] & 0xFFFF0000u);
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T (rows: tile tokens 16*m2 + 4*g4 + i; column: this lane's query)
    f32x4 s[2];
#pragma unroll
    for (int m2 = 0; m2 < 2; ++m2) {
      s[m2] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(Ks + (16 * m2 + l16) * KLD + 32 * ks + 8 * g4);
        s[m2] = mfma_16x16x32(a, qf[ks], s[m2]);
      }
    }
    // ---- online softmax (base 2)
    float mx = -INFINITY;
#pragma unroll
    for (int m2 = 0; m2 < 2; ++m2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 16 * m2 + 4 * g4 + i;
        const float x = t < T ? s[m2][i] * sl2 : -INFINITY;
        s[m2][i] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
    bf16x8 pb;
#pragma unroll
    for (int m2 = 0; m2 < 2; ++m2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pr = exp2f(s[m2][i] - m_new);
        psum += pr;
        pb[4 * m2 + i] = static_cast<bf16>(pr);
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    // ---- O^T += Z~^T P^T
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const uint32_t* zr = Zt + (16 * m + l16) * ZLD;
      const u32x2 lo = *reinterpret_cast<const u32x2*>(zr + 2 * g4);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(zr + 8 + 2 * g4);
      const u32x4 av = {lo[0], lo[1], hi[0], hi[1]};
      acc[m] = mfma_16x16x32(__builtin_bit_cast(bf16x8, av), pb, acc[m] * alpha);
    }
    __syncthreads();
  }

  // ---- normalise and rotate back: O^T = R_h U^T
  float lsum = l_run + __shfl_xor(l_run, 16, kWave);
  lsum += __shfl_xor(lsum, 32, kWave);
  const float inv = 1.f / lsum;
  bf16x8 ub[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ub[ks][i] = static_cast<bf16>(acc[2 * ks][i] * inv);
      ub[ks][4 + i] = static_cast<bf16>(acc[2 * ks + 1][i] * inv);
    }
  const bf16* Rh = static_cast<const bf16*>(p.R) + static_cast<size_t>(h) * DH * DH;
  const size_t obase = ((static_cast<size_t>(b) * p.Tq + (qvalid ? qq : 0)) * H + h) * DH + 4 * g4;
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    const bf16* rr = Rh + (16 * m + l16) * DH + 4 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x2 lo = *reinterpret_cast<const u32x2*>(rr + 32 * ks);
      const u32x2 hi = *reinterpret_cast<const u32x2*>(rr + 32 * ks + 16);
      const u32x4 av = {lo[0], lo[1], hi[0], hi[1]};
      o = mfma_16x16x32(__builtin_bit_cast(bf16x8, av), ub[ks], o);
    }
    if (qvalid) {
      if (p.out_f32) {
        *reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + obase + 16 * m) = o;
      } else {
        bf16x4 ov;
        ov[0] = static_cast<bf16>(o[0]);
        ov[1] = static_cast<bf16>(o[1]);
        ov[2] = static_cast<bf16>(o[2]);
        ov[3] = static_cast<bf16>(o[3]);
        *reinterpret_cast<bf16x4*>(static_cast<bf16*>(p.out) + obase + 16 * m) = ov;
      }
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
  for (int t = 0; t < T; ++t) {
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
    const dim3 grid(static_cast<unsigned>(p.B * p.H), static_cast<unsigned>((p.Tq + 63) / 64));
    if (p.dh == 128)
      hipLaunchKernelGGL(k_attend_bf16<128>, grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL(k_attend_bf16<64>, grid, dim3(256), 0, s, p);
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
