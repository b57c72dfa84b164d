// Role-conditioned routing scores and group selection.
//
//   a     = softmax(W_r h + b_r)                       (Eq. latentrole)
//   gamma = router(h, a, pooled language state)        (Sec. 3.4, Eq. routingscore)
//   keep the K_i highest-scoring groups                (Sec. 3.4, Sec. 3.5)
//
// Two algebraic rewrites keep per-token work small; both are exact in real
// arithmetic:
//   * the language term depends only on the sample, so it is computed once per
//     sample (cb), not once per token;
//   * the role-mixed vector enters linearly: W1_e (sum_c a_c E_c) = F a with
//     F = W1_e E^T (Hr x C), computed once per call.
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

constexpr int kLang = 1;

// ---------------------------------------------------------------------------
// Language pool (Sec. 3.4): hbar[b] = mean of the sample's language rows of h
// (zero when it has none). 1D grid: B x ceil(d / (64*VEC)) blocks. A block
// owns 64*VEC columns of one sample; its language rows are listed in LDS in
// ascending order, the four waves take every fourth listed row, and the wave
// partial sums are added in wave order (deterministic).
//
// With PCB (bf16 MLP2 router, d a multiple of 512, Hr 64 or 128) the
// block also forms its columns' share of the language term,
//   pcb[cblk][b][j] = W1[j, d+d_e + cols] . hbar[b][cols],
// while the pooled columns are still in registers, and blocks past B*ncb fold
// the role term F = W1_e E^T (one thread per entry). cb is then the sum of the
// ncb shares plus b1, added by the MFMA router itself or by k_route_cbsum.
template <class T, bool PCB>
__global__ __launch_bounds__(256) void k_route_pool(RouteParams p) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int TCH = 1024;  // tokens listed per pass
  constexpr int RU = 16;     // row loads in flight per wave
  __shared__ int s_rows[TCH];
  __shared__ int s_wcnt[4];
  __shared__ float s_part[4][64 * VEC];
  const int ncb = (p.d + 64 * VEC - 1) / (64 * VEC);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // F[j][c] = W1[j, d : d+d_e] . E[c] (entry e = j*C + c); d_e a multiple of
  // 8, rows 16-byte aligned
  auto fold_F = [&](int e) {
    const int j = e / p.C, c = e - j * p.C;
    const bool ok = j < p.Hr;
    const uint32_t W1s = 2u * p.d + p.d_e;
    const rsrc_t r_w = make_rsrc(p.W1, static_cast<uint32_t>(p.Hr) * W1s * sizeof(T));
    const rsrc_t r_e = make_rsrc(p.E, static_cast<uint32_t>(p.C * p.d_e) * sizeof(T));
    const uint32_t ow = (static_cast<uint32_t>(j) * W1s + p.d) * sizeof(T);
    const uint32_t oe = static_cast<uint32_t>(c * p.d_e) * sizeof(T);
    float acc = 0.f;
    // 16 loads of each operand in flight: one round trip for d_e <= 16*VEC
    for (int m0 = 0; m0 < p.d_e; m0 += 16 * VEC) {
      u32x4 wv[16], ev[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const bool in = ok && m0 + u * VEC < p.d_e;
        const uint32_t m = static_cast<uint32_t>(m0 + u * VEC) * sizeof(T);
        wv[u] = bload16(r_w, oob_unless(in, ow + m));
        ev[u] = bload16(r_e, oob_unless(in, oe + m));
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const T* a = reinterpret_cast<const T*>(&wv[u]);
        const T* x = reinterpret_cast<const T*>(&ev[u]);
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc = fmaf(tof(a[i]), tof(x[i]), acc);
      }
    }
    if (ok) p.F[j * p.C + c] = acc;
  };
  if (PCB && blockIdx.x >= static_cast<unsigned>(p.B * ncb)) {
    const int fb = blockIdx.x - p.B * ncb;
    fold_F(fb * 256 + tid);
    // the split-K router's per-tile counters start each call at zero
    if (p.rcnt) {
      const int ntiles = static_cast<int>((static_cast<size_t>(p.B) * p.T + kRouteSkTok - 1) / kRouteSkTok);
      const int nfb = (p.Hr * p.C + 255) / 256;
      for (int i = fb * 256 + tid; i < ntiles; i += nfb * 256) p.rcnt[i] = 0;
    }
    return;
  }
  const int b = blockIdx.x / ncb, cb = blockIdx.x % ncb;
  const uint8_t* ty = p.types + static_cast<size_t>(b) * p.T;
  const int col = cb * 64 * VEC + lane * VEC;
  u32x4 wraw[PCB ? 2 : 1][16];
  const bool vec = (p.d % VEC) == 0;
  const T* hsample = static_cast<const T*>(p.h) + static_cast<size_t>(b) * p.T * p.d;
  const rsrc_t r_h = make_rsrc(hsample, static_cast<uint32_t>(p.T) * p.d * sizeof(T));
  float acc[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
  int n_total = 0;
  for (int c0 = 0; c0 < p.T; c0 += TCH) {
    const int nc = min(TCH, p.T - c0);
    // ascending list of this chunk's language rows (wave ballots + prefix)
    int base = 0;
    for (int s0 = 0; s0 < nc; s0 += 256) {
      const int t = c0 + s0 + tid;
      const bool lang = (s0 + tid < nc) && ty[t] == kLang;
      const uint64_t bal = __ballot(lang);
      const int pre = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) s_wcnt[w] = __popcll(bal);
      __syncthreads();
      int woff = base;
      for (int i = 0; i < w; ++i) woff += s_wcnt[i];
      if (lang) s_rows[woff + pre] = t;
      base += s_wcnt[0] + s_wcnt[1] + s_wcnt[2] + s_wcnt[3];
      __syncthreads();
    }
    n_total += base;
    if (vec && col < p.d) {
      // wave w sums listed rows w, w+4, ...; RU loads in flight per step
      for (int i0 = w; i0 < base; i0 += 4 * RU) {
        u32x4 raw[RU];
#pragma unroll
        for (int u = 0; u < RU; ++u) {
          const int i = i0 + 4 * u;
          raw[u] = bload16(r_h, i < base ? static_cast<uint32_t>((static_cast<size_t>(s_rows[i]) * p.d + col) * sizeof(T)) : kOOB);
        }
#pragma unroll
        for (int u = 0; u < RU; ++u) {
          const T* v = reinterpret_cast<const T*>(&raw[u]);
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] += tof(v[e]);
        }
      }
    } else if (!vec) {
      for (int i = w; i < base; i += 4)
        for (int e = 0; e < VEC; ++e)
          if (col + e < p.d) acc[e] += tof(hsample[static_cast<size_t>(s_rows[i]) * p.d + col + e]);
    }
    __syncthreads();
  }
  if constexpr (PCB) {
    // The language-term weights this block needs (Hr <= 128 rows of its
    // 64*VEC columns), requested after the row loads: loads of a wave
    // complete in issue order, so requested first (128 KB per block) they
    // held back the token types and language rows behind them.
    const uint32_t W1s = 2u * p.d + p.d_e;
    const rsrc_t r_w = make_rsrc(p.W1, static_cast<uint32_t>(p.Hr) * W1s * sizeof(T));
    const uint32_t ol = static_cast<uint32_t>(p.d + p.d_e + col) * sizeof(T);
#pragma unroll
    for (int jb = 0; jb < 2; ++jb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int j = 64 * jb + 16 * w + i;
        wraw[jb][i] = bload16(r_w, oob_unless(j < p.Hr, static_cast<uint32_t>(j) * W1s * sizeof(T) + ol));
      }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) s_part[w][lane * VEC + e] = acc[e];
  __syncthreads();
  const float inv = n_total ? 1.f / static_cast<float>(n_total) : 0.f;
  for (int i = tid; i < 64 * VEC; i += 256) {
    const int c = cb * 64 * VEC + i;
    if (c < p.d)
      p.hbar[static_cast<size_t>(b) * p.d + c] = (((s_part[0][i] + s_part[1][i]) + s_part[2][i]) + s_part[3][i]) * inv;
  }
  if constexpr (PCB) {
    // lane holds pooled columns col..col+VEC-1; wave w takes rows jb+16*w+i
    __shared__ float s_red[4][16][65];
    float hv[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int i = lane * VEC + e;
      hv[e] = (((s_part[0][i] + s_part[1][i]) + s_part[2][i]) + s_part[3][i]) * inv;
    }
    float* dst = p.pcb + (static_cast<size_t>(cb) * p.B + b) * p.Hr;
#pragma unroll
    for (int jh = 0; jh < 2; ++jh) {
      const int jb = 64 * jh;
      if (jb >= p.Hr) break;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const T* v = reinterpret_cast<const T*>(&wraw[jh][i]);
        float pd = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) pd = fmaf(tof(v[e]), hv[e], pd);
        s_red[w][i][lane] = pd;
      }
      __syncthreads();
      // lane (r = lane/4, q = lane%4) adds lanes 16q..16q+15 of row r, then the
      // four quarters are combined as (q0+q1)+(q2+q3)
      const int r = lane >> 2, q = lane & 3;
      float sum = 0.f;
#pragma unroll
      for (int k = 0; k < 16; ++k) sum += s_red[w][r][16 * q + k];
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      if (q == 0) dst[jb + 16 * w + r] = sum;
      __syncthreads();
    }
  }
}

// cb[b][j] = b1[j] + sum over column blocks s (in order) of pcb[s][b][j].
// One thread per (b, j).
__global__ __launch_bounds__(256) void k_route_cbsum(RouteParams p, int ncb) {
  const int n = p.B * p.Hr;
  const int i = blockIdx.x * 256 + threadIdx.x;
  const bool ok = i < n;
  const rsrc_t r_p = make_rsrc(p.pcb, static_cast<uint32_t>(ncb) * n * 4u);
  float acc = 0.f;
  for (int s0 = 0; s0 < ncb; s0 += 8) {
    uint32_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = bload4(r_p, oob_unless(ok && s0 + u < ncb, static_cast<uint32_t>((s0 + u) * n + i) * 4u));
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += __uint_as_float(v[u]);
  }
  if (ok) p.cb[i] = acc + tof(static_cast<const bf16*>(p.b1)[i % p.Hr]);
}

// Per-sample language term and folded role term. 1D grid:
//   blocks [0, B*nrb): 8 output rows of one sample (2 per wave),
//     MLP2:     cb[b][j] = W1[j, d+d_e : 2d+d_e] . hbar[b] + b1[j]
//     ADDITIVE: cb[b][s] = alpha_lang (W_lang[s] . hbar[b] + b_lang[s])
//   blocks [B*nrb, ...): F rows, one per wave,
//     MLP2:     F[j][c] = W1[j, d : d+d_e] . E[c]      (so W1_e e = F a)
//     ADDITIVE: F[s][c] = alpha_role W_role[s][c]
template <class T>
__global__ __launch_bounds__(256) void k_route_proj(RouteParams p) {
  extern __shared__ float hs[];
  constexpr int VEC = 16 / sizeof(T);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nout = p.kind == 0 ? p.Hr : p.G;
  const int nrb = (nout + 7) / 8;
  const size_t W1s = 2 * static_cast<size_t>(p.d) + p.d_e;
  if (blockIdx.x >= static_cast<unsigned>(p.B * nrb)) {
    const int j = (blockIdx.x - p.B * nrb) * 4 + wave;
    if (p.kind == 0) {
      // E staged in LDS (f32) once per block; each wave then dots its W1_e row
      // with every role vector. Loads are batched before use.
      const T* E = static_cast<const T*>(p.E);
      const int ne = p.C * p.d_e;
      float* Es = hs;  // p.d floats of dynamic LDS; C * d_e <= d is checked on the host
      for (int i0 = 0; i0 < ne; i0 += 256 * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = i0 + u * 256 + tid;
          v[u] = i < ne ? tof(E[i]) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = i0 + u * 256 + tid;
          if (i < ne) Es[i] = v[u];
        }
      }
      __syncthreads();
      if (j >= p.Hr) return;
      const T* w1 = static_cast<const T*>(p.W1) + j * W1s + p.d;
      for (int m0 = 0; m0 < p.d_e; m0 += 64 * 4) {
        float wv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int m = m0 + u * 64 + lane;
          wv[u] = m < p.d_e ? tof(w1[m]) : 0.f;
        }
        for (int c = 0; c < p.C; ++c) {
          float acc = 0.f;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int m = m0 + u * 64 + lane;
            if (m < p.d_e) acc += wv[u] * Es[c * p.d_e + m];
          }
          acc = wave_sum(acc);
          if (lane == 0) {
            if (m0 == 0) p.F[j * p.C + c] = acc;
            else p.F[j * p.C + c] += acc;
          }
        }
      }
    } else {
      if (j >= p.G) return;
      const T* Wro = static_cast<const T*>(p.W_role);
      for (int c = lane; c < p.C; c += 64) p.F[j * p.C + c] = p.alpha_role * tof(Wro[j * p.C + c]);
    }
    return;
  }
  const int b = blockIdx.x / nrb, j0 = (blockIdx.x % nrb) * 8;
  const float* hb = p.hbar + static_cast<size_t>(b) * p.d;
  const bool vec = (p.d % (64 * VEC)) == 0;
  // In the vector path lane L multiplies weights k = BK*i + VEC*L + e (one
  // 16-byte load) with hbar[k]; hbar is stored lane-interleaved,
  // hs[BK*i + 64*e + L], so those LDS reads hit consecutive banks.
  constexpr int BK = 64 * VEC;
  auto pos = [&](int k) { return vec ? (k / BK) * BK + (k % VEC) * 64 + (k % BK) / VEC : k; };
  {
    // stage hbar: all of a thread's loads issued before its LDS stores
    const rsrc_t r_hb = make_rsrc(hb, static_cast<uint32_t>(p.d) * 4u);
    for (int k0 = 0; k0 < p.d; k0 += 256 * 4 * 8) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + (u * 256 + tid) * 4;
        v[u] = bload16(r_hb, k + 4 <= p.d ? 4u * k : kOOB);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + (u * 256 + tid) * 4;
        if (k + 4 <= p.d) {
          const u32x4 x = v[u];
          hs[pos(k)] = __uint_as_float(x.x);
          hs[pos(k + 1)] = __uint_as_float(x.y);
          hs[pos(k + 2)] = __uint_as_float(x.z);
          hs[pos(k + 3)] = __uint_as_float(x.w);
        }
      }
    }
    for (int k = (p.d / 4) * 4 + tid; k < p.d; k += 256) hs[pos(k)] = hb[k];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int j = j0 + 2 * wave + r;
    if (j >= nout) break;
    const T* wrow;
    float bias, scale;
    if (p.kind == 0) {
      wrow = static_cast<const T*>(p.W1) + j * W1s + p.d + p.d_e;
      bias = tof(static_cast<const T*>(p.b1)[j]);
      scale = 1.f;
    } else {
      wrow = static_cast<const T*>(p.W_lang) + static_cast<size_t>(j) * p.d;
      bias = tof(static_cast<const T*>(p.b_lang)[j]);
      scale = p.alpha_lang;
    }
    float acc = 0.f;
    if (vec && (reinterpret_cast<uintptr_t>(wrow) & 15) == 0) {
#pragma unroll 8
      for (int k0 = 0; k0 < p.d; k0 += BK) {
        const u32x4 raw = *reinterpret_cast<const u32x4*>(wrow + k0 + lane * VEC);
        const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc += tof(v[i]) * hs[k0 + 64 * i + lane];
      }
    } else {
      for (int k = lane; k < p.d; k += 64) acc += tof(wrow[k]) * hs[pos(k)];
    }
    acc = wave_sum(acc);
    if (lane == 0) p.cb[static_cast<size_t>(b) * nout + j] = scale * (acc + bias);
  }
}

__device__ __forceinline__ void write_selection(const RouteParams& p, size_t tok, uint32_t m) {
  p.mask[tok] = m;
  if (p.count) p.count[tok] = static_cast<uint8_t>(__popc(m));
  if (p.idx) {
    uint8_t* o = p.idx + tok * p.G;
    int r = 0;
    for (int s = 0; s < p.G; ++s)
      if ((m >> s) & 1u) o[r++] = static_cast<uint8_t>(s);
    for (; r < p.G; ++r) o[r] = 0xFF;
  }
}

// Full selection for one token whose G scores sit in registers of one thread.
// NP >= G bounds the unrolled loops.
template <int NP>
__device__ __forceinline__ uint32_t select_token(const RouteParams& p, const float* g, int type) {
  int n_above = 0;
#pragma unroll
  for (int s = 0; s < NP; ++s)
    if (s < p.G) n_above += g[s] > p.tau;
  const int K = budget_k(p.mode, p.k_by_type, type, p.tau, p.kmin, p.kmax, p.G, n_above);
  if (p.mode == 1 && K == n_above) {
    // Every group above the threshold ranks before every group at or below it,
    // so the top-K set is exactly the groups above the threshold.
    uint32_t m = 0;
#pragma unroll
    for (int s = 0; s < NP; ++s)
      if (s < p.G && g[s] > p.tau) m |= 1u << s;
    return m;
  }
  return top_k_pairs<NP>(g, p.G, K);
}

// ---------------------------------------------------------------------------
// Selection only, from given scores. A one-wave workgroup takes kSelTok
// consecutive tokens: their scores are read (and copied to scores_out) with
// consecutive lanes on consecutive 16-byte pieces, all of a lane's pieces in
// flight together, staged in LDS with a row stride of G + 1 floats (odd, so
// one token per lane reads its row without bank conflicts), ranked one token
// per lane, and the idx bytes are staged in LDS and written out in 16-byte
// pieces. Reading a token's G scores per lane directly would put consecutive
// lanes G * 4 bytes apart. Small workgroups keep many in flight per CU. The
// ranking is vector-ALU bound (a wave runs it when any of its tokens needs
// it); NP >= G sizes its unrolled pairs, and the occupancy hint keeps the
// register count where no spills occur.
constexpr int kSelTok = 64;
constexpr int kSelPieces = kSelTok * 32 / 4 / kSelTok;  // 16-byte score pieces per lane at G = 32

__device__ __forceinline__ bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; }

template <int NP>
__global__ __launch_bounds__(kSelTok) __attribute__((amdgpu_waves_per_eu(NP == 32 ? 3 : 5))) void k_select(RouteParams p) {
  __shared__ __attribute__((aligned(16))) float sg[kSelTok * 33];  // scores, then the idx bytes
  uint8_t* sidx = reinterpret_cast<uint8_t*>(sg);
  const size_t N = static_cast<size_t>(p.B) * p.T;
  const size_t tok0 = static_cast<size_t>(blockIdx.x) * kSelTok;
  const int tid = threadIdx.x, G = p.G;
  const int ntok = static_cast<int>(N - tok0 < kSelTok ? N - tok0 : kSelTok);
  const int nval = ntok * G;
  const float* src = p.scores_in + tok0 * G;
  float* dst = p.scores_out ? p.scores_out + tok0 * G : nullptr;
  const bool vec = (G & 3) == 0 && aligned16(p.scores_in) && (!dst || aligned16(p.scores_out));
  if (vec) {
    // tok0 * G * 4 bytes is a multiple of 16; at most kSelPieces pieces per lane
    f32x4 v[kSelPieces];
#pragma unroll
    for (int i = 0; i < kSelPieces; ++i) {
      const int q = tid + i * kSelTok;
      if (4 * q < nval) v[i] = *reinterpret_cast<const f32x4*>(src + 4 * q);
    }
#pragma unroll
    for (int i = 0; i < kSelPieces; ++i) {
      const int q = tid + i * kSelTok;
      if (4 * q < nval) {
        if (dst) *reinterpret_cast<f32x4*>(dst + 4 * q) = v[i];
        const int t = (4 * q) / G, s0 = 4 * q - t * G;  // the 4 values share a token (G % 4 == 0)
#pragma unroll
        for (int j = 0; j < 4; ++j) sg[t * (G + 1) + s0 + j] = v[i][j];
      }
    }
  } else {
    for (int e = tid; e < nval; e += kSelTok) {
      const float x = src[e];
      if (dst) dst[e] = x;
      const int t = e / G;
      sg[t * (G + 1) + (e - t * G)] = x;
    }
  }
  __syncthreads();
  const bool valid = tid < ntok;
  float g[NP];
#pragma unroll
  for (int s = 0; s < NP; ++s) g[s] = (valid && s < G) ? sg[tid * (G + 1) + s] : 0.f;
  const size_t tok = tok0 + tid;
  uint32_t m = 0;
  if (valid) {
    m = select_token<NP>(p, g, p.types ? p.types[tok] : 0);
    p.mask[tok] = m;
    if (p.count) p.count[tok] = static_cast<uint8_t>(__popc(m));
  }
  if (p.idx) {
    __syncthreads();  // every lane has its scores in registers before sidx overwrites them
    if (valid) {
      uint8_t* row = sidx + tid * G;
      int r = 0;
      for (int s = 0; s < G; ++s)
        if ((m >> s) & 1u) row[r++] = static_cast<uint8_t>(s);
      for (; r < G; ++r) row[r] = 0xFF;
    }
    __syncthreads();
    // tok0 * G bytes is a multiple of 64: 16-byte pieces, then the tail
    const int nb = ntok * G;
    uint8_t* out = p.idx + tok0 * G;
    const int nv = aligned16(p.idx) ? nb / 16 : 0;
    for (int q = tid; q < nv; q += kSelTok)
      *reinterpret_cast<u32x4*>(out + 16 * q) = *reinterpret_cast<const u32x4*>(sidx + 16 * q);
    for (int e = nv * 16 + tid; e < nb; e += kSelTok) out[e] = sidx[e];
  }
}

// ---------------------------------------------------------------------------
// Generic router: one workgroup per token, vector ALU. Any shape, either
// router kind; the f32 path and unusual bf16 shapes use it.
template <class T>
__global__ __launch_bounds__(256) void k_route_generic(RouteParams p) {
  extern __shared__ float sh[];
  __shared__ float a[64];
  const int tid = threadIdx.x;
  const size_t tok = blockIdx.x;
  const int b = static_cast<int>(tok / p.T);
  const int d = p.d, C = p.C, G = p.G;
  const int nmain = p.kind == 0 ? p.Hr : G;
  float* hs = sh;
  float* dots = hs + d;
  float* gl = dots + nmain + C;
  float* gam = gl + (p.kind == 0 ? p.Hr : 0);
  const T* h = static_cast<const T*>(p.h) + tok * d;
  for (int k = tid; k < d; k += 256) hs[k] = tof(h[k]);
  __syncthreads();
  const size_t W1s = 2 * static_cast<size_t>(d) + p.d_e;
  for (int o = tid; o < nmain + C; o += 256) {
    const T* wrow;
    if (o < nmain)
      wrow = p.kind == 0 ? static_cast<const T*>(p.W1) + o * W1s
                         : static_cast<const T*>(p.W_tok) + static_cast<size_t>(o) * d;
    else
      wrow = static_cast<const T*>(p.W_r) + static_cast<size_t>(o - nmain) * d;
    float acc = 0.f;
    for (int k = 0; k < d; ++k) acc += tof(wrow[k]) * hs[k];
    dots[o] = acc;
  }
  __syncthreads();
  if (tid == 0) {
    const T* br = static_cast<const T*>(p.b_r);
    float mx = -INFINITY;
    for (int c = 0; c < C; ++c) mx = fmaxf(mx, dots[nmain + c] + tof(br[c]));
    float sm = 0.f;
    for (int c = 0; c < C; ++c) {
      a[c] = expf(dots[nmain + c] + tof(br[c]) - mx);
      sm += a[c];
    }
    for (int c = 0; c < C; ++c) a[c] /= sm;
    if (p.priority) {
      const T* wp = static_cast<const T*>(p.w_pri);
      float pr = 0.f;
      for (int c = 0; c < C; ++c) pr = fmaf(tof(wp[c]), a[c], pr);
      p.priority[tok] = pr;
    }
  }
  __syncthreads();
  if (p.kind == 0) {
    for (int j = tid; j < p.Hr; j += 256) {
      float x = dots[j] + p.cb[static_cast<size_t>(b) * p.Hr + j];
      for (int c = 0; c < C; ++c) x += p.F[j * C + c] * a[c];
      gl[j] = gelu_exact(x);
    }
    __syncthreads();
    const T* W2 = static_cast<const T*>(p.W2);
    const T* b2 = static_cast<const T*>(p.b2);
    for (int s = tid; s < G; s += 256) {
      float acc = 0.f;
      for (int j = 0; j < p.Hr; ++j) acc += tof(W2[static_cast<size_t>(s) * p.Hr + j]) * gl[j];
      gam[s] = acc + tof(b2[s]);
    }
  } else {
    const T* bt = static_cast<const T*>(p.b_tok);
    for (int s = tid; s < G; s += 256) {
      float x = dots[s] + tof(bt[s]);
      float r = 0.f;
      for (int c = 0; c < C; ++c) r += p.F[s * C + c] * a[c];
      gam[s] = x + r + p.cb[static_cast<size_t>(b) * G + s];
    }
  }
  __syncthreads();
  if (tid == 0) {
    float g[32];
#pragma unroll
    for (int s = 0; s < 32; ++s) g[s] = s < G ? gam[s] : 0.f;
    if (p.mask) write_selection(p, tok, select_token<32>(p, g, p.types[tok]));
    if (p.scores_out)
      for (int s = 0; s < G; ++s) p.scores_out[tok * G + s] = gam[s];
  }
}

// ---------------------------------------------------------------------------
// bf16 matrix-core router (MLP2, Hr = 128, C <= 16, d % 64 == 0).
//
// The token-independent product is computed transposed: for 64 tokens per
// workgroup, [W1_h ; W_r] (144 x d, rows 128+C.. zero) times h^T (d x 64) on
// 16x16x32 bf16 MFMA with f32 accumulation. The operands stream through a
// ring of kRtNB LDS stages, each holding one 64-column chunk of the 144
// weight rows and of the 64 token rows. Stages are filled by asynchronous
// LDS DMA (16 bytes per lane) issued kRtNB-1 chunks ahead, so about 100 KB
// per workgroup is in flight without spending registers. Rows are stored with
// their 16-byte pieces XOR-swizzled (piece c of row r at c ^ ((r >> 1) & 7)),
// which makes the fragment reads of 16 consecutive rows conflict-free.
// After the K loop lane (t, q) of wave w holds 36 outputs of token 16w + t:
// hidden units 16m+4q+i (m < 8) and role logits 4q+i (m = 8). The epilogue
// (role softmax, F a + cb, GELU, W2, selection) runs on those registers with
// the four lanes of a token exchanging partial sums by cross-lane shuffles.
constexpr int kRtTok = 64, kRtKc = 64, kRtRows = 144, kRtNB = 5;
constexpr int kRtWBytes = kRtRows * 128, kRtHBytes = kRtTok * 128, kRtStage = kRtWBytes + kRtHBytes;
constexpr int kRtLoads = kRtRows / 8 + kRtTok / 8;  // 1 KB wave-loads per stage (26)

__device__ __forceinline__ int rt_swz(int r) { return (r >> 1) & 7; }

// Epilogue operands, written into the (then idle) ring after the K loop:
// F zero-padded to 16 role columns and W2 transposed to [Hr][GP], both with a
// row stride of 4 extra floats so that the 4 rows read by one instruction
// (lanes of one token quarter share a row) fall on distinct LDS banks.
constexpr int kFsStride = 20;

template <int GP, bool PS>
__global__ __launch_bounds__(256) void k_route_mlp2_bf16(RouteParams p, int npcb) {
  constexpr int Hr = 128, kW2Stride = GP + 4;
  static_assert(Hr * (kFsStride + kW2Stride) * 4 <= kRtNB * kRtStage, "epilogue tiles fit the ring");
  __shared__ __attribute__((aligned(16))) char ring[kRtNB * kRtStage];
  __shared__ float b2s[GP], brs[16], wps[16];
  __shared__ __attribute__((aligned(16))) float cbs[PS ? 2 : 1][Hr];
  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, g4 = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform
  const int d = p.d, C = p.C, G = p.G;
  const size_t W1s = 2 * static_cast<size_t>(d) + p.d_e;

  const int N = p.B * p.T;
  const int tok0 = blockIdx.x * kRtTok;
  const int tok = tok0 + 16 * w + l16;
  const bool valid = tok < N;
  const int nvalid = min(kRtTok, N - tok0);
  const int b = valid ? tok / p.T : 0;
  const int type = p.types[valid ? tok : 0];

  // Epilogue operands are loaded now and held in registers through the K
  // loop: F (entry e = j*16 + c), W2 transposed (entry e = s*Hr + j) and
  // either this lane's 32 per-sample language terms cb[b][16m + 4q + i] or,
  // with PS, this thread's share of the block's language terms: the npcb
  // (at most 8) column-block partials of unit j = tid % 128 for sample
  // tok0 / T + tid / 128 (a block spans at most two samples when T >= 64).
  float fv[8], w2v[GP / 2], cbv[PS ? 1 : 32], ps[PS ? 8 : 1], b1v = 0.f;
  const int b0 = tok0 / p.T;
  {
    const rsrc_t r_F = make_rsrc(p.F, static_cast<uint32_t>(Hr * C) * 4u);
    const rsrc_t r_W2 = make_rsrc(p.W2, static_cast<uint32_t>(G * Hr) * 2u);
    const rsrc_t r_cb = make_rsrc(p.cb, static_cast<uint32_t>(p.B * Hr) * 4u);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = u * 256 + tid, j = e >> 4, c = e & 15;
      fv[u] = __uint_as_float(bload4(r_F, c < C ? 4u * (j * C + c) : kOOB));
    }
#pragma unroll
    for (int u = 0; u < GP / 2; ++u) {
      const int e = u * 256 + tid, sg = e >> 7, j = e & 127;
      const uint32_t x = bload4(r_W2, sg < G ? 4u * ((sg * Hr + j) >> 1) : kOOB);
      w2v[u] = __uint_as_float((j & 1) ? (x & 0xffff0000u) : (x << 16));
    }
    if constexpr (PS) {
      const int bs = b0 + (tid >> 7), jj = tid & 127;
      const rsrc_t r_p = make_rsrc(p.pcb, static_cast<uint32_t>(npcb * p.B * Hr) * 4u);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        ps[u] = __uint_as_float(bload4(r_p, oob_unless(bs < p.B && u < npcb, 4u * ((u * p.B + bs) * Hr + jj))));
      b1v = tof(static_cast<const bf16*>(p.b1)[jj]);
    } else {
#pragma unroll
      for (int m = 0; m < 8; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          cbv[4 * m + i] = __uint_as_float(bload4(r_cb, 4u * (b * Hr + 16 * m + 4 * g4 + i)));
    }
    if (tid < GP) b2s[tid] = tid < G ? tof(static_cast<const bf16*>(p.b2)[tid]) : 0.f;
    if (tid < 16) brs[tid] = tid < C ? tof(static_cast<const bf16*>(p.b_r)[tid]) : 0.f;
    if (tid < 16) wps[tid] = (p.priority && tid < C) ? tof(static_cast<const bf16*>(p.w_pri)[tid]) : 0.f;
  }

  const rsrc_t r_h = make_rsrc(static_cast<const bf16*>(p.h) + static_cast<size_t>(tok0) * d,
                               static_cast<uint32_t>(nvalid) * d * 2);
  const rsrc_t r_w1 = make_rsrc(p.W1, static_cast<uint32_t>(Hr * W1s * 2));
  const rsrc_t r_wr = make_rsrc(p.W_r, static_cast<uint32_t>(C) * d * 2);
  const int nch = d / kRtKc;
  const uint32_t ring_base = lds_addr(ring);

  // This wave's wave-loads of a stage: j = w, w+4, ... < kRtLoads (7 for waves
  // 0-1, 6 for waves 2-3). Load j < 18 brings weight rows 8j..8j+7 (W1 for
  // j < 16, W_r rows for j = 16, 17), load j >= 18 token rows 8(j-18).. .
  // Lane i carries row 8j + i/8, LDS piece i%8, global piece (i%8) ^ swizzle.
  const int nld = (kRtLoads - w + 3) / 4;
  uint32_t base_off[7];
#pragma unroll
  for (int u = 0; u < 7; ++u) {
    const int jj = w + 4 * u;
    const int ri = lane >> 3, piece = lane & 7;
    uint32_t off = kOOB;
    if (jj < 16) {
      const int r = 8 * jj + ri;
      off = static_cast<uint32_t>((r * W1s + 8 * (piece ^ rt_swz(r))) * 2);
    } else if (jj < 18) {
      const int r = 8 * jj + ri, rr = r - Hr;
      if (rr < C) off = static_cast<uint32_t>((rr * d + 8 * (piece ^ rt_swz(r))) * 2);
    } else if (jj < kRtLoads) {
      const int t = 8 * (jj - 18) + ri;
      if (t < nvalid) off = static_cast<uint32_t>((t * d + 8 * (piece ^ rt_swz(t))) * 2);
    }
    base_off[u] = off;
  }
  // Wave-loads u = 0..3 are always W1 rows (j <= 15); u = 4 is W_r rows for
  // waves 0-1 and token rows for waves 2-3; u = 5, 6 are token rows. Each call
  // site below uses one fixed buffer resource so it stays in scalar registers.
  auto issue_one = [&](int c, int u) {
    const uint32_t sbase = ring_base + (c % kRtNB) * kRtStage;
    const bool ok = c < nch;  // chunks past the end are all-out-of-range dummies
    const uint32_t kb = static_cast<uint32_t>(c) * kRtKc * 2;
    const uint32_t off = (ok && base_off[u] != kOOB) ? base_off[u] + kb : kOOB;
    const int jj = w + 4 * u;
    const uint32_t dst = sbase + (jj < 18 ? jj * 1024 : kRtWBytes + (jj - 18) * 1024);
    if (u < 4) dma16(r_w1, off, dst);
    else if (u == 4 && w < 2) dma16(r_wr, off, dst);
    else if (u == 4 || u == 5 || (u == 6 && w < 2)) dma16(r_h, off, dst);
  };
  auto issue = [&](int c) {
#pragma unroll
    for (int u = 0; u < 7; ++u) issue_one(c, u);
  };

  f32x4 acc[9], acc_lo[9];
#pragma unroll
  for (int m = 0; m < 9; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto step = [&](int c) {
    // chunk c has landed once at most (kRtNB - 2) younger stages are pending
    if (nld == 7) wait_vmcnt<7 * (kRtNB - 2)>();
    else wait_vmcnt<6 * (kRtNB - 2)>();
    __syncthreads();
    // All fragment reads first; then the 18 MFMAs with this wave's 7 refill
    // DMAs of chunk c + kRtNB - 1 spread between them (the stage they fill was
    // released at this barrier). Issued as one burst after the MFMAs, the
    // DMAs of the four waves queued at the texture unit (about 64 B per
    // clock) while the matrix cores idled, and the other way round.
    const char* st = ring + (c % kRtNB) * kRtStage;
    const int th = 16 * w + l16;
    bf16x8 hb[2], af[2][9];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      hb[ks] = *reinterpret_cast<const bf16x8*>(st + kRtWBytes + th * 128 + 16 * ((4 * ks + g4) ^ rt_swz(th)));
#pragma unroll
      for (int m = 0; m < 9; ++m) {
        const int r = 16 * m + l16;
        af[ks][m] = *reinterpret_cast<const bf16x8*>(st + r * 128 + 16 * ((4 * ks + g4) ^ rt_swz(r)));
      }
    }
#pragma unroll
    for (int i = 0; i < 18; ++i) {
      acc[i % 9] = mfma_16x16x32(af[i / 9][i % 9], hb[i / 9], acc[i % 9]);
      if (i % 3 == 1) issue_one(c + kRtNB - 1, i / 3);
    }
    issue_one(c + kRtNB - 1, 6);
  };

#pragma unroll
  for (int c = 0; c < kRtNB - 1; ++c) issue(c);
  // the two halves of the hidden size are summed separately and added at the
  // end, as the split-K form does; one loop per half keeps the first half's
  // sums out of the loop-carried state of the second
  const int nlo = nch / 2;
  for (int c = 0; c < nlo; ++c) step(c);
#pragma unroll
  for (int m = 0; m < 9; ++m) {
    acc_lo[m] = acc[m];
    acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int c = nlo; c < nch; ++c) step(c);
  wait_vmcnt<0>();  // trailing dummy loads land before the LDS is released
  __syncthreads();  // every wave is done with the ring
#pragma unroll
  for (int m = 0; m < 9; ++m) acc[m] = acc_lo[m] + acc[m];

  float* Fs = reinterpret_cast<float*>(ring);
  float* W2t = Fs + Hr * kFsStride;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int e = u * 256 + tid;
    Fs[(e >> 4) * kFsStride + (e & 15)] = fv[u];
  }
#pragma unroll
  for (int u = 0; u < GP / 2; ++u) {
    const int e = u * 256 + tid;
    W2t[(e & 127) * kW2Stride + (e >> 7)] = w2v[u];
  }
  if constexpr (PS) {
    // partials added in block order; out-of-range ones read as zero
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += ps[u];
    cbs[tid >> 7][tid & 127] = sum + b1v;
  }
  __syncthreads();
  float cbl[32];
  if constexpr (PS) {
    const float* src = cbs[valid ? b - b0 : 0];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(src + 16 * m + 4 * g4);
#pragma unroll
      for (int i = 0; i < 4; ++i) cbl[4 * m + i] = v[i];
    }
  } else {
#pragma unroll
    for (int i = 0; i < 32; ++i) cbl[i] = cbv[i];
  }

  // ---- epilogue: lanes l16, l16+16, l16+32, l16+48 hold token `tok`;
  // lane quarter q = g4 owns hidden units 16m + 4q + i and role logits 4q + i.
  float ex[4], mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = 4 * g4 + i;
    const float lg = acc[8][i] + brs[c];
    ex[i] = c < C ? lg : -INFINITY;
    mx = fmaxf(mx, ex[i]);
  }
  mx = max_xor32(max_xor16(mx));
  float sm = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float e = expf(ex[i] - mx);
    ex[i] = (4 * g4 + i < C) ? e : 0.f;
    sm += ex[i];
  }
  sm = add_xor32(add_xor16(sm));
  const float isum = 1.f / sm;
  float a[16];  // role mixture weights; zero past C
#pragma unroll
  for (int c = 0; c < 16; ++c) a[c] = __shfl(ex[c & 3], l16 + 16 * (c >> 2), kWave) * isum;
  if (p.priority) {  // role priority w^T a (weights zero past C)
    float pr = 0.f;
#pragma unroll
    for (int c = 0; c < 16; ++c) pr = fmaf(wps[c], a[c], pr);
    if (valid && g4 == 0) p.priority[tok] = pr;
  }

  // F a on the f32 matrix cores: the accumulator layout is that of a 16x16x4
  // MFMA with A = F (rows 16m + t, roles k0 + q) and B = a (role k0 + q of the
  // lane's token), so x += F a costs ceil(C / 4) MFMAs per 16 hidden units.
  // Lane quarter q takes a[k0 + q] by a bitwise blend (a select chain on q
  // would be turned into an indexed access and move a[] to scratch memory).
  float ab[4];
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) v |= (g4 == q ? ~0u : 0u) & __float_as_uint(a[4 * k4 + q]);
    ab[k4] = __uint_as_float(v);
  }
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    if (4 * k4 < C) {
#pragma unroll
      for (int m = 0; m < 8; ++m)
        acc[m] = __builtin_amdgcn_mfma_f32_16x16x4f32(Fs[(16 * m + l16) * kFsStride + 4 * k4 + g4], ab[k4],
                                                      acc[m], 0, 0, 0);
    }
  }
  float gam[GP];
#pragma unroll
  for (int s = 0; s < GP; ++s) gam[s] = 0.f;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * m + 4 * g4 + i;
      const float gl = gelu_exact(acc[m][i] + cbl[4 * m + i]);
      const f32x4* wr = reinterpret_cast<const f32x4*>(W2t + j * kW2Stride);
#pragma unroll
      for (int s4 = 0; s4 < GP / 4; ++s4) {
        const f32x4 w2 = wr[s4];
        gam[4 * s4] += w2[0] * gl;
        gam[4 * s4 + 1] += w2[1] * gl;
        gam[4 * s4 + 2] += w2[2] * gl;
        gam[4 * s4 + 3] += w2[3] * gl;
      }
    }
  }
  int n_above = 0;
#pragma unroll
  for (int s = 0; s < GP; ++s) {
    gam[s] = add_xor32(add_xor16(gam[s]));
    gam[s] += b2s[s];
    n_above += static_cast<int>((s < G) & (gam[s] > p.tau));
  }
  // the four lanes of a token now hold bitwise-identical scores; lane quarter
  // q ranks groups s = 4u + q
  // (a bitwise blend: a select chain on q gets turned into an indexed access,
  // which would move gam to scratch memory)
  float mine[GP / 4];
  uint32_t qsel[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) qsel[q] = g4 == q ? ~0u : 0u;
#pragma unroll
  for (int u = 0; u < GP / 4; ++u) {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) v |= qsel[q] & __float_as_uint(gam[4 * u + q]);
    mine[u] = __uint_as_float(v);
  }
  const int K = budget_k(p.mode, p.k_by_type, type, p.tau, p.kmin, p.kmax, G, n_above);
  uint32_t msk = 0;
  if (p.mode == 1 && K == n_above) {
#pragma unroll
    for (int s = 0; s < GP; ++s) msk |= static_cast<uint32_t>((s < G) & (gam[s] > p.tau)) << s;
  } else {
#pragma unroll
    for (int u = 0; u < GP / 4; ++u) {
      const int s = 4 * u + g4;
      int rank = 0;
#pragma unroll
      for (int t = 0; t < GP; ++t)
        rank += static_cast<int>((t < G) & (key_above(gam[t], mine[u]) | ((t < s) & key_equal(gam[t], mine[u]))));
      msk |= static_cast<uint32_t>((s < G) & (rank < K)) << s;
    }
    msk = or_xor32(or_xor16(msk));
  }
  if (valid) {
    if (p.scores_out) {
#pragma unroll
      for (int u = 0; u < GP / 4; ++u) {
        const int s = 4 * u + g4;
        if (s < G) p.scores_out[static_cast<size_t>(tok) * G + s] = mine[u];
      }
    }
    if (g4 == 0 && p.mask) write_selection(p, tok, msk);
  }
}

// ---------------------------------------------------------------------------
// Split-K form of the same router (language terms as column-block partials,
// T >= 96, d a multiple of 128). A tile of 96 tokens is computed by two
// workgroups of six waves (16 tokens each), each over one half of the hidden
// size: a workgroup reads half of the weight panel (0.6 MB rather than
// 1.2 MB per 64 tokens), and 64 prefixes of 177 tokens make 236 workgroups,
// one per CU on almost every CU. Both halves store their partial products
// and take a ticket (one atomic counter per tile). The first to finish waits
// a bounded time for the other; if it comes, each adds the other's partials
// for 48 of the 96 tokens and runs their epilogue (three waves each, one per
// SIMD, instead of six waves on four SIMDs for all 96); if not, the first
// gives the tile up (a compare-and-swap decides against a late arrival) and
// the second completes all of it. The single kernel accumulates the two
// halves separately too, so all forms give the same bits: every product,
// sum and epilogue step is the same per token.
constexpr int kSkW = 6, kSkNB = 4;
constexpr int kSkHBytes = kRouteSkTok * 128, kSkStage = kRtWBytes + kSkHBytes;
constexpr int kSkLoads = kRtRows / 8 + kRouteSkTok / 8;  // 1 KB wave-loads per stage (30: five per wave)
static_assert(kSkLoads == 5 * kSkW, "stage loads split evenly over the waves");

template <int GP>
__global__ __launch_bounds__(64 * kSkW) void k_route_mlp2_sk(RouteParams p, int npcb) {
  constexpr int Hr = 128, kW2Stride = GP + 4;
  static_assert(Hr * (kFsStride + kW2Stride) * 4 <= kSkNB * kSkStage, "epilogue tiles fit the ring");
  __shared__ __attribute__((aligned(16))) char ring[kSkNB * kSkStage];
  __shared__ float b2s[GP], brs[16], wps[16];
  __shared__ __attribute__((aligned(16))) float cbs[kSkW / 2][Hr];
  __shared__ int s_ticket, s_state;
  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, g4 = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform
  const int d = p.d, C = p.C, G = p.G;
  const size_t W1s = 2 * static_cast<size_t>(d) + p.d_e;
  const int tile = blockIdx.x >> 1, half = blockIdx.x & 1;

  const int N = p.B * p.T;
  const int tok0 = tile * kRouteSkTok;
  const int tok = tok0 + 16 * w + l16;
  const bool valid = tok < N;
  const int nvalid = min(kRouteSkTok, N - tok0);
  const int b = valid ? tok / p.T : 0;
  const int type = p.types[valid ? tok : 0];

  // epilogue operands, as in the single kernel: F and W2 by threads 0..255,
  // the language terms of the (at most three) samples the tile touches by all
  float fv[8] = {}, w2v[GP / 2] = {}, ps[8] = {};
  const int b0 = tok0 / p.T;
  {
    const int bs = b0 + (tid >> 7), jj = tid & 127;
    const rsrc_t r_p = make_rsrc(p.pcb, static_cast<uint32_t>(npcb * p.B * Hr) * 4u);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      ps[u] = __uint_as_float(bload4(r_p, oob_unless(bs < p.B && u < npcb, 4u * ((u * p.B + bs) * Hr + jj))));
  }
  const float b1v = tof(static_cast<const bf16*>(p.b1)[tid & 127]);
  if (tid < 256) {
    const rsrc_t r_F = make_rsrc(p.F, static_cast<uint32_t>(Hr * C) * 4u);
    const rsrc_t r_W2 = make_rsrc(p.W2, static_cast<uint32_t>(G * Hr) * 2u);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = u * 256 + tid, j = e >> 4, c = e & 15;
      fv[u] = __uint_as_float(bload4(r_F, c < C ? 4u * (j * C + c) : kOOB));
    }
#pragma unroll
    for (int u = 0; u < GP / 2; ++u) {
      const int e = u * 256 + tid, sg = e >> 7, j = e & 127;
      const uint32_t x = bload4(r_W2, sg < G ? 4u * ((sg * Hr + j) >> 1) : kOOB);
      w2v[u] = __uint_as_float((j & 1) ? (x & 0xffff0000u) : (x << 16));
    }
    if (tid < GP) b2s[tid] = tid < G ? tof(static_cast<const bf16*>(p.b2)[tid]) : 0.f;
    if (tid < 16) brs[tid] = tid < C ? tof(static_cast<const bf16*>(p.b_r)[tid]) : 0.f;
    if (tid < 16) wps[tid] = (p.priority && tid < C) ? tof(static_cast<const bf16*>(p.w_pri)[tid]) : 0.f;
  }

  const rsrc_t r_h = make_rsrc(static_cast<const bf16*>(p.h) + static_cast<size_t>(tok0) * d,
                               static_cast<uint32_t>(nvalid) * d * 2);
  const rsrc_t r_w1 = make_rsrc(p.W1, static_cast<uint32_t>(Hr * W1s * 2));
  const rsrc_t r_wr = make_rsrc(p.W_r, static_cast<uint32_t>(C) * d * 2);
  const int nh = d / kRtKc / 2, cbase = half * nh;  // this half's chunks
  const uint32_t ring_base = lds_addr(ring);

  // This wave's wave-loads of a stage: j = w + 6u, u < 5. Load j < 18 brings
  // weight rows 8j..8j+7 (W1 for j < 16, W_r rows for j = 16, 17), load
  // j >= 18 token rows 8(j-18).. . Lane i carries row 8j + i/8, LDS piece
  // i%8, global piece (i%8) ^ swizzle. u = 0, 1: W1 rows; u = 2: W1 rows for
  // waves 0-3, W_r rows for waves 4-5; u = 3, 4: token rows.
  uint32_t base_off[5];
#pragma unroll
  for (int u = 0; u < 5; ++u) {
    const int jj = w + kSkW * u;
    const int ri = lane >> 3, piece = lane & 7;
    uint32_t off = kOOB;
    if (jj < 16) {
      const int r = 8 * jj + ri;
      off = static_cast<uint32_t>((r * W1s + 8 * (piece ^ rt_swz(r))) * 2);
    } else if (jj < 18) {
      const int r = 8 * jj + ri, rr = r - Hr;
      if (rr < C) off = static_cast<uint32_t>((rr * d + 8 * (piece ^ rt_swz(r))) * 2);
    } else {
      const int t = 8 * (jj - 18) + ri;
      if (t < nvalid) off = static_cast<uint32_t>((t * d + 8 * (piece ^ rt_swz(t))) * 2);
    }
    base_off[u] = off;
  }
  auto issue_one = [&](int i, int u) {
    const uint32_t sbase = ring_base + (i % kSkNB) * kSkStage;
    const bool ok = i < nh;  // stages past this half are all-out-of-range dummies
    const uint32_t kb = static_cast<uint32_t>(cbase + i) * kRtKc * 2;
    const uint32_t off = (ok && base_off[u] != kOOB) ? base_off[u] + kb : kOOB;
    const int jj = w + kSkW * u;
    const uint32_t dst = sbase + (jj < 18 ? jj * 1024 : kRtWBytes + (jj - 18) * 1024);
    if (u < 2) dma16(r_w1, off, dst);
    else if (u == 2) {
      if (w < 4) dma16(r_w1, off, dst);
      else dma16(r_wr, off, dst);
    } else dma16(r_h, off, dst);
  };
  auto issue = [&](int i) {
#pragma unroll
    for (int u = 0; u < 5; ++u) issue_one(i, u);
  };

  f32x4 acc[9];
#pragma unroll
  for (int m = 0; m < 9; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < kSkNB - 1; ++i) issue(i);
  for (int i = 0; i < nh; ++i) {
    // stage i has landed once at most (kSkNB - 2) younger stages are pending
    wait_vmcnt<5 * (kSkNB - 2)>();
    __syncthreads();
    const char* st = ring + (i % kSkNB) * kSkStage;
    const int th = 16 * w + l16;
    bf16x8 hb[2], af[2][9];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      hb[ks] = *reinterpret_cast<const bf16x8*>(st + kRtWBytes + th * 128 + 16 * ((4 * ks + g4) ^ rt_swz(th)));
#pragma unroll
      for (int m = 0; m < 9; ++m) {
        const int r = 16 * m + l16;
        af[ks][m] = *reinterpret_cast<const bf16x8*>(st + r * 128 + 16 * ((4 * ks + g4) ^ rt_swz(r)));
      }
    }
    // the refill DMAs of stage i + kSkNB - 1 spread between the MFMAs
#pragma unroll
    for (int q = 0; q < 18; ++q) {
      acc[q % 9] = mfma_16x16x32(af[q / 9][q % 9], hb[q / 9], acc[q % 9]);
      if (q % 4 == 1) issue_one(i + kSkNB - 1, q / 4);
    }
  }
  wait_vmcnt<0>();  // trailing dummy loads land before the LDS is released
  __syncthreads();  // every wave is done with the ring

  // Both halves store their partial products; whoever completes a token adds
  // the other half's (a + b: the same bits in either order), both halves for
  // 48 tokens each or the second to finish for all 96 (see the kernel's
  // header). The two workgroups of a tile may sit on different XCDs, whose L2 caches
  // are not coherent with each other: the partials are written and read with
  // system-scope cache bits (written through to memory, read past the
  // caches), and the ticket is a system-scope atomic. No fence is needed for
  // them, and none of the XCD's cached weights is written back or dropped.
  constexpr int kSys = 1 | 16;  // sc0 | sc1: system scope
  const uint32_t part_bytes = static_cast<uint32_t>(9 * kSkW * 64 * 16);
  const size_t ntiles = (static_cast<size_t>(N) + kRouteSkTok - 1) / kRouteSkTok;
  const rsrc_t r_part = make_rsrc(p.rpart, clamp_bytes(ntiles * 2 * static_cast<size_t>(part_bytes)));
  {
    const uint32_t o = static_cast<uint32_t>(blockIdx.x) * part_bytes + static_cast<uint32_t>(w * 64 + lane) * 16u;
#pragma unroll
    for (int m = 0; m < 9; ++m)
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[m]), r_part, o + m * kSkW * 64 * 16, 0, kSys);
  }
  wait_vmcnt<0>();  // this wave's partial has been written
  __syncthreads();
  // Ticket states: 0 none arrived, 1 the first arrived and waits, 2 both
  // arrived (shared epilogue), 3 the first gave up (4 once the second came).
  if (tid == 0) s_ticket = __hip_atomic_fetch_add(p.rcnt + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __syncthreads();
  bool shared_epi = s_ticket == 1;  // second to arrive: 1 = the first waits for it, 3 = it gave up
  if (s_ticket == 0) {
    // first to arrive: poll the counter (system scope, past the caches) up
    // to sk_polls times, then give the tile up unless the other came first
    if (tid == 0) {
      int st = 1;
      for (int i = 0; i < p.sk_polls && st == 1; ++i) {
        __builtin_amdgcn_s_sleep(4);
        st = __hip_atomic_load(p.rcnt + tile, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
      if (st == 1) {
        int expect = 1;
        st = __hip_atomic_compare_exchange_strong(p.rcnt + tile, &expect, 3, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_SYSTEM)
                 ? 3
                 : expect;
      }
      s_state = st;
    }
    __syncthreads();
    if (s_state == 3) return;  // the other half completes the tile
    shared_epi = true;
  }
  // with a shared epilogue half 0 finishes the tile's tokens 0..47 (waves
  // 0-2), half 1 tokens 48..95 (waves 3-5)
  const bool my_share = !shared_epi || ((w < kSkW / 2) == (half == 0));
  if (my_share) {
    const uint32_t o = static_cast<uint32_t>(blockIdx.x ^ 1) * part_bytes + static_cast<uint32_t>(w * 64 + lane) * 16u;
#pragma unroll
    for (int m = 0; m < 9; ++m)
      acc[m] = acc[m] + __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                      r_part, static_cast<int>(o + m * kSkW * 64 * 16), 0, kSys));
  }

  float* Fs = reinterpret_cast<float*>(ring);
  float* W2t = Fs + Hr * kFsStride;
  if (tid < 256) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = u * 256 + tid;
      Fs[(e >> 4) * kFsStride + (e & 15)] = fv[u];
    }
#pragma unroll
    for (int u = 0; u < GP / 2; ++u) {
      const int e = u * 256 + tid;
      W2t[(e & 127) * kW2Stride + (e >> 7)] = w2v[u];
    }
  }
  {
    // partials added in block order; out-of-range ones read as zero
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += ps[u];
    cbs[tid >> 7][tid & 127] = sum + b1v;
  }
  __syncthreads();
  if (!my_share) return;  // no barrier follows
  float cbl[32];
  {
    const float* src = cbs[valid ? b - b0 : 0];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(src + 16 * m + 4 * g4);
#pragma unroll
      for (int i = 0; i < 4; ++i) cbl[4 * m + i] = v[i];
    }
  }

  // ---- epilogue: lanes l16, l16+16, l16+32, l16+48 hold token `tok`;
  // lane quarter q = g4 owns hidden units 16m + 4q + i and role logits 4q + i.
  float ex[4], mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = 4 * g4 + i;
    const float lg = acc[8][i] + brs[c];
    ex[i] = c < C ? lg : -INFINITY;
    mx = fmaxf(mx, ex[i]);
  }
  mx = max_xor32(max_xor16(mx));
  float sm = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float e = expf(ex[i] - mx);
    ex[i] = (4 * g4 + i < C) ? e : 0.f;
    sm += ex[i];
  }
  sm = add_xor32(add_xor16(sm));
  const float isum = 1.f / sm;
  float a[16];  // role mixture weights; zero past C
#pragma unroll
  for (int c = 0; c < 16; ++c) a[c] = __shfl(ex[c & 3], l16 + 16 * (c >> 2), kWave) * isum;
  if (p.priority) {  // role priority w^T a (weights zero past C)
    float pr = 0.f;
#pragma unroll
    for (int c = 0; c < 16; ++c) pr = fmaf(wps[c], a[c], pr);
    if (valid && g4 == 0) p.priority[tok] = pr;
  }

  // F a on the f32 matrix cores: the accumulator layout is that of a 16x16x4
  // MFMA with A = F (rows 16m + t, roles k0 + q) and B = a (role k0 + q of the
  // lane's token), so x += F a costs ceil(C / 4) MFMAs per 16 hidden units.
  // Lane quarter q takes a[k0 + q] by a bitwise blend (a select chain on q
  // would be turned into an indexed access and move a[] to scratch memory).
  float ab[4];
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) v |= (g4 == q ? ~0u : 0u) & __float_as_uint(a[4 * k4 + q]);
    ab[k4] = __uint_as_float(v);
  }
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    if (4 * k4 < C) {
#pragma unroll
      for (int m = 0; m < 8; ++m)
        acc[m] = __builtin_amdgcn_mfma_f32_16x16x4f32(Fs[(16 * m + l16) * kFsStride + 4 * k4 + g4], ab[k4],
                                                      acc[m], 0, 0, 0);
    }
  }
  float gam[GP];
#pragma unroll
  for (int s = 0; s < GP; ++s) gam[s] = 0.f;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * m + 4 * g4 + i;
      const float gl = gelu_exact(acc[m][i] + cbl[4 * m + i]);
      const f32x4* wr = reinterpret_cast<const f32x4*>(W2t + j * kW2Stride);
#pragma unroll
      for (int s4 = 0; s4 < GP / 4; ++s4) {
        const f32x4 w2 = wr[s4];
        gam[4 * s4] += w2[0] * gl;
        gam[4 * s4 + 1] += w2[1] * gl;
        gam[4 * s4 + 2] += w2[2] * gl;
        gam[4 * s4 + 3] += w2[3] * gl;
      }
    }
  }
  int n_above = 0;
#pragma unroll
  for (int s = 0; s < GP; ++s) {
    gam[s] = add_xor32(add_xor16(gam[s]));
    gam[s] += b2s[s];
    n_above += static_cast<int>((s < G) & (gam[s] > p.tau));
  }
  // the four lanes of a token now hold bitwise-identical scores; lane quarter
  // q ranks groups s = 4u + q
  // (a bitwise blend: a select chain on q gets turned into an indexed access,
  // which would move gam to scratch memory)
  float mine[GP / 4];
  uint32_t qsel[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) qsel[q] = g4 == q ? ~0u : 0u;
#pragma unroll
  for (int u = 0; u < GP / 4; ++u) {
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) v |= qsel[q] & __float_as_uint(gam[4 * u + q]);
    mine[u] = __uint_as_float(v);
  }
  const int K = budget_k(p.mode, p.k_by_type, type, p.tau, p.kmin, p.kmax, G, n_above);
  uint32_t msk = 0;
  if (p.mode == 1 && K == n_above) {
#pragma unroll
    for (int s = 0; s < GP; ++s) msk |= static_cast<uint32_t>((s < G) & (gam[s] > p.tau)) << s;
  } else {
#pragma unroll
    for (int u = 0; u < GP / 4; ++u) {
      const int s = 4 * u + g4;
      int rank = 0;
#pragma unroll
      for (int t = 0; t < GP; ++t)
        rank += static_cast<int>((t < G) & (key_above(gam[t], mine[u]) | ((t < s) & key_equal(gam[t], mine[u]))));
      msk |= static_cast<uint32_t>((s < G) & (rank < K)) << s;
    }
    msk = or_xor32(or_xor16(msk));
  }
  if (valid) {
    if (p.scores_out) {
#pragma unroll
      for (int u = 0; u < GP / 4; ++u) {
        const int s = 4 * u + g4;
        if (s < G) p.scores_out[static_cast<size_t>(tok) * G + s] = mine[u];
      }
    }
    if (g4 == 0 && p.mask) write_selection(p, tok, msk);
  }
}
}  // namespace

hipError_t launch_route(const RouteParams& p, bool bf16, hipStream_t s) {
  const size_t ntok = static_cast<size_t>(p.B) * p.T;
  if (ntok == 0) return hipSuccess;
  const bool mfma_ok = bf16 && p.kind == 0 && p.Hr == 128 && p.C >= 1 && p.C <= 16 &&
                       p.G <= 32 && p.d % kRtKc == 0 && ntok < (1u << 30);
  const int vec = bf16 ? 8 : 4;
  const int ncb = (p.d + 64 * vec - 1) / (64 * vec);
  const bool pcb_ok = bf16 && p.kind == 0 && p.pcb && p.d % (64 * vec) == 0 && p.d_e % 8 == 0 &&
                      p.Hr % 64 == 0 && p.Hr <= 128 && p.C >= 1 &&
                      static_cast<size_t>(p.Hr) * (2 * static_cast<size_t>(p.d) + p.d_e) * 2 < (1ull << 31) &&
                      static_cast<size_t>(ncb) * p.B * p.Hr * 4 < (1ull << 31) &&
                      ((reinterpret_cast<uintptr_t>(p.W1) | reinterpret_cast<uintptr_t>(p.E)) & 15) == 0;
  // the MFMA router adds the partial language terms itself when a block of
  // its tokens spans at most two samples and there are at most 8 partials
  const bool ps = mfma_ok && pcb_ok && p.T >= kRtTok && ncb <= 8;
  {
    const dim3 gpool(static_cast<unsigned>(p.B * ncb));
    const int nout = p.kind == 0 ? p.Hr : p.G;
    const int nF = ((p.kind == 0 ? p.Hr : p.G) + 3) / 4;
    const dim3 gproj(static_cast<unsigned>(p.B * ((nout + 7) / 8) + nF));
    const size_t shm = static_cast<size_t>(p.d) * sizeof(float);
    if (pcb_ok) {
      const unsigned nfb = static_cast<unsigned>((p.Hr * p.C + 255) / 256);
      hipLaunchKernelGGL((k_route_pool<rolesub::bf16, true>), dim3(gpool.x + nfb), dim3(256), 0, s, p);
      if (!ps)
        hipLaunchKernelGGL(k_route_cbsum, dim3(static_cast<unsigned>((p.B * p.Hr + 255) / 256)), dim3(256), 0,
                           s, p, ncb);
    } else if (bf16) {
      hipLaunchKernelGGL((k_route_pool<rolesub::bf16, false>), gpool, dim3(256), 0, s, p);
      hipLaunchKernelGGL(k_route_proj<rolesub::bf16>, gproj, dim3(256), shm, s, p);
    } else {
      hipLaunchKernelGGL((k_route_pool<float, false>), gpool, dim3(256), 0, s, p);
      hipLaunchKernelGGL(k_route_proj<float>, gproj, dim3(256), shm, s, p);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (mfma_ok && ps && p.rpart && p.rcnt && p.T >= kRouteSkMinT && p.d % (2 * kRtKc) == 0) {
    const dim3 grid(static_cast<unsigned>(2 * route_sk_tiles(p.B, p.T)));
    if (p.G <= 8) hipLaunchKernelGGL(k_route_mlp2_sk<8>, grid, dim3(64 * kSkW), 0, s, p, ncb);
    else if (p.G <= 16) hipLaunchKernelGGL(k_route_mlp2_sk<16>, grid, dim3(64 * kSkW), 0, s, p, ncb);
    else hipLaunchKernelGGL(k_route_mlp2_sk<32>, grid, dim3(64 * kSkW), 0, s, p, ncb);
  } else if (mfma_ok) {
    const dim3 grid(static_cast<unsigned>((ntok + kRtTok - 1) / kRtTok));
    if (ps) {
      if (p.G <= 8) hipLaunchKernelGGL((k_route_mlp2_bf16<8, true>), grid, dim3(256), 0, s, p, ncb);
      else if (p.G <= 16) hipLaunchKernelGGL((k_route_mlp2_bf16<16, true>), grid, dim3(256), 0, s, p, ncb);
      else hipLaunchKernelGGL((k_route_mlp2_bf16<32, true>), grid, dim3(256), 0, s, p, ncb);
    } else {
      if (p.G <= 8) hipLaunchKernelGGL((k_route_mlp2_bf16<8, false>), grid, dim3(256), 0, s, p, 0);
      else if (p.G <= 16) hipLaunchKernelGGL((k_route_mlp2_bf16<16, false>), grid, dim3(256), 0, s, p, 0);
      else hipLaunchKernelGGL((k_route_mlp2_bf16<32, false>), grid, dim3(256), 0, s, p, 0);
    }
  } else {
    const int nmain = p.kind == 0 ? p.Hr : p.G;
    const size_t shm = sizeof(float) * (static_cast<size_t>(p.d) + nmain + p.C +
                                        (p.kind == 0 ? p.Hr : 0) + p.G);
    if (bf16)
      hipLaunchKernelGGL(k_route_generic<rolesub::bf16>, dim3(static_cast<unsigned>(ntok)), dim3(256), shm, s, p);
    else
      hipLaunchKernelGGL(k_route_generic<float>, dim3(static_cast<unsigned>(ntok)), dim3(256), shm, s, p);
  }
  return hipGetLastError();
}

size_t route_generic_shm(int d, int G, int C, int Hr, int kind) {
  const int nmain = kind == 0 ? Hr : G;
  return sizeof(float) * (static_cast<size_t>(d) + nmain + C + (kind == 0 ? Hr : 0) + G);
}

hipError_t launch_select(const RouteParams& p, hipStream_t s) {
  const size_t ntok = static_cast<size_t>(p.B) * p.T;
  if (ntok == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((ntok + kSelTok - 1) / kSelTok));
  if (p.G <= 8) hipLaunchKernelGGL(k_select<8>, grid, dim3(kSelTok), 0, s, p);
  else if (p.G <= 16) hipLaunchKernelGGL(k_select<16>, grid, dim3(kSelTok), 0, s, p);
  else hipLaunchKernelGGL(k_select<32>, grid, dim3(kSelTok), 0, s, p);
  return hipGetLastError();
}

}  // namespace rolesub
