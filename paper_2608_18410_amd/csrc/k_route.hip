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
// Blocks 0..B-1: hl = mean of the sample's language rows of h (zero if none),
//   MLP2:     cb[b][j] = W1[j, d+d_e : 2d+d_e] . hl + b1[j]
//   ADDITIVE: cb[b][s] = alpha_lang (W_lang[s] . hl + b_lang[s])
// Block B:  MLP2 F[j][c] = W1[j, d : d+d_e] . E[c];  ADDITIVE F[s][c] = alpha_role W_role[s][c]
template <class T>
__global__ __launch_bounds__(256) void k_route_prep(RouteParams p) {
  extern __shared__ float hl[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t W1s = 2 * static_cast<size_t>(p.d) + p.d_e;
  if (blockIdx.x == static_cast<unsigned>(p.B)) {
    if (p.kind == 0) {
      const T* W1 = static_cast<const T*>(p.W1);
      const T* E = static_cast<const T*>(p.E);
      for (int o = tid; o < p.Hr * p.C; o += 256) {
        const int j = o / p.C, c = o % p.C;
        float acc = 0.f;
        for (int m = 0; m < p.d_e; ++m)
          acc += tof(W1[j * W1s + p.d + m]) * tof(E[static_cast<size_t>(c) * p.d_e + m]);
        p.F[o] = acc;
      }
    } else {
      const T* Wro = static_cast<const T*>(p.W_role);
      for (int o = tid; o < p.G * p.C; o += 256) p.F[o] = p.alpha_role * tof(Wro[o]);
    }
    return;
  }
  const int b = blockIdx.x;
  const T* h = static_cast<const T*>(p.h) + static_cast<size_t>(b) * p.T * p.d;
  const uint8_t* ty = p.types + static_cast<size_t>(b) * p.T;
  int n = 0;
  for (int t = 0; t < p.T; ++t) n += (ty[t] == kLang);
  const float inv = n ? 1.f / static_cast<float>(n) : 0.f;
  for (int col = tid; col < p.d; col += 256) {
    float acc = 0.f;
    for (int t = 0; t < p.T; ++t)
      if (ty[t] == kLang) acc += tof(h[static_cast<size_t>(t) * p.d + col]);
    hl[col] = acc * inv;
  }
  __syncthreads();
  const int nout = p.kind == 0 ? p.Hr : p.G;
  for (int o = wave; o < nout; o += 4) {
    const T* wrow;
    float bias, scale;
    if (p.kind == 0) {
      wrow = static_cast<const T*>(p.W1) + o * W1s + p.d + p.d_e;
      bias = tof(static_cast<const T*>(p.b1)[o]);
      scale = 1.f;
    } else {
      wrow = static_cast<const T*>(p.W_lang) + static_cast<size_t>(o) * p.d;
      bias = tof(static_cast<const T*>(p.b_lang)[o]);
      scale = p.alpha_lang;
    }
    float acc = 0.f;
    for (int k = lane; k < p.d; k += 64) acc += tof(wrow[k]) * hl[k];
    acc = wave_sum(acc);
    if (lane == 0) p.cb[static_cast<size_t>(b) * nout + o] = scale * (acc + bias);
  }
}

// Rank-based selection of one token's groups from scores held in registers.
__device__ __forceinline__ uint32_t select_from(const float* g, int G, int K) {
  uint32_t m = 0;
#pragma unroll
  for (int s = 0; s < 32; ++s) {
    if (s < G) {
      int rank = 0;
#pragma unroll
      for (int t = 0; t < 32; ++t)
        if (t < G) rank += key_above(g[t], g[s]) || (t < s && key_equal(g[t], g[s]));
      if (rank < K) m |= 1u << s;
    }
  }
  return m;
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
__device__ __forceinline__ uint32_t select_token(const RouteParams& p, const float* g, int type) {
  int n_above = 0;
#pragma unroll
  for (int s = 0; s < 32; ++s)
    if (s < p.G) n_above += g[s] > p.tau;
  const int K = budget_k(p.mode, p.k_by_type, type, p.tau, p.kmin, p.kmax, p.G, n_above);
  if (p.mode == 1 && K == n_above) {
    // Every group above the threshold ranks before every group at or below it,
    // so the top-K set is exactly the groups above the threshold.
    uint32_t m = 0;
#pragma unroll
    for (int s = 0; s < 32; ++s)
      if (s < p.G && g[s] > p.tau) m |= 1u << s;
    return m;
  }
  return select_from(g, p.G, K);
}

// ---------------------------------------------------------------------------
// Selection only, from given scores. One thread per token.
__global__ __launch_bounds__(256) void k_select(RouteParams p) {
  const size_t N = static_cast<size_t>(p.B) * p.T;
  const size_t tok = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (tok >= N) return;
  float g[32];
  const float* src = p.scores_in + tok * p.G;
  if ((p.G & 3) == 0) {
#pragma unroll
    for (int s = 0; s < 32; s += 4) {
      if (s < p.G) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(src + s);
        g[s] = v[0]; g[s + 1] = v[1]; g[s + 2] = v[2]; g[s + 3] = v[3];
      } else {
        g[s] = g[s + 1] = g[s + 2] = g[s + 3] = 0.f;
      }
    }
  } else {
#pragma unroll
    for (int s = 0; s < 32; ++s) g[s] = s < p.G ? src[s] : 0.f;
  }
  const uint32_t m = select_token(p, g, p.types ? p.types[tok] : 0);
  write_selection(p, tok, m);
  if (p.scores_out) {
    float* dst = p.scores_out + tok * p.G;
    for (int s = 0; s < p.G; ++s) dst[s] = src[s];
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
    const uint32_t m = select_token(p, g, p.types[tok]);
    write_selection(p, tok, m);
    if (p.scores_out)
      for (int s = 0; s < G; ++s) p.scores_out[tok * G + s] = gam[s];
  }
}

// ---------------------------------------------------------------------------
// bf16 matrix-core router (MLP2, Hr = 128, C <= 16, d % 64 == 0).
//
// The token-independent product is computed transposed: for 64 tokens per
// workgroup, [W1_h ; W_r] (144 x d, rows 128+C.. zero) times h^T (d x 64) on
// 16x16x32 bf16 MFMA with f32 accumulation. Weight chunks of 64 columns are
// staged through LDS (double buffered) and shared by the four waves; each wave
// streams the hidden states of its own 16 tokens straight into B fragments.
// After the K loop lane (t, q) of a wave holds 36 outputs of token t:
// hidden units 16m+4q+i (m < 8) and role logits 4q+i (m = 8). The epilogue
// (role softmax, F a + cb, GELU, W2, selection) runs on those registers with
// the four lanes of a token exchanging partial sums by cross-lane shuffles.
constexpr int kRtTok = 64, kRtKc = 64, kRtRows = 144, kRtLd = kRtKc + 8;

__global__ __launch_bounds__(256) void k_route_mlp2_bf16(RouteParams p) {
  __shared__ __attribute__((aligned(16))) bf16 Ws[2][kRtRows * kRtLd];
  __shared__ float Fs[128 * 16];
  __shared__ bf16 W2s[32 * 128];
  __shared__ float b2s[32], brs[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int d = p.d, C = p.C, G = p.G;
  constexpr int Hr = 128;
  const size_t W1s = 2 * static_cast<size_t>(d) + p.d_e;
  const bf16* W1 = static_cast<const bf16*>(p.W1);
  const bf16* Wr = static_cast<const bf16*>(p.W_r);
  for (int i = tid; i < Hr * C; i += 256) Fs[i] = p.F[i];
  for (int i = tid; i < G * Hr; i += 256) W2s[i] = static_cast<const bf16*>(p.W2)[i];
  if (tid < G) b2s[tid] = tof(static_cast<const bf16*>(p.b2)[tid]);
  if (tid < C) brs[tid] = tof(static_cast<const bf16*>(p.b_r)[tid]);

  const int N = p.B * p.T;
  const int tok = blockIdx.x * kRtTok + 16 * w + l16;
  const bool valid = tok < N;
  const bf16* hrow = static_cast<const bf16*>(p.h) + static_cast<size_t>(valid ? tok : 0) * d + 8 * g4;

  u32x4 wr[5];
  auto load_w = [&](int kc) {
#pragma unroll
    for (int r = 0; r < 5; ++r) {
      const int pc = tid + 256 * r;
      u32x4 val = {0u, 0u, 0u, 0u};
      if (pc < kRtRows * 8) {
        const int row = pc >> 3, c8 = pc & 7;
        if (row < Hr)
          val = *reinterpret_cast<const u32x4*>(W1 + row * W1s + kc + 8 * c8);
        else if (row - Hr < C)
          val = *reinterpret_cast<const u32x4*>(Wr + static_cast<size_t>(row - Hr) * d + kc + 8 * c8);
      }
      wr[r] = val;
    }
  };
  auto store_w = [&](int buf) {
#pragma unroll
    for (int r = 0; r < 5; ++r) {
      const int pc = tid + 256 * r;
      if (pc < kRtRows * 8) {
        const int row = pc >> 3, c8 = pc & 7;
        *reinterpret_cast<u32x4*>(&Ws[buf][row * kRtLd + 8 * c8]) = wr[r];
      }
    }
  };
  bf16x8 hb0, hb1;
  auto load_h = [&](int kc) {
    const bf16x8 zero = {};
    hb0 = valid ? *reinterpret_cast<const bf16x8*>(hrow + kc) : zero;
    hb1 = valid ? *reinterpret_cast<const bf16x8*>(hrow + kc + 32) : zero;
  };

  f32x4 acc[9];
#pragma unroll
  for (int m = 0; m < 9; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nch = d / kRtKc;
  load_w(0);
  load_h(0);
  store_w(0);
  for (int c = 0; c < nch; ++c) {
    __syncthreads();
    const bf16x8 h0 = hb0, h1 = hb1;
    if (c + 1 < nch) {
      load_w((c + 1) * kRtKc);
      load_h((c + 1) * kRtKc);
    }
    const bf16* Wb = Ws[c & 1];
#pragma unroll
    for (int m = 0; m < 9; ++m) {
      const bf16* ar = Wb + (16 * m + l16) * kRtLd + 8 * g4;
      acc[m] = mfma_16x16x32(*reinterpret_cast<const bf16x8*>(ar), h0, acc[m]);
      acc[m] = mfma_16x16x32(*reinterpret_cast<const bf16x8*>(ar + 32), h1, acc[m]);
    }
    if (c + 1 < nch) store_w((c + 1) & 1);
  }

  // ---- epilogue: lanes l16, l16+16, l16+32, l16+48 hold token `tok`
  const int b = valid ? tok / p.T : 0;
  const int type = valid ? p.types[tok] : 0;
  float ex[4], mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = 4 * g4 + i;
    ex[i] = c < C ? acc[8][i] + brs[c] : -INFINITY;
    mx = fmaxf(mx, ex[i]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
  mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
  float sm = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ex[i] = (4 * g4 + i < C) ? expf(ex[i] - mx) : 0.f;
    sm += ex[i];
  }
  sm += __shfl_xor(sm, 16, kWave);
  sm += __shfl_xor(sm, 32, kWave);
  const float isum = 1.f / sm;
  float a[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) a[c] = __shfl(ex[c & 3], l16 + 16 * (c >> 2), kWave) * isum;

  const float* cb = p.cb + static_cast<size_t>(b) * Hr;
  float gam[32];
#pragma unroll
  for (int s = 0; s < 32; ++s) gam[s] = 0.f;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 16 * m + 4 * g4 + i;
      float x = acc[m][i] + cb[j];
#pragma unroll
      for (int c = 0; c < 16; ++c)
        if (c < C) x += Fs[j * C + c] * a[c];
      const float gl = gelu_exact(x);
#pragma unroll
      for (int s = 0; s < 32; ++s)
        if (s < G) gam[s] += tof(W2s[s * Hr + j]) * gl;
    }
  }
  int n_above = 0;
#pragma unroll
  for (int s = 0; s < 32; ++s) {
    if (s < G) {
      gam[s] += __shfl_xor(gam[s], 16, kWave);
      gam[s] += __shfl_xor(gam[s], 32, kWave);
      gam[s] += b2s[s];
      n_above += gam[s] > p.tau;
    }
  }
  // the four lanes of a token now hold bitwise-identical scores
  const int K = budget_k(p.mode, p.k_by_type, type, p.tau, p.kmin, p.kmax, G, n_above);
  uint32_t m = 0;
  if (p.mode == 1 && K == n_above) {
#pragma unroll
    for (int s = 0; s < 32; ++s)
      if (s < G && gam[s] > p.tau) m |= 1u << s;
  } else {
#pragma unroll
    for (int s = 0; s < 32; ++s) {
      if (s < G && (s & 3) == g4) {
        int rank = 0;
#pragma unroll
        for (int t = 0; t < 32; ++t)
          if (t < G) rank += key_above(gam[t], gam[s]) || (t < s && key_equal(gam[t], gam[s]));
        if (rank < K) m |= 1u << s;
      }
    }
    m |= __shfl_xor(m, 16, kWave);
    m |= __shfl_xor(m, 32, kWave);
  }
  if (valid) {
    if (p.scores_out) {
#pragma unroll
      for (int s = 0; s < 32; ++s)
        if (s < G && (s & 3) == g4) p.scores_out[static_cast<size_t>(tok) * G + s] = gam[s];
    }
    if (g4 == 0) write_selection(p, tok, m);
  }
}

}  // namespace

hipError_t launch_route(const RouteParams& p, bool bf16, hipStream_t s) {
  const size_t ntok = static_cast<size_t>(p.B) * p.T;
  if (ntok == 0) return hipSuccess;
  const size_t prep_shm = static_cast<size_t>(p.d) * sizeof(float);
  if (bf16)
    hipLaunchKernelGGL(k_route_prep<rolesub::bf16>, dim3(p.B + 1), dim3(256), prep_shm, s, p);
  else
    hipLaunchKernelGGL(k_route_prep<float>, dim3(p.B + 1), dim3(256), prep_shm, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool mfma_ok = bf16 && p.kind == 0 && p.Hr == 128 && p.C >= 1 && p.C <= 16 &&
                       p.G <= 32 && p.d % kRtKc == 0 && ntok < (1u << 30);
  if (mfma_ok) {
    const unsigned nblk = static_cast<unsigned>((ntok + kRtTok - 1) / kRtTok);
    hipLaunchKernelGGL(k_route_mlp2_bf16, dim3(nblk), dim3(256), 0, s, p);
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
  hipLaunchKernelGGL(k_select, dim3(static_cast<unsigned>((ntok + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace rolesub
