// Role-driven within-type budget allocation (Sec. 3.5) followed by the Top-K_i
// group selection (Sec. 3.4).
//
// For every sample and token type m the B_m = K_m * n_m value groups of the
// type's n_m tokens are apportioned by integer priority weights
// w_i = floor(min(max(p_i, 0), 256) * 2^16) (NaN as 0): a token whose share
// B * w_i / Q exceeds G keeps G and the remaining groups are shared again
// among the others; the shares are then rounded by largest remainders, equal
// remainders to the lower token index. All-zero weights count as equal.
// K_m = 0 and K_m >= G need no allocation; tokens of a type other than the four
// keep all G groups. Everything is exact integer arithmetic, so the result does
// not depend on the order of any sum.
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

using u64 = unsigned long long;

__device__ __forceinline__ uint32_t priority_weight(float x) {
  if (!(x > 0.f)) return 0u;  // NaN, zero and negative priorities
  // x * 2^16 <= 2^24 is exact in f32, and so is its floor
  return static_cast<uint32_t>(floorf(fminf(x, 256.f) * 65536.f));
}

// Sum over the 256 threads of the workgroup; every thread gets the total.
__device__ __forceinline__ u64 block_sum(u64 x, u64* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  const u64 s = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return s;
}

// One workgroup per (sample, m): m = 0..3 the token types, m = 4 every token of
// another type. Tokens of the type are listed in index order in LDS; each
// thread owns list entries j = tid, tid + 256, ...
__global__ __launch_bounds__(256) void k_allocate(AllocParams p) {
  constexpr uint8_t kCap = 0xFF;
  __shared__ uint32_t wq[kAllocMaxT];  // integer priority weights
  __shared__ u64 rem[kAllocMaxT];      // remainders of the proportional shares
  __shared__ uint16_t tok[kAllocMaxT]; // token index in the sample
  __shared__ uint8_t kk[kAllocMaxT];   // allocated K (kCap while capped)
  __shared__ u64 red[4];
  __shared__ int wsum[4];
  const int b = blockIdx.x / 5, m = blockIdx.x % 5;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int G = p.G, T = p.T;
  const uint8_t* ty = p.types + static_cast<size_t>(b) * T;
  const float* pr = p.priority + static_cast<size_t>(b) * T;
  const int km = m < 4 ? min(p.k_by_type[m], G) : G;
  const bool alloc = km > 0 && km < G;

  // the type's tokens in index order (block-wide scan of membership flags)
  int n = 0;
  for (int c0 = 0; c0 < T; c0 += 256) {
    const int t = c0 + tid;
    const int tt = t < T ? static_cast<int>(ty[t]) : -1;
    const bool mine = m < 4 ? tt == m : tt > 3;
    const uint64_t bal = __ballot(mine);
    if (lane == 0) wsum[w] = __popcll(bal);
    __syncthreads();
    int off = n + __popcll(bal & ((1ull << lane) - 1ull));
    for (int v = 0; v < w; ++v) off += wsum[v];
    if (mine) {
      tok[off] = static_cast<uint16_t>(t);
      wq[off] = alloc ? priority_weight(pr[t]) : 0u;
      kk[off] = 0;
    }
    n += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
  }
  if (n == 0) return;  // n is the same in every thread

  if (!alloc) {
    for (int j = tid; j < n; j += 256) kk[j] = static_cast<uint8_t>(km);
  } else {
    // capping rounds: every round caps at least one token, at most n rounds
    u64 Bm = static_cast<u64>(km) * n;
    u64 Q = 1;
    bool uni = false;
    for (int round = 0; round <= n; ++round) {
      u64 part = 0;  // active weight sum (low 40 bits) and active count (high bits)
      for (int j = tid; j < n; j += 256)
        if (kk[j] != kCap) part += wq[j] + (1ull << 40);
      part = block_sum(part, red);
      const u64 qs = part & ((1ull << 40) - 1), na = part >> 40;
      uni = qs == 0;
      Q = uni ? na : qs;
      u64 over = 0;
      for (int j = tid; j < n; j += 256) {
        if (kk[j] == kCap) continue;
        const u64 wj = uni ? 1ull : wq[j];
        if (Bm * wj > static_cast<u64>(G) * Q) {
          kk[j] = kCap;
          ++over;
        }
      }
      over = block_sum(over, red);
      if (over == 0 || na == over) break;  // the second never holds while K_m < G
      Bm -= static_cast<u64>(G) * over;
    }
    // proportional shares of the uncapped tokens: floor and remainder
    u64 fsum = 0;
    for (int j = tid; j < n; j += 256) {
      if (kk[j] == kCap) {
        kk[j] = static_cast<uint8_t>(G);
        rem[j] = 0;
      } else {
        const u64 prod = Bm * (uni ? 1ull : wq[j]);
        const u64 f = prod / Q;
        rem[j] = prod - f * Q;
        kk[j] = static_cast<uint8_t>(f);
        fsum += f;
      }
    }
    const u64 left = Bm - block_sum(fsum, red);  // < number of positive remainders
    if (left > 0) {
      // one more group to the `left` largest remainders, lower index first
      // (capped tokens carry remainder 0 and never rank above a positive one)
      for (int j = tid; j < n; j += 256) {
        const u64 r = rem[j];
        u64 rank = 0;
        for (int i = 0; i < n; ++i) {
          const u64 ri = rem[i];
          rank += static_cast<u64>((ri > r) | ((ri == r) & (i < j)));
        }
        if (rank < left) kk[j] = static_cast<uint8_t>(kk[j] + 1);
      }
    }
  }

  // K_i out, then the K_i highest-scoring groups of each token
  for (int j = tid; j < n; j += 256) {
    const size_t t = static_cast<size_t>(b) * T + tok[j];
    const int K = kk[j];
    if (p.k_out) p.k_out[t] = static_cast<uint8_t>(K);
    if (!p.scores) continue;
    float g[32];
    const float* src = p.scores + t * G;
#pragma unroll
    for (int s = 0; s < 32; ++s) g[s] = s < G ? src[s] : 0.f;
    uint32_t msk = 0;
#pragma unroll
    for (int s = 0; s < 32; ++s) {
      int rank = 0;
#pragma unroll
      for (int u = 0; u < 32; ++u) {
        const bool before = key_above(g[u], g[s]) || (u < s && key_equal(g[u], g[s]));
        rank += static_cast<int>(u < G && before);
      }
      msk |= static_cast<uint32_t>((s < G) & (rank < K)) << s;
    }
    p.mask[t] = msk;
    if (p.count) p.count[t] = static_cast<uint8_t>(__popc(msk));
    if (p.idx) {
      uint8_t* o = p.idx + t * G;
      int r = 0;
      for (int s = 0; s < G; ++s)
        if ((msk >> s) & 1u) o[r++] = static_cast<uint8_t>(s);
      for (; r < G; ++r) o[r] = 0xFF;
    }
  }
}

}  // namespace

hipError_t launch_allocate(const AllocParams& p, hipStream_t s) {
  if (p.B == 0 || p.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_allocate, dim3(static_cast<unsigned>(p.B) * 5u), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace rolesub
