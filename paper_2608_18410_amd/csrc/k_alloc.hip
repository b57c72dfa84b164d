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
typedef u64 u64x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t priority_weight(float x) {
  if (!(x > 0.f)) return 0u;  // NaN, zero and negative priorities
  // x * 2^16 <= 2^24 is exact in f32, and so is its floor
  return static_cast<uint32_t>(floorf(fminf(x, 256.f) * 65536.f));
}

__device__ __forceinline__ u64 wave_sum(u64 x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}

// Sum over the 256 threads of the workgroup; every thread gets the total. One
// barrier: `slot` must not be written again until every thread has passed
// another barrier.
__device__ __forceinline__ u64 block_sum(u64 x, u64* slot) {
  x = wave_sum(x);
  if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = x;
  __syncthreads();
  return slot[0] + slot[1] + slot[2] + slot[3];
}

// The K highest-scoring of a token's G scores (larger first, equal scores to
// the lower group index, -0 equal to +0, NaN last) as a bit mask.
template <int GP>
__device__ __forceinline__ uint32_t top_k_mask(const float (&g)[GP], int G, int K) {
  return top_k_pairs<GP>(g, G, K);
}

template <int GP>
__device__ __forceinline__ void load_scores(const float* src, int G, float (&g)[GP]) {
  if ((G & 3) == 0) {
#pragma unroll
    for (int s = 0; s < GP; s += 4) {
      const f32x4 v = s < G ? *reinterpret_cast<const f32x4*>(src + s) : f32x4{0.f, 0.f, 0.f, 0.f};
      g[s] = v[0];
      g[s + 1] = v[1];
      g[s + 2] = v[2];
      g[s + 3] = v[3];
    }
  } else {
#pragma unroll
    for (int s = 0; s < GP; ++s) g[s] = s < G ? src[s] : 0.f;
  }
}

// One workgroup per (sample, m): m = 0..3 the token types, m = 4 every token of
// another type. Tokens of the type are listed in index order in LDS; each
// thread owns list entries j = tid, tid + 256, ... GP >= G bounds the unrolled
// selection loops.
template <int GP>
__global__ __launch_bounds__(256) void k_allocate(AllocParams p) {
  constexpr uint8_t kCap = 0xFF;
  constexpr u64 kLow40 = (1ull << 40) - 1;
  __shared__ uint32_t wq[kAllocMaxT];  // integer priority weights
  __shared__ __attribute__((aligned(16))) u64 rem[kAllocMaxT + 2];  // remainders of the shares
  __shared__ uint16_t tok[kAllocMaxT]; // token index in the sample
  __shared__ uint8_t kk[kAllocMaxT];   // allocated K (kCap while capped)
  // block-sum slots: 0 and 1 alternate over the capping rounds, 2 the floors,
  // 3 the listing
  __shared__ u64 red[4][4];
  __shared__ int wsum[4];
  const int b = blockIdx.x / 5, m = blockIdx.x % 5;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int G = p.G, T = p.T;
  const uint8_t* ty = p.types + static_cast<size_t>(b) * T;
  const float* pr = p.priority + static_cast<size_t>(b) * T;
  const int km = m < 4 ? min(p.k_by_type[m], G) : G;
  const bool alloc = km > 0 && km < G;

  // the type's tokens in index order (block-wide scan of membership flags),
  // with the sum of their weights
  int n = 0;
  u64 qsum = 0;
  for (int c0 = 0; c0 < T; c0 += 256) {
    const int t = c0 + tid;
    // both loads issued together (the priority is not needed for most tokens)
    const int tt = t < T ? static_cast<int>(ty[t]) : -1;
    const float pv = (t < T && alloc) ? pr[t] : 0.f;
    const bool mine = m < 4 ? tt == m : tt > 3;
    const uint32_t wt = mine ? priority_weight(pv) : 0u;
    const uint64_t bal = __ballot(mine);
    const u64 ws = wave_sum(static_cast<u64>(wt));
    if (lane == 0) {
      wsum[w] = __popcll(bal);
      red[3][w] = ws;
    }
    __syncthreads();
    int off = n + __popcll(bal & ((1ull << lane) - 1ull));
    for (int v = 0; v < w; ++v) off += wsum[v];
    if (mine) {
      tok[off] = static_cast<uint16_t>(t);
      wq[off] = wt;
      kk[off] = 0;
    }
    n += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    qsum += red[3][0] + red[3][1] + red[3][2] + red[3][3];
    __syncthreads();
  }
  if (n == 0) return;  // n is the same in every thread

  // this thread's first token's scores, in flight during the allocation
  float g0[GP];
  const bool sel = p.scores != nullptr;
  if (sel && tid < n) load_scores<GP>(p.scores + (static_cast<size_t>(b) * T + tok[tid]) * G, G, g0);

  if (!alloc) {
    for (int j = tid; j < n; j += 256) kk[j] = static_cast<uint8_t>(km);
  } else {
    // capping rounds; every round that caps a token removes its weight and
    // its G groups, so one packed sum per round (capped weight, count) keeps
    // Q, the active count and the budget current
    u64 Bm = static_cast<u64>(km) * n, Q = qsum, na = static_cast<u64>(n);
    for (int round = 0; round <= n; ++round) {
      const bool uni = Q == 0;  // only zero weights left: equal shares
      const u64 QQ = uni ? na : Q;
      u64 part = 0;
      for (int j = tid; j < n; j += 256) {
        if (kk[j] == kCap) continue;
        const u64 wj = uni ? 1ull : wq[j];
        if (Bm * wj > static_cast<u64>(G) * QQ) {
          kk[j] = kCap;
          part += wq[j] + (1ull << 40);
        }
      }
      part = block_sum(part, red[round & 1]);
      const u64 over = part >> 40;
      if (over == 0 || over == na) break;  // the second never holds while K_m < G
      Q -= part & kLow40;
      na -= over;
      Bm -= static_cast<u64>(G) * over;
    }
    // proportional shares of the uncapped tokens: floor and remainder
    const bool uni = Q == 0;
    const u64 QQ = uni ? na : Q;
    u64 fsum = 0;
    for (int j = tid; j < n; j += 256) {
      if (kk[j] == kCap) {
        kk[j] = static_cast<uint8_t>(G);
        rem[j] = 0;
      } else {
        const u64 prod = Bm * (uni ? 1ull : wq[j]);
        const u64 f = prod / QQ;
        rem[j] = prod - f * QQ;
        kk[j] = static_cast<uint8_t>(f);
        fsum += f;
      }
    }
    // pad to an even count: remainder 0 past every token never ranks before one
    if (tid == 0) rem[n] = 0;
    const u64 left = Bm - block_sum(fsum, red[2]);  // < number of positive remainders
    if (left > 0 && n <= 128) {
      // one more group to the `left` largest remainders, lower index first
      // (capped tokens carry remainder 0 and never rank above a positive one,
      // and a token with remainder 0 never gets one). Short lists: tpt lanes
      // of one wave share a token, each counting over every tpt-th pair.
      int tpt = 1;
      while (tpt < 64 && 2 * tpt * n <= 256) tpt *= 2;
      const int j = tid / tpt, sub = tid % tpt;
      const u64 r = j < n ? rem[j] : 0;
      int rank = 0;
      if (j < n && r != 0) {
        for (int i = 2 * sub; i < n; i += 2 * tpt) {
          const u64x2 ri = *reinterpret_cast<const u64x2*>(rem + i);
          rank += static_cast<int>((ri[0] > r) | ((ri[0] == r) & (i < j)));
          rank += static_cast<int>((ri[1] > r) | ((ri[1] == r) & (i + 1 < j)));
        }
      }
      for (int o = 1; o < tpt; o <<= 1) rank += __shfl_xor(rank, o, kWave);
      if (j < n && sub == 0 && r != 0 && rank < static_cast<int>(left)) kk[j] = static_cast<uint8_t>(kk[j] + 1);
      __syncthreads();  // kk[j] is read below by thread j, not by the lane that updated it
    } else if (left > 0) {
      for (int j = tid; j < n; j += 256) {
        const u64 r = rem[j];
        if (r == 0) continue;
        int rank = 0;
#pragma unroll 4
        for (int i = 0; i < n; i += 2) {
          const u64x2 ri = *reinterpret_cast<const u64x2*>(rem + i);  // same address in every lane
          rank += static_cast<int>((ri[0] > r) | ((ri[0] == r) & (i < j)));
          rank += static_cast<int>((ri[1] > r) | ((ri[1] == r) & (i + 1 < j)));
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
    if (!sel) continue;
    float g[GP];
    if (j == tid) {
#pragma unroll
      for (int s = 0; s < GP; ++s) g[s] = g0[s];
    } else {
      load_scores<GP>(p.scores + t * G, G, g);
    }
    const uint32_t msk = top_k_mask<GP>(g, G, K);
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
  const dim3 grid(static_cast<unsigned>(p.B) * 5u);
  if (p.G <= 8) hipLaunchKernelGGL(k_allocate<8>, grid, dim3(256), 0, s, p);
  else if (p.G <= 16) hipLaunchKernelGGL(k_allocate<16>, grid, dim3(256), 0, s, p);
  else hipLaunchKernelGGL(k_allocate<32>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace rolesub
