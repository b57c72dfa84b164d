// Token-level retention ahead of the routed path (Sec. 3.1; Sec. 4.1):
// per sample and per segment of consecutive tokens (a camera view), keep the
// highest-scoring tokens, then gather the kept tokens' rows.
#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

// Order-preserving unsigned key of a score: a larger score gives a larger
// key, -0 and +0 give the same key, and NaN gives 0, below every number.
__device__ __forceinline__ uint32_t score_key(float x) {
  if (x != x) return 0u;
  const uint32_t u = __float_as_uint(x == 0.f ? 0.f : x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// One workgroup per (sample, segment). Token i of the segment is kept when
// fewer than keep tokens rank before it: a larger key, or an equal key at a
// lower index. Kept tokens are written in index order (block-wide scan of the
// keep flags).
__global__ __launch_bounds__(256) void k_retain(RetainParams p) {
  __shared__ __attribute__((aligned(16))) uint32_t keys[kRetainMaxSeg + 4];
  __shared__ int wsum[4];
  const int b = blockIdx.x / p.n_seg, sg = blockIdx.x % p.n_seg;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = p.seg_len[sg], start = p.seg_start[sg], keep = p.seg_keep[sg];
  const float* sc = p.scores + static_cast<size_t>(b) * p.N + start;
  for (int i = tid; i < n; i += 256) keys[i] = score_key(sc[i]);
  // padding up to a multiple of 4: key 0 at an index past every token never
  // ranks before one (0 is not above any key, and equal keys need j < i)
  if (tid < 4) keys[n + tid] = 0u;
  __syncthreads();
  int32_t* out = p.keep_idx + static_cast<size_t>(b) * p.K + p.seg_out[sg];
  int base = 0;  // kept tokens before this chunk
  for (int c0 = 0; c0 < n; c0 += 256) {
    const int i = c0 + tid;
    bool kept = false;
    if (i < n && keep > 0) {
      const uint32_t ki = keys[i];
      int rank = 0;
      // four keys per 16-byte read; the same address in every lane is a broadcast
#pragma unroll 4
      for (int j = 0; j < n; j += 4) {
        const u32x4 kj = *reinterpret_cast<const u32x4*>(keys + j);
#pragma unroll
        for (int e = 0; e < 4; ++e) rank += (kj[e] > ki) | ((kj[e] == ki) & (j + e < i));
      }
      kept = rank < keep;
    }
    const uint64_t bal = __ballot(kept);
    const int pre = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[w] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int v = 0; v < w; ++v) off += wsum[v];
    if (kept) out[off + pre] = start + i;
    base += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
  }
}

// dst[b, j, :] = src[b, idx[b, j], :], rows of row_bytes (a multiple of 4).
// One workgroup per (sample, kept token); 16-byte pieces when row_bytes allows.
// An index outside [0, N) falls outside the sample's buffer resource and
// gives a zero row.
__global__ __launch_bounds__(256) void k_gather_rows(GatherParams p) {
  const size_t row = blockIdx.x;
  const int b = static_cast<int>(row / p.K);
  const int32_t t = p.idx[row];
  const uint32_t rb = static_cast<uint32_t>(p.row_bytes);
  const rsrc_t r_src = make_rsrc(static_cast<const char*>(p.src) + static_cast<size_t>(b) * p.N * p.row_bytes,
                                 clamp_bytes(static_cast<size_t>(p.N) * p.row_bytes));
  const rsrc_t r_dst = make_rsrc(static_cast<char*>(p.dst) + row * p.row_bytes, rb);
  const bool in = (t >= 0) & (t < p.N);
  const uint32_t so = in ? static_cast<uint32_t>(t) * rb : kOOB;
  if ((rb & 15u) == 0) {
    // four 16-byte loads in flight per thread before their stores
    for (uint32_t o0 = 16u * threadIdx.x; o0 < rb; o0 += 4u * 16u * 256u) {
      u32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t o = o0 + u * 16u * 256u;
        v[u] = bload16(r_src, (so == kOOB) | (o >= rb) ? kOOB : so + o);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t o = o0 + u * 16u * 256u;
        __builtin_amdgcn_raw_buffer_store_b128(v[u], r_dst, o < rb ? o : kOOB, 0, 0);
      }
    }
  } else {
    for (uint32_t o = 4u * threadIdx.x; o < rb; o += 4u * 256u) {
      const uint32_t v = bload4(r_src, so == kOOB ? kOOB : so + o);
      __builtin_amdgcn_raw_buffer_store_b32(v, r_dst, o, 0, 0);
    }
  }
}

}  // namespace

hipError_t launch_retain(const RetainParams& p, hipStream_t s) {
  if (p.B == 0 || p.n_seg == 0 || p.K == 0) return hipSuccess;
  hipLaunchKernelGGL(k_retain, dim3(static_cast<unsigned>(p.B * p.n_seg)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const GatherParams& p, hipStream_t s) {
  if (p.B == 0 || p.K == 0 || p.row_bytes == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows, dim3(static_cast<unsigned>(static_cast<size_t>(p.B) * p.K)), dim3(256), 0, s,
                     p);
  return hipGetLastError();
}

}  // namespace rolesub
