// Compact group-indexed value cache: the kept groups of z~ = M z (Sec. 3.2).
//
// offsets[b, i] = sum_{j<i} popcount(mask[b, j]) (group units, shared by all
// heads); Vp[b, h, offsets[b, i] + r] = r-th kept group (ascending id) of
// token i, head h. The copy is byte-exact, so it is dtype-agnostic.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace rolesub {
namespace {

__device__ __forceinline__ uint32_t group_mask(int G) { return G >= 32 ? 0xFFFFFFFFu : ((1u << G) - 1u); }

// One workgroup per sample: exclusive scan of the per-token kept counts,
// 256 tokens per step (wave scans + a carry).
__global__ __launch_bounds__(256) void k_pack_offsets(const uint32_t* __restrict__ mask,
                                                      int32_t* __restrict__ off, int T, int G) {
  __shared__ int wsum[4];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint32_t gm = group_mask(G);
  const uint32_t* mb = mask + static_cast<size_t>(b) * T;
  int32_t* ob = off + static_cast<size_t>(b) * (T + 1);
  int carry = 0;
  for (int base = 0; base < T; base += 256) {
    const int t = base + tid;
    const int c = t < T ? __popc(mb[t] & gm) : 0;
    int x = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, kWave);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int pre = 0;
    for (int i = 0; i < w; ++i) pre += wsum[i];
    const int tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    if (t < T) ob[t] = carry + pre + x - c;
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) ob[T] = carry;
}

// Scatter. A workgroup owns (sample b, 64 tokens, 8 heads). It first builds a
// slot -> (token, group) table for its tokens in LDS, then copies: consecutive
// threads take consecutive VB-byte pieces of consecutive slots of one head, so
// the writes into Vp[b, h, :] are contiguous.
constexpr int kPkT = 64, kPkH = 8;

template <int VB>
__global__ __launch_bounds__(256) void k_pack_scatter(const char* __restrict__ z,
                                                      const uint32_t* __restrict__ mask,
                                                      const int32_t* __restrict__ off,
                                                      char* __restrict__ Vp, int T, int H, int dh,
                                                      int G, int esz, int64_t cap) {
  typedef typename std::conditional<VB == 16, u32x4, typename std::conditional<VB == 8, u32x2, uint32_t>::type>::type V;
  __shared__ uint16_t src_of_slot[kPkT * 32];
  const int b = blockIdx.y, t0 = blockIdx.x * kPkT, h0 = blockIdx.z * kPkH;
  const int nt = min(kPkT, T - t0), nh = min(kPkH, H - h0);
  const int ds = dh / G, gbytes = ds * esz, pieces = gbytes / VB;
  const uint32_t gm = group_mask(G);
  const int32_t* ob = off + static_cast<size_t>(b) * (T + 1);
  const int base = ob[t0];
  const int n = ob[t0 + nt] - base;
  if (static_cast<int>(threadIdx.x) < nt) {
    const int t = t0 + threadIdx.x;
    uint32_t m = mask[static_cast<size_t>(b) * T + t] & gm;
    int o = ob[t] - base;
    while (m) {
      const int g = __ffs(m) - 1;
      src_of_slot[o++] = static_cast<uint16_t>((threadIdx.x << 5) | g);
      m &= m - 1;
    }
  }
  __syncthreads();
  const uint32_t zrow = static_cast<uint32_t>(H) * dh * esz;
  // this workgroup's source rows; out-of-range items load as zero and are not stored
  const rsrc_t r_z = make_rsrc(z + (static_cast<size_t>(b) * T + t0) * zrow, static_cast<uint32_t>(nt) * zrow);
  const int items = nh * n * pieces;
  constexpr int U = 4;  // loads issued before their stores
  for (int i0 = threadIdx.x; i0 < items; i0 += 256 * U) {
    V val[U];
    char* dst[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + 256 * u;
      const int piece = i % pieces;
      const int rest = i / pieces;
      const int sl = n ? rest % n : 0;
      const int h = h0 + (n ? rest / n : 0);
      const int64_t slot = static_cast<int64_t>(base) + sl;
      const bool ok = i < items && slot < cap;
      const int e = src_of_slot[ok ? sl : 0];
      const int tl = e >> 5, g = e & 31;
      const uint32_t so = static_cast<uint32_t>(tl) * zrow + static_cast<uint32_t>((h * dh + g * ds) * esz + piece * VB);
      const uint32_t off = ok ? so : kOOB;
      if constexpr (VB == 16) val[u] = bload16(r_z, off);
      else if constexpr (VB == 8) val[u] = bload8(r_z, off);
      else val[u] = bload4(r_z, off);
      dst[u] = ok ? Vp + ((static_cast<size_t>(b) * H + h) * cap + slot) * gbytes + piece * VB : nullptr;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (dst[u]) *reinterpret_cast<V*>(dst[u]) = val[u];
  }
}

}  // namespace

hipError_t launch_pack_offsets(int B, int T, int G, const uint32_t* mask, int32_t* offsets, hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_offsets, dim3(B), dim3(256), 0, s, mask, offsets, T, G);
  return hipGetLastError();
}

hipError_t launch_pack(bool bf16, int B, int T, int H, int dh, int G, const void* z,
                       const uint32_t* mask, int32_t* offsets, void* Vp, int64_t cap,
                       hipStream_t s) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_offsets, dim3(B), dim3(256), 0, s, mask, offsets, T, G);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || T == 0 || H == 0 || cap == 0) return e;
  const int esz = bf16 ? 2 : 4;
  const int gbytes = (dh / G) * esz;
  const dim3 grid((T + kPkT - 1) / kPkT, B, (H + kPkH - 1) / kPkH);
  const char* zc = static_cast<const char*>(z);
  char* vc = static_cast<char*>(Vp);
  if (gbytes % 16 == 0)
    hipLaunchKernelGGL(k_pack_scatter<16>, grid, dim3(256), 0, s, zc, mask, offsets, vc, T, H, dh, G, esz, cap);
  else if (gbytes % 8 == 0)
    hipLaunchKernelGGL(k_pack_scatter<8>, grid, dim3(256), 0, s, zc, mask, offsets, vc, T, H, dh, G, esz, cap);
  else
    hipLaunchKernelGGL(k_pack_scatter<4>, grid, dim3(256), 0, s, zc, mask, offsets, vc, T, H, dh, G, esz, cap);
  return hipGetLastError();
}

}  // namespace rolesub
