// Shared device types and helpers of librolesub (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rolesub {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float tof(float x) { return x; }
__device__ __forceinline__ float tof(bf16 x) { return static_cast<float>(x); }

template <class T> __device__ __forceinline__ T fromf(float x);
template <> __device__ __forceinline__ float fromf<float>(float x) { return x; }
// float -> bf16 conversion rounds to nearest even (v_cvt_pk_bf16_f32 on gfx950).
template <> __device__ __forceinline__ bf16 fromf<bf16>(float x) { return static_cast<bf16>(x); }

// D = A(16x32) * B(32x16) + C on the bf16 matrix cores.
// Lane l holds: A row l%16, k = 8*(l/16) .. +8;  B column l%16, same k;
//               C/D column l%16, rows 4*(l/16) .. +4.
__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16 a = static_cast<bf16>(lo), b = static_cast<bf16>(hi);
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, a)) |
         (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b)) << 16);
}

// Raw buffer loads. A load whose byte offset is at or past the resource's
// size returns zeros without touching memory, so masked or out-of-range
// elements need no branch around the load (a branch would force a wait for
// every outstanding load at its join). Resources must cover < 2 GiB so that
// kOOB is always out of range.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;  // gfx9 family: 32-bit data format, untyped access

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), kRsrcWord3);
}
__device__ __forceinline__ u32x4 bload16(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0));
}
__device__ __forceinline__ u32x2 bload8(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(off), 0, 0));
}
__device__ __forceinline__ uint32_t bload4(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, static_cast<int>(off), 0, 0);
}
// Offset v for lanes with ok, else kOOB. The empty asm pins v as computed
// unconditionally: otherwise the compiler may move an expensive operand (a
// division, a 64-bit product) under a branch, and a branch around memory
// operations makes later waits cover every outstanding one.
__device__ __forceinline__ uint32_t oob_unless(bool ok, uint32_t v) {
  asm volatile("" : "+v"(v));
  return ok ? v : kOOB;
}
__device__ __forceinline__ uint32_t clamp_bytes(size_t n) {
  return n < kOOB ? static_cast<uint32_t>(n) : kOOB;
}

// Asynchronous copy of 16 bytes per lane from a buffer resource into LDS:
// lane i writes LDS bytes [lds_base + 16 i, lds_base + 16 i + 16); an
// out-of-range offset writes zeros. The load is issued through inline
// assembly so that the compiler does not serialise later LDS reads behind it;
// the caller waits with wait_vmcnt<N>() before reading the data.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>((uintptr_t)((__attribute__((address_space(3))) const char*)p));
}
__device__ __forceinline__ void dma16(rsrc_t r, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(r)
               : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// Group-selection order (top-K_i, Sec. 3.4): a larger score ranks first,
// -0 and +0 are equal, NaN ranks after every number, equal keys go to the
// lower group index.
__device__ __forceinline__ bool key_above(float a, float b) {
  return !__builtin_isnan(a) && (__builtin_isnan(b) || a > b);
}
__device__ __forceinline__ bool key_equal(float a, float b) {
  return (a == b) || (__builtin_isnan(a) && __builtin_isnan(b));
}

// The same order as an unsigned integer: order_key(a) > order_key(b) exactly
// when key_above(a, b), and equal keys exactly when key_equal(a, b). Sign and
// magnitude become one monotone code (negatives bit-flipped, positives with
// the top bit set); every NaN maps to 0, below -inf's code.
__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t u = x == 0.f ? 0u : __float_as_uint(x);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return __builtin_isnan(x) ? 0u : u;
}

// Top-K of the first G of NP scores, in the order above, as a bit mask. Each
// unordered pair s < t is compared once: s wins when its key is at least t's
// (equal keys go to the lower index), and the loser's rank (the number of
// groups ranked before it) goes up by one. Entries past G get key 0 and lose
// to every real group, which sits at a lower index; rank[s] starts at the
// number of later entries and drops by one per later entry s beats.
template <int NP>
__device__ __forceinline__ uint32_t top_k_pairs(const float* g, int G, int K) {
  uint32_t key[NP];
  int rank[NP];
#pragma unroll
  for (int s = 0; s < NP; ++s) {
    key[s] = s < G ? order_key(g[s]) : 0u;
    rank[s] = NP - 1 - s;
  }
#pragma unroll
  for (int s = 0; s < NP; ++s) {
#pragma unroll
    for (int t = s + 1; t < NP; ++t) {
      const int c = key[s] >= key[t];
      rank[t] += c;
      rank[s] -= c;
    }
  }
  uint32_t m = 0;
#pragma unroll
  for (int s = 0; s < NP; ++s) m |= static_cast<uint32_t>((s < G) & (rank[s] < K)) << s;
  return m;
}

// Number of groups kept by one token (Sec. 3.5).
__device__ __forceinline__ int budget_k(int mode, const int* k_by_type, int type, float tau,
                                        int kmin, int kmax, int G, int n_above) {
  int k;
  if (mode == 0) {
    k = (type >= 0 && type < 4) ? k_by_type[type] : G;
  } else {
    k = n_above < kmin ? kmin : (n_above > kmax ? kmax : n_above);
  }
  return k < G ? k : G;
}

// Pairwise combination with the lane 16 (or 32) positions away, i.e.
// x op (x of lane l ^ 16): v_permlane16_swap / v_permlane32_swap exchange the
// 16-lane rows (32-lane halves) of two copies of x in one VALU instruction,
// leaving each lane with {x, partner} in some order; op is commutative, so the
// result is bitwise that of the operands in either order (a cross-lane
// shuffle goes through the LDS crossbar and costs an LDS round trip).
__device__ __forceinline__ void swap16(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void swap32(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ float add_xor16(float x) {
  uint32_t a, b;
  swap16(__float_as_uint(x), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}
__device__ __forceinline__ float add_xor32(float x) {
  uint32_t a, b;
  swap32(__float_as_uint(x), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}
__device__ __forceinline__ float max_xor16(float x) {
  uint32_t a, b;
  swap16(__float_as_uint(x), a, b);
  return fmaxf(__uint_as_float(a), __uint_as_float(b));
}
__device__ __forceinline__ float max_xor32(float x) {
  uint32_t a, b;
  swap32(__float_as_uint(x), a, b);
  return fmaxf(__uint_as_float(a), __uint_as_float(b));
}
__device__ __forceinline__ uint32_t or_xor16(uint32_t x) {
  uint32_t a, b;
  swap16(x, a, b);
  return a | b;
}
__device__ __forceinline__ uint32_t or_xor32(uint32_t x) {
  uint32_t a, b;
  swap32(x, a, b);
  return a | b;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}

// GELU(x) = x Phi(x) = x erfc(-x / sqrt 2) / 2, the exact (erf-based) form.
// erfc is evaluated without branches with the Chebyshev-fitted approximation
// of Numerical Recipes (erfcc; fractional error below 1.2e-7 for z >= 0),
// erfc(z) = t exp(-z^2 + P(t)) with t = 1 / (1 + z/2), and erfc(-z) =
// 2 - erfc(z). A branch-free form matters here: a divergent branch inside the
// per-hidden-unit loop of the router epilogue serialises its LDS reads.
__device__ __forceinline__ float gelu_exact(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(1.f + 0.5f * z);
  float P = 0.17087277f;
  P = fmaf(P, t, -0.82215223f);
  P = fmaf(P, t, 1.48851587f);
  P = fmaf(P, t, -1.13520398f);
  P = fmaf(P, t, 0.27886807f);
  P = fmaf(P, t, -0.18628806f);
  P = fmaf(P, t, 0.09678418f);
  P = fmaf(P, t, 0.37409196f);
  P = fmaf(P, t, 1.00002368f);
  P = fmaf(P, t, -1.26551223f);
  // exp through the hardware base-2 exponential (about 1 ulp); the argument
  // is at most ~30 in magnitude, so rounding it after the scaling by log2(e)
  // changes the result by about 2e-6 relative, well inside the erfc fit
  const float ec = t * __builtin_amdgcn_exp2f(fmaf(-z, z, P) * 1.44269504088896341f);
  return 0.5f * x * (x >= 0.f ? 2.f - ec : ec);
}

// Workgroup-to-XCD placement: consecutive workgroup ids go round-robin to the
// 8 XCDs. Given a linear id over `n` items that are naturally grouped by a
// "key" (heads) of size nkey, return an item order that keeps every key on a
// single XCD so its shared operands stay in that XCD's L2.
__device__ __forceinline__ void xcd_split(int lin, int nkey, int& key, int& rest) {
  if ((nkey & 7) == 0) {
    const int xcd = lin & 7, slot = lin >> 3, per = nkey >> 3;
    key = xcd + 8 * (slot % per);
    rest = slot / per;
  } else {
    key = lin % nkey;
    rest = lin / nkey;
  }
}

}  // namespace rolesub
