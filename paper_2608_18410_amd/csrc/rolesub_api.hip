// C ABI of librolesub: host-side validation, then asynchronous launches on the
// caller's stream. No allocation, no state between calls.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <string>

#include "launch.hpp"
#include "rolesub.h"

using namespace rolesub;

// Route workspace of rolesub_route_noalloc, for callers that cannot allocate
// device memory. Each device holds its own copy for the life of the process.
// In host code this name is only a stand-in for the symbol: kernels and
// copies take the device address that hipGetSymbolAddress returns for it.
__device__ __align__(256) char scratch[ROLESUB_ROUTE_NOALLOC_MAX_BYTES];

namespace {

thread_local std::string g_err;

rolesub_status fail(rolesub_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

rolesub_status from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return ROLESUB_OK;
  return fail(ROLESUB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool valid_dtype(rolesub_dtype t) { return t == ROLESUB_F32 || t == ROLESUB_BF16; }
size_t esize(rolesub_dtype t) { return t == ROLESUB_F32 ? 4 : 2; }
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }
// Kernels address each sample's (or workgroup's) slice of a tensor through a
// buffer resource that must cover less than 2 GiB.
constexpr size_t kMaxRegion = static_cast<size_t>(1) << 31;

// B, T >= 0; H >= 1; dh in {64, 128}.
rolesub_status check_value_dims(const rolesub_dims* d, const char* fn) {
  if (!d) return fail(ROLESUB_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  if (d->B < 0 || d->T < 0 || d->H < 1)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: need B >= 0, T >= 0, H >= 1 (got B=%d T=%d H=%d)", fn,
                d->B, d->T, d->H);
  if (d->dh != 64 && d->dh != 128)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: head dim %d not supported (64 or 128)", fn, d->dh);
  return ROLESUB_OK;
}

rolesub_status check_groups(const rolesub_dims* d, const char* fn, bool need_dh) {
  if (d->G < 1 || d->G > 32)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: G=%d groups not supported (1..32)", fn, d->G);
  if (need_dh && d->dh % d->G != 0)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: G=%d does not divide dh=%d", fn, d->G, d->dh);
  return ROLESUB_OK;
}

rolesub_status check_budget(const rolesub_budget* bu, int G, const char* fn) {
  if (!bu) return fail(ROLESUB_ERR_INVALID_ARG, "%s: budget is NULL", fn);
  if (bu->mode == ROLESUB_BUDGET_TOPK) {
    for (int t = 0; t < 4; ++t)
      if (bu->k_by_type[t] < 0 || bu->k_by_type[t] > G)
        return fail(ROLESUB_ERR_INVALID_ARG, "%s: k_by_type[%d]=%d outside 0..G=%d", fn, t,
                    bu->k_by_type[t], G);
  } else if (bu->mode == ROLESUB_BUDGET_THRESHOLD) {
    if (bu->kmin < 0 || bu->kmin > bu->kmax || bu->kmax > G)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: need 0 <= kmin <= kmax <= G (kmin=%d kmax=%d G=%d)",
                  fn, bu->kmin, bu->kmax, G);
    if (std::isnan(bu->tau)) return fail(ROLESUB_ERR_INVALID_ARG, "%s: tau is NaN", fn);
  } else {
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: unknown budget mode %d", fn, bu->mode);
  }
  return ROLESUB_OK;
}

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* x = static_cast<const char*>(a);
  const char* y = static_cast<const char*>(b);
  return x < y + nb && y < x + na;
}

// Packed-cache capacity against the budget (only when both are given).
rolesub_status check_capacity(const rolesub_dims* dims, const rolesub_budget* budget, const int32_t* type_counts,
                              int64_t cap_groups, const char* fn) {
  if (!budget || !type_counts) return ROLESUB_OK;
  rolesub_status st = check_budget(budget, dims->G, fn);
  if (st) return st;
  int64_t need = 0;
  if (budget->mode == ROLESUB_BUDGET_TOPK) {
    for (int t = 0; t < 4; ++t) {
      if (type_counts[t] < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: type_counts[%d] < 0", fn, t);
      need += static_cast<int64_t>(type_counts[t]) * std::min(budget->k_by_type[t], dims->G);
    }
  } else {
    need = static_cast<int64_t>(dims->T) * std::min(budget->kmax, dims->G);
  }
  if (cap_groups < need)
    return fail(ROLESUB_ERR_CAPACITY, "%s: cap_groups=%lld below the budget of %lld groups", fn,
                static_cast<long long>(cap_groups), static_cast<long long>(need));
  return ROLESUB_OK;
}

// Route workspace: cb, F, hbar and the partial language terms, then (with
// split) the partial products and tile counters of the split-K router.
size_t route_ws_bytes(const rolesub_dims* d, const rolesub_router* r, bool split = true) {
  if (!d || !r || d->B <= 0) return 0;
  const int T = d->T > 0 ? d->T : 0;
  return align256(route_cb_floats(d->B, r->Hr, d->G, r->kind) * sizeof(float)) +
         align256(route_F_floats(r->Hr, d->G, r->C, r->kind) * sizeof(float)) +
         align256(route_hbar_floats(d->B, d->d > 0 ? d->d : 0) * sizeof(float)) +
         align256(route_pcb_floats(d->B, d->d > 0 ? d->d : 0, r->Hr, r->kind) * sizeof(float)) +
         (split ? align256(route_sk_part_floats(d->B, T, r->Hr, r->kind) * sizeof(float)) +
                      align256(route_sk_cnt_ints(d->B, T, r->Hr, r->kind) * sizeof(int))
                : 0);
}

// Polls the first half of a split-K router tile makes for the second before
// leaving the tile to it (a poll is one round trip to memory, about a
// microsecond; the halves of a tile usually finish within a few of each
// other). ROLESUB_SK_POLLS overrides it (0 to 1000); with 0 the halves share
// the epilogue only when the second has already arrived.
int route_sk_polls() {
  const char* e = std::getenv("ROLESUB_SK_POLLS");
  if (e && *e) return std::min(1000, std::max(0, std::atoi(e)));
  return 32;
}

// Checks the router and hidden states and fills the router part of p (B, T,
// d, G already set); the route workspace sits at the start of `workspace`.
rolesub_status setup_router(const char* fn, const rolesub_dims* dims, rolesub_dtype dtype,
                            const rolesub_router* router, const void* h, void* workspace, size_t ws_bytes,
                            RouteParams& p, bool split = true) {
  if (!h) return fail(ROLESUB_ERR_INVALID_ARG, "%s: h must be non-NULL", fn);
  if (dims->d < 1) return fail(ROLESUB_ERR_INVALID_ARG, "%s: hidden size d=%d", fn, dims->d);
  if (router->C < 1 || router->C > 64)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: C=%d latent roles not supported (1..64)", fn, router->C);
  if (!router->W_r || !router->b_r) return fail(ROLESUB_ERR_INVALID_ARG, "%s: W_r/b_r are NULL", fn);
  if (router->kind == ROLESUB_ROUTER_MLP2) {
    if (router->d_e < 1 || router->Hr < 1)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: need d_e >= 1 and Hr >= 1", fn);
    if (!router->E || !router->W1 || !router->b1 || !router->W2 || !router->b2)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: MLP2 router weights are NULL", fn);
    if (static_cast<int64_t>(router->C) * router->d_e > dims->d)
      return fail(ROLESUB_ERR_UNSUPPORTED, "%s: C*d_e=%d exceeds d=%d", fn, router->C * router->d_e, dims->d);
  } else if (router->kind == ROLESUB_ROUTER_ADDITIVE) {
    if (!router->W_tok || !router->b_tok || !router->W_role || !router->W_lang || !router->b_lang)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: additive router weights are NULL", fn);
  } else {
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: unknown router kind %d", fn, router->kind);
  }
  if (route_generic_shm(dims->d, dims->G, router->C, router->Hr, router->kind) > 64 * 1024 ||
      static_cast<size_t>(dims->d) * sizeof(float) > 64 * 1024)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: hidden size d=%d too large", fn, dims->d);
  if (static_cast<size_t>(dims->T) * dims->d * esize(dtype) >= kMaxRegion ||
      static_cast<size_t>(router->Hr) * (2 * static_cast<size_t>(dims->d) + router->d_e) * esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: one sample's hidden states exceed 2 GiB", fn);
  const size_t need = route_ws_bytes(dims, router, split);
  if (ws_bytes < need || (need && !workspace))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws_bytes);

  p.d_e = router->d_e;
  p.Hr = router->Hr;
  p.C = router->C;
  p.kind = router->kind;
  p.alpha_role = router->alpha_role;
  p.alpha_lang = router->alpha_lang;
  p.h = h;
  p.W_r = router->W_r;
  p.b_r = router->b_r;
  p.E = router->E;
  p.W1 = router->W1;
  p.b1 = router->b1;
  p.W2 = router->W2;
  p.b2 = router->b2;
  p.W_tok = router->W_tok;
  p.b_tok = router->b_tok;
  p.W_role = router->W_role;
  p.W_lang = router->W_lang;
  p.b_lang = router->b_lang;
  char* ws = static_cast<char*>(workspace);
  p.cb = reinterpret_cast<float*>(ws);
  const size_t off_F = align256(route_cb_floats(p.B, p.Hr, p.G, p.kind) * sizeof(float));
  const size_t off_h = off_F + align256(route_F_floats(p.Hr, p.G, p.C, p.kind) * sizeof(float));
  const size_t off_p = off_h + align256(route_hbar_floats(p.B, p.d) * sizeof(float));
  p.F = reinterpret_cast<float*>(ws + off_F);
  p.hbar = reinterpret_cast<float*>(ws + off_h);
  p.pcb = reinterpret_cast<float*>(ws + off_p);
  p.rpart = nullptr;
  p.rcnt = nullptr;
  if (split && route_sk_cnt_ints(p.B, p.T, p.Hr, p.kind)) {
    const size_t off_s = off_p + align256(route_pcb_floats(p.B, p.d, p.Hr, p.kind) * sizeof(float));
    const size_t off_c = off_s + align256(route_sk_part_floats(p.B, p.T, p.Hr, p.kind) * sizeof(float));
    p.rpart = reinterpret_cast<float*>(ws + off_s);
    p.rcnt = reinterpret_cast<int*>(ws + off_c);
    p.sk_polls = route_sk_polls();
  }
  return ROLESUB_OK;
}

// Device address of the current device's copy of `scratch`, looked up once
// per device (with that device current) and kept. The caller's stream must
// belong to the current device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

rolesub_status scratch_on_current_device(const char* fn, hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return from_hip(e, fn);
  if (dev < 0 || dev >= kMaxDevices)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: device %d is beyond the %d supported", fn, dev, kMaxDevices);
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return from_hip(e, fn);
    if (sdev != dev)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: the stream belongs to device %d, the current device is %d", fn,
                  static_cast<int>(sdev), dev);
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return from_hip(e, fn);
    if (!ptr) return fail(ROLESUB_ERR_HIP, "%s: no device address for the scratch array", fn);
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return ROLESUB_OK;
}

rolesub_status check_alloc(const char* fn, int32_t B, int32_t T, int32_t G, const int32_t* k_by_type) {
  if (B < 0 || T < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: need B >= 0, T >= 0", fn);
  if (G < 1 || G > 32) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: G=%d groups not supported (1..32)", fn, G);
  if (!k_by_type) return fail(ROLESUB_ERR_INVALID_ARG, "%s: k_by_type is NULL", fn);
  for (int t = 0; t < 4; ++t)
    if (k_by_type[t] < 0 || k_by_type[t] > G)
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: k_by_type[%d]=%d outside 0..G=%d", fn, t, k_by_type[t], G);
  if (T > kAllocMaxT)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: T=%d tokens per sample above %d", fn, T, kAllocMaxT);
  if (static_cast<int64_t>(B) * 5 > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B too large", fn);
  return ROLESUB_OK;
}

AllocParams alloc_params(int32_t B, int32_t T, int32_t G, const int32_t* k_by_type) {
  AllocParams a = {};
  a.B = B;
  a.T = T;
  a.G = G;
  for (int t = 0; t < 4; ++t) a.k_by_type[t] = k_by_type[t];
  return a;
}

size_t route_allocate_ws_bytes(const rolesub_dims* d, const rolesub_router* r) {
  if (!d || !r || d->B <= 0 || d->T <= 0 || d->G < 1) return 0;
  const size_t ntok = static_cast<size_t>(d->B) * d->T;
  return route_ws_bytes(d, r) + align256(ntok * d->G * sizeof(float)) + align256(ntok * sizeof(float));
}

// Shapes the full-width kernels take; fills the shape part of p.
rolesub_status full_setup(const char* fn, const rolesub_dims* dims, rolesub_dtype dtype, int64_t cap,
                          void* workspace, size_t ws_bytes, FullParams& p) {
  if (!dims) return fail(ROLESUB_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  if (dtype != ROLESUB_BF16) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: bf16 only", fn);
  if (dims->B < 0 || dims->T < 0 || dims->H < 1)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: need B >= 0, T >= 0, H >= 1", fn);
  if (dims->dh != 128) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: head dim %d not supported (128)", fn, dims->dh);
  const int64_t dv = static_cast<int64_t>(dims->H) * dims->dh;
  const int S = dims->G;
  if (S < 1 || S > 32 || dv % S != 0 || (dv / S) % 128 != 0)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: S=%d groups of d_v=%lld: need 1 <= S <= 32 and d_v/S a multiple of 128",
                fn, S, static_cast<long long>(dv));
  if (dims->T > kFullMaxT || dims->B > kFullMaxB)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: at most %d prefixes of %d tokens", fn, kFullMaxB, kFullMaxT);
  if (cap < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: cap_groups < 0", fn);
  const int64_t ds = dv / S;
  if (static_cast<int64_t>(dims->B) * dims->T * dv * 2 >= static_cast<int64_t>(kMaxRegion) ||
      static_cast<int64_t>(dims->B) * cap * ds * 2 >= static_cast<int64_t>(kMaxRegion) ||
      dv * dv * 2 >= static_cast<int64_t>(kMaxRegion))
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: values, cache or R exceed 2 GiB", fn);
  const size_t need = rolesub_full_workspace_size(dims->B, dims->T, S);
  if (ws_bytes < need || (need && !workspace))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws_bytes);
  p = FullParams{};
  p.B = dims->B;
  p.T = dims->T;
  p.H = dims->H;
  p.dv = static_cast<int>(dv);
  p.S = S;
  p.ds = static_cast<int>(ds);
  p.cap = cap;
  char* ws = static_cast<char*>(workspace);
  const size_t b = static_cast<size_t>(dims->B);
  size_t o = 0;
  p.counts = reinterpret_cast<int32_t*>(ws + o);
  o += align256(b * sizeof(int32_t));
  p.rlist = reinterpret_cast<int32_t*>(ws + o);
  o += align256(b * dims->T * sizeof(int32_t));
  p.counts_g = reinterpret_cast<int32_t*>(ws + o);
  o += align256(b * S * sizeof(int32_t));
  p.starts_g = reinterpret_cast<int32_t*>(ws + o);
  o += align256(b * S * sizeof(int32_t));
  p.pairs = reinterpret_cast<int32_t*>(ws + o);
  return ROLESUB_OK;
}

}  // namespace

namespace {

// rolesub_route and rolesub_route_noalloc: with use_scratch the workspace is
// this device's `scratch` array (no allocation anywhere on the path).
rolesub_status route_impl(const char* fn, const rolesub_dims* dims, rolesub_dtype dtype,
                          const rolesub_router* router, const rolesub_budget* budget, const void* h,
                          const uint8_t* token_type, const float* scores_in, float* scores_out, uint32_t* mask,
                          uint8_t* idx, uint8_t* count, void* workspace, size_t ws_bytes, bool use_scratch,
                          void* stream) {
  if (!dims) return fail(ROLESUB_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  if (dims->B < 0 || dims->T < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: need B >= 0, T >= 0", fn);
  rolesub_status st = check_groups(dims, fn, false);
  if (st) return st;
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  st = check_budget(budget, dims->G, fn);
  if (st) return st;
  const size_t ntok = static_cast<size_t>(dims->B) * dims->T;
  if (ntok == 0) return ROLESUB_OK;
  if (ntok > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B*T too large", fn);
  if (!mask) return fail(ROLESUB_ERR_INVALID_ARG, "%s: mask must be non-NULL", fn);
  const bool need_types = budget->mode == ROLESUB_BUDGET_TOPK || scores_in == nullptr;
  if (need_types && !token_type)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: token_type must be non-NULL", fn);

  RouteParams p = {};
  p.B = dims->B;
  p.T = dims->T;
  p.d = dims->d;
  p.G = dims->G;
  p.types = token_type;
  p.mode = budget->mode;
  for (int t = 0; t < 4; ++t) p.k_by_type[t] = budget->k_by_type[t];
  p.tau = budget->tau;
  p.kmin = budget->kmin;
  p.kmax = budget->kmax;
  p.scores_in = scores_in;
  p.scores_out = scores_out;
  p.mask = mask;
  p.idx = idx;
  p.count = count;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (scores_in) return from_hip(launch_select(p, s), fn);

  if (!router) return fail(ROLESUB_ERR_INVALID_ARG, "%s: router is NULL and no scores_in given", fn);
  // the no-alloc call runs the single-kernel router (its array holds no
  // split-K partials); both forms give bitwise-equal results
  if (use_scratch) {
    const size_t need = route_ws_bytes(dims, router, false);
    if (need > ROLESUB_ROUTE_NOALLOC_MAX_BYTES)
      return fail(ROLESUB_ERR_UNSUPPORTED, "%s: needs %zu bytes of route workspace, above the %zu bytes it holds", fn,
                  need, static_cast<size_t>(ROLESUB_ROUTE_NOALLOC_MAX_BYTES));
    st = scratch_on_current_device(fn, s, &workspace);
    if (st) return st;
    ws_bytes = ROLESUB_ROUTE_NOALLOC_MAX_BYTES;
  }
  st = setup_router(fn, dims, dtype, router, h, workspace, ws_bytes, p, !use_scratch);
  if (st) return st;
  return from_hip(launch_route(p, dtype == ROLESUB_BF16, s), fn);
}

}  // namespace

extern "C" {

const char* rolesub_status_str(rolesub_status s) {
  switch (s) {
    case ROLESUB_OK: return "ROLESUB_OK";
    case ROLESUB_ERR_INVALID_ARG: return "ROLESUB_ERR_INVALID_ARG";
    case ROLESUB_ERR_UNSUPPORTED: return "ROLESUB_ERR_UNSUPPORTED";
    case ROLESUB_ERR_CAPACITY: return "ROLESUB_ERR_CAPACITY";
    case ROLESUB_ERR_HIP: return "ROLESUB_ERR_HIP";
  }
  return "ROLESUB_UNKNOWN_STATUS";
}

const char* rolesub_last_error(void) { return g_err.c_str(); }

int32_t rolesub_version(void) { return 100; }

rolesub_status rolesub_rotate_values(const rolesub_dims* dims, rolesub_dtype dtype, const void* v,
                                     const void* R, void* z, void* stream) {
  const char* fn = "rolesub_rotate_values";
  rolesub_status st = check_value_dims(dims, fn);
  if (st) return st;
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  const size_t ntok = static_cast<size_t>(dims->B) * dims->T;
  if (ntok == 0) return ROLESUB_OK;
  if (!v || !R || !z) return fail(ROLESUB_ERR_INVALID_ARG, "%s: v, R and z must be non-NULL", fn);
  if (ntok > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B*T too large", fn);
  const size_t bytes = ntok * dims->H * dims->dh * esize(dtype);
  if (ranges_overlap(v, bytes, z, bytes)) return fail(ROLESUB_ERR_INVALID_ARG, "%s: z overlaps v", fn);
  if (static_cast<size_t>(512) * dims->H * dims->dh * esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: too many heads", fn);
  return from_hip(launch_rotate(dtype == ROLESUB_BF16, static_cast<int>(ntok), dims->H, dims->dh, v, R,
                                z, static_cast<hipStream_t>(stream)),
                  fn);
}

size_t rolesub_route_workspace_size(const rolesub_dims* dims, const rolesub_router* router) {
  return route_ws_bytes(dims, router);
}

rolesub_status rolesub_route(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_router* router,
                             const rolesub_budget* budget, const void* h, const uint8_t* token_type,
                             const float* scores_in, float* scores_out, uint32_t* mask, uint8_t* idx,
                             uint8_t* count, void* workspace, size_t ws_bytes, void* stream) {
  return route_impl("rolesub_route", dims, dtype, router, budget, h, token_type, scores_in, scores_out, mask, idx,
                    count, workspace, ws_bytes, false, stream);
}

rolesub_status rolesub_route_noalloc(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_router* router,
                                     const rolesub_budget* budget, const void* h, const uint8_t* token_type,
                                     const float* scores_in, float* scores_out, uint32_t* mask, uint8_t* idx,
                                     uint8_t* count, void* stream) {
  return route_impl("rolesub_route_noalloc", dims, dtype, router, budget, h, token_type, scores_in, scores_out,
                    mask, idx, count, nullptr, 0, true, stream);
}

rolesub_status rolesub_allocate_groups(int32_t B, int32_t T, int32_t G, const int32_t* k_by_type,
                                       const float* priority, const uint8_t* token_type, const float* scores,
                                       uint8_t* k_out, uint32_t* mask, uint8_t* idx, uint8_t* count, void* stream) {
  const char* fn = "rolesub_allocate_groups";
  rolesub_status st = check_alloc(fn, B, T, G, k_by_type);
  if (st) return st;
  if (static_cast<int64_t>(B) * T == 0) return ROLESUB_OK;
  if (!priority || !token_type) return fail(ROLESUB_ERR_INVALID_ARG, "%s: priority and token_type must be non-NULL", fn);
  if (scores && !mask) return fail(ROLESUB_ERR_INVALID_ARG, "%s: scores given but mask is NULL", fn);
  if (!scores && (mask || idx || count))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: selection outputs given without scores", fn);
  if (!scores && !k_out) return fail(ROLESUB_ERR_INVALID_ARG, "%s: nothing to write (k_out and scores NULL)", fn);
  AllocParams a = alloc_params(B, T, G, k_by_type);
  a.priority = priority;
  a.types = token_type;
  a.scores = scores;
  a.k_out = k_out;
  a.mask = mask;
  a.idx = idx;
  a.count = count;
  return from_hip(launch_allocate(a, static_cast<hipStream_t>(stream)), fn);
}

size_t rolesub_route_allocate_workspace_size(const rolesub_dims* dims, const rolesub_router* router) {
  return route_allocate_ws_bytes(dims, router);
}

rolesub_status rolesub_route_allocate(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_router* router,
                                      const void* w_pri, const int32_t* k_by_type, const void* h,
                                      const uint8_t* token_type, float* priority_out, float* scores_out,
                                      uint8_t* k_out, uint32_t* mask, uint8_t* idx, uint8_t* count,
                                      void* workspace, size_t ws_bytes, void* stream) {
  const char* fn = "rolesub_route_allocate";
  if (!dims) return fail(ROLESUB_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  rolesub_status st = check_alloc(fn, dims->B, dims->T, dims->G, k_by_type);
  if (st) return st;
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  const size_t ntok = static_cast<size_t>(dims->B) * dims->T;
  if (ntok == 0) return ROLESUB_OK;
  if (ntok > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B*T too large", fn);
  if (!router) return fail(ROLESUB_ERR_INVALID_ARG, "%s: router is NULL", fn);
  if (!w_pri) return fail(ROLESUB_ERR_INVALID_ARG, "%s: w_pri is NULL", fn);
  if (!token_type || !mask) return fail(ROLESUB_ERR_INVALID_ARG, "%s: token_type and mask must be non-NULL", fn);
  const size_t need = route_allocate_ws_bytes(dims, router);
  if (ws_bytes < need || !workspace)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws_bytes);

  RouteParams p = {};
  p.B = dims->B;
  p.T = dims->T;
  p.d = dims->d;
  p.G = dims->G;
  p.types = token_type;
  st = setup_router(fn, dims, dtype, router, h, workspace, ws_bytes, p);
  if (st) return st;
  // scores and priorities go to the caller's buffers or to the workspace tail
  char* tail = static_cast<char*>(workspace) + route_ws_bytes(dims, router);
  float* sc = scores_out ? scores_out : reinterpret_cast<float*>(tail);
  float* pr = priority_out ? priority_out : reinterpret_cast<float*>(tail + align256(ntok * dims->G * sizeof(float)));
  p.mode = ROLESUB_BUDGET_TOPK;
  for (int t = 0; t < 4; ++t) p.k_by_type[t] = k_by_type[t];
  p.scores_out = sc;
  p.w_pri = w_pri;
  p.priority = pr;
  p.mask = nullptr;  // the selection waits for the allocation
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = from_hip(launch_route(p, dtype == ROLESUB_BF16, s), fn);
  if (st) return st;
  AllocParams a = alloc_params(dims->B, dims->T, dims->G, k_by_type);
  a.priority = pr;
  a.types = token_type;
  a.scores = sc;
  a.k_out = k_out;
  a.mask = mask;
  a.idx = idx;
  a.count = count;
  return from_hip(launch_allocate(a, s), fn);
}

// ---------------------------------------------------------------------------
// Full-width routing space

size_t rolesub_full_workspace_size(int32_t B, int32_t T, int32_t S) {
  if (B <= 0 || T <= 0 || S <= 0) return 0;
  const size_t b = static_cast<size_t>(B);
  return align256(b * sizeof(int32_t)) + align256(b * T * sizeof(int32_t)) + 2 * align256(b * S * sizeof(int32_t)) +
         align256(b * T * S * sizeof(int32_t));
}

rolesub_status rolesub_full_transpose(int32_t n, rolesub_dtype dtype, const void* R, void* Rt, void* stream) {
  const char* fn = "rolesub_full_transpose";
  if (dtype != ROLESUB_BF16) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: bf16 only", fn);
  if (n < 0 || n % 64 != 0) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: n=%d must be a multiple of 64", fn, n);
  if (n == 0) return ROLESUB_OK;
  if (!R || !Rt) return fail(ROLESUB_ERR_INVALID_ARG, "%s: R and Rt must be non-NULL", fn);
  if (ranges_overlap(R, static_cast<size_t>(n) * n * 2, Rt, static_cast<size_t>(n) * n * 2))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: Rt overlaps R", fn);
  return from_hip(launch_transpose(R, Rt, n, static_cast<hipStream_t>(stream)), fn);
}

rolesub_status rolesub_full_rotate_pack(const rolesub_dims* dims, rolesub_dtype dtype, const void* Rt,
                                        const void* v, const uint32_t* mask, int32_t* offsets, void* Vp,
                                        int64_t cap_groups, const rolesub_budget* budget,
                                        const int32_t* type_counts, void* workspace, size_t ws_bytes,
                                        void* stream) {
  const char* fn = "rolesub_full_rotate_pack";
  FullParams p;
  rolesub_status st = full_setup(fn, dims, dtype, cap_groups, workspace, ws_bytes, p);
  if (st) return st;
  if (static_cast<int64_t>(p.B) * p.T == 0) return ROLESUB_OK;
  if (!Rt || !v || !mask || !offsets || !Vp)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: Rt, v, mask, offsets and Vp must be non-NULL", fn);
  st = check_capacity(dims, budget, type_counts, cap_groups, fn);
  if (st) return st;
  if (ranges_overlap(v, static_cast<size_t>(p.B) * p.T * p.dv * 2, Vp, static_cast<size_t>(p.B) * cap_groups * p.ds * 2))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: Vp overlaps v", fn);
  p.mask = mask;
  p.offsets = offsets;
  p.v = v;
  p.Rm = Rt;
  p.Vp = Vp;
  return from_hip(launch_full(p, 0, static_cast<hipStream_t>(stream)), fn);
}

rolesub_status rolesub_full_values(const rolesub_dims* dims, rolesub_dtype dtype, const void* R,
                                   const uint32_t* mask, const int32_t* offsets, const void* Vp, int64_t cap_groups,
                                   void* Vh, void* workspace, size_t ws_bytes, void* stream) {
  const char* fn = "rolesub_full_values";
  FullParams p;
  rolesub_status st = full_setup(fn, dims, dtype, cap_groups, workspace, ws_bytes, p);
  if (st) return st;
  if (static_cast<int64_t>(p.B) * p.T == 0) return ROLESUB_OK;
  if (!R || !mask || !offsets || !Vp || !Vh)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: R, mask, offsets, Vp and Vh must be non-NULL", fn);
  if (ranges_overlap(Vh, static_cast<size_t>(p.B) * p.T * p.dv * 2, Vp, static_cast<size_t>(p.B) * cap_groups * p.ds * 2))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: Vh overlaps Vp", fn);
  p.mask = mask;
  p.offsets = const_cast<int32_t*>(offsets);
  p.Rm = R;
  p.Vp = const_cast<void*>(Vp);
  p.Vh = Vh;
  return from_hip(launch_full(p, 1, static_cast<hipStream_t>(stream)), fn);
}

rolesub_status rolesub_pack_kv(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_budget* budget,
                               const int32_t* type_counts, const void* z, const uint32_t* mask,
                               int32_t* offsets, void* Vp, int64_t cap_groups, void* stream) {
  const char* fn = "rolesub_pack_kv";
  rolesub_status st = check_value_dims(dims, fn);
  if (st) return st;
  st = check_groups(dims, fn, true);
  if (st) return st;
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  if (cap_groups < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: cap_groups < 0", fn);
  st = check_capacity(dims, budget, type_counts, cap_groups, fn);
  if (st) return st;
  if (dims->B == 0) return ROLESUB_OK;
  if (!mask || !offsets || (dims->T > 0 && !z) || (cap_groups > 0 && dims->T > 0 && !Vp))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: z, mask, offsets and Vp must be non-NULL", fn);
  if (static_cast<size_t>(dims->B) * dims->T > 0x7FFFFFFF)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B*T too large", fn);
  if (static_cast<size_t>(dims->H) * cap_groups * (dims->dh / dims->G) * esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: one sample's packed cache exceeds 2 GiB", fn);
  return from_hip(launch_pack(dtype == ROLESUB_BF16, dims->B, dims->T, dims->H, dims->dh, dims->G, z, mask,
                              offsets, Vp, cap_groups, static_cast<hipStream_t>(stream)),
                  fn);
}

rolesub_status rolesub_rotate_pack(const rolesub_dims* dims, rolesub_dtype dtype, const rolesub_budget* budget,
                                   const int32_t* type_counts, const void* v, const void* R,
                                   const uint32_t* mask, int32_t* offsets, void* Vp, int64_t cap_groups,
                                   void* stream) {
  const char* fn = "rolesub_rotate_pack";
  rolesub_status st = check_value_dims(dims, fn);
  if (st) return st;
  st = check_groups(dims, fn, true);
  if (st) return st;
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  if (cap_groups < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: cap_groups < 0", fn);
  st = check_capacity(dims, budget, type_counts, cap_groups, fn);
  if (st) return st;
  if (dims->B == 0) return ROLESUB_OK;
  if (!mask || !offsets || (dims->T > 0 && (!v || !R)) || (cap_groups > 0 && dims->T > 0 && !Vp))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: v, R, mask, offsets and Vp must be non-NULL", fn);
  if (static_cast<size_t>(dims->B) * dims->T > 0x7FFFFFFF)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: B*T too large", fn);
  if (static_cast<size_t>(512) * dims->H * dims->dh * esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: too many heads", fn);
  // a 16-token tile spans at most 15/T + 2 samples of the cache
  if (static_cast<size_t>(15 / std::max(dims->T, 1) + 2) * dims->H * cap_groups * (dims->dh / dims->G) *
          esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: packed cache too large", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return from_hip(launch_rotate_pack(dtype == ROLESUB_BF16, dims->B, dims->T, dims->H, dims->dh, dims->G, v, R,
                                     mask, offsets, Vp, cap_groups, s),
                  fn);
}

size_t rolesub_attend_workspace_size(const rolesub_dims* dims, int32_t Tq) {
  (void)dims;
  (void)Tq;
  return 0;
}

static rolesub_status attend_call(const char* fn, bool causal, bool dense, const rolesub_dims* dims,
                                  rolesub_dtype dtype,
                                  int32_t Tq, const void* q, const void* k, const uint32_t* mask,
                                  const int32_t* offsets, const void* Vp, int64_t cap_groups, const void* R,
                                  float scale, void* out, rolesub_dtype out_dtype, void* workspace,
                                  size_t ws_bytes, void* stream) {
  (void)workspace;
  (void)ws_bytes;
  rolesub_status st = check_value_dims(dims, fn);
  if (st) return st;
  if (!dense) {
    st = check_groups(dims, fn, true);
    if (st) return st;
  }
  if (!valid_dtype(dtype)) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: unknown dtype %d", fn, dtype);
  if (dense && dtype != ROLESUB_BF16) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: bf16 only", fn);
  if (out_dtype != ROLESUB_F32 && out_dtype != dtype)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: out_dtype must be f32 or the input dtype", fn);
  if (Tq < 0 || cap_groups < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: Tq and cap_groups must be >= 0", fn);
  if (!std::isfinite(scale)) return fail(ROLESUB_ERR_INVALID_ARG, "%s: scale is not finite", fn);
  if (dims->B == 0 || Tq == 0) return ROLESUB_OK;
  if (dims->T < 1) return fail(ROLESUB_ERR_INVALID_ARG, "%s: attention over T=0 tokens is undefined", fn);
  if (!q || !k || !out || (cap_groups > 0 && !Vp) || (!dense && (!mask || !offsets || !R)))
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: a tensor pointer is NULL", fn);
  if (static_cast<size_t>(dims->B) * dims->H > 0x7FFFFFFF ||
      static_cast<size_t>(dims->B) * dims->H * Tq > 0x7FFFFFFF)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: grid too large", fn);
  if (static_cast<size_t>(dims->T) * dims->H * dims->dh * esize(dtype) >= kMaxRegion ||
      static_cast<size_t>(Tq) * dims->H * dims->dh * esize(dtype) >= kMaxRegion ||
      static_cast<size_t>(cap_groups) * (dims->dh / dims->G) * esize(dtype) >= kMaxRegion)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: one sample's keys, queries or packed cache exceed 2 GiB", fn);
  AttendParams p = {};
  p.B = dims->B;
  p.T = dims->T;
  p.H = dims->H;
  p.dh = dims->dh;
  p.G = dense ? 1 : dims->G;
  p.Tq = Tq;
  p.q = q;
  p.k = k;
  p.mask = mask;
  p.offsets = offsets;
  p.Vp = Vp;
  p.cap = cap_groups;
  p.R = R;
  p.scale = scale == 0.f ? 1.f / std::sqrt(static_cast<float>(dims->dh)) : scale;
  p.out = out;
  p.out_f32 = out_dtype == ROLESUB_F32;
  p.causal = causal ? 1 : 0;
  p.dense = dense ? 1 : 0;
  return from_hip(launch_attend(p, dtype == ROLESUB_BF16, static_cast<hipStream_t>(stream)), fn);
}

rolesub_status rolesub_attend(const rolesub_dims* dims, rolesub_dtype dtype, int32_t Tq, const void* q,
                              const void* k, const uint32_t* mask, const int32_t* offsets, const void* Vp,
                              int64_t cap_groups, const void* R, float scale, void* out,
                              rolesub_dtype out_dtype, void* workspace, size_t ws_bytes, void* stream) {
  return attend_call("rolesub_attend", false, false, dims, dtype, Tq, q, k, mask, offsets, Vp, cap_groups, R, scale, out,
                     out_dtype, workspace, ws_bytes, stream);
}

rolesub_status rolesub_attend_values(const rolesub_dims* dims, rolesub_dtype dtype, int32_t Tq, const void* q,
                                     const void* k, const void* V, float scale, void* out, rolesub_dtype out_dtype,
                                     void* stream) {
  if (!dims) return fail(ROLESUB_ERR_INVALID_ARG, "rolesub_attend_values: dims is NULL");
  return attend_call("rolesub_attend_values", false, true, dims, dtype, Tq, q, k, nullptr, nullptr, V, dims->T,
                     nullptr, scale, out, out_dtype, nullptr, 0, stream);
}

rolesub_status rolesub_attend_causal(const rolesub_dims* dims, rolesub_dtype dtype, const void* q,
                                     const void* k, const uint32_t* mask, const int32_t* offsets,
                                     const void* Vp, int64_t cap_groups, const void* R, float scale,
                                     void* out, rolesub_dtype out_dtype, void* workspace, size_t ws_bytes,
                                     void* stream) {
  const char* fn = "rolesub_attend_causal";
  if (!dims) return fail(ROLESUB_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  if (dims->T == 0) return ROLESUB_OK;  // no prefix tokens, no queries
  return attend_call(fn, true, false, dims, dtype, dims->T, q, k, mask, offsets, Vp, cap_groups, R, scale, out,
                     out_dtype, workspace, ws_bytes, stream);
}

rolesub_status rolesub_retain_tokens(int32_t B, int32_t N, int32_t n_seg, const int32_t* seg_len,
                                     const int32_t* seg_keep, const float* scores, int32_t* keep_idx,
                                     void* stream) {
  const char* fn = "rolesub_retain_tokens";
  if (B < 0 || N < 0) return fail(ROLESUB_ERR_INVALID_ARG, "%s: B and N must be >= 0", fn);
  if (n_seg < 1 || n_seg > kRetainMaxSegments)
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: n_seg=%d outside [1, %d]", fn, n_seg, kRetainMaxSegments);
  if (!seg_len || !seg_keep) return fail(ROLESUB_ERR_INVALID_ARG, "%s: seg_len or seg_keep is NULL", fn);
  RetainParams p = {};
  p.B = B;
  p.N = N;
  p.n_seg = n_seg;
  int64_t start = 0, out = 0;
  for (int s_ = 0; s_ < n_seg; ++s_) {
    if (seg_len[s_] < 0 || seg_keep[s_] < 0 || seg_keep[s_] > seg_len[s_])
      return fail(ROLESUB_ERR_INVALID_ARG, "%s: segment %d: need 0 <= keep (%d) <= length (%d)", fn, s_,
                  seg_keep[s_], seg_len[s_]);
    if (seg_len[s_] > kRetainMaxSeg)
      return fail(ROLESUB_ERR_UNSUPPORTED, "%s: segment %d has %d tokens (at most %d)", fn, s_, seg_len[s_],
                  kRetainMaxSeg);
    p.seg_start[s_] = static_cast<int>(start);
    p.seg_len[s_] = seg_len[s_];
    p.seg_keep[s_] = seg_keep[s_];
    p.seg_out[s_] = static_cast<int>(out);
    start += seg_len[s_];
    out += seg_keep[s_];
  }
  if (start != N) return fail(ROLESUB_ERR_INVALID_ARG, "%s: segment lengths sum to %lld, not N=%d", fn,
                              static_cast<long long>(start), N);
  p.K = static_cast<int>(out);
  if (B == 0 || p.K == 0) return ROLESUB_OK;
  if (!scores || !keep_idx) return fail(ROLESUB_ERR_INVALID_ARG, "%s: a tensor pointer is NULL", fn);
  if (static_cast<size_t>(B) * n_seg > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: grid too large", fn);
  p.scores = scores;
  p.keep_idx = keep_idx;
  return from_hip(launch_retain(p, static_cast<hipStream_t>(stream)), fn);
}

rolesub_status rolesub_gather_tokens(int32_t B, int32_t N, int32_t K, int64_t row_bytes, const int32_t* keep_idx,
                                     const void* src, void* dst, void* stream) {
  const char* fn = "rolesub_gather_tokens";
  if (B < 0 || N < 0 || K < 0 || row_bytes < 0)
    return fail(ROLESUB_ERR_INVALID_ARG, "%s: sizes must be >= 0", fn);
  if (row_bytes % 4 != 0) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: row_bytes must be a multiple of 4", fn);
  if (B == 0 || K == 0 || row_bytes == 0) return ROLESUB_OK;
  if (!keep_idx || !src || !dst) return fail(ROLESUB_ERR_INVALID_ARG, "%s: a tensor pointer is NULL", fn);
  if (static_cast<size_t>(N) * row_bytes >= kMaxRegion || row_bytes >= static_cast<int64_t>(kMaxRegion))
    return fail(ROLESUB_ERR_UNSUPPORTED, "%s: one sample's rows exceed 2 GiB", fn);
  if (static_cast<size_t>(B) * K > 0x7FFFFFFF) return fail(ROLESUB_ERR_UNSUPPORTED, "%s: grid too large", fn);
  GatherParams p = {};
  p.B = B;
  p.N = N;
  p.K = K;
  p.row_bytes = row_bytes;
  p.idx = keep_idx;
  p.src = src;
  p.dst = dst;
  return from_hip(launch_gather_rows(p, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
