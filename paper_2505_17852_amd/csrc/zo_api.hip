// C ABI entry points: argument validation on the host, then kernel launches
// on the caller's stream. Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/zo.h"
#include "zo_common.hpp"
#include "zo_kernels.hpp"
#include "zo_profile.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return ZO_OK;
}

int device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(ZO_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Shape rules of the kernels: every matrix dimension that a K tile or a
// column tile walks is a multiple of 32 (so that a 32-element probe word
// never straddles two weight rows).
int check_config(const zo_config* c) {
  if (!zo::config_valid(c)) return fail(ZO_EINVAL, "invalid zo_config");
  if (c->embed % 32 || c->hidden % 32)
    return fail(ZO_ESHAPE, "embed (%d) and hidden (%d) must be multiples of 32", c->embed,
                c->hidden);
  return ZO_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Workspace of zo_perturbed_losses_noalloc: a fixed device array, one copy per
// device, held until the process ends. In host code `scratch` names a host
// stand-in; its device address on the current device comes from
// hipGetSymbolAddress, once per device, and only that address is ever used.
constexpr size_t kScratchBytes = (size_t)ZO_NOALLOC_WORKSPACE_BYTES;
__device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (looked up on the first call on that
// device, with the device current).
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(ZO_EDEVICE, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return device_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(ZO_EDEVICE, "no device address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ZO_OK;
}

}  // namespace

extern "C" {

size_t zo_param_count(const zo_config* cfg) {
  if (!zo::config_valid(cfg)) return 0;
  return (size_t)zo::make_layout(*cfg).total;
}

// Both estimators' passes fit: central (2N passes) and forward (N + 1) differences.
static zo::WsPlan plan_for(const zo_config* cfg, int32_t N, int32_t B, int32_t C, bool fd) {
  return zo::plan_workspace(*cfg, zo::make_rows(N, B, zo::row_granule(*cfg, fd), fd), C);
}

size_t zo_workspace_bytes(const zo_config* cfg, int32_t N, int32_t B, int32_t C) {
  if (!zo::config_valid(cfg) || N < 1 || B < 1 || C < 1) return 0;
  return std::max(plan_for(cfg, N, B, C, false).total, plan_for(cfg, N, B, C, true).total);
}

size_t zo_workspace_bytes_min(const zo_config* cfg, int32_t N, int32_t B, int32_t C) {
  if (!zo::config_valid(cfg) || N < 1 || B < 1 || C < 1) return 0;
  return std::max(plan_for(cfg, N, B, C, false).min_total, plan_for(cfg, N, B, C, true).min_total);
}

int zo_init(const zo_config* cfg, void* theta, uint64_t seed, void* stream) {
  zo::PhaseRange range("zo_init");
  int st = check_config(cfg);
  if (st) return st;
  if (!theta) return fail(ZO_EINVAL, "theta is NULL");
  const uint64_t P = zo::make_layout(*cfg).total;
  const float scale = (float)(1.0 / std::sqrt((double)cfg->hidden));
  return device_status(zo::launch_init(cfg->wdtype, theta, P, seed, scale, (hipStream_t)stream),
                       "zo_init");
}

static int forward_call(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                        uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                        float* L1, float* L2, void* workspace, size_t ws_bytes, int32_t products,
                        void* stream, bool fd, const char* name) {
  zo::PhaseRange range(name);
  int st = check_config(cfg);
  if (st) return st;
  // the bf16 forward walks K in tiles of 64
  if (cfg->wdtype == ZO_WBF16 && (cfg->embed % 64 || cfg->hidden % 64))
    return fail(ZO_ESHAPE, "bf16 weights: embed (%d) and hidden (%d) must be multiples of 64",
                cfg->embed, cfg->hidden);
  if (!theta || !tokens || !L1 || !L2 || !workspace)
    return fail(ZO_EINVAL, "a required pointer is NULL");
  if (!aligned16(theta) || !aligned16(workspace))
    return fail(ZO_EINVAL, "theta and workspace must be 16-byte aligned");
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(ZO_EINVAL, "eps must be finite and > 0");
  if (cfg->wdtype == ZO_WBF16 && eps < ZO_BF16_EPS_MIN)
    return fail(ZO_EINVAL, "bf16 weights: eps (%g) must be >= %g (fp16 probe operands)", (double)eps,
                (double)ZO_BF16_EPS_MIN);
  if (products != ZO_PRODUCTS_AUTO && products != ZO_PRODUCTS_FUSED && products != ZO_PRODUCTS_SPLIT)
    return fail(ZO_EINVAL, "unknown products mode %d", products);
  if (fd && cfg->wdtype == ZO_WFP32 && products == ZO_PRODUCTS_SPLIT)
    return fail(ZO_EINVAL, "fp32 weights: forward differences have no two-stream form");
  if (N < 1 || B < 1 || C < 1) return fail(ZO_EINVAL, "N, B and C must be >= 1");
  if ((uint64_t)i0 + (uint64_t)N > 0x100000000ull)
    return fail(ZO_EINVAL, "probe indices i0 .. i0+N-1 must fit in 32 bits");
  const zo::Rows rows = zo::make_rows(N, B, zo::row_granule(*cfg, fd), fd);
  if (rows.M > (int64_t)1 << 30) return fail(ZO_ESHAPE, "rows of all passes too many");
  const zo::WsPlan plan = zo::plan_workspace(*cfg, rows, C);
  if (ws_bytes < plan.min_total)
    return fail(ZO_ENOMEM, "workspace of %zu bytes < %zu required", ws_bytes, plan.min_total);
  zo::ForwardArgs a;
  a.cfg = *cfg;
  a.lay = zo::make_layout(*cfg);
  a.rows = rows;
  a.ws = plan;
  a.theta = theta;
  a.seed = seed;
  a.eps = eps;
  a.i0 = i0;
  a.tokens = tokens;
  a.mask = mask;
  a.C = C;
  a.Lplus = L1;
  a.Lminus = L2;
  a.work = (char*)workspace;
  // bf16 weights: the fused form fp16(W + s eps z) down to its floor, the
  // two-stream form below it; fp32 weights: fused (w +- eps z in fp32)
  if (products == ZO_PRODUCTS_AUTO)
    a.split = cfg->wdtype == ZO_WBF16 && eps < ZO_BF16_FUSED_EPS_MIN;
  else
    a.split = products == ZO_PRODUCTS_SPLIT;
  // the probe cache is used when the workspace has room for it
  a.zc = (zo::probe_cache_kind(*cfg) && ws_bytes >= plan.total) ? (char*)workspace + plan.zcache : nullptr;
  a.bits = (zo::bit_cache_kind(*cfg) && ws_bytes >= plan.total) ? (uint32_t*)((char*)workspace + plan.bits) : nullptr;
  a.zmap = zo::make_zcache_map(*cfg);
  a.w16 = cfg->wdtype == ZO_WBF16 ? (char*)workspace + plan.w16 : nullptr;
  return device_status(zo::launch_forward(a, (hipStream_t)stream), name);
}

int zo_perturbed_losses(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                        uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                        float* Lplus, float* Lminus, void* workspace, size_t ws_bytes, void* stream) {
  return forward_call(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, Lplus, Lminus, workspace, ws_bytes,
                      ZO_PRODUCTS_AUTO, stream, false, "zo_perturbed_losses");
}

int zo_perturbed_losses_ex(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                           uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                           float* Lplus, float* Lminus, void* workspace, size_t ws_bytes, int32_t products,
                           void* stream) {
  return forward_call(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, Lplus, Lminus, workspace, ws_bytes,
                      products, stream, false, "zo_perturbed_losses_ex");
}

int zo_perturbed_losses_noalloc(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N,
                                uint32_t i0, const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C,
                                float* Lplus, float* Lminus, void* stream) {
  int st = check_config(cfg);
  if (st) return st;
  if (N < 1 || B < 1 || C < 1) return fail(ZO_EINVAL, "N, B and C must be >= 1");
  // the sizes are checked before the scratch array is first touched
  const size_t need = zo_workspace_bytes_min(cfg, N, B, C);
  if (need == 0) return fail(ZO_EINVAL, "invalid workspace request");
  if (need > kScratchBytes)
    return fail(ZO_ENOMEM, "zo_perturbed_losses_noalloc: %zu bytes of workspace needed, the fixed scratch holds %zu",
                need, kScratchBytes);
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st) return st;
  // the probe cache too when it fits (the results are the same either way)
  const size_t full = zo_workspace_bytes(cfg, N, B, C);
  const size_t bytes = full <= kScratchBytes ? full : need;
  zo::g_profile_suppressed = true;
  st = forward_call(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, Lplus, Lminus, ws, bytes, ZO_PRODUCTS_AUTO,
                    stream, false, "zo_perturbed_losses_noalloc");
  zo::g_profile_suppressed = false;
  return st;
}

int zo_fd_losses(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N, uint32_t i0,
                 const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C, float* L, float* L0,
                 void* workspace, size_t ws_bytes, void* stream) {
  return forward_call(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, L, L0, workspace, ws_bytes,
                      ZO_PRODUCTS_AUTO, stream, true, "zo_fd_losses");
}

int zo_fd_losses_ex(const zo_config* cfg, const void* theta, uint64_t seed, float eps, int32_t N, uint32_t i0,
                    const int32_t* tokens, const uint8_t* mask, int32_t B, int32_t C, float* L, float* L0,
                    void* workspace, size_t ws_bytes, int32_t products, void* stream) {
  return forward_call(cfg, theta, seed, eps, N, i0, tokens, mask, B, C, L, L0, workspace, ws_bytes, products,
                      stream, true, "zo_fd_losses_ex");
}

int zo_update(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
              uint32_t i0, const float* Lplus, const float* Lminus, int32_t* skipped_out,
              void* stream) {
  zo::PhaseRange range("zo_update");
  int st = check_config(cfg);
  if (st) return st;
  if (!theta || !Lplus || !Lminus) return fail(ZO_EINVAL, "a required pointer is NULL");
  if (!aligned16(theta)) return fail(ZO_EINVAL, "theta must be 16-byte aligned");
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(ZO_EINVAL, "eps must be finite and > 0");
  if (!std::isfinite(lr)) return fail(ZO_EINVAL, "lr must be finite");
  if (N < 1) return fail(ZO_EINVAL, "N must be >= 1");
  if ((uint64_t)i0 + (uint64_t)N > 0x100000000ull)
    return fail(ZO_EINVAL, "probe indices i0 .. i0+N-1 must fit in 32 bits");
  const uint64_t P = zo::make_layout(*cfg).total;
  return device_status(zo::launch_update(cfg->wdtype, cfg->probe, theta, P, seed, eps, lr, N, i0,
                                         Lplus, Lminus, skipped_out, (hipStream_t)stream),
                       "zo_update");
}

size_t zo_probe_bits_offset(const zo_config* cfg, int32_t N, int32_t B, int32_t C) {
  if (!zo::config_valid(cfg) || N < 1 || B < 1 || C < 1 || !zo::bit_cache_kind(*cfg)) return 0;
  return plan_for(cfg, N, B, C, false).bits;
}

int zo_update_cached(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                     uint32_t i0, const float* Lplus, const float* Lminus, int32_t* skipped_out,
                     const uint32_t* probe_bits, void* stream) {
  zo::PhaseRange range("zo_update_cached");
  int st = check_config(cfg);
  if (st) return st;
  if (cfg->probe != ZO_RADEMACHER) return fail(ZO_EINVAL, "zo_update_cached: sign probes only");
  if (!theta || !Lplus || !Lminus || !probe_bits) return fail(ZO_EINVAL, "a required pointer is NULL");
  if (!aligned16(theta) || !aligned16(probe_bits))
    return fail(ZO_EINVAL, "theta and probe_bits must be 16-byte aligned");
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(ZO_EINVAL, "eps must be finite and > 0");
  if (!std::isfinite(lr)) return fail(ZO_EINVAL, "lr must be finite");
  if (N < 1) return fail(ZO_EINVAL, "N must be >= 1");
  if ((uint64_t)i0 + (uint64_t)N > 0x100000000ull)
    return fail(ZO_EINVAL, "probe indices i0 .. i0+N-1 must fit in 32 bits");
  const uint64_t P = zo::make_layout(*cfg).total;
  return device_status(zo::launch_update(cfg->wdtype, cfg->probe, theta, P, seed, eps, lr, N, i0, Lplus, Lminus,
                                         skipped_out, (hipStream_t)stream, 1, probe_bits),
                       "zo_update_cached");
}

int zo_fd_update(const zo_config* cfg, void* theta, uint64_t seed, float eps, float lr, int32_t N,
                 uint32_t i0, const float* L, const float* L0, int32_t* skipped_out, void* stream) {
  zo::PhaseRange range("zo_fd_update");
  int st = check_config(cfg);
  if (st) return st;
  if (!theta || !L || !L0) return fail(ZO_EINVAL, "a required pointer is NULL");
  if (!aligned16(theta)) return fail(ZO_EINVAL, "theta must be 16-byte aligned");
  if (!(eps > 0.0f) || !std::isfinite(eps)) return fail(ZO_EINVAL, "eps must be finite and > 0");
  if (!std::isfinite(lr)) return fail(ZO_EINVAL, "lr must be finite");
  if (N < 1) return fail(ZO_EINVAL, "N must be >= 1");
  if ((uint64_t)i0 + (uint64_t)N > 0x100000000ull)
    return fail(ZO_EINVAL, "probe indices i0 .. i0+N-1 must fit in 32 bits");
  const uint64_t P = zo::make_layout(*cfg).total;
  // the update kernels divide by 2 eps; eps / 2 (exact in fp32) gives (L_n - L0) / eps
  return device_status(zo::launch_update(cfg->wdtype, cfg->probe, theta, P, seed, 0.5f * eps, lr, N, i0, L,
                                         L0, skipped_out, (hipStream_t)stream, 0),
                       "zo_fd_update");
}

int zo_debug_probe(int32_t probe, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n, float* out,
                   void* stream) {
  if (probe != ZO_RADEMACHER && probe != ZO_GAUSSIAN) return fail(ZO_EINVAL, "unknown probe kind");
  if (!out && n) return fail(ZO_EINVAL, "out is NULL");
  if (n > ((uint64_t)1 << 30)) return fail(ZO_EINVAL, "n must be <= 2^30");
  return device_status(zo::launch_debug_probe(probe, seed, i, j0, n, out, (hipStream_t)stream),
                       "zo_debug_probe");
}

int zo_debug_gauss_pairs(const uint32_t* words, uint64_t n_pairs, float* out, void* stream) {
  if ((!words || !out) && n_pairs) return fail(ZO_EINVAL, "a required pointer is NULL");
  if (n_pairs > ((uint64_t)1 << 30)) return fail(ZO_EINVAL, "n_pairs must be <= 2^30");
  return device_status(zo::launch_debug_gauss_pairs(words, n_pairs, out, (hipStream_t)stream),
                       "zo_debug_gauss_pairs");
}

const char* zo_last_error(void) { return g_err; }

}  // extern "C"
