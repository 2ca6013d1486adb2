// Drives the host side of the C ABI (paper_2505_17852_amd/csrc/zo_api.hip,
// built for the host only under AddressSanitizer and UBSan) through every
// entry point: argument errors, and valid arguments that reach the kernel
// launchers, which are stubbed here to report a device error (no GPU is
// touched). Prints "api sanitizer driver ok" when every call returned the
// expected status.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>

#include "../../include/zo.h"
#include "../../paper_2505_17852_amd/csrc/zo_kernels.hpp"

namespace zo {
static int launches = 0;
hipError_t launch_debug_probe(int, uint64_t, uint32_t, uint64_t, uint64_t, float*, hipStream_t) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_debug_gauss_pairs(const uint32_t*, uint64_t, float*, hipStream_t) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_init(int, void*, uint64_t, uint64_t, float, hipStream_t) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_update(int, int, void*, uint64_t, uint64_t, float, float, int32_t, uint32_t, const float*,
                         const float*, int32_t*, hipStream_t, int, const uint32_t*) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_bits_fill(uint32_t*, uint64_t, uint64_t, uint32_t, int32_t, hipStream_t) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_forward(const ForwardArgs&, hipStream_t) {
  ++launches;
  return hipErrorInvalidValue;
}
hipError_t launch_embed_bf16(const ForwardArgs&, int, void*, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_gate_bf16(const ForwardArgs&, int, const void*, const void*, void*, float*, const float*,
                            hipStream_t) {
  return hipErrorInvalidValue;
}
hipError_t launch_head_bf16(const ForwardArgs&, const void*, int, int, const float*, float*, float*, float*,
                            hipStream_t) {
  return hipErrorInvalidValue;
}
}  // namespace zo

static int failures = 0;
static void expect(int got, int want, const char* what) {
  if (got != want) {
    std::printf("FAIL %s: status %d, expected %d (%s)\n", what, got, want, zo_last_error());
    ++failures;
  }
}

int main() {
  void* fake = (void*)0x10000;
  const int32_t* tok = (const int32_t*)fake;
  float* L = (float*)fake;
  const zo_config c1 = {1, 256, 32, 64, ZO_WFP32, ZO_RADEMACHER};
  const zo_config bf = {2, 300, 64, 128, ZO_WBF16, ZO_RADEMACHER};
  const zo_config bfg = {2, 300, 64, 128, ZO_WBF16, ZO_GAUSSIAN};
  const zo_config bad[] = {{0, 256, 32, 64, 0, 0}, {65, 256, 32, 64, 0, 0}, {1, 0, 32, 64, 0, 0},
                           {1, 256, 32, 64, 2, 0}, {1, 256, 32, 64, 0, 3}, {1, 256, 20, 64, 0, 0}};
  for (const zo_config& b : bad) {
    const bool shape_only = b.embed == 20;  // a valid config the kernels' tiles do not fit
    if (!shape_only) expect(zo_param_count(&b) == 0 ? 0 : 1, 0, "param count of an invalid config");
    expect(zo_perturbed_losses(&b, fake, 1, 1e-3f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, nullptr),
           shape_only ? ZO_ESHAPE : ZO_EINVAL, "bad config");
  }
  expect(zo_param_count(nullptr) == 0 ? 0 : 1, 0, "param count of NULL");
  expect(zo_workspace_bytes(nullptr, 1, 1, 1) == 0 ? 0 : 1, 0, "workspace of NULL");
  // argument errors of the forward calls
  expect(zo_perturbed_losses(&c1, nullptr, 1, 1e-3f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, nullptr),
         ZO_EINVAL, "NULL theta");
  expect(zo_perturbed_losses(&c1, fake, 1, 0.0f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, nullptr),
         ZO_EINVAL, "eps 0");
  expect(zo_perturbed_losses(&c1, fake, 1, 1e-3f, 0, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, nullptr),
         ZO_EINVAL, "N 0");
  expect(zo_perturbed_losses(&c1, fake, 1, 1e-3f, 2, 0xFFFFFFFFu, tok, nullptr, 2, 4, L, L, fake, 1ull << 40,
                             nullptr),
         ZO_EINVAL, "probe index overflow");
  expect(zo_perturbed_losses(&c1, fake, 1, 1e-3f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 16, nullptr), ZO_ENOMEM,
         "small workspace");
  expect(zo_perturbed_losses(&bf, fake, 1, 1e-6f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, nullptr),
         ZO_EINVAL, "bf16 eps floor");
  expect(zo_perturbed_losses_ex(&bf, fake, 1, 1e-3f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, 9, nullptr),
         ZO_EINVAL, "products mode");
  expect(zo_fd_losses_ex(&c1, fake, 1, 1e-3f, 2, 0, tok, nullptr, 2, 4, L, L, fake, 1ull << 40, ZO_PRODUCTS_SPLIT,
                         nullptr),
         ZO_EINVAL, "fp32 forward-difference split");
  // valid arguments reach the (stubbed) launcher
  const zo_config* ok[] = {&c1, &bf, &bfg};
  for (const zo_config* c : ok) {
    const size_t ws = zo_workspace_bytes(c, 3, 5, 7);
    expect(ws > 0 ? 0 : 1, 0, "workspace bytes");
    expect(zo_perturbed_losses(c, fake, 1, 1e-3f, 3, 2, tok, nullptr, 5, 7, L, L, fake, ws, nullptr), ZO_EDEVICE,
           "losses reach the launcher");
    expect(zo_perturbed_losses(c, fake, 1, 1e-4f, 3, 2, tok, nullptr, 5, 7, L, L, fake,
                               zo_workspace_bytes_min(c, 3, 5, 7), nullptr),
           ZO_EDEVICE, "losses with the smallest workspace");
    expect(zo_fd_losses(c, fake, 1, 1e-3f, 3, 2, tok, nullptr, 5, 7, L, L, fake, ws, nullptr), ZO_EDEVICE,
           "forward differences reach the launcher");
    expect(zo_update(c, fake, 1, 1e-3f, 1e-3f, 3, 2, L, L, nullptr, nullptr), ZO_EDEVICE, "update");
    expect(zo_fd_update(c, fake, 1, 1e-3f, 1e-3f, 3, 2, L, L, nullptr, nullptr), ZO_EDEVICE, "fd update");
    expect(zo_init(c, fake, 1, nullptr), ZO_EDEVICE, "init");
  }
  expect(zo_update_cached(&bf, fake, 1, 1e-3f, 1e-3f, 3, 2, L, L, nullptr, (const uint32_t*)fake, nullptr),
         ZO_EDEVICE, "cached update");
  expect(zo_update_cached(&bfg, fake, 1, 1e-3f, 1e-3f, 3, 2, L, L, nullptr, (const uint32_t*)fake, nullptr),
         ZO_EINVAL, "cached update of normal probes");
  expect(zo_probe_bits_offset(&bf, 3, 5, 7) > 0 ? 0 : 1, 0, "bits offset");
  expect(zo_update(&c1, fake, 1, 1e-3f, 1.0f / 0.0f, 3, 0, L, L, nullptr, nullptr), ZO_EINVAL, "infinite lr");
  expect(zo_debug_probe(7, 1, 0, 0, 4, L, nullptr), ZO_EINVAL, "probe kind");
  expect(zo_debug_probe(0, 1, 0, 0, 4, L, nullptr), ZO_EDEVICE, "probe dump");
  expect(zo_debug_gauss_pairs(nullptr, 4, L, nullptr), ZO_EINVAL, "NULL words");
  // the allocation-free entry point: sizes beyond its scratch, bad sizes
  const zo_config c4 = {6, 50000, 4096, 4096, ZO_WBF16, ZO_RADEMACHER};
  expect(zo_perturbed_losses_noalloc(&c4, fake, 1, 1e-3f, 16, 0, tok, nullptr, 256, 1024, L, L, nullptr), ZO_ENOMEM,
         "noalloc beyond the scratch");
  expect(zo_perturbed_losses_noalloc(&c1, fake, 1, 1e-3f, 0, 0, tok, nullptr, 4, 32, L, L, nullptr), ZO_EINVAL,
         "noalloc N 0");
  // within the scratch: the device lookup fails without a GPU, else the launcher stub does
  expect(zo_perturbed_losses_noalloc(&c1, fake, 1, 1e-3f, 2, 0, tok, nullptr, 4, 32, L, L, nullptr), ZO_EDEVICE,
         "noalloc within the scratch");
  // timing records
  expect(zo_profile_enable(-1), ZO_EINVAL, "profile every < 0");
  double ms;
  int64_t n1, n2;
  expect(zo_profile_read(99, &ms, &n1, &n2), ZO_EINVAL, "profile class");
  expect(zo_profile_enable(0), ZO_OK, "profile off");
  if (std::strlen(zo_last_error()) > 511) ++failures;
  if (zo::launches == 0) ++failures;
  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("api sanitizer driver ok (%d launcher calls)\n", zo::launches);
  return 0;
}
