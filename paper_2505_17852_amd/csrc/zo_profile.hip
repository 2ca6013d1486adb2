// Event-based kernel timing behind zo_profile_enable / zo_profile_read.
#include "zo_profile.hpp"

#include <rocprofiler-sdk-roctx/roctx.h>

#include <mutex>
#include <vector>

#include "../../include/zo.h"

namespace zo {

std::atomic<int> g_profile_on{0};
thread_local bool g_profile_suppressed = false;

namespace {
struct Slot {
  hipEvent_t a, b;
  int cls;
};
std::mutex g_mu;
std::vector<Slot> g_slots;  // event pairs, reused across enable/read cycles
size_t g_used = 0;
int64_t g_all[kKClasses] = {};  // launches per class since the last enable
}  // namespace

PhaseRange::PhaseRange(const char* name) { roctxRangePushA(name); }
PhaseRange::~PhaseRange() { roctxRangePop(); }

int prof_begin(KernelClass k, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_mu);
  const int every = g_profile_on.load(std::memory_order_relaxed);
  if (every <= 0) return -1;
  if (g_all[k]++ % every != 0) return -1;
  if (g_used == g_slots.size()) {
    Slot sl{};
    if (hipEventCreate(&sl.a) != hipSuccess || hipEventCreate(&sl.b) != hipSuccess) return -1;
    g_slots.push_back(sl);
  }
  Slot& sl = g_slots[g_used];
  sl.cls = (int)k;
  if (hipEventRecord(sl.a, s) != hipSuccess) return -1;
  return (int)g_used++;
}

void prof_end(int slot, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_mu);
  (void)hipEventRecord(g_slots[(size_t)slot].b, s);
}

}  // namespace zo

extern "C" {

int zo_profile_enable(int32_t every) {
  if (every < 0) return ZO_EINVAL;
  std::lock_guard<std::mutex> lk(zo::g_mu);
  zo::g_used = 0;
  for (auto& n : zo::g_all) n = 0;
  zo::g_profile_on.store(every);
  return ZO_OK;
}

int zo_profile_read(int32_t kernel_class, double* timed_ms, int64_t* timed_launches, int64_t* all_launches) {
  if (!timed_ms || !timed_launches || !all_launches || kernel_class < 0 || kernel_class >= zo::kKClasses)
    return ZO_EINVAL;
  std::lock_guard<std::mutex> lk(zo::g_mu);
  double ms = 0.0;
  int64_t n = 0;
  for (size_t i = 0; i < zo::g_used; ++i) {
    const auto& sl = zo::g_slots[i];
    if (sl.cls != kernel_class) continue;
    if (hipEventSynchronize(sl.b) != hipSuccess) return ZO_EDEVICE;
    float e = 0.f;
    if (hipEventElapsedTime(&e, sl.a, sl.b) != hipSuccess) return ZO_EDEVICE;
    ms += e;
    ++n;
  }
  *timed_ms = ms;
  *timed_launches = n;
  *all_launches = zo::g_all[kernel_class];
  return ZO_OK;
}

}  // extern "C"
