// Optional kernel timing: while enabled, launchers bracket selected kernel
// launches with HIP events recorded on the launch stream, and
// zo_profile_read() turns them into per-class totals. Disabled by default;
// when disabled the hooks cost one relaxed atomic load.
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>

namespace zo {

enum KernelClass { kKGate = 0, kKHead = 1, kKEmbed = 2, kKCombine = 3, kKUpdate = 4, kKProbeCache = 5,
                   kKClasses = 6 };

extern std::atomic<int> g_profile_on;

// Returns a slot index to pass to prof_end, or -1 when profiling is off.
int prof_begin(KernelClass k, hipStream_t s);
void prof_end(int slot, hipStream_t s);

struct ProfScope {
  int slot;
  hipStream_t s;
  ProfScope(KernelClass k, hipStream_t st)
      : slot(g_profile_on.load(std::memory_order_relaxed) ? prof_begin(k, st) : -1), s(st) {}
  ~ProfScope() {
    if (slot >= 0) prof_end(slot, s);
  }
};

}  // namespace zo
