// Optional kernel timing: while enabled, launchers count their launches per
// kernel class and bracket every n-th one with HIP events recorded on the
// launch stream; zo_profile_read() turns them into per-class totals. Disabled
// by default; when disabled the hooks cost one relaxed atomic load.
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>

namespace zo {

enum KernelClass { kKGate = 0, kKHead = 1, kKEmbed = 2, kKCombine = 3, kKUpdate = 4, kKProbeCache = 5,
                   kKWeights16 = 6, kKClasses = 7 };

extern std::atomic<int> g_profile_on;  // 0: off; n >= 1: time every n-th launch of a class
// Set by entry points that must not allocate (timing creates HIP events on
// first use): their launches are neither counted nor timed.
extern thread_local bool g_profile_suppressed;

// Counts the launch; returns a slot index to pass to prof_end when this launch
// is timed, else -1.
int prof_begin(KernelClass k, hipStream_t s);
void prof_end(int slot, hipStream_t s);

struct ProfScope {
  int slot;
  hipStream_t s;
  ProfScope(KernelClass k, hipStream_t st)
      : slot(g_profile_on.load(std::memory_order_relaxed) && !g_profile_suppressed ? prof_begin(k, st) : -1),
        s(st) {}
  ~ProfScope() {
    if (slot >= 0) prof_end(slot, s);
  }
};

// A named phase range for profilers that trace markers (rocprofv3
// --marker-trace): pushed on construction, popped on destruction, on the
// calling host thread. The forward's phases and the entry points carry one;
// without a tracing tool attached a range costs one library call each way.
struct PhaseRange {
  explicit PhaseRange(const char* name);
  ~PhaseRange();
  PhaseRange(const PhaseRange&) = delete;
  PhaseRange& operator=(const PhaseRange&) = delete;
};

}  // namespace zo
