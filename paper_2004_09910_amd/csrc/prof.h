// Optional per-launch timing with HIP events, for measurement only.  When
// enabled on the calling thread, the kernel launched (with TGP_LAUNCH)
// inside a ProfScope records a start and a stop event; tgp_profile_read sums
// the durations per kernel together with the algorithmic FLOPs and bytes the
// launcher attributes to each launch.  Disabled, a ProfScope does nothing.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

namespace tgpk {

bool prof_enabled();

// Launch-failure injection, for tests of the error path only
// (tgp_debug_fail_launch): once armed for the n-th launch, that launch and
// every later one on the thread are skipped (nothing reaches the device)
// until a launcher collects the failure through launch_status(), which the
// launchers return in place of hipGetLastError().
bool launch_skipped();
hipError_t launch_status();

class ProfScope {
 public:
  ProfScope(const char* name, double flops, double bytes, hipStream_t st);
  bool active() const { return rec_ >= 0; }
  hipEvent_t start_event() const;
  hipEvent_t stop_event() const;
  void mark_launched();

 private:
  int rec_ = -1;
};

// Launches `kernel` on `st`; when the scope is active the dispatch itself
// records the scope's start and stop events around the kernel
// (hipExtLaunchKernelGGL), so a duration is the kernel's own, without the
// queue gaps an event recorded before and after the launch would add.
#define TGP_LAUNCH(ps, kernel, grid, block, shmem, st, ...)                                   \
  do {                                                                                       \
    if (::tgpk::launch_skipped()) break;                                                     \
    if ((ps).active()) {                                                                     \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, (ps).start_event(),              \
                            (ps).stop_event(), 0, __VA_ARGS__);                              \
      (ps).mark_launched();                                                                  \
    } else {                                                                                 \
      hipLaunchKernelGGL(kernel, grid, block, shmem, st, __VA_ARGS__);                       \
    }                                                                                        \
  } while (0)

}  // namespace tgpk
