// Optional per-launch timing with HIP events, for measurement only.  When
// enabled on the calling thread, every kernel launch made through a
// ProfScope is bracketed by two events on its stream; tgp_profile_read sums
// the durations per kernel together with the algorithmic FLOPs and bytes the
// launcher attributes to each launch.  Disabled, a ProfScope does nothing.
#pragma once
#include <hip/hip_runtime.h>

namespace tgpk {

bool prof_enabled();

class ProfScope {
 public:
  ProfScope(const char* name, double flops, double bytes, hipStream_t st);
  ~ProfScope();

 private:
  int rec_ = -1;
  hipStream_t st_;
};

}  // namespace tgpk
