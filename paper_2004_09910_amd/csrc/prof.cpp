#include "prof.h"

#include <cstring>
#include <string>
#include <vector>

#include "tgp.h"

namespace tgpk {
namespace {

struct Rec {
  std::string name;
  double flops, bytes;
  hipEvent_t a, b;
  bool launched;
};

struct State {
  bool on = false;
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

thread_local State g;

// launch-failure injection: launches left before the injected failure
// (0 = disarmed), and the failure pending collection
thread_local int g_fail_in = 0;
thread_local hipError_t g_failed = hipSuccess;

}  // namespace

bool prof_enabled() { return g.on; }

bool launch_skipped() {
  if (g_failed != hipSuccess) return true;
  if (g_fail_in > 0 && --g_fail_in == 0) {
    g_failed = hipErrorLaunchFailure;
    return true;
  }
  return false;
}

hipError_t launch_status() {
  if (g_failed != hipSuccess) {
    const hipError_t e = g_failed;
    g_failed = hipSuccess;
    return e;
  }
  return hipGetLastError();
}

ProfScope::ProfScope(const char* name, double flops, double bytes, hipStream_t) {
  if (!g.on) return;
  hipEvent_t a = g.get(), b = g.get();
  if (!a || !b) return;
  g.recs.push_back({name, flops, bytes, a, b, false});
  rec_ = (int)g.recs.size() - 1;
}

hipEvent_t ProfScope::start_event() const { return rec_ >= 0 ? g.recs[rec_].a : nullptr; }
hipEvent_t ProfScope::stop_event() const { return rec_ >= 0 ? g.recs[rec_].b : nullptr; }
void ProfScope::mark_launched() {
  if (rec_ >= 0) g.recs[rec_].launched = true;
}

}  // namespace tgpk

extern "C" {

int tgp_debug_fail_launch(int n) {
  const int prev = tgpk::g_fail_in;
  tgpk::g_fail_in = n > 0 ? n : 0;
  tgpk::g_failed = hipSuccess;
  return prev;
}

tgp_status tgp_profile_enable(int enable) {
  tgpk::g.on = enable != 0;
  return TGP_OK;
}

tgp_status tgp_profile_clear(void) {
  using tgpk::g;
  for (auto& r : g.recs) {
    g.pool.push_back(r.a);
    g.pool.push_back(r.b);
  }
  g.recs.clear();
  return TGP_OK;
}

tgp_status tgp_profile_read(tgp_kernel_stat* out, int cap, int* count) {
  using tgpk::g;
  if (!count) return TGP_EINVAL;
  std::vector<tgp_kernel_stat> agg;
  for (auto& r : g.recs) {
    if (!r.launched) {   // a scope that launched nothing (early return)
      g.pool.push_back(r.a);
      g.pool.push_back(r.b);
      continue;
    }
    if (hipEventSynchronize(r.b) != hipSuccess) return TGP_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return TGP_EHIP;
    tgp_kernel_stat* s = nullptr;
    for (auto& a : agg)
      if (r.name == a.name) s = &a;
    if (!s) {
      agg.push_back(tgp_kernel_stat{});
      s = &agg.back();
      strncpy(s->name, r.name.c_str(), sizeof(s->name) - 1);
    }
    s->launches += 1;
    s->ms += ms;
    s->flops += r.flops;
    s->bytes += r.bytes;
    g.pool.push_back(r.a);
    g.pool.push_back(r.b);
  }
  g.recs.clear();
  *count = (int)agg.size();
  for (int k = 0; k < (int)agg.size() && k < cap; ++k) out[k] = agg[k];
  return *count <= cap ? TGP_OK : TGP_EINVAL;
}

}  // extern "C"
