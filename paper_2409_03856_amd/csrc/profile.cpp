// Per-kernel timing: when enabled, the kernels of every ProfScope carry a pair of HIP events
// on their own dispatches (see profile.h).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sirius.h"
#include "profile.h"

namespace sirius {

thread_local ProfScope* t_prof = nullptr;
thread_local bool t_prof_off = false;

namespace {

struct Rec {
  const char* name;
  hipEvent_t a, b;
  bool used;  // false until a kernel carried the events
};

std::atomic<bool> g_on{false};
std::mutex g_mu;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_free;

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

int prof_open(const char* name) {
  if (t_prof_off || !g_on.load(std::memory_order_relaxed)) return -1;
  std::lock_guard<std::mutex> lk(g_mu);
  Rec r{name, take_event(), take_event(), false};
  if (r.a == nullptr || r.b == nullptr) {
    if (r.a != nullptr) g_free.push_back(r.a);
    if (r.b != nullptr) g_free.push_back(r.b);
    return -1;
  }
  g_recs.push_back(r);
  return (int)g_recs.size() - 1;
}

bool prof_events(int id, hipEvent_t* start, hipEvent_t* stop) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (id < 0 || id >= (int)g_recs.size()) return false;
  *start = g_recs[id].a;
  *stop = g_recs[id].b;
  return true;
}

void prof_close(int id, bool launched) {
  if (id < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (id < (int)g_recs.size()) g_recs[id].used = launched;
}

}  // namespace sirius

extern "C" {

int sirius_profile_enable(int on) {
  sirius::g_on.store(on != 0);
  return SIRIUS_OK;
}

int sirius_profile_reset(void) {
  std::lock_guard<std::mutex> lk(sirius::g_mu);
  for (auto& r : sirius::g_recs) {
    if (r.used) (void)hipEventSynchronize(r.b);
    sirius::g_free.push_back(r.a);
    sirius::g_free.push_back(r.b);
  }
  sirius::g_recs.clear();
  return SIRIUS_OK;
}

int sirius_profile_query(const char* kernel, double* total_ms, int64_t* launches) {
  if (kernel == nullptr || total_ms == nullptr || launches == nullptr) return SIRIUS_EINVAL;
  std::lock_guard<std::mutex> lk(sirius::g_mu);
  double tot = 0.0;
  int64_t n = 0;
  for (auto& r : sirius::g_recs) {
    if (!r.used || std::strcmp(r.name, kernel) != 0) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return SIRIUS_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return SIRIUS_EHIP;
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return SIRIUS_OK;
}

}  // extern "C"
