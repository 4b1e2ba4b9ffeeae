// Per-kernel timing: when enabled, every library kernel launch is bracketed by a pair of
// HIP events recorded on the stream the kernel is launched on.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sirius.h"
#include "profile.h"

namespace sirius {
namespace {

struct Rec {
  const char* name;
  hipEvent_t a, b;
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

int prof_begin(const char* name, hipStream_t s) {
  if (!g_on.load(std::memory_order_relaxed)) return -1;
  std::lock_guard<std::mutex> lk(g_mu);
  Rec r{name, take_event(), take_event()};
  if (r.a == nullptr || r.b == nullptr) return -1;
  if (hipEventRecord(r.a, s) != hipSuccess) return -1;
  g_recs.push_back(r);
  return (int)g_recs.size() - 1;
}

void prof_end(int id, hipStream_t s) {
  if (id < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (id < (int)g_recs.size()) (void)hipEventRecord(g_recs[id].b, s);
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
    (void)hipEventSynchronize(r.b);
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
    if (std::strcmp(r.name, kernel) != 0) continue;
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
