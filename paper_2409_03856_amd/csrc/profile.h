// Internal: per-kernel timing hooks (see sirius_profile_enable in sirius.h).
//
// Every library kernel is launched through klaunch() inside a ProfScope. While timing is on,
// the scope's pair of HIP events is attached to the kernel's own dispatch
// (hipExtLaunchKernel): the start event takes the first kernel's start timestamp and the end
// event the last kernel's end timestamp, so an elapsed time is the kernels' execution time as
// a kernel trace reports it, without the gap between a separately recorded event and the
// dispatch. While timing is off, klaunch is a plain launch.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sirius {

int prof_open(const char* name);
bool prof_events(int id, hipEvent_t* start, hipEvent_t* stop);
void prof_close(int id, bool launched);

struct ProfScope;
extern thread_local ProfScope* t_prof;
extern thread_local bool t_prof_off;

// While alive, the calling thread's kernels carry no timing events even if timing is on (for the
// entry point that must create nothing).
struct ProfSuppress {
  bool prev;
  ProfSuppress() : prev(t_prof_off) { t_prof_off = true; }
  ~ProfSuppress() { t_prof_off = prev; }
  ProfSuppress(const ProfSuppress&) = delete;
  ProfSuppress& operator=(const ProfSuppress&) = delete;
};

// Times the kernels launched through klaunch while it is alive: ProfScope p("name", stream);
struct ProfScope {
  int id;
  bool launched = false;
  ProfScope* prev;
  ProfScope(const char* name, hipStream_t) : id(prof_open(name)), prev(t_prof) { t_prof = this; }
  ~ProfScope() {
    t_prof = prev;
    prof_close(id, launched);
  }
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;
};

template <typename... KArgs, typename... Args>
inline void klaunch(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t shmem,
                    hipStream_t stream, Args... args) {
  ProfScope* p = t_prof;
  hipEvent_t a = nullptr, b = nullptr;
  if (p != nullptr && p->id >= 0 && prof_events(p->id, &a, &b)) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, p->launched ? nullptr : a, b, 0u,
                          static_cast<KArgs>(args)...);
    p->launched = true;
  } else {
    kernel<<<grid, block, shmem, stream>>>(static_cast<KArgs>(args)...);
  }
}

}  // namespace sirius
