// Internal: per-kernel event timing hooks (see sirius_profile_enable in sirius.h).
#pragma once

#include <hip/hip_runtime.h>

namespace sirius {

int prof_begin(const char* name, hipStream_t s);
void prof_end(int id, hipStream_t s);

// Brackets one kernel launch: ProfScope p("name", stream); kernel<<<..., stream>>>(...);
struct ProfScope {
  int id;
  hipStream_t s;
  ProfScope(const char* name, hipStream_t stream) : id(prof_begin(name, stream)), s(stream) {}
  ~ProfScope() { prof_end(id, s); }
};

}  // namespace sirius
