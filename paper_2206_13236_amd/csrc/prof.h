// Opt-in per-kernel timing: when enabled (rnnt_profile_enable), every named
// launch is bracketed by two HIP events recorded on the launch stream.
// Disabled by default, in which case the brackets cost one branch.
#pragma once

#include <hip/hip_runtime.h>

void prof_begin(hipStream_t s, const char* name);
void prof_end(hipStream_t s, const char* name);

struct ProfScope {
  hipStream_t s;
  const char* name;
  ProfScope(hipStream_t s_, const char* n) : s(s_), name(n) { prof_begin(s, name); }
  ~ProfScope() { prof_end(s, name); }
};

#define RNNT_PROF(stream, name) ProfScope _rnnt_prof_scope((stream), (name))
