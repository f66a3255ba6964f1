// Opt-in per-kernel timing: while enabled, each kernel launch is bracketed by
// HIP events recorded on the launch stream (see linsimp_timing_enable).
#pragma once
#include <hip/hip_runtime.h>

namespace linsimp {

bool timing_on();
void timing_mark(const char* name, hipStream_t st, bool begin);

struct ProfScope {
  const char* name;
  hipStream_t st;
  ProfScope(const char* n, hipStream_t s) : name(n), st(s) { if (timing_on()) timing_mark(name, st, true); }
  ~ProfScope() { if (timing_on()) timing_mark(name, st, false); }
};

}  // namespace linsimp
