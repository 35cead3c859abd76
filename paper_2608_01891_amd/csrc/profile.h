// Opt-in per-kernel timing: while a profile session is active, launches whose
// name is selected are bracketed by HIP events on their stream.
#pragma once
#include <hip/hip_runtime.h>

namespace aflex {

bool profile_wants(const char* name);
void profile_mark(const char* name, hipStream_t stream, bool begin);
hipError_t profile_release();

struct ProfScope {
  const char* name;
  hipStream_t stream;
  bool on;
  ProfScope(const char* n, hipStream_t s) : name(n), stream(s), on(profile_wants(n)) {
    if (on) profile_mark(name, stream, true);
  }
  ~ProfScope() {
    if (on) profile_mark(name, stream, false);
  }
};

}  // namespace aflex
