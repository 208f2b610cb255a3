// Internal hooks of the step profiler (include/tfm_prof.h).
#pragma once

#include <hip/hip_runtime.h>

namespace tfm {

// Brackets one launch step with events on stream s while profiling is on; no-ops otherwise.
void prof_begin(const char* name, hipStream_t s);
void prof_end(hipStream_t s);

}  // namespace tfm
