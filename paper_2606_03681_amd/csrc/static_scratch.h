// Library-owned device scratch of the allocation-free forward entry point.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "tfm_layer.h"

namespace tfm {

constexpr size_t kStaticScratchBytes = TFM_NOALLOC_SCRATCH_BYTES;

// Device address of the scratch array on the current device (looked up on the first call per
// device).  Fails with hipErrorInvalidDevice when `stream` belongs to another device than the
// current one.
hipError_t static_scratch(hipStream_t stream, void** ptr);

}  // namespace tfm
