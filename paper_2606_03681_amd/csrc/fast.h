// MFMA (bfloat16) path of the layer: launch sequences for the forward and backward pass.
#pragma once

#include <stddef.h>

#include "common.h"

namespace tfm {

// Scratch bytes that the MFMA path needs inside the workspace.
size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16);

}  // namespace tfm
