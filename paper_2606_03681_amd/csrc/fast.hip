// MFMA (bfloat16) path of the layer.
#include "fast.h"

namespace tfm {

size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16) {
  (void)B; (void)R; (void)S; (void)E; (void)heads; (void)H; (void)bf16;
  return 0;
}

}  // namespace tfm
