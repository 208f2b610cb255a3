// Kernels of the optimiser step (C ABI in include/tfm_optim.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tfm {

constexpr int OPT_CHUNK = 4096;  // elements per workgroup of the element-wise kernels
inline int64_t opt_blocks(int64_t n) { return (n + OPT_CHUNK - 1) / OPT_CHUNK; }

constexpr int SF_MAXSEG = 64;
// Segments of one schedule-free AdamW call: segment k covers entries [off[k], off[k] + len) of
// the vectors; start[k] is its first index in the concatenation (start[nseg] = total).
struct SfSegs {
  int64_t off[SF_MAXSEG];
  int64_t start[SF_MAXSEG + 1];
  int32_t nseg;
};
struct SfScalars {
  float beta2, eps, wd;
  float c;      // averaging weight s_t^2 / sum s_i^2
  float gamma;  // step rate s_t sqrt(1 - beta2^t)
  float ycoef;  // gamma (beta1 (1 - c) - 1)
};

struct MuonGeo {
  int32_t count, rows, cols;
  int32_t tall;        // rows > cols: the operand is the transpose
  int32_t nesterov;
  float momentum, eps;
  float shrink;        // 1 - lr weight_decay
  float step;          // lr max(1, rows / cols)^(1/2)
};

// part[b] = sum of squares of g over [b OPT_CHUNK, (b + 1) OPT_CHUNK)
hipError_t launch_sumsq(const float* g, int64_t n, float* part, hipStream_t s);
// scale = min(1, max_norm / (sqrt(sum part) + 1e-6)), norm (nullable) = sqrt(sum part)
hipError_t launch_clip_final(const float* part, int64_t np, float max_norm, float* scale,
                             float* norm, hipStream_t s);
hipError_t launch_sfadamw(const SfSegs& sg, const SfScalars& sc, float* y, float* z, float* v,
                          const float* grad, const float* gscale, hipStream_t s);
// ptr: device int64 [3 count] = (W, G, buf) of each matrix; X: [count][rows * cols];
// part: [count][opt_blocks(rows * cols)]
hipError_t launch_muon_prep(const MuonGeo& mg, const int64_t* ptr, const float* gscale, float* X,
                            float* part, hipStream_t s);
hipError_t launch_muon_norm(const MuonGeo& mg, const float* part, float* X, hipStream_t s);
hipError_t launch_muon_apply(const MuonGeo& mg, const int64_t* ptr, const float* X,
                             hipStream_t s);

}  // namespace tfm
