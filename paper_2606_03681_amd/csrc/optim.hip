// Kernels of the optimiser step (C ABI in include/tfm_optim.h): global-norm clipping, the
// schedule-free AdamW update and the element-wise parts of Muon (momentum, Nesterov input,
// Frobenius scaling, the final update).  The Newton–Schulz products run on the float32 matrix
// cores through the batched GEMM of ends.hip.  Every kernel here is HBM-bound element-wise work
// or a small reduction; sums are taken in a fixed order.
#include "optim.h"

#include <hip/hip_runtime.h>

namespace tfm {
namespace {

// Block-wide sum of one value per thread in a fixed order (tree over the 256 threads).
__device__ __forceinline__ float block_sum(float v, float* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const float s = red[0];
  __syncthreads();
  return s;
}

// part[b] = sum of squares of g over elements [b * OPT_CHUNK, (b + 1) * OPT_CHUNK).
__global__ __launch_bounds__(256) void k_sumsq(const float* __restrict__ g, int64_t n,
                                               float* __restrict__ part) {
  __shared__ float red[256];
  const int64_t b0 = (int64_t)blockIdx.x * OPT_CHUNK;
  float s = 0.f;
  for (int i = threadIdx.x; i < OPT_CHUNK; i += 256) {
    const int64_t k = b0 + i;
    if (k < n) s = fmaf(g[k], g[k], s);
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_clip_final(const float* __restrict__ part, int64_t np,
                                                    float max_norm, float* __restrict__ scale,
                                                    float* __restrict__ norm) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < np; i += 256) s += part[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double nrm = sqrt(red[0]);
    const double f = (double)max_norm / (nrm + 1e-6);
    scale[0] = (float)(f < 1.0 ? f : 1.0);
    if (norm) norm[0] = (float)nrm;
  }
}

__global__ __launch_bounds__(256) void k_sfadamw(SfSegs sg, SfScalars sc, float* __restrict__ y,
                                                 float* __restrict__ z, float* __restrict__ v,
                                                 const float* __restrict__ grad,
                                                 const float* __restrict__ gscale) {
  const float gs = gscale ? gscale[0] : 1.f;
  const int64_t total = sg.start[sg.nseg];
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    int k = 0;
    while (k + 1 < sg.nseg && sg.start[k + 1] <= i) ++k;
    const int64_t j = sg.off[k] + (i - sg.start[k]);
    const float g = gs * grad[j];
    const float vv = fmaf(sc.beta2, v[j], (1.f - sc.beta2) * g * g);
    v[j] = vv;
    const float yy = y[j], zz = z[j];
    const float u = g / (sqrtf(vv) + sc.eps) + sc.wd * yy;
    y[j] = yy + sc.c * (zz - yy) + sc.ycoef * u;
    z[j] = zz - sc.gamma * u;
  }
}

// Muon, element-wise parts.  Matrix i has pointers ptr[3 i] (W), ptr[3 i + 1] (G),
// ptr[3 i + 2] (buf); X[i] holds its Newton–Schulz operand in the wide orientation
// (n = min(rows, cols) rows of m = max(rows, cols)).
__global__ __launch_bounds__(256) void k_muon_prep(MuonGeo mg, const int64_t* __restrict__ ptr,
                                                   const float* __restrict__ gscale,
                                                   float* __restrict__ X,
                                                   float* __restrict__ part) {
  __shared__ float red[256];
  const int i = blockIdx.y;
  const float* G = (const float*)ptr[3 * i + 1];
  float* buf = (float*)ptr[3 * i + 2];
  float* Xi = X + (int64_t)i * mg.rows * mg.cols;
  const float gs = gscale ? gscale[0] : 1.f;
  const int64_t nel = (int64_t)mg.rows * mg.cols;
  const int64_t b0 = (int64_t)blockIdx.x * OPT_CHUNK;
  float s = 0.f;
  for (int e = threadIdx.x; e < OPT_CHUNK; e += 256) {
    const int64_t k = b0 + e;
    if (k < nel) {
      const float g = gs * G[k];
      const float bb = fmaf(mg.momentum, buf[k], (1.f - mg.momentum) * g);
      buf[k] = bb;
      const float u = mg.nesterov ? fmaf(mg.momentum, bb, (1.f - mg.momentum) * g) : bb;
      const int64_t r = k / mg.cols, c = k - r * mg.cols;
      Xi[mg.tall ? c * mg.rows + r : k] = u;
      s = fmaf(u, u, s);
    }
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) part[(int64_t)i * gridDim.x + blockIdx.x] = s;
}

// X[i] *= 1 / (||U_i||_F + eps); every block sums matrix i's partials in the same order.
__global__ __launch_bounds__(256) void k_muon_norm(MuonGeo mg, const float* __restrict__ part,
                                                   float* __restrict__ X) {
  __shared__ float inv;
  const int i = blockIdx.y;
  if (threadIdx.x == 0) {
    float s = 0.f;
    for (int k = 0; k < (int)gridDim.x; ++k) s += part[(int64_t)i * gridDim.x + k];
    inv = 1.f / (sqrtf(s) + mg.eps);
  }
  __syncthreads();
  const int64_t nel = (int64_t)mg.rows * mg.cols;
  float* Xi = X + (int64_t)i * nel;
  const int64_t b0 = (int64_t)blockIdx.x * OPT_CHUNK;
  for (int e = threadIdx.x; e < OPT_CHUNK; e += 256) {
    const int64_t k = b0 + e;
    if (k < nel) Xi[k] *= inv;
  }
}

__global__ __launch_bounds__(256) void k_muon_apply(MuonGeo mg, const int64_t* __restrict__ ptr,
                                                    const float* __restrict__ X) {
  const int i = blockIdx.y;
  float* W = (float*)ptr[3 * i];
  const int64_t nel = (int64_t)mg.rows * mg.cols;
  const float* Xi = X + (int64_t)i * nel;
  const int64_t b0 = (int64_t)blockIdx.x * OPT_CHUNK;
  for (int e = threadIdx.x; e < OPT_CHUNK; e += 256) {
    const int64_t k = b0 + e;
    if (k < nel) {
      const int64_t r = k / mg.cols, c = k - r * mg.cols;
      const float o = Xi[mg.tall ? c * mg.rows + r : k];
      W[k] = fmaf(W[k], mg.shrink, -mg.step * o);
    }
  }
}

}  // namespace

hipError_t launch_sumsq(const float* g, int64_t n, float* part, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  k_sumsq<<<(unsigned)opt_blocks(n), 256, 0, s>>>(g, n, part);
  return hipGetLastError();
}

hipError_t launch_clip_final(const float* part, int64_t np, float max_norm, float* scale,
                             float* norm, hipStream_t s) {
  k_clip_final<<<1, 256, 0, s>>>(part, np, max_norm, scale, norm);
  return hipGetLastError();
}

hipError_t launch_sfadamw(const SfSegs& sg, const SfScalars& sc, float* y, float* z, float* v,
                          const float* grad, const float* gscale, hipStream_t s) {
  const int64_t total = sg.start[sg.nseg];
  if (total <= 0) return hipSuccess;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  k_sfadamw<<<(unsigned)blocks, 256, 0, s>>>(sg, sc, y, z, v, grad, gscale);
  return hipGetLastError();
}

hipError_t launch_muon_prep(const MuonGeo& mg, const int64_t* ptr, const float* gscale, float* X,
                            float* part, hipStream_t s) {
  dim3 grid((unsigned)opt_blocks((int64_t)mg.rows * mg.cols), (unsigned)mg.count);
  k_muon_prep<<<grid, 256, 0, s>>>(mg, ptr, gscale, X, part);
  return hipGetLastError();
}

hipError_t launch_muon_norm(const MuonGeo& mg, const float* part, float* X, hipStream_t s) {
  dim3 grid((unsigned)opt_blocks((int64_t)mg.rows * mg.cols), (unsigned)mg.count);
  k_muon_norm<<<grid, 256, 0, s>>>(mg, part, X);
  return hipGetLastError();
}

hipError_t launch_muon_apply(const MuonGeo& mg, const int64_t* ptr, const float* X,
                             hipStream_t s) {
  dim3 grid((unsigned)opt_blocks((int64_t)mg.rows * mg.cols), (unsigned)mg.count);
  k_muon_apply<<<grid, 256, 0, s>>>(mg, ptr, X);
  return hipGetLastError();
}

}  // namespace tfm
