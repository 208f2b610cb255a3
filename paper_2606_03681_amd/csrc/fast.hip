// Small kernels of the MFMA path: weight casts, strided reductions, zero fill.
#include "fast.h"

namespace tfm {

WOff weight_offsets(int E, int H) {
  WOff o;
  int64_t x = 0;
  o.qkv_f = x; x += 3LL * E * E;
  o.o_f = x; x += (int64_t)E * E;
  o.qkv_i = x; x += 3LL * E * E;
  o.o_i = x; x += (int64_t)E * E;
  o.w1 = x; x += (int64_t)H * E;
  o.w2 = x; x += (int64_t)E * H;
  o.total = x;
  return o;
}

// One thread per weight element: src (fp32, packed parameter order) -> w (same layout, bf16)
// and wt (each matrix transposed, bf16).
__global__ void k_weight_prep(const float* __restrict__ p, int E, int H, WOff wo,
                              bf16* __restrict__ w, bf16* __restrict__ wt) {
  // packed parameter offsets of the six matrices
  const int64_t E2 = (int64_t)E * E;
  const int64_t src[6] = {0, 3 * E2 + 3 * E, 4 * E2 + 4 * E, 7 * E2 + 7 * E, 8 * E2 + 8 * E,
                          8 * E2 + 8 * E + (int64_t)H * E + H};
  const int64_t dst[6] = {wo.qkv_f, wo.o_f, wo.qkv_i, wo.o_i, wo.w1, wo.w2};
  const int rows[6] = {3 * E, E, 3 * E, E, H, E};
  const int cols[6] = {E, E, E, E, E, H};
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int k = 0; k < 6; ++k) {
    int64_t n = (int64_t)rows[k] * cols[k];
    if (t < n) {
      int r = (int)(t / cols[k]), c = (int)(t % cols[k]);
      uint16_t v = f2bf(p[src[k] + t]);
      w[dst[k] + t] = v;
      wt[dst[k] + (int64_t)c * rows[k] + r] = v;
      return;
    }
    t -= n;
  }
}

hipError_t launch_weight_prep(const float* params, int E, int H, bf16* w, bf16* wt,
                              hipStream_t s) {
  WOff wo = weight_offsets(E, H);
  unsigned grid = (unsigned)((wo.total + 255) / 256);
  k_weight_prep<<<grid, 256, 0, s>>>(params, E, H, wo, w, wt);
  return hipGetLastError();
}

__global__ void k_reduce_strided(int Z, int64_t count, int64_t stride,
                                 const float* __restrict__ part, float* __restrict__ grad,
                                 int accumulate) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  float s = 0.f;
  for (int z = 0; z < Z; ++z) s += part[(int64_t)z * stride + i];
  grad[i] = (accumulate ? grad[i] : 0.f) + s;
}

hipError_t launch_reduce_strided(int Z, int64_t count, int64_t stride, const float* part,
                                 float* grad, int accumulate, hipStream_t s) {
  k_reduce_strided<<<(unsigned)((count + 255) / 256), 256, 0, s>>>(Z, count, stride, part, grad,
                                                                   accumulate);
  return hipGetLastError();
}

// One thread per native cell; inactive cells get E zeros (16-byte stores).
__global__ void k_zero_inactive(Geo g, bf16* __restrict__ x) {
  int64_t cell = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (cell >= (int64_t)g.B * g.R * g.S) return;
  int c = (int)(cell % g.S);
  int b = (int)(cell / ((int64_t)g.R * g.S));
  if (g.colmap[b * g.S + c] >= 0) return;
  uint4 z = make_uint4(0, 0, 0, 0);
  uint4* p = reinterpret_cast<uint4*>(x + cell * g.E);
  for (int i = 0; i < g.E / 8; ++i) p[i] = z;
}

hipError_t launch_zero_inactive(const Geo& g, bf16* native, hipStream_t s) {
  int64_t n = (int64_t)g.B * g.R * g.S;
  k_zero_inactive<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(g, native);
  return hipGetLastError();
}

size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16) {
  (void)heads;
  if (!bf16) return 0;
  WOff wo = weight_offsets(E, H);
  int64_t tiles = ((int64_t)B * R * S + 127) / 128;
  size_t bytes = 2 * (size_t)wo.total * 2 + 1024;   // w and wt
  bytes += (size_t)tiles * 2 * E * 4 + 256;         // LN-backward column partials
  return bytes;
}

}  // namespace tfm
