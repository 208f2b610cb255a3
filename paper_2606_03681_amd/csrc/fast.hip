// Small kernels of the MFMA path: weight casts, strided reductions, zero fill.
#include "fast.h"
#include "mfma.h"

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

// One wave per cell, 8 waves per block, LN_CELLS cells per block; each lane holds up to 4 of
// the E <= 256 values of a cell and keeps running column sums across the block's cells.
constexpr int LN_CELLS = 256;

__global__ __launch_bounds__(512) void k_ln_out_bwd(Geo g, const bf16* __restrict__ dY,
                                                    const bf16* __restrict__ xhat,
                                                    const float* __restrict__ rstd,
                                                    const float* __restrict__ gamma,
                                                    bf16* __restrict__ dz,
                                                    float* __restrict__ part) {
  __shared__ float red[8][2][256];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int E = g.E;
  float cs1[4] = {0.f, 0.f, 0.f, 0.f}, cs2[4] = {0.f, 0.f, 0.f, 0.f};
  float gm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) gm[i] = lane + 64 * i < E ? gamma[lane + 64 * i] : 0.f;
  const int64_t c0 = (int64_t)blockIdx.x * LN_CELLS;
  for (int cc = w; cc < LN_CELLS; cc += 8) {
    const int64_t p = c0 + cc;
    if (p >= g.N) break;
    const int64_t src = native_cell(g, p) * E;
    float dy[4], xv[4];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + 64 * i;
      dy[i] = 0.f;
      xv[i] = 0.f;
      if (e < E) {
        dy[i] = bf2f(dY[src + e]);
        xv[i] = bf2f(xhat[p * E + e]);
        cs1[i] += dy[i] * xv[i];
        cs2[i] += dy[i];
        s1 += dy[i] * gm[i];
        s2 += dy[i] * gm[i] * xv[i];
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      s1 += __shfl_xor(s1, o, 64);
      s2 += __shfl_xor(s2, o, 64);
    }
    const float m1 = s1 / E, m2 = s2 / E, rs = rstd[p];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + 64 * i;
      if (e < E) dz[p * E + e] = f2bf(rs * (dy[i] * gm[i] - m1 - xv[i] * m2));
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    red[w][0][lane + 64 * i] = cs1[i];
    red[w][1][lane + 64 * i] = cs2[i];
  }
  __syncthreads();
  if (threadIdx.x < 2 * E) {
    const int t = threadIdx.x / E, e = threadIdx.x % E;
    float s = 0.f;
#pragma unroll
    for (int ww = 0; ww < 8; ++ww) s += red[ww][t][e];
    part[(int64_t)blockIdx.x * 2 * E + t * E + e] = s;
  }
}

hipError_t launch_ln_out_bwd(const Geo& g, const bf16* dY, const bf16* xhat, const float* rstd,
                             const float* gamma, bf16* dz, float* part, int* nblocks,
                             hipStream_t s) {
  const int64_t nb = (g.N + LN_CELLS - 1) / LN_CELLS;
  *nblocks = (int)nb;
  k_ln_out_bwd<<<(unsigned)nb, 512, 0, s>>>(g, dY, xhat, rstd, gamma, dz, part);
  return hipGetLastError();
}

size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16) {
  (void)heads;
  if (!bf16) return 0;
  WOff wo = weight_offsets(E, H);
  const int64_t tiles = gemm_row_tiles((int64_t)B * R * S);
  size_t bytes = 2 * (size_t)wo.total * 2 + 1024;   // w and wt
  bytes += (size_t)tiles * 2 * E * 4 + 256;         // LN-backward column partials
  const int64_t cells = (int64_t)B * R * S;
  const int64_t zw = (cells + WGRAD_CHUNK - 1) / WGRAD_CHUNK;
  const int64_t maxw = 3LL * E * E > (int64_t)H * E ? 3LL * E * E : (int64_t)H * E;
  const int64_t maxn = 3LL * E > H ? 3LL * E : H;
  bytes += (size_t)zw * maxw * 4 + 256;                // weight-gradient partials
  bytes += (size_t)zw * maxn * 4 + 256;                // bias-gradient partials
  return bytes;
}

}  // namespace tfm
