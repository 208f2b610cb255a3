// Straightforward HIP kernels of the layer: fp32 arithmetic on VALU, any storage type.
// They serve the float32 mode, whose 1e-4 parity needs true fp32 products, and they are the
// baseline that the MFMA kernels of the bfloat16 mode are measured against.
#include <math.h>

#include "kernels.h"

namespace tfm {

namespace {

inline unsigned grid_for(int64_t n, int per_block = TFM_BLOCK) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (unsigned)g;
}

__device__ __forceinline__ int64_t gtid() {
  return (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
}
__device__ __forceinline__ int64_t gstride() { return (int64_t)gridDim.x * blockDim.x; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace

// ============================================================================ metadata
struct UploadChunk {
  int32_t n, off;
  int32_t v[504];
};

__global__ void k_upload(UploadChunk c, int32_t* dst) {
  for (int i = threadIdx.x; i < c.n; i += blockDim.x) dst[c.off + i] = c.v[i];
}

hipError_t launch_upload(const int32_t* host, int64_t count, int32_t* dst, hipStream_t s) {
  for (int64_t o = 0; o < count; o += 504) {
    UploadChunk c;
    c.n = (int32_t)((count - o) < 504 ? (count - o) : 504);
    c.off = (int32_t)o;
    for (int i = 0; i < c.n; ++i) c.v[i] = host[o + i];
    k_upload<<<1, TFM_BLOCK, 0, s>>>(c, dst);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ void k_expand_meta(const int32_t* blob, int B, int R, int S, int W, DsInfo* ds,
                              int32_t* col_ds, int32_t* col_c, int32_t* colmap,
                              int64_t* col_cell0, int32_t* col_ntr) {
  int64_t t = gtid();
  if (t >= (int64_t)B * S) return;
  int b = (int)(t / S), c = (int)(t % S);
  const int32_t* e = blob + (int64_t)b * (3 + W);
  const uint32_t* bits = (const uint32_t*)(e + 3);
  if (c == 0) ds[b] = DsInfo{e[0], e[1], e[2], 0};
  bool on = (bits[c >> 5] >> (c & 31)) & 1u;
  if (!on) {
    colmap[t] = -1;
    return;
  }
  int k = 0;
  for (int w = 0; w < (c >> 5); ++w) k += __popc(bits[w]);
  k += __popc(bits[c >> 5] & ((1u << (c & 31)) - 1u));
  int gcol = e[1] + k;
  col_ds[gcol] = b;
  col_c[gcol] = c;
  colmap[t] = gcol;
  col_cell0[gcol] = (int64_t)b * R * S + c;
  col_ntr[gcol] = e[0];
}

hipError_t launch_expand_meta(const int32_t* blob, int B, int R, int S, int words, DsInfo* ds,
                              int32_t* col_ds, int32_t* col_c, int32_t* colmap,
                              int64_t* col_cell0, int32_t* col_ntr, hipStream_t s) {
  k_expand_meta<<<grid_for((int64_t)B * S), TFM_BLOCK, 0, s>>>(blob, B, R, S, words, ds, col_ds,
                                                                 col_c, colmap, col_cell0,
                                                                 col_ntr);
  return hipGetLastError();
}

// ============================================================================ gather / scatter
template <class T>
__global__ void k_gather(Geo g, const T* __restrict__ src, T* __restrict__ dst) {
  int64_t total = g.N * g.E;
  for (int64_t i = gtid(); i < total; i += gstride()) {
    int64_t p = i / g.E;
    int e = (int)(i - p * g.E);
    dst[i] = src[native_cell(g, p) * g.E + e];
  }
}

template <class T>
hipError_t launch_gather(const Geo& g, const T* native, T* cells, hipStream_t s) {
  k_gather<T><<<grid_for(g.N * g.E), TFM_BLOCK, 0, s>>>(g, native, cells);
  return hipGetLastError();
}

template <class T>
__global__ void k_scatter(Geo g, const T* __restrict__ a, const T* __restrict__ b,
                          T* __restrict__ dst) {
  int64_t total = (int64_t)g.B * g.R * g.S * g.E;
  for (int64_t i = gtid(); i < total; i += gstride()) {
    int64_t cell = i / g.E;
    int e = (int)(i - cell * g.E);
    int c = (int)(cell % g.S);
    int64_t br = cell / g.S;
    int r = (int)(br % g.R);
    int bb = (int)(br / g.R);
    int gcol = g.colmap[bb * g.S + c];
    float v = 0.f;
    if (gcol >= 0) {
      int64_t p = ((int64_t)gcol * g.R + r) * g.E + e;
      v = ld(a + p);
      if (b) v += ld(b + p);
    }
    st(dst + i, v);
  }
}

template <class T>
hipError_t launch_scatter(const Geo& g, const T* a, const T* b, T* native, hipStream_t s) {
  k_scatter<T><<<grid_for((int64_t)g.B * g.R * g.S * g.E), TFM_BLOCK, 0, s>>>(g, a, b, native);
  return hipGetLastError();
}

// ============================================================================ linear
// 64 x 64 output tile per block, 4 x 4 outputs per thread, K in steps of 16 through LDS.
template <class TA, class TO, bool ITEM>
__global__ __launch_bounds__(256) void k_linear(int64_t M, int Nout, int K,
                                                const TA* __restrict__ A, int64_t lda,
                                                const float* __restrict__ w, int64_t wsj,
                                                int64_t wsi, const float* __restrict__ bias,
                                                TO* __restrict__ out, int64_t ldo, Geo g,
                                                TO* __restrict__ kout, TO* __restrict__ vout) {
  __shared__ float As[16][65];
  __shared__ float Ws[16][65];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int64_t m0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int i = threadIdx.x; i < 1024; i += 256) {
      int mm = i >> 4, kk = i & 15;
      int64_t m = m0 + mm;
      int k = k0 + kk;
      As[kk][mm] = (m < M && k < K) ? ld(A + m * lda + k) : 0.f;
      int n = n0 + mm;
      Ws[kk][mm] = (n < Nout && k < K) ? w[n * wsj + (int64_t)k * wsi] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Ws[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int64_t m = m0 + ty + 16 * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int n = n0 + tx + 16 * j;
      if (n >= Nout) continue;
      float v = acc[i][j] + (bias ? bias[n] : 0.f);
      if (!ITEM) {
        st(out + m * ldo + n, v);
      } else {
        int part = n / g.E, within = n - part * g.E;
        int head = within / g.d, jj = within - head * g.d;
        int64_t col = m / g.R;
        int r = (int)(m - col * g.R);
        if (part > 0 && r >= g.col_ntr[col]) continue;
        TO* base = part == 0 ? out : (part == 1 ? kout : vout);
        st(base + (((int64_t)col * g.heads + head) * g.R + r) * g.d + jj, v);
      }
    }
  }
}

template <class TA, class TO>
hipError_t launch_linear(int64_t M, int Nout, int K, const TA* A, int64_t lda, const float* w,
                         int64_t wsj, int64_t wsi, const float* bias, TO* out, int64_t ldo,
                         hipStream_t s) {
  if (M <= 0) return hipSuccess;
  dim3 grid((unsigned)((M + 63) / 64), (unsigned)((Nout + 63) / 64));
  Geo g{};
  k_linear<TA, TO, false><<<grid, 256, 0, s>>>(M, Nout, K, A, lda, w, wsj, wsi, bias, out, ldo,
                                               g, nullptr, nullptr);
  return hipGetLastError();
}

template <class T>
hipError_t launch_linear_item_qkv(const Geo& g, const T* A, const float* w, const float* bias,
                                  T* q, T* k, T* v, hipStream_t s) {
  if (g.N <= 0) return hipSuccess;
  dim3 grid((unsigned)((g.N + 63) / 64), (unsigned)((3 * g.E + 63) / 64));
  k_linear<T, T, true><<<grid, 256, 0, s>>>(g.N, 3 * g.E, g.E, A, g.E, w, g.E, 1, bias, q, 0,
                                            g, k, v);
  return hipGetLastError();
}

// ============================================================================ reductions
template <class T>
__global__ __launch_bounds__(256) void k_wgrad(int64_t M, int Nj, int Ki,
                                               const T* __restrict__ dY, int64_t ldy,
                                               const T* __restrict__ X, int64_t ldx,
                                               int64_t chunk, float* __restrict__ part) {
  __shared__ float Ys[16][65];
  __shared__ float Xs[16][65];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int j0 = blockIdx.x * 64, i0 = blockIdx.y * 64;
  const int64_t mb = (int64_t)blockIdx.z * chunk;
  const int64_t me = (mb + chunk < M) ? mb + chunk : M;
  float acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = 0.f;
  for (int64_t m0 = mb; m0 < me; m0 += 16) {
    for (int t = threadIdx.x; t < 1024; t += 256) {
      int mm = t >> 6, jj = t & 63;
      int64_t m = m0 + mm;
      Ys[mm][jj] = (m < me && j0 + jj < Nj) ? ld(dY + m * ldy + j0 + jj) : 0.f;
      Xs[mm][jj] = (m < me && i0 + jj < Ki) ? ld(X + m * ldx + i0 + jj) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int mm = 0; mm < 16; ++mm) {
      float a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = Ys[mm][ty + 16 * q];
#pragma unroll
      for (int q = 0; q < 4; ++q) b[q] = Xs[mm][tx + 16 * q];
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[p][q] = fmaf(a[p], b[q], acc[p][q]);
    }
    __syncthreads();
  }
  float* out = part + (int64_t)blockIdx.z * Nj * Ki;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    int j = j0 + ty + 16 * p;
    if (j >= Nj) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int i = i0 + tx + 16 * q;
      if (i < Ki) out[(int64_t)j * Ki + i] = acc[p][q];
    }
  }
}

template <class T>
hipError_t launch_wgrad(int64_t M, int Nj, int Ki, const T* dY, int64_t ldy, const T* X,
                        int64_t ldx, int64_t chunk, float* partial, hipStream_t s) {
  int64_t Z = (M + chunk - 1) / chunk;
  if (Z < 1) Z = 1;
  dim3 grid((unsigned)((Nj + 63) / 64), (unsigned)((Ki + 63) / 64), (unsigned)Z);
  k_wgrad<T><<<grid, 256, 0, s>>>(M, Nj, Ki, dY, ldy, X, ldx, chunk, partial);
  return hipGetLastError();
}

template <class T>
__global__ void k_colsum(int64_t M, int Nj, const T* __restrict__ A, int64_t lda,
                         const T* __restrict__ B, int64_t ldb, int64_t chunk,
                         float* __restrict__ part) {
  int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= Nj) return;
  int64_t mb = (int64_t)blockIdx.y * chunk;
  int64_t me = (mb + chunk < M) ? mb + chunk : M;
  float acc = 0.f;
  for (int64_t m = mb; m < me; ++m) {
    float v = ld(A + m * lda + j);
    if (B) v *= ld(B + m * ldb + j);
    acc += v;
  }
  part[(int64_t)blockIdx.y * Nj + j] = acc;
}

template <class T>
hipError_t launch_colsum(int64_t M, int Nj, const T* A, int64_t lda, const T* B, int64_t ldb,
                         int64_t chunk, float* partial, hipStream_t s) {
  int64_t Z = (M + chunk - 1) / chunk;
  if (Z < 1) Z = 1;
  dim3 grid((unsigned)((Nj + 255) / 256), (unsigned)Z);
  k_colsum<T><<<grid, 256, 0, s>>>(M, Nj, A, lda, B, ldb, chunk, partial);
  return hipGetLastError();
}

__global__ void k_reduce_partials(int Z, int64_t count, const float* __restrict__ part,
                                  float* __restrict__ grad, int accumulate) {
  for (int64_t i = gtid(); i < count; i += gstride()) {
    float acc = accumulate ? grad[i] : 0.f;
    float sum = 0.f;
    for (int z = 0; z < Z; ++z) sum += part[(int64_t)z * count + i];
    grad[i] = acc + sum;
  }
}

hipError_t launch_reduce_partials(int Z, int64_t count, const float* partial, float* grad,
                                  int accumulate, hipStream_t s) {
  k_reduce_partials<<<grid_for(count), TFM_BLOCK, 0, s>>>(Z, count, partial, grad, accumulate);
  return hipGetLastError();
}

// ============================================================================ LayerNorm, GELU
// One wave per cell; each lane holds up to 4 of the E <= 256 values.
template <class T>
__global__ __launch_bounds__(256) void k_add_ln(int64_t N, int E, const T* __restrict__ a,
                                                const T* __restrict__ b,
                                                const float* __restrict__ gamma,
                                                const float* __restrict__ beta,
                                                T* __restrict__ h, T* __restrict__ xhat,
                                                float* __restrict__ rstd) {
  const int lane = threadIdx.x & 63;
  const int64_t cell = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (cell >= N) return;
  float u[4];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int e = lane + 64 * i;
    u[i] = 0.f;
    if (e < E) {
      u[i] = ld(a + cell * E + e) + (b ? ld(b + cell * E + e) : 0.f);
      s += u[i];
    }
  }
  const float mean = wave_sum(s) / E;
  float v = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int e = lane + 64 * i;
    if (e < E) v += (u[i] - mean) * (u[i] - mean);
  }
  const float rs = 1.0f / sqrtf(wave_sum(v) / E + 1e-5f);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int e = lane + 64 * i;
    if (e < E) {
      float x = (u[i] - mean) * rs;
      st(xhat + cell * E + e, x);
      st(h + cell * E + e, fmaf(gamma[e], x, beta[e]));
    }
  }
  if (lane == 0) rstd[cell] = rs;
}

template <class T>
hipError_t launch_add_ln(int64_t N, int E, const T* a, const T* b, const float* gamma,
                         const float* beta, T* h, T* xhat, float* rstd, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  k_add_ln<T><<<(unsigned)((N + 3) / 4), 256, 0, s>>>(N, E, a, b, gamma, beta, h, xhat, rstd);
  return hipGetLastError();
}

template <class T>
__global__ __launch_bounds__(256) void k_ln_bwd(int64_t N, int E, const T* __restrict__ dya,
                                                const T* __restrict__ dyb,
                                                const T* __restrict__ xhat,
                                                const float* __restrict__ rstd,
                                                const float* __restrict__ gamma,
                                                T* __restrict__ du, T* __restrict__ dysum) {
  const int lane = threadIdx.x & 63;
  const int64_t cell = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (cell >= N) return;
  float gv[4], xv[4];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int e = lane + 64 * i;
    gv[i] = 0.f;
    xv[i] = 0.f;
    if (e < E) {
      float dy = ld(dya + cell * E + e) + (dyb ? ld(dyb + cell * E + e) : 0.f);
      if (dysum) st(dysum + cell * E + e, dy);
      gv[i] = dy * gamma[e];
      xv[i] = ld(xhat + cell * E + e);
      s1 += gv[i];
      s2 += gv[i] * xv[i];
    }
  }
  const float m1 = wave_sum(s1) / E, m2 = wave_sum(s2) / E;
  const float rs = rstd[cell];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int e = lane + 64 * i;
    if (e < E) st(du + cell * E + e, rs * (gv[i] - m1 - xv[i] * m2));
  }
}

template <class T>
hipError_t launch_ln_bwd(int64_t N, int E, const T* dya, const T* dyb, const T* xhat,
                         const float* rstd, const float* gamma, T* du, T* dysum, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  k_ln_bwd<T><<<(unsigned)((N + 3) / 4), 256, 0, s>>>(N, E, dya, dyb, xhat, rstd, gamma, du,
                                                       dysum);
  return hipGetLastError();
}

template <class T>
__global__ void k_gelu(int64_t n, const T* __restrict__ g, T* __restrict__ u) {
  for (int64_t i = gtid(); i < n; i += gstride()) {
    float x = ld(g + i);
    st(u + i, 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)));
  }
}

template <class T>
hipError_t launch_gelu(int64_t count, const T* g, T* u, hipStream_t s) {
  k_gelu<T><<<grid_for(count), TFM_BLOCK, 0, s>>>(count, g, u);
  return hipGetLastError();
}

template <class T>
__global__ void k_gelu_bwd(int64_t n, const T* __restrict__ g, T* __restrict__ du) {
  for (int64_t i = gtid(); i < n; i += gstride()) {
    float x = ld(g + i);
    float cdf = 0.5f * (1.0f + erff(x * 0.70710678118654752f));
    float pdf = 0.39894228040143268f * expf(-0.5f * x * x);
    st(du + i, ld(du + i) * (cdf + x * pdf));
  }
}

template <class T>
hipError_t launch_gelu_bwd(int64_t count, const T* g, T* du, hipStream_t s) {
  k_gelu_bwd<T><<<grid_for(count), TFM_BLOCK, 0, s>>>(count, g, du);
  return hipGetLastError();
}

// ============================================================================ feature attention
// One thread per (row, head, query cell).  The cells of row (b, r) are
// p = (col0[b] + k) * R + r; q/k/v of cell p sit at qkv[p*3E + {0, E, 2E} + head*d].
template <class T, int D>
__global__ __launch_bounds__(256) void k_feat_attn_fwd(Geo g, const T* __restrict__ qkv,
                                                       T* __restrict__ o,
                                                       float* __restrict__ lse) {
  int64_t t = gtid();
  int64_t total = (int64_t)g.B * g.R * g.heads * g.S;
  if (t >= total) return;
  const int kq = (int)(t % g.S);
  t /= g.S;
  const int head = (int)(t % g.heads);
  const int64_t rho = t / g.heads;
  const int b = (int)(rho / g.R), r = (int)(rho % g.R);
  const DsInfo di = g.ds[b];
  if (kq >= di.S) return;
  const int E = g.E, E3 = 3 * g.E;
  const float tau = 1.0f / sqrtf((float)D);
  const int64_t pq = (int64_t)(di.col0 + kq) * g.R + r;
  float qv[D];
#pragma unroll
  for (int j = 0; j < D; ++j) qv[j] = ld(qkv + pq * E3 + head * D + j) * tau;
  float mx = -INFINITY;
  for (int kk = 0; kk < di.S; ++kk) {
    const T* kp = qkv + ((int64_t)(di.col0 + kk) * g.R + r) * E3 + E + head * D;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) s = fmaf(qv[j], ld(kp + j), s);
    mx = fmaxf(mx, s);
  }
  float acc[D];
#pragma unroll
  for (int j = 0; j < D; ++j) acc[j] = 0.f;
  float sum = 0.f;
  for (int kk = 0; kk < di.S; ++kk) {
    const T* kp = qkv + ((int64_t)(di.col0 + kk) * g.R + r) * E3 + E + head * D;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) s = fmaf(qv[j], ld(kp + j), s);
    float p = expf(s - mx);
    sum += p;
    const T* vp = kp + E;
#pragma unroll
    for (int j = 0; j < D; ++j) acc[j] = fmaf(p, ld(vp + j), acc[j]);
  }
  const float inv = 1.0f / sum;
#pragma unroll
  for (int j = 0; j < D; ++j) st(o + pq * E + head * D + j, acc[j] * inv);
  lse[pq * g.heads + head] = mx + logf(sum);
}

template <class T>
hipError_t launch_feat_attn_fwd_simple(const Geo& g, const T* qkv, T* o, float* lse,
                                       hipStream_t s) {
  int64_t total = (int64_t)g.B * g.R * g.heads * g.S;
  if (g.d == 16)
    k_feat_attn_fwd<T, 16><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, lse);
  else if (g.d == 32)
    k_feat_attn_fwd<T, 32><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, lse);
  else
    k_feat_attn_fwd<T, 64><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, lse);
  return hipGetLastError();
}

// One thread per (row, head, cell i): dQ_i as a query, dK_i and dV_i as a key.
template <class T, int D>
__global__ __launch_bounds__(256) void k_feat_attn_bwd(Geo g, const T* __restrict__ qkv,
                                                       const T* __restrict__ o,
                                                       const T* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       T* __restrict__ dqkv) {
  int64_t t = gtid();
  int64_t total = (int64_t)g.B * g.R * g.heads * g.S;
  if (t >= total) return;
  const int ki = (int)(t % g.S);
  t /= g.S;
  const int head = (int)(t % g.heads);
  const int64_t rho = t / g.heads;
  const int b = (int)(rho / g.R), r = (int)(rho % g.R);
  const DsInfo di = g.ds[b];
  if (ki >= di.S) return;
  const int E = g.E, E3 = 3 * g.E, hd = head * D;
  const float tau = 1.0f / sqrtf((float)D);
  const int64_t pi = (int64_t)(di.col0 + ki) * g.R + r;
  float qi[D], kv[D], vv[D], doi[D];
  float Di = 0.f;
#pragma unroll
  for (int j = 0; j < D; ++j) {
    qi[j] = ld(qkv + pi * E3 + hd + j);
    kv[j] = ld(qkv + pi * E3 + E + hd + j);
    vv[j] = ld(qkv + pi * E3 + 2 * E + hd + j);
    doi[j] = ld(dout + pi * E + hd + j);
    Di = fmaf(doi[j], ld(o + pi * E + hd + j), Di);
  }
  const float lsei = lse[pi * g.heads + head];
  float dq[D], dk[D], dv[D];
#pragma unroll
  for (int j = 0; j < D; ++j) dq[j] = dk[j] = dv[j] = 0.f;
  for (int kk = 0; kk < di.S; ++kk) {
    const int64_t pk = (int64_t)(di.col0 + kk) * g.R + r;
    const T* base = qkv + pk * E3 + hd;
    // cell i as the query, cell kk as the key
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      s = fmaf(qi[j], ld(base + E + j), s);
      dp = fmaf(doi[j], ld(base + 2 * E + j), dp);
    }
    float p = expf(s * tau - lsei);
    float ds = p * (dp - Di);
#pragma unroll
    for (int j = 0; j < D; ++j) dq[j] = fmaf(ds * tau, ld(base + E + j), dq[j]);
    // cell kk as the query, cell i as the key
    float s2 = 0.f, dp2 = 0.f, Dk = 0.f;
    const T* dok = dout + pk * E + hd;
    const T* ok = o + pk * E + hd;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      float qk = ld(base + j);
      float dokj = ld(dok + j);
      s2 = fmaf(qk, kv[j], s2);
      dp2 = fmaf(dokj, vv[j], dp2);
      Dk = fmaf(dokj, ld(ok + j), Dk);
    }
    float p2 = expf(s2 * tau - lse[pk * g.heads + head]);
    float ds2 = p2 * (dp2 - Dk);
#pragma unroll
    for (int j = 0; j < D; ++j) {
      dk[j] = fmaf(ds2 * tau, ld(base + j), dk[j]);
      dv[j] = fmaf(p2, ld(dok + j), dv[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < D; ++j) {
    st(dqkv + pi * E3 + hd + j, dq[j]);
    st(dqkv + pi * E3 + E + hd + j, dk[j]);
    st(dqkv + pi * E3 + 2 * E + hd + j, dv[j]);
  }
}

template <class T>
hipError_t launch_feat_attn_bwd_simple(const Geo& g, const T* qkv, const T* o, const T* dout,
                                       const float* lse, T* dqkv, hipStream_t s) {
  int64_t total = (int64_t)g.B * g.R * g.heads * g.S;
  if (g.d == 16)
    k_feat_attn_bwd<T, 16><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  else if (g.d == 32)
    k_feat_attn_bwd<T, 32><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  else
    k_feat_attn_bwd<T, 64><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  return hipGetLastError();
}

// ============================================================================ item attention
// One thread per (column, head, query row); keys are the train rows t < n_train.
template <class T, int D>
__global__ __launch_bounds__(256) void k_item_attn_fwd(Geo g, const T* __restrict__ q,
                                                       const T* __restrict__ k,
                                                       const T* __restrict__ v,
                                                       T* __restrict__ o,
                                                       float* __restrict__ lse) {
  int64_t t = gtid();
  if (t >= (int64_t)g.NC * g.heads * g.R) return;
  const int r = (int)(t % g.R);
  const int64_t ch = t / g.R;  // col * heads + head
  const int head = (int)(ch % g.heads);
  const int64_t col = ch / g.heads;
  const int n = g.col_ntr[col];
  const float tau = 1.0f / sqrtf((float)D);
  const int64_t base = ch * g.R;
  float qv[D];
#pragma unroll
  for (int j = 0; j < D; ++j) qv[j] = ld(q + (base + r) * D + j) * tau;
  float mx = -INFINITY;
  for (int tt = 0; tt < n; ++tt) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) s = fmaf(qv[j], ld(k + (base + tt) * D + j), s);
    mx = fmaxf(mx, s);
  }
  float acc[D];
#pragma unroll
  for (int j = 0; j < D; ++j) acc[j] = 0.f;
  float sum = 0.f;
  for (int tt = 0; tt < n; ++tt) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) s = fmaf(qv[j], ld(k + (base + tt) * D + j), s);
    float p = expf(s - mx);
    sum += p;
#pragma unroll
    for (int j = 0; j < D; ++j) acc[j] = fmaf(p, ld(v + (base + tt) * D + j), acc[j]);
  }
  const float inv = 1.0f / sum;
  const int64_t p = col * g.R + r;
#pragma unroll
  for (int j = 0; j < D; ++j) st(o + p * g.E + head * D + j, acc[j] * inv);
  lse[base + r] = mx + logf(sum);
}

template <class T>
hipError_t launch_item_attn_fwd_simple(const Geo& g, const T* q, const T* k, const T* v, T* o,
                                       float* lse, hipStream_t s) {
  int64_t total = (int64_t)g.NC * g.heads * g.R;
  if (g.d == 16)
    k_item_attn_fwd<T, 16><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, q, k, v, o, lse);
  else if (g.d == 32)
    k_item_attn_fwd<T, 32><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, q, k, v, o, lse);
  else
    k_item_attn_fwd<T, 64><<<grid_for(total), TFM_BLOCK, 0, s>>>(g, q, k, v, o, lse);
  return hipGetLastError();
}

template <class T, int D>
__global__ void k_item_rowdot(Geo g, const T* __restrict__ o, const T* __restrict__ dout,
                              float* __restrict__ Dv) {
  int64_t t = gtid();
  if (t >= (int64_t)g.NC * g.heads * g.R) return;
  const int r = (int)(t % g.R);
  const int64_t ch = t / g.R;
  const int head = (int)(ch % g.heads);
  const int64_t col = ch / g.heads;
  const int64_t p = (col * g.R + r) * g.E + head * D;
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < D; ++j) acc = fmaf(ld(o + p + j), ld(dout + p + j), acc);
  Dv[t] = acc;
}

template <class T, int D>
__global__ __launch_bounds__(256) void k_item_attn_dq(Geo g, const T* __restrict__ q,
                                                      const T* __restrict__ k,
                                                      const T* __restrict__ v,
                                                      const T* __restrict__ dout,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ Dv,
                                                      T* __restrict__ dq) {
  int64_t t = gtid();
  if (t >= (int64_t)g.NC * g.heads * g.R) return;
  const int r = (int)(t % g.R);
  const int64_t ch = t / g.R;
  const int head = (int)(ch % g.heads);
  const int64_t col = ch / g.heads;
  const int n = g.col_ntr[col];
  const float tau = 1.0f / sqrtf((float)D);
  const int64_t base = ch * g.R;
  float qv[D], dov[D], acc[D];
  const int64_t p = (col * g.R + r) * g.E + head * D;
#pragma unroll
  for (int j = 0; j < D; ++j) {
    qv[j] = ld(q + (base + r) * D + j) * tau;
    dov[j] = ld(dout + p + j);
    acc[j] = 0.f;
  }
  const float L = lse[base + r], Dr = Dv[t];
  for (int tt = 0; tt < n; ++tt) {
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      s = fmaf(qv[j], ld(k + (base + tt) * D + j), s);
      dp = fmaf(dov[j], ld(v + (base + tt) * D + j), dp);
    }
    float ds = expf(s - L) * (dp - Dr) * tau;
#pragma unroll
    for (int j = 0; j < D; ++j) acc[j] = fmaf(ds, ld(k + (base + tt) * D + j), acc[j]);
  }
#pragma unroll
  for (int j = 0; j < D; ++j) st(dq + (base + r) * D + j, acc[j]);
}

template <class T, int D>
__global__ __launch_bounds__(256) void k_item_attn_dkv(Geo g, const T* __restrict__ q,
                                                       const T* __restrict__ k,
                                                       const T* __restrict__ v,
                                                       const T* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       const float* __restrict__ Dv,
                                                       T* __restrict__ dk,
                                                       T* __restrict__ dv) {
  int64_t t = gtid();
  if (t >= (int64_t)g.NC * g.heads * g.R) return;
  const int tk = (int)(t % g.R);
  const int64_t ch = t / g.R;
  const int head = (int)(ch % g.heads);
  const int64_t col = ch / g.heads;
  const int n = g.col_ntr[col];
  if (tk >= n) return;
  const float tau = 1.0f / sqrtf((float)D);
  const int64_t base = ch * g.R;
  float kv[D], vv[D], ak[D], av[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    kv[j] = ld(k + (base + tk) * D + j) * tau;
    vv[j] = ld(v + (base + tk) * D + j);
    ak[j] = av[j] = 0.f;
  }
  for (int r = 0; r < g.R; ++r) {
    const T* qr = q + (base + r) * D;
    const T* dor = dout + (col * g.R + r) * g.E + head * D;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      s = fmaf(ld(qr + j), kv[j], s);
      dp = fmaf(ld(dor + j), vv[j], dp);
    }
    float p = expf(s - lse[base + r]);
    float ds = p * (dp - Dv[base + r]) * tau;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      ak[j] = fmaf(ds, ld(qr + j), ak[j]);
      av[j] = fmaf(p, ld(dor + j), av[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < D; ++j) {
    st(dk + (base + tk) * D + j, ak[j]);
    st(dv + (base + tk) * D + j, av[j]);
  }
}

template <class T>
hipError_t launch_item_attn_bwd_simple(const Geo& g, const T* q, const T* k, const T* v,
                                       const T* o, const T* dout, const float* lse, float* D,
                                       T* dq, T* dk, T* dv, hipStream_t s) {
  int64_t total = (int64_t)g.NC * g.heads * g.R;
  unsigned grid = grid_for(total);
  if (g.d == 16) {
    k_item_rowdot<T, 16><<<grid, TFM_BLOCK, 0, s>>>(g, o, dout, D);
    k_item_attn_dq<T, 16><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dq);
    k_item_attn_dkv<T, 16><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dk, dv);
  } else if (g.d == 32) {
    k_item_rowdot<T, 32><<<grid, TFM_BLOCK, 0, s>>>(g, o, dout, D);
    k_item_attn_dq<T, 32><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dq);
    k_item_attn_dkv<T, 32><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dk, dv);
  } else {
    k_item_rowdot<T, 64><<<grid, TFM_BLOCK, 0, s>>>(g, o, dout, D);
    k_item_attn_dq<T, 64><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dq);
    k_item_attn_dkv<T, 64><<<grid, TFM_BLOCK, 0, s>>>(g, q, k, v, dout, lse, D, dk, dv);
  }
  return hipGetLastError();
}

template <class T>
__global__ void k_item_dqkv_to_cells(Geo g, const T* __restrict__ dq, const T* __restrict__ dk,
                                     const T* __restrict__ dv, T* __restrict__ dqkv) {
  const int E3 = 3 * g.E;
  int64_t total = g.N * E3;
  for (int64_t i = gtid(); i < total; i += gstride()) {
    int64_t p = i / E3;
    int nn = (int)(i - p * E3);
    int part = nn / g.E, within = nn - part * g.E;
    int head = within / g.d, j = within - head * g.d;
    int64_t col = p / g.R;
    int r = (int)(p - col * g.R);
    const T* src = part == 0 ? dq : (part == 1 ? dk : dv);
    if (part > 0 && r >= g.col_ntr[col]) {
      st(dqkv + i, 0.f);
    } else {
      dqkv[i] = src[((col * g.heads + head) * g.R + r) * g.d + j];
    }
  }
}

template <class T>
hipError_t launch_item_dqkv_to_cells(const Geo& g, const T* dq, const T* dk, const T* dv,
                                     T* dqkv, hipStream_t s) {
  k_item_dqkv_to_cells<T><<<grid_for(g.N * 3 * g.E), TFM_BLOCK, 0, s>>>(g, dq, dk, dv, dqkv);
  return hipGetLastError();
}

// ============================================================================ instantiations
#define INST(T)                                                                               \
  template hipError_t launch_gather<T>(const Geo&, const T*, T*, hipStream_t);              \
  template hipError_t launch_scatter<T>(const Geo&, const T*, const T*, T*, hipStream_t);   \
  template hipError_t launch_linear<T, T>(int64_t, int, int, const T*, int64_t,             \
                                          const float*, int64_t, int64_t, const float*, T*,  \
                                          int64_t, hipStream_t);                             \
  template hipError_t launch_linear_item_qkv<T>(const Geo&, const T*, const float*,         \
                                                const float*, T*, T*, T*, hipStream_t);      \
  template hipError_t launch_wgrad<T>(int64_t, int, int, const T*, int64_t, const T*,        \
                                      int64_t, int64_t, float*, hipStream_t);                \
  template hipError_t launch_colsum<T>(int64_t, int, const T*, int64_t, const T*, int64_t,   \
                                       int64_t, float*, hipStream_t);                        \
  template hipError_t launch_add_ln<T>(int64_t, int, const T*, const T*, const float*,      \
                                       const float*, T*, T*, float*, hipStream_t);           \
  template hipError_t launch_ln_bwd<T>(int64_t, int, const T*, const T*, const T*,          \
                                       const float*, const float*, T*, T*, hipStream_t);     \
  template hipError_t launch_gelu<T>(int64_t, const T*, T*, hipStream_t);                   \
  template hipError_t launch_gelu_bwd<T>(int64_t, const T*, T*, hipStream_t);               \
  template hipError_t launch_feat_attn_fwd_simple<T>(const Geo&, const T*, T*, float*,      \
                                                     hipStream_t);                           \
  template hipError_t launch_feat_attn_bwd_simple<T>(const Geo&, const T*, const T*,        \
                                                     const T*, const float*, T*,             \
                                                     hipStream_t);                           \
  template hipError_t launch_item_attn_fwd_simple<T>(const Geo&, const T*, const T*,        \
                                                     const T*, T*, float*, hipStream_t);     \
  template hipError_t launch_item_attn_bwd_simple<T>(const Geo&, const T*, const T*,        \
                                                     const T*, const T*, const T*,           \
                                                     const float*, float*, T*, T*, T*,       \
                                                     hipStream_t);                           \
  template hipError_t launch_item_dqkv_to_cells<T>(const Geo&, const T*, const T*,          \
                                                   const T*, T*, hipStream_t);

INST(float)
INST(bf16)

}  // namespace tfm
