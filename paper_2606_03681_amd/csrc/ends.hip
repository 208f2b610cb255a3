// Kernels of the two ends of the stack (declarations and layout in ends.h).
//
// Encoder forward: one workgroup per ENC_ROWS data rows of one dataset; it stages the rows'
// feature values and the encoder weights in LDS and writes whole rows of the stack input with
// 16-byte stores (feature cells, zero padding cells, the target cell).  HBM-write bound.
// Encoder backward: the same row slabs; each thread owns one 8-wide slice of E and a lane of
// cells, accumulates the weight and bias gradients in registers, and the workgroup folds its
// lanes in a fixed order into one partial row (summed over slabs in a fixed order afterwards).
// HBM-read bound.
// Decoder: gather of the decoder input, float32 GEMMs on the MFMA with bias/GELU epilogues, a
// masked softmax cross entropy per row, and a scatter that writes the whole dY.
#include "ends.h"

#include <hip/hip_runtime.h>

namespace tfm {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void ld8(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void ld8(const bf16* p, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void st8(float* p, const float* v) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void st8(bf16* p, const float* v) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f2bf(v[2 * i]) | ((uint32_t)f2bf(v[2 * i + 1]) << 16);
  *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}

// Dataset of decoder row t: the last dataset whose first decoder row is <= t (datasets without
// test rows share their successor's first row and are skipped that way).
__device__ __forceinline__ int dataset_of(const EndsGeo& g, int64_t t) {
  int lo = 0, hi = g.B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (g.ds[mid].test0 <= t) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Mean of the labelled data rows' labels: an integer sum (exact, so independent of the order),
// one division.  Contains barriers: every thread of the block calls it.
__device__ float train_label_mean(const int32_t* lab, int ntr, int64_t* red) {
  int64_t sum = 0;
  for (int i = threadIdx.x; i < ntr; i += blockDim.x) sum += lab[i];
  red[threadIdx.x] = sum;
  __syncthreads();
  for (int w = blockDim.x >> 1; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const float mean = (float)((double)red[0] / (double)ntr);
  __syncthreads();
  return mean;
}

// Shifts of the groups reduced mod m, so that column (c + o) mod m = c + om, minus m on wrap.
__device__ __forceinline__ void shifts_mod(const EndsGeo& g, int m, int* om) {
#pragma unroll
  for (int k = 0; k < ENDS_GMAX; ++k) om[k] = k < g.G ? g.off[k] % m : 0;
}

// Stages the feature values of rows [i0, i0 + nrow) of dataset b (columns [0, m)).
__device__ __forceinline__ void stage_rows(const EndsGeo& g, const float* x, int b, int i0,
                                           int nrow, int m, float (*sx)[256]) {
  const int Rd = g.R - g.T;
  for (int i = threadIdx.x; i < nrow * m; i += blockDim.x) {
    const int rr = i / m, c = i - rr * m;
    sx[rr][c] = x[((int64_t)b * Rd + i0 + rr) * g.F + c];
  }
}

// ---- encoder ----------------------------------------------------------------------------------
template <class T>
__global__ __launch_bounds__(256) void k_encode_fwd(EndsGeo g, const float* __restrict__ x,
                                                    const int32_t* __restrict__ lab,
                                                    const float* __restrict__ prm,
                                                    T* __restrict__ X) {
  __shared__ float sW[256 * ENDS_GMAX];
  __shared__ float sb[256], stw[256], stb[256];
  __shared__ float sx[ENC_ROWS][256];
  __shared__ int64_t red[256];
  const int b = blockIdx.y;
  const EndsDs md = g.ds[b];
  const int E = g.E, G = g.G, m = md.n_feat, C = g.S - 1;
  const int Rd = g.R - g.T, ntr = md.n_train - g.T;
  const int i0 = blockIdx.x * ENC_ROWS;
  const int nrow = Rd - i0 < ENC_ROWS ? Rd - i0 : ENC_ROWS;
  for (int i = threadIdx.x; i < E * G; i += 256) sW[i] = prm[i];
  for (int i = threadIdx.x; i < E; i += 256) {
    sb[i] = prm[E * G + i];
    stw[i] = prm[E * G + E + i];
    stb[i] = prm[E * G + 2 * E + i];
  }
  stage_rows(g, x, b, i0, nrow, m, sx);
  const float mean = train_label_mean(lab + (int64_t)b * Rd, ntr, red);  // barriers inside
  int om[ENDS_GMAX];
  shifts_mod(g, m, om);
  const int nch = E >> 3, nvec = g.S * nch;
  for (int rr = 0; rr < nrow; ++rr) {
    const int i = i0 + rr;
    const float tval = i < ntr ? (float)lab[(int64_t)b * Rd + i] : mean;
    T* row = X + ((int64_t)b * g.R + g.T + i) * g.S * E;
    for (int v = threadIdx.x; v < nvec; v += 256) {
      const int c = v / nch, e0 = (v - c * nch) << 3;
      float o[8];
      if (c < m) {
        float xg[ENDS_GMAX];
#pragma unroll
        for (int k = 0; k < ENDS_GMAX; ++k) {
          int j = c + om[k];
          j = j >= m ? j - m : j;
          xg[k] = k < G ? sx[rr][j] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          float a = sb[e0 + q];
#pragma unroll
          for (int k = 0; k < ENDS_GMAX; ++k)
            if (k < G) a = fmaf(sW[(e0 + q) * G + k], xg[k], a);
          o[q] = a;
        }
      } else if (c == C) {
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = fmaf(tval, stw[e0 + q], stb[e0 + q]);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = 0.f;
      }
      st8(row + (int64_t)c * E + e0, o);
    }
  }
}

// Folds one 8-wide register slice per (lane, slice) over the lanes in a fixed order and writes
// out[e * os] for e in [0, E).  Contains barriers: every thread of the block calls it.
__device__ __forceinline__ void fold_lanes(const float* v, bool act, int lane, int ch, int L,
                                           int E, float* sred, float* out, int os) {
  if (act) {
#pragma unroll
    for (int q = 0; q < 8; ++q) sred[lane * E + ch * 8 + q] = v[q];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 256) {
    float s = 0.f;
    for (int l = 0; l < L; ++l) s += sred[l * E + e];
    out[(int64_t)e * os] = s;
  }
  __syncthreads();
}

template <class T>
__global__ __launch_bounds__(256) void k_encode_bwd(EndsGeo g, const float* __restrict__ x,
                                                    const int32_t* __restrict__ lab,
                                                    const T* __restrict__ dX,
                                                    float* __restrict__ part) {
  __shared__ float sx[ENC_ROWS][256];
  __shared__ float sred[2048];
  __shared__ int64_t red[256];
  const int b = blockIdx.y;
  const EndsDs md = g.ds[b];
  const int E = g.E, G = g.G, m = md.n_feat, C = g.S - 1;
  const int Rd = g.R - g.T, ntr = md.n_train - g.T;
  const int i0 = blockIdx.x * ENC_ROWS;
  const int nrow = Rd - i0 < ENC_ROWS ? Rd - i0 : ENC_ROWS;
  stage_rows(g, x, b, i0, nrow, m, sx);
  const float mean = train_label_mean(lab + (int64_t)b * Rd, ntr, red);  // barriers inside
  int om[ENDS_GMAX];
  shifts_mod(g, m, om);
  const int nch = E >> 3, L = 256 / nch;
  const int ch = threadIdx.x % nch, lane = threadIdx.x / nch;
  const bool act = lane < L;
  float aw[8][ENDS_GMAX], ab[8], atw[8], atb[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    ab[q] = atw[q] = atb[q] = 0.f;
#pragma unroll
    for (int k = 0; k < ENDS_GMAX; ++k) aw[q][k] = 0.f;
  }
  if (act) {
    for (int rr = 0; rr < nrow; ++rr) {
      const int i = i0 + rr;
      const T* row = dX + ((int64_t)b * g.R + g.T + i) * g.S * E + ch * 8;
      for (int c = lane; c < m; c += L) {
        float d[8], xg[ENDS_GMAX];
        ld8(row + (int64_t)c * E, d);
#pragma unroll
        for (int k = 0; k < ENDS_GMAX; ++k) {
          int j = c + om[k];
          j = j >= m ? j - m : j;
          xg[k] = k < G ? sx[rr][j] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          ab[q] += d[q];
#pragma unroll
          for (int k = 0; k < ENDS_GMAX; ++k) aw[q][k] = fmaf(d[q], xg[k], aw[q][k]);
        }
      }
      if (lane == 0) {
        const float tval = i < ntr ? (float)lab[(int64_t)b * Rd + i] : mean;
        float d[8];
        ld8(row + (int64_t)C * E, d);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          atb[q] += d[q];
          atw[q] = fmaf(d[q], tval, atw[q]);
        }
      }
    }
  }
  float* out = part + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * ((int64_t)E * (G + 3));
#pragma unroll
  for (int k = 0; k < ENDS_GMAX; ++k) {
    if (k < G) {  // uniform over the block
      float v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = aw[q][k];
      fold_lanes(v, act, lane, ch, L, E, sred, out + k, G);
    }
  }
  fold_lanes(ab, act, lane, ch, L, E, sred, out + (int64_t)E * G, 1);
  fold_lanes(atw, act, lane, ch, L, E, sred, out + (int64_t)E * (G + 1), 1);
  fold_lanes(atb, act, lane, ch, L, E, sred, out + (int64_t)E * (G + 2), 1);
}

// ---- decoder ----------------------------------------------------------------------------------
// One wave per decoder row.
template <class T>
__global__ __launch_bounds__(256) void k_decode_gather(EndsGeo g, const T* __restrict__ Y,
                                                       float* __restrict__ Z) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= g.Ttot) return;
  const int lane = threadIdx.x & 63;
  const int b = dataset_of(g, t);
  const EndsDs md = g.ds[b];
  const int r = md.n_train + (int)(t - md.test0);
  const T* row = Y + ((int64_t)b * g.R + r) * g.S * g.E;
  for (int e = lane; e < g.E; e += 64) {
    float v;
    if (g.mean) {
      float s = 0.f;
      for (int c = 0; c < md.n_feat; ++c) s += ld(row + (int64_t)c * g.E + e);
      v = s / (float)md.n_feat;
    } else {
      v = ld(row + (int64_t)(g.S - 1) * g.E + e);
    }
    Z[t * g.E + e] = v;
  }
}

// One workgroup per row (b, r) of dY.
template <class T>
__global__ __launch_bounds__(256) void k_decode_scatter(EndsGeo g, const float* __restrict__ dZ,
                                                        T* __restrict__ dY) {
  const int b = blockIdx.y, r = blockIdx.x;
  const EndsDs md = g.ds[b];
  const int E = g.E, C = g.S - 1, m = md.n_feat;
  T* row = dY + ((int64_t)b * g.R + r) * g.S * E;
  const bool test = r >= md.n_train;
  const float* z = dZ + (test ? (int64_t)(md.test0 + r - md.n_train) * E : 0);
  const int nch = E >> 3, nvec = g.S * nch;
  for (int v = threadIdx.x; v < nvec; v += 256) {
    const int c = v / nch, e0 = (v - c * nch) << 3;
    float o[8];
    const bool hit = test && (g.mean ? c < m : c == C);
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = 0.f;
    if (hit) {
#pragma unroll
      for (int q = 0; q < 8; ++q) o[q] = g.mean ? z[e0 + q] / (float)m : z[e0 + q];
    }
    st8(row + (int64_t)c * E + e0, o);
  }
}

__global__ __launch_bounds__(256) void k_cross_entropy(EndsGeo g, const float* __restrict__ lg,
                                                       const int32_t* __restrict__ lab,
                                                       float* __restrict__ lrow,
                                                       float* __restrict__ dlog) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= g.Ttot) return;
  const int b = dataset_of(g, t);
  const EndsDs md = g.ds[b];
  const int nc = md.n_class, K = g.K;
  const int r = md.n_train + (int)(t - md.test0);
  const int y = lab[(int64_t)b * (g.R - g.T) + (r - g.T)];
  const float* z = lg + t * K;
  float mx = -INFINITY;
  for (int k = 0; k < nc; ++k) mx = fmaxf(mx, z[k]);
  float se = 0.f;
  for (int k = 0; k < nc; ++k) se += expf(z[k] - mx);
  const float lse = mx + logf(se);
  const float zy = (y >= 0 && y < nc) ? z[y] : 0.f;
  const float invT = 1.0f / (float)g.Ttot;
  lrow[t] = (lse - zy) * invT;
  const float rse = 1.0f / se;
  for (int k = 0; k < K; ++k) {
    float d = 0.f;
    if (k < nc) d = (expf(z[k] - mx) * rse - (k == y ? 1.f : 0.f)) * invT;
    dlog[t * K + k] = d;
  }
}

// ---- float32 GEMM on the MFMA ---------------------------------------------------------------
// 64 x 64 output tile per workgroup, four waves of 32 x 32 (2 x 2 blocks of
// v_mfma_f32_16x16x4f32), K staged through LDS 16 at a time with zero fill past the edges.
// Operand lanes: A[i][k] from lane i + 16 k, B[k][j] from lane j + 16 k; result D[i][j] in
// lane j + 16 (i / 4), element i % 4.
__device__ __forceinline__ float gelu_exact(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_exact_grad(float v) {
  const float cdf = 0.5f * (1.0f + erff(v * 0.70710678118654752f));
  return cdf + v * 0.39894228040143268f * expf(-0.5f * v * v);
}

template <bool TA, bool TB, int EPI>
__global__ __launch_bounds__(256) void k_sgemm(SgemmArgs a) {
  __shared__ float As[16][68];
  __shared__ float Bs[16][68];
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  const int kb = a.kchunk ? (int)blockIdx.z * a.kchunk : 0;
  const int ke = a.kchunk ? (kb + a.kchunk < a.K ? kb + a.kchunk : a.K) : a.K;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int wm = (w >> 1) * 32, wn = (w & 1) * 32;
  v4f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int k0 = kb; k0 < ke; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + 256 * q;
      int mm, kk;
      if (TA) { mm = idx & 63; kk = idx >> 6; }
      else { kk = idx & 15; mm = idx >> 4; }
      int gm = m0 + mm, gk = k0 + kk;
      float v = 0.f;
      if (gm < a.M && gk < ke)
        v = TA ? a.A[(int64_t)gk * a.lda + gm] : a.A[(int64_t)gm * a.lda + gk];
      As[kk][mm] = v;
      int nn;
      if (TB) { kk = idx & 15; nn = idx >> 4; }
      else { nn = idx & 63; kk = idx >> 6; }
      const int gn = n0 + nn;
      gk = k0 + kk;
      float u = 0.f;
      if (gn < a.N && gk < ke)
        u = TB ? a.B[(int64_t)gn * a.ldb + gk] : a.B[(int64_t)gk * a.ldb + gn];
      Bs[kk][nn] = u;
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kr = ks * 4 + (l >> 4);
      float av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) av[i] = As[kr][wm + i * 16 + (l & 15)];
#pragma unroll
      for (int j = 0; j < 2; ++j) bv[j] = Bs[kr][wn + j * 16 + (l & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  float* C = a.C + (int64_t)blockIdx.z * a.zstride;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = m0 + wm + i * 16 + 4 * (l >> 4) + q;
        const int col = n0 + wn + j * 16 + (l & 15);
        if (row < a.M && col < a.N) {
          const int64_t o = (int64_t)row * a.ldc + col;
          float v = acc[i][j][q];
          if (EPI == SG_GELU_GRAD) {
            C[o] = v * gelu_exact_grad(a.aux[o]);
          } else {
            if (a.bias) v += a.bias[col];
            C[o] = v;
            if (EPI == SG_GELU) a.C2[o] = gelu_exact(v);
          }
        }
      }
}

__global__ __launch_bounds__(256) void k_fill(float* __restrict__ p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = v;
}

}  // namespace

// ---- launchers --------------------------------------------------------------------------------
template <class T>
hipError_t launch_encode_fwd(const EndsGeo& g, const float* x, const int32_t* lab,
                             const float* prm, T* X, hipStream_t s) {
  const int Rd = g.R - g.T;
  dim3 grid((unsigned)((Rd + ENC_ROWS - 1) / ENC_ROWS), (unsigned)g.B);
  k_encode_fwd<T><<<grid, 256, 0, s>>>(g, x, lab, prm, X);
  return hipGetLastError();
}

int64_t encode_bwd_parts(const EndsGeo& g) {
  const int Rd = g.R - g.T;
  return (int64_t)g.B * ((Rd + ENC_ROWS - 1) / ENC_ROWS);
}

template <class T>
hipError_t launch_encode_bwd(const EndsGeo& g, const float* x, const int32_t* lab, const T* dX,
                             float* part, hipStream_t s) {
  const int Rd = g.R - g.T;
  dim3 grid((unsigned)((Rd + ENC_ROWS - 1) / ENC_ROWS), (unsigned)g.B);
  k_encode_bwd<T><<<grid, 256, 0, s>>>(g, x, lab, dX, part);
  return hipGetLastError();
}

template <class T>
hipError_t launch_decode_gather(const EndsGeo& g, const T* Y, float* Z, hipStream_t s) {
  if (g.Ttot == 0) return hipSuccess;
  k_decode_gather<T><<<(unsigned)((g.Ttot + 3) / 4), 256, 0, s>>>(g, Y, Z);
  return hipGetLastError();
}

template <class T>
hipError_t launch_decode_scatter(const EndsGeo& g, const float* dZ, T* dY, hipStream_t s) {
  k_decode_scatter<T><<<dim3((unsigned)g.R, (unsigned)g.B), 256, 0, s>>>(g, dZ, dY);
  return hipGetLastError();
}

hipError_t launch_cross_entropy(const EndsGeo& g, const float* logits, const int32_t* lab,
                                float* lrow, float* dlog, hipStream_t s) {
  if (g.Ttot == 0) return hipSuccess;
  k_cross_entropy<<<(unsigned)((g.Ttot + 255) / 256), 256, 0, s>>>(g, logits, lab, lrow, dlog);
  return hipGetLastError();
}

hipError_t launch_sgemm(const SgemmArgs& a, bool ta, bool tb, int epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  const unsigned nz = a.kchunk ? (unsigned)((a.K + a.kchunk - 1) / a.kchunk) : 1u;
  dim3 grid((unsigned)((a.M + 63) / 64), (unsigned)((a.N + 63) / 64), nz ? nz : 1u);
  if (!ta && tb && epi == SG_GELU) k_sgemm<false, true, SG_GELU><<<grid, 256, 0, s>>>(a);
  else if (!ta && tb && epi == SG_BIAS) k_sgemm<false, true, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else if (!ta && !tb && epi == SG_GELU_GRAD)
    k_sgemm<false, false, SG_GELU_GRAD><<<grid, 256, 0, s>>>(a);
  else if (!ta && !tb && epi == SG_BIAS) k_sgemm<false, false, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else if (ta && !tb && epi == SG_BIAS) k_sgemm<true, false, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  k_fill<<<(unsigned)(blocks < 4096 ? blocks : 4096), 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

#define TFM_ENDS_INST(T)                                                                      \
  template hipError_t launch_encode_fwd<T>(const EndsGeo&, const float*, const int32_t*,      \
                                           const float*, T*, hipStream_t);                    \
  template hipError_t launch_encode_bwd<T>(const EndsGeo&, const float*, const int32_t*,      \
                                           const T*, float*, hipStream_t);                    \
  template hipError_t launch_decode_gather<T>(const EndsGeo&, const T*, float*, hipStream_t); \
  template hipError_t launch_decode_scatter<T>(const EndsGeo&, const float*, T*, hipStream_t);
TFM_ENDS_INST(float)
TFM_ENDS_INST(bf16)
#undef TFM_ENDS_INST

}  // namespace tfm
