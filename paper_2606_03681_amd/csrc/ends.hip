// Kernels of the two ends of the stack (declarations and layout in ends.h).
//
// Encoder forward: one workgroup per ENC_ROWS data rows of one dataset; it stages the rows'
// feature values in LDS, keeps each thread's 8-wide slice of the encoder weights in registers
// and writes whole rows of the stack input with 16-byte stores (feature cells, zero padding
// cells, the target cell).  HBM-write bound.
// Encoder backward: the same row slabs and slices; each thread accumulates its slice of the
// weight and bias gradients in registers over a lane of cells, and the workgroup folds its lanes
// in a fixed order into one partial row (summed over slabs in a fixed order afterwards).
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
template <int G>
__device__ __forceinline__ void shifts_mod(const EndsGeo& g, int m, int* om) {
#pragma unroll
  for (int k = 0; k < G; ++k) om[k] = g.off[k] % m;
}

// Stages the feature values (columns [0, m)) of the workgroup's rows i0 + rr * rs, rr < nrow,
// of dataset b.
__device__ __forceinline__ void stage_rows(const EndsGeo& g, const float* x, int b, int i0,
                                           int rs, int nrow, int m, float (*sx)[256]) {
  const int Rd = g.R - g.T;
  for (int i = threadIdx.x; i < nrow * m; i += blockDim.x) {
    const int rr = i / m, c = i - rr * m;
    sx[rr][c] = x[((int64_t)b * Rd + i0 + rr * rs) * g.F + c];
  }
}

// Rows of an encoder workgroup: workgroup j of a dataset takes the data rows j, j + rs, ...
// (rs = workgroups per dataset, at most ENC_ROWS rows), so that the workgroups running at one
// time stream through neighbouring rows of HBM instead of a thousand separate regions.
__device__ __forceinline__ int slab_rows(int Rd, int i0, int rs) {
  const int n = (Rd - i0 + rs - 1) / rs;
  return n < ENC_ROWS ? n : ENC_ROWS;
}

// ---- encoder ----------------------------------------------------------------------------------
// Thread layout of both encoder kernels: thread t owns the 8-wide slice ch = t % (E/8) of the
// embedding and serves cell lane t / (E/8); the L = 256 / (E/8) lanes of a workgroup walk the
// (row, cell) pairs of its slab, so that a wave touches consecutive 16-byte pieces of whole cells.
struct Lanes {
  int nch, L, ch, lane;
  bool act;
};
__device__ __forceinline__ Lanes lanes_of(int E) {
  Lanes l;
  l.nch = E >> 3;
  l.L = 256 / l.nch;
  l.ch = threadIdx.x % l.nch;
  l.lane = threadIdx.x / l.nch;
  l.act = l.lane < l.L;
  return l;
}

template <class T, int G>
__global__ __launch_bounds__(256) void k_encode_fwd(EndsGeo g, const float* __restrict__ x,
                                                    const int32_t* __restrict__ lab,
                                                    const float* __restrict__ prm,
                                                    T* __restrict__ X) {
  __shared__ float sx[ENC_ROWS][256];
  __shared__ float stv[ENC_ROWS];
  __shared__ int64_t red[256];
  const int b = blockIdx.y;
  const EndsDs md = g.ds[b];
  const int E = g.E, m = md.n_feat, C = g.S - 1, S = g.S;
  const int Rd = g.R - g.T, ntr = md.n_train - g.T;
  const int i0 = blockIdx.x, rs = gridDim.x;
  const int nrow = slab_rows(Rd, i0, rs);
  const Lanes ln = lanes_of(E);
  // this thread's slice of the encoder weights, in registers
  const int e0 = ln.ch * 8;
  float w[8][G], bf[8], tw[8], tb[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
#pragma unroll
    for (int k = 0; k < G; ++k) w[q][k] = prm[(e0 + q) * G + k];
    bf[q] = prm[E * G + e0 + q];
    tw[q] = prm[E * G + E + e0 + q];
    tb[q] = prm[E * G + 2 * E + e0 + q];
  }
  stage_rows(g, x, b, i0, rs, nrow, m, sx);
  const float mean = train_label_mean(lab + (int64_t)b * Rd, ntr, red);  // barriers inside
  if (threadIdx.x < nrow) {
    const int i = i0 + threadIdx.x * rs;
    stv[threadIdx.x] = i < ntr ? (float)lab[(int64_t)b * Rd + i] : mean;
  }
  __syncthreads();
  if (!ln.act) return;
  int om[G];
  shifts_mod<G>(g, m, om);
  T* base = X + ((int64_t)b * g.R + g.T + i0) * S * E + e0;
  const int64_t rstep = (int64_t)rs * S * E;
  const int tot = nrow * S;
  for (int p = ln.lane; p < tot; p += ln.L) {
    const int rr = p / S, c = p - rr * S;
    float o[8];
    if (c < m) {
      float xg[G];
#pragma unroll
      for (int k = 0; k < G; ++k) {
        int j = c + om[k];
        j = j >= m ? j - m : j;
        xg[k] = sx[rr][j];
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float a = bf[q];
#pragma unroll
        for (int k = 0; k < G; ++k) a = fmaf(w[q][k], xg[k], a);
        o[q] = a;
      }
    } else if (c == C) {
      const float tv = stv[rr];
#pragma unroll
      for (int q = 0; q < 8; ++q) o[q] = fmaf(tv, tw[q], tb[q]);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) o[q] = 0.f;
    }
    st8(base + rr * rstep + (int64_t)c * E, o);
  }
}

// Folds one 8-wide register slice per (lane, slice) over the lanes in a fixed order and writes
// out[e * os] for e in [0, E).  Contains barriers: every thread of the block calls it.
__device__ __forceinline__ void fold_lanes(const float* v, const Lanes& ln, int E, float* sred,
                                           float* out, int os) {
  if (ln.act) {
#pragma unroll
    for (int q = 0; q < 8; ++q) sred[ln.lane * E + ln.ch * 8 + q] = v[q];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += 256) {
    float s = 0.f;
    for (int l = 0; l < ln.L; ++l) s += sred[l * E + e];
    out[(int64_t)e * os] = s;
  }
  __syncthreads();
}

// Feature cells per unrolled step of the encoder backward: their loads are issued together.
constexpr int ENC_BWD_UNROLL = 4;

template <class T, int G>
__global__ __launch_bounds__(256) void k_encode_bwd(EndsGeo g, const float* __restrict__ x,
                                                    const int32_t* __restrict__ lab,
                                                    const T* __restrict__ dX,
                                                    float* __restrict__ part) {
  __shared__ float sx[ENC_ROWS][256];
  __shared__ float stv[ENC_ROWS];
  __shared__ float sred[2048];
  __shared__ int64_t red[256];
  const int b = blockIdx.y;
  const EndsDs md = g.ds[b];
  const int E = g.E, m = md.n_feat, C = g.S - 1, S = g.S;
  const int Rd = g.R - g.T, ntr = md.n_train - g.T;
  const int i0 = blockIdx.x, rs = gridDim.x;
  const int nrow = slab_rows(Rd, i0, rs);
  const Lanes ln = lanes_of(E);
  stage_rows(g, x, b, i0, rs, nrow, m, sx);
  const float mean = train_label_mean(lab + (int64_t)b * Rd, ntr, red);  // barriers inside
  if (threadIdx.x < nrow) {
    const int i = i0 + threadIdx.x * rs;
    stv[threadIdx.x] = i < ntr ? (float)lab[(int64_t)b * Rd + i] : mean;
  }
  __syncthreads();
  int om[G];
  shifts_mod<G>(g, m, om);
  float aw[8][G], ab[8], atw[8], atb[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    ab[q] = atw[q] = atb[q] = 0.f;
#pragma unroll
    for (int k = 0; k < G; ++k) aw[q][k] = 0.f;
  }
  const T* base = dX + ((int64_t)b * g.R + g.T + i0) * S * E + ln.ch * 8;
  const int64_t rstep = (int64_t)rs * S * E;
  if (ln.act) {
    // feature cells: (row, cell) pairs of the slab, ENC_BWD_UNROLL loads in flight per lane;
    // a pair past the end reloads the first pair of the step and is not accumulated
    const int tot = nrow * m;
    for (int p0 = ln.lane; p0 < tot; p0 += ENC_BWD_UNROLL * ln.L) {
      float d[ENC_BWD_UNROLL][8];
      int rrs[ENC_BWD_UNROLL], cs[ENC_BWD_UNROLL];
#pragma unroll
      for (int u = 0; u < ENC_BWD_UNROLL; ++u) {
        const int p = p0 + u * ln.L < tot ? p0 + u * ln.L : p0;
        rrs[u] = p / m;
        cs[u] = p - rrs[u] * m;
        ld8(base + rrs[u] * rstep + (int64_t)cs[u] * E, d[u]);
      }
#pragma unroll
      for (int u = 0; u < ENC_BWD_UNROLL; ++u) {
        if (p0 + u * ln.L < tot) {
          float xg[G];
#pragma unroll
          for (int k = 0; k < G; ++k) {
            int j = cs[u] + om[k];
            j = j >= m ? j - m : j;
            xg[k] = sx[rrs[u]][j];
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            ab[q] += d[u][q];
#pragma unroll
            for (int k = 0; k < G; ++k) aw[q][k] = fmaf(d[u][q], xg[k], aw[q][k]);
          }
        }
      }
    }
    // target cells, one row per lane
    for (int rr = ln.lane; rr < nrow; rr += ln.L) {
      float d[8];
      ld8(base + rr * rstep + (int64_t)C * E, d);
      const float tv = stv[rr];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        atb[q] += d[q];
        atw[q] = fmaf(d[q], tv, atw[q]);
      }
    }
  }
  float* out = part + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * ((int64_t)E * (G + 3));
#pragma unroll
  for (int k = 0; k < G; ++k) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = aw[q][k];
    fold_lanes(v, ln, E, sred, out + k, G);
  }
  fold_lanes(ab, ln, E, sred, out + (int64_t)E * G, 1);
  fold_lanes(atw, ln, E, sred, out + (int64_t)E * (G + 1), 1);
  fold_lanes(atb, ln, E, sred, out + (int64_t)E * (G + 2), 1);
}

// ---- decoder ----------------------------------------------------------------------------------
// Decoder input: each thread reads one 8-wide slice of E of one decoder row (the lanes of a
// workgroup take consecutive rows), summing the feature cells in ascending order for the mean.
template <class T>
__global__ __launch_bounds__(256) void k_decode_gather(EndsGeo g, const T* __restrict__ Y,
                                                       float* __restrict__ Z) {
  const Lanes ln = lanes_of(g.E);
  const int64_t t = (int64_t)blockIdx.x * ln.L + ln.lane;
  if (!ln.act || t >= g.Ttot) return;
  const int b = dataset_of(g, t);
  const EndsDs md = g.ds[b];
  const int E = g.E, m = md.n_feat;
  const int r = md.n_train + (int)(t - md.test0);
  const T* row = Y + ((int64_t)b * g.R + r) * g.S * E + ln.ch * 8;
  float v[8];
  if (g.mean) {
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = 0.f;
    int c = 0;
    for (; c + 4 <= m; c += 4) {
      float d[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) ld8(row + (int64_t)(c + u) * E, d[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] += d[u][q];
    }
    for (; c < m; ++c) {
      float d[8];
      ld8(row + (int64_t)c * E, d);
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] += d[q];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = v[q] / (float)m;
  } else {
    ld8(row + (int64_t)(g.S - 1) * E, v);
  }
  st8(Z + t * E + ln.ch * 8, v);
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
  // batch entry (kchunk == 0; the strides are 0 for a single product) or K chunk
  a.A += (int64_t)blockIdx.z * a.bsa;
  a.B += (int64_t)blockIdx.z * a.bsb;
  if (a.aux) a.aux += (int64_t)blockIdx.z * a.bsaux;
  const int kb = a.kchunk ? (int)blockIdx.z * a.kchunk : 0;
  const int ke = a.kchunk ? (kb + a.kchunk < a.K ? kb + a.kchunk : a.K) : a.K;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int wm = (w >> 1) * 32, wn = (w & 1) * 32;
  v4f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  // staging coordinates of this thread's four A and four B elements of a K step
  int a_mm[4], a_kk[4], b_nn[4], b_kk[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + 256 * q;
    if (TA) { a_mm[q] = idx & 63; a_kk[q] = idx >> 6; }
    else { a_kk[q] = idx & 15; a_mm[q] = idx >> 4; }
    if (TB) { b_kk[q] = idx & 15; b_nn[q] = idx >> 4; }
    else { b_nn[q] = idx & 63; b_kk[q] = idx >> 6; }
  }
  // the next K step's elements are loaded into registers while the current one is multiplied;
  // every load reads a valid element (out-of-range ones read element 0 and are zeroed)
  float ra[4], rb[4];
  auto gload = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gm = m0 + a_mm[q], gk = k0 + a_kk[q];
      const bool oka = gm < a.M && gk < ke;
      const int64_t oa = TA ? (int64_t)gk * a.lda + gm : (int64_t)gm * a.lda + gk;
      const float va = a.A[oka ? oa : 0];
      ra[q] = oka ? va : 0.f;
      const int gn = n0 + b_nn[q], gkb = k0 + b_kk[q];
      const bool okb = gn < a.N && gkb < ke;
      const int64_t ob = TB ? (int64_t)gn * a.ldb + gkb : (int64_t)gkb * a.ldb + gn;
      const float vb = a.B[okb ? ob : 0];
      rb[q] = okb ? vb : 0.f;
    }
  };
  if (kb < ke) gload(kb);
  for (int k0 = kb; k0 < ke; k0 += 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      As[a_kk[q]][a_mm[q]] = ra[q];
      Bs[b_kk[q]][b_nn[q]] = rb[q];
    }
    __syncthreads();
    if (k0 + 16 < ke) gload(k0 + 16);
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
          } else if (EPI == SG_AXPBY) {
            C[o] = fmaf(a.alpha, v, a.beta * a.aux[o]);
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
  switch (g.G) {
#define TFM_ENC_G(G_) \
  case G_: k_encode_fwd<T, G_><<<grid, 256, 0, s>>>(g, x, lab, prm, X); break;
    TFM_ENC_G(1) TFM_ENC_G(2) TFM_ENC_G(3) TFM_ENC_G(4)
    TFM_ENC_G(5) TFM_ENC_G(6) TFM_ENC_G(7) TFM_ENC_G(8)
#undef TFM_ENC_G
    default: return hipErrorInvalidValue;
  }
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
  switch (g.G) {
#define TFM_ENC_G(G_) \
  case G_: k_encode_bwd<T, G_><<<grid, 256, 0, s>>>(g, x, lab, dX, part); break;
    TFM_ENC_G(1) TFM_ENC_G(2) TFM_ENC_G(3) TFM_ENC_G(4)
    TFM_ENC_G(5) TFM_ENC_G(6) TFM_ENC_G(7) TFM_ENC_G(8)
#undef TFM_ENC_G
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class T>
hipError_t launch_decode_gather(const EndsGeo& g, const T* Y, float* Z, hipStream_t s) {
  if (g.Ttot == 0) return hipSuccess;
  const int L = 256 / (g.E >> 3);
  k_decode_gather<T><<<(unsigned)((g.Ttot + L - 1) / L), 256, 0, s>>>(g, Y, Z);
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
  const unsigned nz = a.kchunk ? (unsigned)((a.K + a.kchunk - 1) / a.kchunk)
                               : (unsigned)(a.batch > 1 ? a.batch : 1);
  dim3 grid((unsigned)((a.M + 63) / 64), (unsigned)((a.N + 63) / 64), nz ? nz : 1u);
  if (!ta && tb && epi == SG_GELU) k_sgemm<false, true, SG_GELU><<<grid, 256, 0, s>>>(a);
  else if (!ta && tb && epi == SG_BIAS) k_sgemm<false, true, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else if (!ta && !tb && epi == SG_GELU_GRAD)
    k_sgemm<false, false, SG_GELU_GRAD><<<grid, 256, 0, s>>>(a);
  else if (!ta && !tb && epi == SG_BIAS) k_sgemm<false, false, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else if (ta && !tb && epi == SG_BIAS) k_sgemm<true, false, SG_BIAS><<<grid, 256, 0, s>>>(a);
  else if (!ta && tb && epi == SG_AXPBY) k_sgemm<false, true, SG_AXPBY><<<grid, 256, 0, s>>>(a);
  else if (!ta && !tb && epi == SG_AXPBY) k_sgemm<false, false, SG_AXPBY><<<grid, 256, 0, s>>>(a);
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
