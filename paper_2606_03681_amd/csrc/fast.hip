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
  o.fb = (x + 7) / 8 * 8; x = o.fb + 2 * (3LL * E + H);
  // the forward and the backward stream of the fused MLP share one region
  int64_t msz = 0;
  if (mlp_fused_ok(E, H))
    msz = mlp_fwd_stream_elems(E, H) > mlp_bwd_stream_elems(E, H) ? mlp_fwd_stream_elems(E, H)
                                                                   : mlp_bwd_stream_elems(E, H);
  o.ms = (x + 127) / 128 * 128; x = o.ms + msz;
  o.total = x;
  return o;
}

// One thread per weight element: src (fp32, packed parameter order) -> w (same layout, bf16)
// and wt (each matrix transposed, bf16).
__global__ void k_weight_prep(const float* __restrict__ p, int E, int H, WOff wo,
                              bf16* __restrict__ w, bf16* __restrict__ wt, WFold fold,
                              int folded) {
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
      const float x = p[src[k] + t];
      const uint16_t v = f2bf(x);
      // the fold scales input column c of Wqkv_i by g1[c] and of W1 by g2[c]
      w[dst[k] + t] = folded && (k == 2 || k == 4) ? f2bf(x * (k == 2 ? fold.g1 : fold.g2)[c]) : v;
      wt[dst[k] + (int64_t)c * rows[k] + r] = v;
      return;
    }
    t -= n;
  }
}

// Folded biases, one wave per output: bqkv_i[n] + sum_k Wqkv_i[n][k] be1[k] for n < 3E, then
// b1[m] + sum_k W1[m][k] be2[k]; float32, lane l summing k = l, l + 64, ... (a coalesced read of
// the weight row), then the lanes' sums added in a fixed butterfly.
__global__ void k_fold_bias(const float* __restrict__ p, int E, int H, WFold fold,
                            float* __restrict__ fb) {
  const int n = blockIdx.x * 4 + wave_id();
  if (n >= 3 * E + H) return;
  const int lane = threadIdx.x & 63;
  const int64_t E2 = (int64_t)E * E;
  const bool q = n < 3 * E;
  const int m = q ? n : n - 3 * E;
  const float* row = p + (q ? 4 * E2 + 4 * E : 8 * E2 + 8 * E) + (int64_t)m * E;
  const float* be = q ? fold.be1 : fold.be2;
  float acc = 0.f;
  for (int k = lane; k < E; k += 64) acc = fmaf(row[k], be[k], acc);
  acc = wave_reduce_sum(acc);
  if (lane == 0) fb[n] = (q ? fold.bqkv_i : fold.b1)[m] + acc;
}

hipError_t launch_weight_prep(const float* params, int E, int H, bf16* w, bf16* wt,
                              const WFold* fold, hipStream_t s) {
  WOff wo = weight_offsets(E, H);
  unsigned grid = (unsigned)((wo.fb + 255) / 256);
  k_weight_prep<<<grid, 256, 0, s>>>(params, E, H, wo, w, wt, fold ? *fold : WFold{}, fold != nullptr);
  if (fold) {
    const int n = 3 * E + H;
    k_fold_bias<<<(n + 3) / 4, 256, 0, s>>>(params, E, H, *fold,
                                                reinterpret_cast<float*>(w + wo.fb));
  }
  return hipGetLastError();
}

// One wave per native row (b, r): the row's S cells are S * E contiguous elements, written in
// 16-byte pieces with consecutive lanes on consecutive pieces, zero where the piece's cell is
// inactive.  Rows of datasets with every cell active leave at once.
__global__ void k_zero_inactive(Geo g, bf16* __restrict__ x) {
  const int64_t row = (int64_t)blockIdx.x * 4 + wave_id();
  if (row >= (int64_t)g.B * g.R) return;
  const int b = (int)(row / g.R);
  if (g.ds[b].S == g.S) return;
  const int lane = threadIdx.x & 63, per = g.E / 8;
  const int32_t* cm = g.colmap + (int64_t)b * g.S;
  uint4* p = reinterpret_cast<uint4*>(x + row * g.S * g.E);
  const uint4 z = make_uint4(0, 0, 0, 0);
  for (int i = lane; i < g.S * per; i += 64)
    if (cm[i / per] < 0) p[i] = z;
}

hipError_t launch_zero_inactive(const Geo& g, bf16* native, hipStream_t s) {
  const int64_t rows = (int64_t)g.B * g.R;
  k_zero_inactive<<<(unsigned)((rows + 3) / 4), 256, 0, s>>>(g, native);
  return hipGetLastError();
}

// LN3 backward from the native dY: 512 threads = 16 half-waves; a half-wave owns one cell at a
// time, lane l holding features 8l .. 8l+7 (E <= 256) in 16-byte pieces.  A block covers
// LN_CELLS consecutive compact cells; half-wave h takes cells h, h + 16, ..., four per batch
// with all their loads in flight, and keeps running column sums of dY * xhat and dY.
constexpr int LN_CELLS = 256;
constexpr int LN_BATCH = 4;

__global__ __launch_bounds__(512) void k_ln_out_bwd(Geo g, const bf16* __restrict__ dY,
                                                    const bf16* __restrict__ xhat,
                                                    const float* __restrict__ rstd,
                                                    const float* __restrict__ gamma,
                                                    bf16* __restrict__ dz,
                                                    float* __restrict__ part) {
  __shared__ float red[16][2][256];
  const int tid = threadIdx.x, hw = tid >> 5, l = tid & 31;
  const int E = g.E;
  const bool act = 8 * l < E;
  float gm[8], cs1[8], cs2[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    gm[j] = act ? gamma[8 * l + j] : 0.f;
    cs1[j] = cs2[j] = 0.f;
  }
  const int64_t c0 = (int64_t)blockIdx.x * LN_CELLS;
  const int col0 = (int)(c0 / g.R), r0 = (int)(c0 - (int64_t)col0 * g.R);
  for (int base = hw; base < LN_CELLS; base += 16 * LN_BATCH) {
    uint4 dyv[LN_BATCH], xv[LN_BATCH];
    float rs[LN_BATCH];
    int64_t pc[LN_BATCH];
    bool ok[LN_BATCH];
#pragma unroll
    for (int u = 0; u < LN_BATCH; ++u) {
      const int cc = base + 16 * u;
      const int64_t p = c0 + cc;
      pc[u] = p;
      ok[u] = cc < LN_CELLS && p < g.N;
      dyv[u] = xv[u] = make_uint4(0, 0, 0, 0);
      rs[u] = 0.f;
      if (ok[u]) {
        int col = col0, r = r0 + cc;
        while (r >= g.R) {
          r -= g.R;
          ++col;
        }
        const int64_t nat = g.col_cell0[col] + (int64_t)r * g.S;
        rs[u] = rstd[p];
        if (act) {
          dyv[u] = ldu4(dY + nat * E + 8 * l);
          xv[u] = ldu4(xhat + p * E + 8 * l);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < LN_BATCH; ++u) {
      float dy[8], x[8];
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        dy[j] = bf2f(u4_elem(dyv[u], j));
        x[j] = bf2f(u4_elem(xv[u], j));
        cs1[j] += dy[j] * x[j];
        cs2[j] += dy[j];
        s1 += dy[j] * gm[j];
        s2 += dy[j] * gm[j] * x[j];
      }
      s1 = half32_sum(s1);
      s2 = half32_sum(s2);
      const float m1 = s1 / E, m2 = s2 / E;
      if (ok[u] && act) {
        uint4 o;
        o.x = pack2(rs[u] * (dy[0] * gm[0] - m1 - x[0] * m2), rs[u] * (dy[1] * gm[1] - m1 - x[1] * m2));
        o.y = pack2(rs[u] * (dy[2] * gm[2] - m1 - x[2] * m2), rs[u] * (dy[3] * gm[3] - m1 - x[3] * m2));
        o.z = pack2(rs[u] * (dy[4] * gm[4] - m1 - x[4] * m2), rs[u] * (dy[5] * gm[5] - m1 - x[5] * m2));
        o.w = pack2(rs[u] * (dy[6] * gm[6] - m1 - x[6] * m2), rs[u] * (dy[7] * gm[7] - m1 - x[7] * m2));
        stu4(dz + pc[u] * E + 8 * l, o);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    red[hw][0][8 * l + j] = cs1[j];
    red[hw][1][8 * l + j] = cs2[j];
  }
  __syncthreads();
  if (tid < 2 * E) {
    const int t = tid / E, e = tid % E;
    float sm = 0.f;
#pragma unroll
    for (int h = 0; h < 16; ++h) sm += red[h][t][e];
    part[(int64_t)blockIdx.x * 2 * E + t * E + e] = sm;
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

// Pre-norm block input: x' = decay * X (native rows) and r = gamma x' / sqrt(mean(x'^2) + eps),
// both written compact, with rstd.  Same thread layout as the LN3 backward above: a half-wave
// per cell, lane l holding features 8l .. 8l+7, four cells per half-wave in flight.
__global__ __launch_bounds__(512) void k_rms_in(Geo g, const bf16* __restrict__ X, float decay,
                                                const float* __restrict__ gamma, float eps,
                                                bf16* __restrict__ xs, bf16* __restrict__ r,
                                                float* __restrict__ rstd) {
  const int tid = threadIdx.x, hw = tid >> 5, l = tid & 31;
  const int E = g.E;
  const bool act = 8 * l < E;
  float gm[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) gm[j] = act ? gamma[8 * l + j] : 0.f;
  const int64_t c0 = (int64_t)blockIdx.x * LN_CELLS;
  const int col0 = (int)(c0 / g.R), r0 = (int)(c0 - (int64_t)col0 * g.R);
  for (int base = hw; base < LN_CELLS; base += 16 * LN_BATCH) {
    uint4 xv[LN_BATCH];
    int64_t pc[LN_BATCH];
    bool ok[LN_BATCH];
#pragma unroll
    for (int u = 0; u < LN_BATCH; ++u) {
      const int cc = base + 16 * u;
      const int64_t p = c0 + cc;
      pc[u] = p;
      ok[u] = cc < LN_CELLS && p < g.N;
      xv[u] = make_uint4(0, 0, 0, 0);
      if (ok[u] && act) {
        int col = col0, rr = r0 + cc;
        while (rr >= g.R) {
          rr -= g.R;
          ++col;
        }
        const int64_t nat = g.col_cell0[col] + (int64_t)rr * g.S;
        xv[u] = ldu4(X + nat * E + 8 * l);
      }
    }
#pragma unroll
    for (int u = 0; u < LN_BATCH; ++u) {
      float x[8];
      float ss = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        x[j] = decay * bf2f(u4_elem(xv[u], j));
        ss += x[j] * x[j];
      }
      ss = half32_sum(ss);
      const float rs = 1.0f / sqrtf(ss / E + eps);
      if (ok[u] && l == 0) rstd[pc[u]] = rs;
      if (ok[u] && act) {
        uint4 a, b;
        a.x = pack2(x[0], x[1]); a.y = pack2(x[2], x[3]);
        a.z = pack2(x[4], x[5]); a.w = pack2(x[6], x[7]);
        b.x = pack2(gm[0] * x[0] * rs, gm[1] * x[1] * rs);
        b.y = pack2(gm[2] * x[2] * rs, gm[3] * x[3] * rs);
        b.z = pack2(gm[4] * x[4] * rs, gm[5] * x[5] * rs);
        b.w = pack2(gm[6] * x[6] * rs, gm[7] * x[7] * rs);
        stu4(xs + pc[u] * E + 8 * l, a);
        stu4(r + pc[u] * E + 8 * l, b);
      }
    }
  }
}

hipError_t launch_rms_in(const Geo& g, const bf16* X, float decay, const float* gamma, float eps,
                         bf16* xs, bf16* r, float* rstd, hipStream_t s) {
  const int64_t nb = (g.N + LN_CELLS - 1) / LN_CELLS;
  if (nb == 0) return hipSuccess;
  k_rms_in<<<(unsigned)nb, 512, 0, s>>>(g, X, decay, gamma, eps, xs, r, rstd);
  return hipGetLastError();
}

// Thinking rows: rows [0, T) of X get the table (float32 [T][E]) at active cell columns and 0 at
// inactive ones; one thread per element of those rows.
template <class TT>
__global__ void k_thinking_fwd(Geo g, int T, const float* __restrict__ table, TT* __restrict__ X) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per = (int64_t)T * g.S * g.E;
  if (i >= per * g.B) return;
  const int b = (int)(i / per);
  const int64_t rest = i - b * per;
  const int t = (int)(rest / ((int64_t)g.S * g.E));
  const int c = (int)(rest / g.E % g.S);
  const int e = (int)(rest % g.E);
  const bool act = g.colmap[b * g.S + c] >= 0;
  st(X + (((int64_t)b * g.R + t) * g.S + c) * g.E + e, act ? table[t * g.E + e] : 0.f);
}

// dtable[t][e] (+)= sum over datasets b and active columns c of dX[b][t][c][e], in (b, c) order.
template <class TT>
__global__ void k_thinking_bwd(Geo g, int T, const TT* __restrict__ dX, float* __restrict__ dtable,
                               int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)T * g.E) return;
  const int t = (int)(i / g.E), e = (int)(i % g.E);
  float s = 0.f;
  for (int b = 0; b < g.B; ++b)
    for (int c = 0; c < g.S; ++c)
      if (g.colmap[b * g.S + c] >= 0) s += ld(dX + (((int64_t)b * g.R + t) * g.S + c) * g.E + e);
  dtable[i] = (accumulate ? dtable[i] : 0.f) + s;
}

template <class TT>
hipError_t launch_thinking_fwd(const Geo& g, int T, const float* table, TT* X, hipStream_t s) {
  const int64_t n = (int64_t)g.B * T * g.S * g.E;
  if (n == 0) return hipSuccess;
  k_thinking_fwd<TT><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(g, T, table, X);
  return hipGetLastError();
}

template <class TT>
hipError_t launch_thinking_bwd(const Geo& g, int T, const TT* dX, float* dtable, int accumulate,
                               hipStream_t s) {
  const int64_t n = (int64_t)T * g.E;
  if (n == 0) return hipSuccess;
  k_thinking_bwd<TT><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(g, T, dX, dtable, accumulate);
  return hipGetLastError();
}

template hipError_t launch_thinking_fwd<float>(const Geo&, int, const float*, float*, hipStream_t);
template hipError_t launch_thinking_fwd<bf16>(const Geo&, int, const float*, bf16*, hipStream_t);
template hipError_t launch_thinking_bwd<float>(const Geo&, int, const float*, float*, int,
                                               hipStream_t);
template hipError_t launch_thinking_bwd<bf16>(const Geo&, int, const bf16*, float*, int,
                                              hipStream_t);

size_t ln_partial_bytes(int64_t cells, int E) {
  // LN-backward GEMM epilogues: [64-cell tiles][2 E]; fused MLP backward: [tiles][4 E]
  const size_t a = (size_t)gemm_row_tiles(cells) * 2 * E * 4;
  const size_t b = (size_t)mlp_bwd_tiles(cells) * 4 * E * 4;
  return (a > b ? a : b) + 256;
}

size_t fast_workspace_bytes(int B, int R, int S, int E, int heads, int H, bool bf16) {
  (void)heads;
  if (!bf16) return 0;
  WOff wo = weight_offsets(E, H);
  const int64_t tiles = gemm_row_tiles((int64_t)B * R * S);
  size_t bytes = 2 * (size_t)wo.total * 2 + 1024;   // w and wt
  (void)tiles;
  bytes += ln_partial_bytes((int64_t)B * R * S, E);  // LN-backward column partials
  const int64_t cells = (int64_t)B * R * S;
  const int64_t zw = wgrad_max_chunks(cells);
  const int64_t maxw = 3LL * E * E > (int64_t)H * E ? 3LL * E * E : (int64_t)H * E;
  const int64_t maxn = 3LL * E > H ? 3LL * E : H;
  bytes += (size_t)zw * maxw * 4 + 256;                // weight-gradient partials
  bytes += (size_t)zw * maxn * 4 + 256;                // bias-gradient partials
  return bytes;
}

}  // namespace tfm
