// bf16 MFMA GEMM over active cells with fused epilogues.
//
//   C[m, n] = sum_k A[m, k] * Bt[n, k]        (A: cells x K, Bt: [N][K] bf16 weights)
//
// Block tile 64 x BN (BN = E, the embedding width, so that one block owns whole cell rows and
// LayerNorm can run in the epilogue), K streamed through LDS in steps of 32 with double
// buffering.  Four waves in a 2 x 2 arrangement; each wave owns a 32 x BN/2 sub-tile held as
// 2 x (BN/32) accumulators of v_mfma_f32_16x16x32_bf16, computed as C^T blocks (weights as
// the A operand) so that a lane holds 4 consecutive output features of one cell: epilogue
// tiles then move through LDS in 8-byte pieces.
#include <math.h>

#include "fast.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr int BM = GEMM_BM;
constexpr int MI = BM / 32;  // 16-row blocks per wave (2 x 2 waves, each BM/2 rows)
constexpr int BK = 32;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row (16-byte pad)
constexpr int CPRK = BK / 8;        // 16-byte chunks per staged row

// Normal CDF Phi(x) = (1 + erf(x / sqrt 2)) / 2 with erf from Abramowitz & Stegun 7.1.26
// (|error| <= 1.5e-7): erf(z) = 1 - t (a1 + t (a2 + ... + t a5)) exp(-z^2), t = 1 / (1 + p z)
// for z >= 0, odd in z.  *e returns exp(-x^2 / 2), which the normal density shares.
__device__ __forceinline__ float norm_cdf(float x, float* e) {
  const float az = fabsf(x) * 0.70710678118654752f;
  *e = __builtin_amdgcn_exp2f(-0.72134752044448170f * x * x);  // exp(-x^2/2) = 2^(-x^2 log2e / 2)
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, az, 1.0f));
  float poly = fmaf(t, 1.061405429f, -1.453152027f);
  poly = fmaf(t, poly, 1.421413741f);
  poly = fmaf(t, poly, -0.284496736f);
  poly = fmaf(t, poly, 0.254829592f);
  const float h = 0.5f * t * poly * *e;  // (1 - erf(|z|)) / 2
  return x >= 0.f ? 1.0f - h : h;
}
// GELU(x) = x Phi(x)
__device__ __forceinline__ float gelu_f(float x) {
  float e;
  return x * norm_cdf(x, &e);
}
// GELU'(x) = Phi(x) + x phi(x), phi(x) = exp(-x^2 / 2) / sqrt(2 pi)
__device__ __forceinline__ float gelu_grad_f(float x) {
  float e;
  const float cdf = norm_cdf(x, &e);
  return fmaf(x * 0.39894228040143268f, e, cdf);
}

__device__ __forceinline__ int64_t row_addr(const Geo& g, int mode, int64_t m, int64_t ld) {
  return mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
}

// Sum over the 16 lanes that share lane / 16.
__device__ __forceinline__ float sum16(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  return v;
}
// Sum over the 4 lanes that share lane % 16.
__device__ __forceinline__ float sum4g(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}
__device__ __forceinline__ f32x4 unpack4(uint2 u) {
  f32x4 r;
  r[0] = __uint_as_float(u.x << 16);
  r[1] = __uint_as_float(u.x & 0xffff0000u);
  r[2] = __uint_as_float(u.y << 16);
  r[3] = __uint_as_float(u.y & 0xffff0000u);
  return r;
}

}  // namespace

template <int BN, int EPI>
__global__ __launch_bounds__(256, 2) void k_gemm(GemmArgs a) {
  constexpr int NB = BN / 32;          // 16-wide column blocks per wave
  constexpr int BCH = BN * CPRK / 256; // 16-byte chunks of the B tile per thread
  constexpr int TS = BN + 8;  // epilogue tile row stride (elements)
  constexpr int MAIN_BYTES = 2 * (BM + BN) * LDS_STRIDE * 2;
  constexpr int TILE_BYTES = BM * TS * 2;
  __shared__ __attribute__((aligned(16))) char smem[MAIN_BYTES > TILE_BYTES ? MAIN_BYTES : TILE_BYTES];
  bf16 (*As)[BM * LDS_STRIDE] = reinterpret_cast<bf16 (*)[BM * LDS_STRIDE]>(smem);
  bf16 (*Bs)[BN * LDS_STRIDE] =
      reinterpret_cast<bf16 (*)[BN * LDS_STRIDE]>(smem + 2 * BM * LDS_STRIDE * 2);
  bf16* tile = reinterpret_cast<bf16*>(smem);  // epilogue: [BM][TS], after the main loop
  __shared__ float red[2][BM];
  __shared__ float cred[2][2][BN];
  __shared__ __attribute__((aligned(16))) float cpar[3][BN];  // bias, gamma, beta of the tile
  __shared__ int64_t rbase[BM];  // epilogue: per-row element offset for the current mode

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const Geo& g = a.g;

  if (EPI == EPI_ITEM_QKV && blockIdx.y > 0) {
    // K and V exist for train rows only: skip tiles made of test rows alone
    int64_t last = m0 + BM - 1 < a.M ? m0 + BM - 1 : a.M - 1;
    int64_t c0 = m0 / g.R, c1 = last / g.R;
    bool any = false;
    for (int64_t c = c0; c <= c1 && !any; ++c) {
      int64_t rlo = c == c0 ? m0 - c0 * g.R : 0;
      any = rlo < g.ds[g.col_ds[c]].n_train;
    }
    if (!any) return;
  }

  // ---- global -> register staging assignment
  constexpr int ACH = BM * CPRK / 256;  // 16-byte chunks of the A tile per thread
  int64_t aoff[ACH];
  bool aval[ACH];
  int arow[ACH], akc[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    int c = tid + 256 * i;
    arow[i] = c / CPRK;
    akc[i] = (c % CPRK) * 8;
    int64_t m = m0 + arow[i];
    aval[i] = m < a.M;
    aoff[i] = aval[i] && a.amode != ROWS_ITEM_HM ? row_addr(g, a.amode, m, a.lda) : 0;
  }
  int brow[BCH], bkc[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    int c = tid + 256 * i;
    brow[i] = c / CPRK;
    bkc[i] = (c % CPRK) * 8;
  }
  const bf16* Bt = a.Bt + (int64_t)n0 * a.K;

  uint4 ra[ACH], rb[BCH];
  // head-major item gradients: per row, the column (global active column) and the row index
  int64_t hcol[ACH];
  int hr[ACH];
  if (a.amode == ROWS_ITEM_HM) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int64_t m = m0 + arow[i];
      hcol[i] = m / g.R;
      hr[i] = (int)(m - hcol[i] * g.R);
    }
  }
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      if (a.amode == ROWS_ITEM_HM) {
        int part = 0;
        const int64_t off = aval[i] ? item_hm_offset(g, hcol[i], hr[i], k0 + akc[i], &part) : -1;
        const bf16* base = part == 0 ? a.A : (part == 1 ? a.A2 : a.A3);
        ra[i] = off >= 0 ? ldu4(base + off) : make_uint4(0, 0, 0, 0);
      } else {
        ra[i] = aval[i] ? ldu4(a.A + aoff[i] + k0 + akc[i]) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) rb[i] = ldu4(Bt + (int64_t)brow[i] * a.K + k0 + bkc[i]);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) stu4(&As[buf][arow[i] * LDS_STRIDE + akc[i]], ra[i]);
#pragma unroll
    for (int i = 0; i < BCH; ++i) stu4(&Bs[buf][brow[i] * LDS_STRIDE + bkc[i]], rb[i]);
  };

  // per-column epilogue parameters of this column tile, staged once
  if (tid < BN) {
    cpar[0][tid] = a.bias ? a.bias[n0 + tid] : 0.f;
    if (EPI == EPI_LN || EPI == EPI_LN_BWD) cpar[1][tid] = a.gamma[tid];
    if (EPI == EPI_LN) cpar[2][tid] = a.beta[tid];
  }

  f32x4 acc[MI][NB];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = zero4();

  const int KT = a.K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 af[MI], bfr[NB];
#pragma unroll
      for (int i = 0; i < MI; ++i)
        af[i] = ld8(&As[cur][(wm * (BM / 2) + i * 16 + lr) * LDS_STRIDE + ks * 32 + lg * 8]);
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bfr[j] = ld8(&Bs[cur][(wn * (BN / 2) + j * 16 + lr) * LDS_STRIDE + ks * 32 + lg * 8]);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = mfma16(bfr[j], af[i], acc[i][j]);
    }
    if (kt + 1 < KT) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogues.  acc[i][j][q] is C[row, col] with
  //   row = m0 + wm*BM/2 + i*16 + lr,  col = n0 + wn*BN/2 + j*16 + lg*4 + q
  // Global traffic goes through the LDS tile [BM][TS] in 16-byte row chunks: residual / x-hat
  // inputs are loaded into it, outputs are written into it and copied out row by row.
  const int cb0 = wn * (BN / 2) + lg * 4;  // tile column of q = 0 for j = 0
  constexpr int CPRW = BN / 8;             // 16-byte chunks per tile row
  auto rloc = [&](int i) { return wm * (BM / 2) + i * 16 + lr; };

  // per-row element offsets: ROWS_COMPACT with leading dimension ld, ROWS_NATIVE, or the
  // head-major item layout (offset of row m's (head 0, dim 0); -1 where K/V do not exist)
  auto set_rows = [&](int mode, int64_t ld, int hm_part) {
    if (tid < BM) {
      const int64_t m = m0 + tid;
      int64_t off = -1;
      if (m < a.M) {
        if (hm_part >= 0) {
          const int64_t col = m / g.R;
          const int r = (int)(m - col * g.R);
          if (hm_part == 0 || r < g.ds[g.col_ds[col]].n_train)
            off = (col * g.heads * g.R + r) * (int64_t)g.d;
        } else {
          off = mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
        }
      }
      rbase[tid] = off;
    }
  };
  // tile <- rows of src (columns [c0, c0 + BN)); rows without an offset read as 0
  auto load_tile = [&](const bf16* src, int c0) {
    for (int ch = tid; ch < BM * CPRW; ch += 256) {
      const int row = ch / CPRW, cc = (ch % CPRW) * 8;
      const int64_t off = rbase[row];
      stu4(&tile[row * TS + cc], off >= 0 ? ldu4(src + off + c0 + cc) : make_uint4(0, 0, 0, 0));
    }
  };
  // rows of dst <- tile (columns [c0, c0 + BN)); head-major destinations when hm is set
  auto store_tile = [&](bf16* dst, int c0, bool hm) {
    for (int ch = tid; ch < BM * CPRW; ch += 256) {
      const int row = ch / CPRW, cc = (ch % CPRW) * 8;
      const int64_t off = rbase[row];
      if (off < 0) continue;
      int64_t o = off + c0 + cc;
      if (hm) {
        const int head = cc / g.d, jj = cc - head * g.d;
        o = off + (int64_t)head * g.R * g.d + jj;
      }
      stu4(dst + o, ldu4(&tile[row * TS + cc]));
    }
  };
  // the lane's 4 consecutive tile elements of block (i, j), and the matching parameters
  auto tile4 = [&](int i, int j) -> f32x4 {
    return unpack4(*reinterpret_cast<const uint2*>(&tile[rloc(i) * TS + cb0 + j * 16]));
  };
  auto put4 = [&](int i, int j, const f32x4& v) {
    *reinterpret_cast<uint2*>(&tile[rloc(i) * TS + cb0 + j * 16]) =
        make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
  };
  auto par4 = [&](int which, int j) -> f32x4 {
    const float4 f = *reinterpret_cast<const float4*>(&cpar[which][cb0 + j * 16]);
    f32x4 r;
    r[0] = f.x; r[1] = f.y; r[2] = f.z; r[3] = f.w;
    return r;
  };

  if (EPI == EPI_BIAS || EPI == EPI_GELU_FWD || EPI == EPI_ITEM_QKV) {
    if (EPI == EPI_ITEM_QKV)
      set_rows(ROWS_COMPACT, 0, blockIdx.y);
    else
      set_rows(ROWS_COMPACT, a.ldo, -1);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f32x4 b = par4(0, j);
#pragma unroll
      for (int i = 0; i < MI; ++i) put4(i, j, acc[i][j] + b);
    }
    lds_barrier();
    if (EPI == EPI_ITEM_QKV) {
      bf16* dst = blockIdx.y == 0 ? a.out : (blockIdx.y == 1 ? a.out2 : a.out3);
      store_tile(dst, 0, true);
      return;
    }
    store_tile(a.out, n0, false);
    if (EPI == EPI_GELU_FWD) {
      // U = GELU of the stored (bf16) pre-activation, computed in place of the accumulators
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const f32x4 x = tile4(i, j);
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[i][j][q] = gelu_f(x[q]);
        }
      lds_barrier();
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) put4(i, j, acc[i][j]);
      lds_barrier();
      store_tile(a.out2, n0, false);
    }
    return;
  }

  if (EPI == EPI_GELU_BWD) {
    set_rows(ROWS_COMPACT, a.ldo, -1);
    lds_barrier();
    load_tile(a.aux, n0);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4 x = tile4(i, j);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][j][q] *= gelu_grad_f(x[q]);
      }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, acc[i][j]);
    lds_barrier();
    store_tile(a.out, n0, false);
    return;
  }

  if (EPI == EPI_DX) {
    set_rows(ROWS_COMPACT, BN, -1);
    lds_barrier();
    load_tile(a.resid, 0);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] += tile4(i, j);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, acc[i][j]);
    set_rows(ROWS_NATIVE, 0, -1);
    lds_barrier();
    store_tile(a.out, 0, false);
    return;
  }

  // ---- LayerNorm epilogues (BN == E, n0 == 0): row statistics across the lane groups of a
  // wave and the two column waves.  The accumulators are overwritten in place.
  auto& val = acc;
  // sum over the row's BN columns of f(i, j) (a 4-vector per block) -> per-row value
  auto row_sum = [&](auto f, float* out) {
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      float sm = 0.f;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4 v = f(i, j);
        sm += (v[0] + v[1]) + (v[2] + v[3]);
      }
      sm = sum4g(sm);
      if (lg == 0) red[wn][rloc(i)] = sm;
    }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i) out[i] = (red[0][rloc(i)] + red[1][rloc(i)]) * (1.0f / BN);
    lds_barrier();
  };

  if (EPI == EPI_LN) {
    set_rows(a.rmode, BN, -1);
    lds_barrier();
    load_tile(a.resid, 0);
    lds_barrier();
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f32x4 b = par4(0, j);
#pragma unroll
      for (int i = 0; i < MI; ++i) val[i][j] = acc[i][j] + b + tile4(i, j);
    }
    float mean[MI], var[MI];
    row_sum([&](int i, int j) { return val[i][j]; }, mean);
    row_sum([&](int i, int j) {
      const f32x4 dv = val[i][j] - mean[i];
      return dv * dv;
    }, var);
    // x-hat in place of val; rstd per row
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const float rs = 1.0f / sqrtf(var[i] + 1e-5f);
#pragma unroll
      for (int j = 0; j < NB; ++j) val[i][j] = (val[i][j] - mean[i]) * rs;
      if (wn == 0 && lg == 0 && m0 + rloc(i) < a.M) a.rstd[m0 + rloc(i)] = rs;
    }
    // h = gamma * x-hat + beta -> out (omode); x-hat -> xhat (compact)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f32x4 gm = par4(1, j), bt = par4(2, j);
#pragma unroll
      for (int i = 0; i < MI; ++i) put4(i, j, gm * val[i][j] + bt);
    }
    set_rows(a.omode, BN, -1);
    lds_barrier();
    store_tile(a.out, 0, false);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, val[i][j]);
    set_rows(ROWS_COMPACT, BN, -1);
    lds_barrier();
    store_tile(a.xhat, 0, false);
    return;
  }

  if (EPI == EPI_LN_BWD) {
    // dh = acc + resid; du = rstd * (g - mean(g) - xhat * mean(g * xhat)), g = dh * gamma;
    // column partial sums of dh * xhat (dgamma) and dh (dbeta) per workgroup
    set_rows(ROWS_COMPACT, BN, -1);
    lds_barrier();
    load_tile(a.resid, 0);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) val[i][j] = acc[i][j] + tile4(i, j);
    lds_barrier();
    load_tile(a.aux, 0);  // x-hat stays in the tile for the rest of the epilogue
    lds_barrier();
    // column sums over the wave's rows: within the lane over i, then over the 16 row lanes
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      f32x4 s1 = zero4(), s2 = zero4();
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        s1 += val[i][j] * tile4(i, j);
        s2 += val[i][j];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float t1 = sum16(s1[q]), t2 = sum16(s2[q]);
        if (lr == 0) {
          cred[0][wm][cb0 + j * 16 + q] = t1;
          cred[1][wm][cb0 + j * 16 + q] = t2;
        }
      }
    }
    float m1[MI], m2[MI];
    row_sum([&](int i, int j) { return val[i][j] * par4(1, j); }, m1);
    if (tid < BN) {
      float* pg = a.part + (int64_t)blockIdx.x * 2 * BN;
      pg[tid] = cred[0][0][tid] + cred[0][1][tid];
      pg[BN + tid] = cred[1][0][tid] + cred[1][1][tid];
    }
    row_sum([&](int i, int j) { return val[i][j] * par4(1, j) * tile4(i, j); }, m2);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const float rs = m0 + rloc(i) < a.M ? a.rstd_in[m0 + rloc(i)] : 0.f;
#pragma unroll
      for (int j = 0; j < NB; ++j)
        val[i][j] = rs * (val[i][j] * par4(1, j) - m1[i] - tile4(i, j) * m2[i]);
    }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, val[i][j]);
    lds_barrier();
    store_tile(a.out, 0, false);
    return;
  }
}

template <int BN>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t s) {
  dim3 grid((unsigned)((a.M + BM - 1) / BM), (unsigned)(a.N / BN));
  switch (a.epi) {
    case EPI_BIAS: k_gemm<BN, EPI_BIAS><<<grid, 256, 0, s>>>(a); break;
    case EPI_GELU_FWD: k_gemm<BN, EPI_GELU_FWD><<<grid, 256, 0, s>>>(a); break;
    case EPI_GELU_BWD: k_gemm<BN, EPI_GELU_BWD><<<grid, 256, 0, s>>>(a); break;
    case EPI_ITEM_QKV: k_gemm<BN, EPI_ITEM_QKV><<<grid, 256, 0, s>>>(a); break;
    case EPI_LN: k_gemm<BN, EPI_LN><<<grid, 256, 0, s>>>(a); break;
    case EPI_LN_BWD: k_gemm<BN, EPI_LN_BWD><<<grid, 256, 0, s>>>(a); break;
    case EPI_DX: k_gemm<BN, EPI_DX><<<grid, 256, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.K % BK || a.N % a.BN) return hipErrorInvalidValue;
  switch (a.BN) {
    case 64: return gemm_dispatch<64>(a, s);
    case 128: return gemm_dispatch<128>(a, s);
    case 192: return gemm_dispatch<192>(a, s);
    case 256: return gemm_dispatch<256>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tfm
