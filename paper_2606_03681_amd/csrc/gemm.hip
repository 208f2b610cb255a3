// bf16 MFMA GEMM over active cells with fused epilogues.
//
//   C[m, n] = sum_k A[m, k] * Bt[n, k]        (A: cells x K, Bt: [N][K] bf16 weights)
//
// Block tile 128 x BN (BN = E, the embedding width, so that one block owns whole cell rows and
// LayerNorm can run in the epilogue), K streamed through LDS in steps of 32 with double
// buffering.  Four waves in a 2 x 2 arrangement; each wave owns a 64 x BN/2 sub-tile held as
// 4 x (BN/32) accumulators of v_mfma_f32_16x16x32_bf16.
#include <math.h>

#include "fast.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr int BM = 128;
constexpr int BK = 32;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row (16-byte pad)

__device__ __forceinline__ float gelu_f(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad_f(float x) {
  float cdf = 0.5f * (1.0f + erff(x * 0.70710678118654752f));
  float pdf = 0.39894228040143268f * __expf(-0.5f * x * x);
  return cdf + x * pdf;
}

__device__ __forceinline__ int64_t row_addr(const Geo& g, int mode, int64_t m, int64_t ld) {
  return mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
}

// Sum over the 16 lanes that share lane / 16 (the 16 columns of one MFMA D block).
__device__ __forceinline__ float sum16(float v) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  return v;
}

}  // namespace

template <int BN, int EPI>
__global__ __launch_bounds__(256, 2) void k_gemm(GemmArgs a) {
  constexpr int NB = BN / 32;          // 16-wide column blocks per wave
  constexpr int BCH = BN * 4 / 256;    // 16-byte chunks of the B tile per thread
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LDS_STRIDE];
  __shared__ float red[2][BM];
  __shared__ float cred[2][2][BN];

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
  int64_t aoff[2];
  bool aval[2];
  int arow[2], akc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int c = tid + 256 * i;
    arow[i] = c >> 2;
    akc[i] = (c & 3) * 8;
    int64_t m = m0 + arow[i];
    aval[i] = m < a.M;
    aoff[i] = aval[i] && a.amode != ROWS_ITEM_HM ? row_addr(g, a.amode, m, a.lda) : 0;
  }
  int brow[BCH], bkc[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    int c = tid + 256 * i;
    brow[i] = c >> 2;
    bkc[i] = (c & 3) * 8;
  }
  const bf16* Bt = a.Bt + (int64_t)n0 * a.K;

  uint4 ra[2], rb[BCH];
  // head-major item gradients: per row, the column (global active column) and the row index
  int64_t hcol[2];
  int hr[2];
  if (a.amode == ROWS_ITEM_HM) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int64_t m = m0 + arow[i];
      hcol[i] = m / g.R;
      hr[i] = (int)(m - hcol[i] * g.R);
    }
  }
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
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
    for (int i = 0; i < 2; ++i) stu4(&As[buf][arow[i] * LDS_STRIDE + akc[i]], ra[i]);
#pragma unroll
    for (int i = 0; i < BCH; ++i) stu4(&Bs[buf][brow[i] * LDS_STRIDE + bkc[i]], rb[i]);
  };

  f32x4 acc[4][NB];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = zero4();

  const int KT = a.K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK);
    bf16x8 af[4], bfr[NB];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      af[i] = ld8(&As[cur][(wm * 64 + i * 16 + lr) * LDS_STRIDE + lg * 8]);
#pragma unroll
    for (int j = 0; j < NB; ++j)
      bfr[j] = ld8(&Bs[cur][(wn * (BN / 2) + j * 16 + lr) * LDS_STRIDE + lg * 8]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = mfma16(af[i], bfr[j], acc[i][j]);
    if (kt + 1 < KT) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogues.  acc[i][j][q] is C[row, col] with
  //   row = m0 + wm*64 + i*16 + lg*4 + q,  col = n0 + wn*BN/2 + j*16 + lr
  const int colb = wn * (BN / 2) + lr;  // column within the tile for j = 0

  if (EPI == EPI_BIAS || EPI == EPI_GELU_FWD || EPI == EPI_GELU_BWD) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
        if (m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = n0 + colb + j * 16;
          float v = acc[i][j][q];
          if (a.bias) v += a.bias[n];
          int64_t o = m * a.ldo + n;
          if (EPI == EPI_GELU_BWD) v *= gelu_grad_f(bf2f(a.aux[o]));
          a.out[o] = f2bf(v);
          if (EPI == EPI_GELU_FWD) a.out2[o] = f2bf(gelu_f(bf2f(a.out[o])));
        }
      }
    return;
  }

  if (EPI == EPI_ITEM_QKV) {
    const int part = blockIdx.y;  // 0 = Q, 1 = K, 2 = V
    bf16* dst = part == 0 ? a.out : (part == 1 ? a.out2 : a.out3);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
        if (m >= a.M) continue;
        int64_t col = m / g.R;
        int r = (int)(m - col * g.R);
        if (part > 0 && r >= g.ds[g.col_ds[col]].n_train) continue;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int within = colb + j * 16;
          int head = within / g.d, jj = within - head * g.d;
          float v = acc[i][j][q] + a.bias[n0 + within];
          dst[((col * g.heads + head) * g.R + r) * g.d + jj] = f2bf(v);
        }
      }
    return;
  }

  if (EPI == EPI_DX) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
        if (m >= a.M) continue;
        int64_t ro = m * (int64_t)BN;
        int64_t oo = native_cell(g, m) * BN;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = colb + j * 16;
          a.out[oo + n] = f2bf(acc[i][j][q] + bf2f(a.resid[ro + n]));
        }
      }
    return;
  }

  // ---- LayerNorm epilogues (BN == E, n0 == 0): row statistics across the two column waves.
  // The accumulators are overwritten in place by the pre-norm values.
  auto& val = acc;
  float gam[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) gam[j] = a.gamma[colb + j * 16];

  if (EPI == EPI_LN) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
        bool ok = m < a.M;
        int64_t ro = ok ? row_addr(g, a.rmode, m, BN) : 0;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = colb + j * 16;
          val[i][j][q] = ok ? acc[i][j][q] + a.bias[n] + bf2f(a.resid[ro + n]) : 0.f;
        }
      }
    // mean
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) s += val[i][j][q];
        s = sum16(s);
        if (lr == 0) red[wn][wm * 64 + i * 16 + lg * 4 + q] = s;
      }
    __syncthreads();
    float mean[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int rl = wm * 64 + i * 16 + lg * 4 + q;
        mean[i][q] = (red[0][rl] + red[1][rl]) * (1.0f / BN);
      }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          float dv = val[i][j][q] - mean[i][q];
          s += dv * dv;
        }
        s = sum16(s);
        if (lr == 0) red[wn][wm * 64 + i * 16 + lg * 4 + q] = s;
      }
    __syncthreads();
    float bet[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) bet[j] = a.beta[colb + j * 16];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int rl = wm * 64 + i * 16 + lg * 4 + q;
        int64_t m = m0 + rl;
        if (m >= a.M) continue;
        float rs = 1.0f / sqrtf((red[0][rl] + red[1][rl]) * (1.0f / BN) + 1e-5f);
        int64_t oo = row_addr(g, a.omode, m, BN);
        int64_t co = m * (int64_t)BN;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = colb + j * 16;
          float xh = (val[i][j][q] - mean[i][q]) * rs;
          a.out[oo + n] = f2bf(fmaf(gam[j], xh, bet[j]));
          a.xhat[co + n] = f2bf(xh);
        }
        if (wn == 0 && lr == 0) a.rstd[m] = rs;
      }
    return;
  }

  if (EPI == EPI_LN_BWD) {
    // dh = acc + resid; du = rstd * (g - mean(g) - xhat * mean(g * xhat)), g = dh * gamma.
    // xhat (aux) is re-read from memory in each pass to keep register pressure down.
    auto xv_at = [&](int i, int j, int q) -> float {
      int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
      return m < a.M ? bf2f(a.aux[m * (int64_t)BN + colb + j * 16]) : 0.f;
    };
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t m = m0 + wm * 64 + i * 16 + lg * 4 + q;
        bool ok = m < a.M;
        int64_t ro = m * (int64_t)BN;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = colb + j * 16;
          val[i][j][q] = ok ? acc[i][j][q] + bf2f(a.resid[ro + n]) : 0.f;
        }
      }
    // column partial sums for dgamma (sum dh * xhat) and dbeta (sum dh)
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          s1 += val[i][j][q] * xv_at(i, j, q);
          s2 += val[i][j][q];
        }
      s1 += __shfl_xor(s1, 16, 64);
      s1 += __shfl_xor(s1, 32, 64);
      s2 += __shfl_xor(s2, 16, 64);
      s2 += __shfl_xor(s2, 32, 64);
      if (lg == 0) {
        cred[0][wm][colb + j * 16] = s1;
        cred[1][wm][colb + j * 16] = s2;
      }
    }
    float m1[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) s += val[i][j][q] * gam[j];
        s = sum16(s);
        if (lr == 0) red[wn][wm * 64 + i * 16 + lg * 4 + q] = s;
      }
    __syncthreads();
    if (tid < BN) {
      float* pg = a.part + (int64_t)blockIdx.x * 2 * BN;
      pg[tid] = cred[0][0][tid] + cred[0][1][tid];
      pg[BN + tid] = cred[1][0][tid] + cred[1][1][tid];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int rl = wm * 64 + i * 16 + lg * 4 + q;
        m1[i][q] = (red[0][rl] + red[1][rl]) * (1.0f / BN);
      }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < NB; ++j) s += val[i][j][q] * gam[j] * xv_at(i, j, q);
        s = sum16(s);
        if (lr == 0) red[wn][wm * 64 + i * 16 + lg * 4 + q] = s;
      }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int rl = wm * 64 + i * 16 + lg * 4 + q;
        int64_t m = m0 + rl;
        if (m >= a.M) continue;
        float m2 = (red[0][rl] + red[1][rl]) * (1.0f / BN);
        float rs = a.rstd_in[m];
        int64_t co = m * (int64_t)BN;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          int n = colb + j * 16;
          float gg = val[i][j][q] * gam[j];
          a.out[co + n] = f2bf(rs * (gg - m1[i][q] - xv_at(i, j, q) * m2));
        }
      }
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
