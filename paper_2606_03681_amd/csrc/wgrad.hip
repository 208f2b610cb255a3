// Weight gradients on bf16 MFMA: dW[n][k] = sum over active cells m of dY[m][n] X[m][k], with
// the bias gradient db[n] = sum_m dY[m][n] formed from the same staged tiles.
//
// The reduction runs over the cells (1.6 M at eval scale) while the output is one E x E tile
// of the weight, so the cells are split into chunks (split-K): workgroup (n-tile, k-tile, z)
// sums chunk z into a float32 partial, and a second kernel adds the partials in a fixed order
// (bitwise reproducible).  The MFMA contraction index is the cell, which is the slow index in
// memory for both operands, so 32-cell slices of dY and X are staged transposed in LDS
// ([n][cell] and [k][cell]); consecutive lanes take consecutive cells so that the transposed
// 16-bit writes of a wave fall on distinct banks.
#include "fast.h"
#include "mfma.h"

namespace tfm {

namespace {
constexpr int MS = 32;       // cells per MFMA step
constexpr int LS = MS + 8;   // LDS row stride (elements)
}  // namespace

// 512 threads = 8 waves in a 2 (n) x 4 (k) arrangement; tile BT x BT with BT = E.
template <int BT>
__global__ __launch_bounds__(512) void k_wgrad(WgradArgs a) {
  constexpr int NBW = BT / 32;   // 16-row blocks per wave along n (BT/2 rows)
  constexpr int KBW = BT / 64;   // 16-col blocks per wave along k (BT/4 cols)
  constexpr int CH = 4 * BT;     // 16-byte chunks per operand slice (MS x BT)
  constexpr int CPT = CH / 256;  // chunks per staging thread (256 threads per operand)
  __shared__ __attribute__((aligned(16))) bf16 As[2][BT * LS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BT * LS];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, lg = lane >> 4;
  const int wn = w >> 2, wk = w & 3;
  const int n0 = blockIdx.x * BT, k0 = blockIdx.y * BT;
  const int64_t mb = (int64_t)blockIdx.z * a.chunk;
  const int64_t me = mb + a.chunk < a.M ? mb + a.chunk : a.M;
  const Geo& g = a.g;

  // staging: threads 0-255 stage dY columns [n0, n0+BT), threads 256-511 stage X columns
  // [k0, k0+BT); chunk ch -> cell offset ch % 32, column block (ch / 32) * 8
  const int op = tid >> 8, st = tid & 255;
  const bf16* src = op == 0 ? a.dY : a.X;
  const int64_t ld = op == 0 ? a.ldy : a.ldx;
  const int mode = op == 0 ? a.ymode : a.xmode;
  const int cb = op == 0 ? n0 : k0;
  bf16* dst0 = op == 0 ? As[0] : Bs[0];
  bf16* dst1 = op == 0 ? As[1] : Bs[1];
  const bool bsum = op == 0 && a.bpart && blockIdx.y == 0;
  float csum[CPT][8];
#pragma unroll
  for (int i = 0; i < CPT; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) csum[i][j] = 0.f;

  uint4 r[CPT];
  auto gload = [&](int64_t m0) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int ch = st + 256 * i;
      const int64_t m = m0 + (ch & 31);
      const int col = cb + (ch >> 5) * 8;
      r[i] = make_uint4(0, 0, 0, 0);
      if (m < me) {
        if (mode == ROWS_ITEM_HM) {
          const int64_t gc = m / g.R;
          int part = 0;
          const int64_t off = item_hm_offset(g, gc, (int)(m - gc * g.R), col, &part);
          const bf16* base = part == 0 ? a.dY : (part == 1 ? a.dY2 : a.dY3);
          if (off >= 0) r[i] = ldu4(base + off);
        } else {
          const int64_t base = mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
          r[i] = ldu4(src + base + col);
        }
      }
    }
  };
  auto sstore = [&](int b) {
    bf16* d = b ? dst1 : dst0;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int ch = st + 256 * i;
      const int mm = ch & 31, cc = (ch >> 5) * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j) d[(cc + j) * LS + mm] = u4_elem(r[i], j);
      if (bsum) {
#pragma unroll
        for (int j = 0; j < 8; ++j) csum[i][j] += bf2f(u4_elem(r[i], j));
      }
    }
  };

  f32x4 acc[NBW][KBW];
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int j = 0; j < KBW; ++j) acc[i][j] = zero4();

  const int64_t steps = (me - mb + MS - 1) / MS;
  if (steps > 0) {
    gload(mb);
    sstore(0);
  }
  lds_barrier();
  for (int64_t s = 0; s < steps; ++s) {
    const int b = (int)(s & 1);
    if (s + 1 < steps) gload(mb + (s + 1) * MS);
    const bf16* A = b ? As[1] : As[0];
    const bf16* B = b ? Bs[1] : Bs[0];
    bf16x8 af[NBW], bfr[KBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i) af[i] = ld8(&A[(wn * (BT / 2) + i * 16 + c) * LS + lg * 8]);
#pragma unroll
    for (int j = 0; j < KBW; ++j) bfr[j] = ld8(&B[(wk * (BT / 4) + j * 16 + c) * LS + lg * 8]);
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < KBW; ++j) acc[i][j] = mfma16(af[i], bfr[j], acc[i][j]);
    if (s + 1 < steps) sstore(b ^ 1);
    lds_barrier();
  }

  // partial tile: lane holds rows n = wn*BT/2 + i*16 + 4*lg + q, column k = wk*BT/4 + j*16 + c
  float* out = a.part + (int64_t)blockIdx.z * a.N * a.K;
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + wn * (BT / 2) + i * 16 + lg * 4 + q;
#pragma unroll
      for (int j = 0; j < KBW; ++j) out[(int64_t)n * a.K + k0 + wk * (BT / 4) + j * 16 + c] = acc[i][j][q];
    }
  if (bsum) {
    // the 32 lanes of a half-wave share a column block; sum over them in a fixed pattern
#pragma unroll
    for (int i = 0; i < CPT; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float v = csum[i][j];
#pragma unroll
        for (int off = 1; off < 32; off <<= 1) v += __shfl_xor(v, off, 64);
        csum[i][j] = v;
      }
    if ((st & 31) == 0) {
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int ch = st + 256 * i;
        float* bp = a.bpart + (int64_t)blockIdx.z * a.N + n0 + (ch >> 5) * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) bp[j] = csum[i][j];
      }
    }
  }
}

// out[i] = (accumulate ? out[i] : 0) + sum over z in [z0, z1) of part[z * stride + i], with
// z0 = blockIdx.y * zc, z1 = min(Z, z0 + zc), and out advanced by blockIdx.y * out_ystride.  A
// block owns 32 groups of four consecutive outputs; 8 z-groups of threads each sum z = z0 + zg,
// z0 + zg + 8, ... with four independent accumulators, combined in a fixed order (bitwise
// reproducible).  out may be the first partial row of the block's own range (the first pass of
// a two-pass sum): every read of the range precedes the barrier, every write follows it, and no
// other block touches the range.
__global__ __launch_bounds__(256) void k_reduce_z(int Z, int zc, int64_t count, int64_t stride,
                                                  const float* part, float* out,
                                                  int64_t out_ystride, int accumulate) {
  __shared__ float4 red[8][32];
  const int o = threadIdx.x & 31, zg = threadIdx.x >> 5;
  const int64_t i4 = ((int64_t)blockIdx.x * 32 + o) * 4;
  const int z0 = (int)blockIdx.y * zc;
  const int z1 = z0 + zc < Z ? z0 + zc : Z;
  out += (int64_t)blockIdx.y * out_ystride;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i4 < count) {
    float4 a[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    const bool full = i4 + 4 <= count && (stride & 3) == 0;
    for (int z = z0 + zg; z < z1; z += 32) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int zz = z + 8 * u;
        if (zz < z1) {
          const float* p = part + (int64_t)zz * stride + i4;
          float4 v;
          if (full) {
            v = *reinterpret_cast<const float4*>(p);
          } else {
            v.x = p[0];
            v.y = i4 + 1 < count ? p[1] : 0.f;
            v.z = i4 + 2 < count ? p[2] : 0.f;
            v.w = i4 + 3 < count ? p[3] : 0.f;
          }
          a[u].x += v.x; a[u].y += v.y; a[u].z += v.z; a[u].w += v.w;
        }
      }
    }
    s.x = (a[0].x + a[1].x) + (a[2].x + a[3].x);
    s.y = (a[0].y + a[1].y) + (a[2].y + a[3].y);
    s.z = (a[0].z + a[1].z) + (a[2].z + a[3].z);
    s.w = (a[0].w + a[1].w) + (a[2].w + a[3].w);
  }
  red[zg][o] = s;
  __syncthreads();
  if (zg == 0 && i4 < count) {
    float4 t = red[0][o];
#pragma unroll
    for (int k = 1; k < 8; ++k) {
      t.x += red[k][o].x; t.y += red[k][o].y; t.z += red[k][o].z; t.w += red[k][o].w;
    }
    const float tv[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (i4 + k < count) out[i4 + k] = (accumulate ? out[i4 + k] : 0.f) + tv[k];
  }
}

int wgrad_chunks(int64_t M) {
  int64_t z = (M + WGRAD_CHUNK - 1) / WGRAD_CHUNK;
  return (int)(z < 1 ? 1 : z);
}

hipError_t launch_wgrad_mfma(const WgradArgs& a, hipStream_t s) {
  const int Z = wgrad_chunks(a.M);
  const int BT = a.g.E;
  if (a.N % BT || a.K % BT) return hipErrorInvalidValue;
  dim3 grid((unsigned)(a.N / BT), (unsigned)(a.K / BT), (unsigned)Z);
  WgradArgs b = a;
  b.chunk = WGRAD_CHUNK;
  switch (BT) {
    case 64: k_wgrad<64><<<grid, 512, 0, s>>>(b); break;
    case 128: k_wgrad<128><<<grid, 512, 0, s>>>(b); break;
    case 192: k_wgrad<192><<<grid, 512, 0, s>>>(b); break;
    case 256: k_wgrad<256><<<grid, 512, 0, s>>>(b); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_reduce_z(int Z, int64_t count, int64_t stride, float* part, float* out,
                           int accumulate, hipStream_t s) {
  if (Z <= 0 || count <= 0) return hipSuccess;
  const unsigned bx = (unsigned)((count + 127) / 128);
  // Few output blocks and many partials: first fold groups of ZC partials into the first row
  // of each group, leaving ceil(Z / ZC) partials ZC rows apart.
  constexpr int ZC = 64;
  if (bx < 512 && Z > 2 * ZC) {
    const unsigned groups = (unsigned)((Z + ZC - 1) / ZC);
    k_reduce_z<<<dim3(bx, groups), 256, 0, s>>>(Z, ZC, count, stride, part, part,
                                                 (int64_t)ZC * stride, 0);
    Z = (int)groups;
    stride *= ZC;
  }
  k_reduce_z<<<dim3(bx, 1), 256, 0, s>>>(Z, Z, count, stride, part, out, 0, accumulate);
  return hipGetLastError();
}

}  // namespace tfm
