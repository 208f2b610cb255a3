// The MLP half of the post-norm block in one kernel per direction, with the hidden layer kept in
// registers (paper Sec. 4.1 and the Fig. 3 caption: after the item-axis attention come a norm,
// the MLP and a norm).  Forward, per active cell:
//
//   z2  = O_i Wo_i^T + bo_i + (g1 xh1 + be1)      item out-projection + residual (H1 from x-hat1)
//   xh2 = (z2 - mean z2) rstd2                     LN2 (x-hat saved, its affine folded onward)
//   G   = xh2 W1'^T + b1'                          W1' = W1 diag(g2), b1' = b1 + W1 be2
//   z3  = GELU(G) W2^T + b2 + (g2 xh2 + be2)
//   xh3 = (z3 - mean z3) rstd3,  Y = g3 xh3 + be3  LN3
//
// Layout (v_mfma_f32_16x16x32_bf16; lane L = 16 g + c):
// * A workgroup is 4 waves, a wave owns 32 cells (two 16-cell blocks that share every weight
//   fragment read); every product is computed transposed,
//   out^T = W x^T, so the weights are the A operand (rows = output features) and the cells the
//   B operand: lane (g, c) holds 8 k values of cell c, and receives output features
//   16 b + 4 g .. + 3 of cell c.
// * The activations never leave registers between the products: two output blocks b, b + 1 of
//   a product give lane (g, c) the features {4 g .. + 3, 16 + 4 g .. + 3} of a 32-block, which
//   is a B fragment of the next product once its k positions are taken in that order; the
//   weights read in the next product carry the same permutation of their input columns
//   (applied when the weight stream is built), so no shuffle or LDS round trip is needed.
// * Weights stream from L2 through a 2-slot LDS ring (global_load_lds, 16 bytes per lane) in
//   stages of 2 E/16 fragments, each fragment 1 KB in lane order (one conflict-free 16-byte
//   read per lane): first Wo_i (two k steps per stage), then per 32 hidden units the 2 E/32
//   W1' fragments of the unit block pair and the E/16 W2 fragments of those units.
#include <math.h>

#include "fast.h"
#include "gelu.h"
#include "mfma.h"

namespace tfm {

namespace {

// k position of slot j (0..7) of lane group g in a B fragment that two D blocks form:
// values 4 g .. 4 g + 3 of the first block, then of the second (16 + ...).
__device__ __forceinline__ int perm_k(int g, int j) { return j < 4 ? 4 * g + j : 16 + 4 * g + (j - 4); }

__device__ __forceinline__ f32x4 unpack4(uint32_t lo, uint32_t hi) {
  f32x4 r;
  r[0] = __uint_as_float(lo << 16);
  r[1] = __uint_as_float(lo & 0xffff0000u);
  r[2] = __uint_as_float(hi << 16);
  r[3] = __uint_as_float(hi & 0xffff0000u);
  return r;
}

__device__ __forceinline__ f32x4 lds4(const float* p) {
  const float4 f = *reinterpret_cast<const float4*>(p);
  f32x4 r;
  r[0] = f.x; r[1] = f.y; r[2] = f.z; r[3] = f.w;
  return r;
}

__device__ __forceinline__ float sum4(const f32x4& v) { return (v[0] + v[1]) + (v[2] + v[3]); }

}  // namespace

// ----------------------------------------------------------------------------- weight stream
// One thread per bf16 element of the stream (see the file comment for the order).
__global__ void k_mlp_fwd_stream(const float* __restrict__ wo, const float* __restrict__ w1,
                                 const float* __restrict__ g2, const float* __restrict__ w2,
                                 int E, int H, bf16* __restrict__ out) {
  const int NE = E / 16, NK = E / 32, FPS = 2 * NE;  // fragments per stage
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)(NK / 2 + H / 32) * FPS * 512;
  if (t >= total) return;
  const int j = (int)(t & 7), lane = (int)((t >> 3) & 63);
  const int64_t f = t >> 9;  // fragment index in the stream
  const int st = (int)(f / FPS), fi = (int)(f % FPS);
  const int g = lane >> 4, r = lane & 15;
  float v;
  if (st < NK / 2) {  // Wo_i: rows = output features, k = input features (natural order)
    const int kk = fi / NE, eb = fi % NE;
    const int row = eb * 16 + r, k = (2 * st + kk) * 32 + 8 * g + j;
    v = wo[(int64_t)row * E + k];
  } else {
    const int c = st - NK / 2;
    if (fi < 2 * NK) {  // W1' = W1 diag(g2): rows = hidden units, k = features (permuted)
      const int hb = fi / NK, ks = fi % NK;
      const int row = c * 32 + hb * 16 + r, k = ks * 32 + perm_k(g, j);
      v = w1[(int64_t)row * E + k] * g2[k];
    } else {  // W2: rows = output features, k = the chunk's hidden units (permuted)
      const int eb = fi - 2 * NK;
      const int row = eb * 16 + r, k = c * 32 + perm_k(g, j);
      v = w2[(int64_t)row * H + k];
    }
  }
  out[t] = f2bf(v);
}

int64_t mlp_fwd_stream_elems(int E, int H) { return (int64_t)(E / 64 + H / 32) * (E / 8) * 512; }

hipError_t launch_mlp_fwd_stream(const float* wo, const float* w1, const float* g2,
                                 const float* w2, int E, int H, bf16* out, hipStream_t s) {
  const int64_t n = mlp_fwd_stream_elems(E, H);
  k_mlp_fwd_stream<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(wo, w1, g2, w2, E, H, out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------- forward
// A workgroup: NW waves of CB 16-cell blocks each (every weight fragment read from LDS feeds CB
// products), TILE = NW * CB * 16 cells.
constexpr int MLP_NW = 4, MLP_CB = 2, MLP_TILE = MLP_NW * MLP_CB * 16;

template <int E, int H>
__global__ __launch_bounds__(MLP_NW * 64, 2) void k_mlp_fwd(MlpFwdArgs a) {
  constexpr int NW = MLP_NW, CB = MLP_CB, NT = NW * 64;
  constexpr int NE = E / 16, NK = E / 32;  // 16-feature output blocks, 32-wide k steps
  constexpr int FPS = 2 * NE;              // fragments per stage
  constexpr int SEL = FPS * 512;           // elements per stage
  constexpr int NP1 = NK / 2;              // stages of the out-projection
  constexpr int NST = NP1 + H / 32;        // stages in all
  constexpr int DPT = FPS * 64 / NT;       // 16-byte DMA pieces per thread and stage
  static_assert(NK % 2 == 0 && H % 32 == 0 && DPT >= 1 && FPS * 64 % NT == 0, "shape");
  constexpr int NSLOT = 2;                 // LDS ring slots
  __shared__ __attribute__((aligned(16))) bf16 ring[NSLOT * SEL];
  // per-feature parameters: bo_i, g1, be1, g2, be2, b2, g3, be3; then b1' per hidden unit
  __shared__ __attribute__((aligned(16))) float pe[8][E];
  __shared__ __attribute__((aligned(16))) float pfb[H];

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int c = lane & 15, g = lane >> 4;
  const int64_t m0 = (int64_t)blockIdx.x * MLP_TILE;
  int64_t cell[CB], crow[CB];
  bool valid[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    cell[cb] = m0 + (w * CB + cb) * 16 + c;
    valid[cb] = cell[cb] < a.M;
    crow[cb] = valid[cb] ? cell[cb] : a.M - 1;  // past the end: read the last cell, store nothing
  }

  auto issue = [&](int st) {
    const bf16* src = a.ws + (int64_t)st * SEL;
    bf16* dst = ring + (st % NSLOT) * SEL;
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int piece = i * NT + w * 64;
      lds_dma16_s(src + piece * 8, (uint32_t)lane * 16, dst + piece * 8);
    }
  };
  issue(0);

  // activations of the out-projection: O_i as B fragments, the residual x-hat1 in the D layout
  bf16x8 ob[CB][NK];
  uint2 xr[CB][NE];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) ob[cb][ks] = ld8(a.oi + crow[cb] * E + ks * 32 + 8 * g);
#pragma unroll
    for (int eb = 0; eb < NE; ++eb)
      xr[cb][eb] = *reinterpret_cast<const uint2*>(a.xh1 + crow[cb] * E + eb * 16 + 4 * g);
  }
  for (int i = tid; i < E; i += NT) {
    pe[0][i] = a.bo[i]; pe[1][i] = a.g1[i]; pe[2][i] = a.be1[i]; pe[3][i] = a.g2[i];
    pe[4][i] = a.be2[i]; pe[5][i] = a.b2[i]; pe[6][i] = a.g3[i]; pe[7][i] = a.be3[i];
  }
  for (int i = tid; i < H; i += NT) pfb[i] = a.fb1[i];

  f32x4 acc[CB][NE];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) acc[cb][eb] = zero4();
  bf16x8 xf[CB][NK];  // x-hat2 as B fragments (k order perm_k within each 32-block)

  // Stage st waits for its own pieces (issued when stage st - 1 began), then the barrier
  // publishes every wave's pieces and frees the slot of stage st - 1, which stage st + 1 refills
  // while stage st computes.
  auto stage_begin = [&](int st) -> const bf16* {
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + 1 < NST) issue(st + 1);
    return ring + (st % NSLOT) * SEL + lane * 8;
  };

  // out-projection, two k steps per stage
#pragma unroll
  for (int st = 0; st < NP1; ++st) {
    const bf16* sl = stage_begin(st);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int eb = 0; eb < NE; ++eb) {
        const bf16x8 af = ld8(sl + (kk * NE + eb) * 512);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          acc[cb][eb] = mfma16(af, ob[cb][2 * st + kk], acc[cb][eb]);
      }
  }
  // z2 = acc + bo_i + g1 xh1 + be1, LN2 -> x-hat2 (saved, and the B fragments of W1')
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    float s = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const int e0 = eb * 16 + 4 * g;
      acc[cb][eb] += lds4(&pe[0][e0]) +
                     lds4(&pe[1][e0]) * unpack4(xr[cb][eb].x, xr[cb][eb].y) + lds4(&pe[2][e0]);
      s += sum4(acc[cb][eb]);
    }
    const float mean = rows4_sum(s) * (1.0f / E);
    float v = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      acc[cb][eb] -= mean;
      v += sum4(acc[cb][eb] * acc[cb][eb]);
    }
    const float rs = 1.0f / sqrtf(rows4_sum(v) * (1.0f / E) + 1e-5f);
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) {
      const f32x4 lo = acc[cb][2 * ks] * rs, hi = acc[cb][2 * ks + 1] * rs;
      uint4 u = make_uint4(pack2(lo[0], lo[1]), pack2(lo[2], lo[3]), pack2(hi[0], hi[1]),
                           pack2(hi[2], hi[3]));
      xf[cb][ks] = *reinterpret_cast<bf16x8*>(&u);
      if (valid[cb] && a.xh2) {
        bf16* row = a.xh2 + cell[cb] * E + ks * 32 + 4 * g;
        *reinterpret_cast<uint2*>(row) = make_uint2(u.x, u.y);
        *reinterpret_cast<uint2*>(row + 16) = make_uint2(u.z, u.w);
      }
    }
    if (valid[cb] && g == 0 && a.rs2) a.rs2[cell[cb]] = rs;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) acc[cb][eb] = zero4();  // now the down-projection sums
  }

  // hidden units [32 hc, 32 hc + 32): G^T = W1' xh2^T + b1', U = GELU(G), acc += W2 U^T
#pragma unroll 1
  for (int hc = 0; hc < H / 32; ++hc) {
    const bf16* sl = stage_begin(NP1 + hc);
    f32x4 gacc[CB][2];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) gacc[cb][0] = gacc[cb][1] = zero4();
#pragma unroll
    for (int ks = 0; ks < NK; ++ks)
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const bf16x8 af = ld8(sl + (hb * NK + ks) * 512);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) gacc[cb][hb] = mfma16(af, xf[cb][ks], gacc[cb][hb]);
      }
    bf16x8 uf[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      uint32_t up[4];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const int u0 = hc * 32 + hb * 16 + 4 * g;
        const f32x4 gv = gacc[cb][hb] + lds4(&pfb[u0]);
        f32x4 uv;
#pragma unroll
        for (int q = 0; q < 4; ++q) uv[q] = gelu_f(gv[q]);
        up[2 * hb] = pack2(uv[0], uv[1]);
        up[2 * hb + 1] = pack2(uv[2], uv[3]);
        if (valid[cb] && a.gout)
          *reinterpret_cast<uint2*>(a.gout + cell[cb] * H + u0) =
              make_uint2(pack2(gv[0], gv[1]), pack2(gv[2], gv[3]));
        if (valid[cb] && a.uout)
          *reinterpret_cast<uint2*>(a.uout + cell[cb] * H + u0) =
              make_uint2(up[2 * hb], up[2 * hb + 1]);
      }
      uint4 uu = make_uint4(up[0], up[1], up[2], up[3]);
      uf[cb] = *reinterpret_cast<bf16x8*>(&uu);
    }
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const bf16x8 af = ld8(sl + (2 * NK + eb) * 512);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[cb][eb] = mfma16(af, uf[cb], acc[cb][eb]);
    }
  }

  // z3 = acc + b2 + g2 xh2 + be2 (x-hat2 as rounded to bf16), LN3 -> x-hat3, Y = g3 xh3 + be3
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    float s = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const int e0 = eb * 16 + 4 * g;
      const uint4 u = *reinterpret_cast<const uint4*>(&xf[cb][eb / 2]);
      const f32x4 xv = (eb & 1) ? unpack4(u.z, u.w) : unpack4(u.x, u.y);
      acc[cb][eb] += lds4(&pe[5][e0]) + lds4(&pe[3][e0]) * xv + lds4(&pe[4][e0]);
      s += sum4(acc[cb][eb]);
    }
    const float mean = rows4_sum(s) * (1.0f / E);
    float v = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      acc[cb][eb] -= mean;
      v += sum4(acc[cb][eb] * acc[cb][eb]);
    }
    const float rs = 1.0f / sqrtf(rows4_sum(v) * (1.0f / E) + 1e-5f);
    if (!valid[cb]) continue;
    if (g == 0 && a.rs3) a.rs3[cell[cb]] = rs;
    bf16* yrow = a.y + native_cell(a.g, cell[cb]) * E;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const int e0 = eb * 16 + 4 * g;
      const f32x4 xh = acc[cb][eb] * rs;
      const f32x4 yv = lds4(&pe[6][e0]) * xh + lds4(&pe[7][e0]);
      *reinterpret_cast<uint2*>(yrow + e0) = make_uint2(pack2(yv[0], yv[1]), pack2(yv[2], yv[3]));
      if (a.xh3)
        *reinterpret_cast<uint2*>(a.xh3 + cell[cb] * E + e0) =
            make_uint2(pack2(xh[0], xh[1]), pack2(xh[2], xh[3]));
    }
  }
}

// ----------------------------------------------------------------------------- backward
// Backward of the same sub-block, from the native upstream gradient dY:
//
//   dz3 = rstd3 (g - mean g - xh3 mean(g xh3)),  g = dY g3         LN3'   (dz3 saved for dW2)
//   G   = xh2 W1'^T + b1' (recomputed),  U = GELU(G)               (U saved for dW2)
//   dG  = (dz3 W2) GELU'(G)                                        (saved for dW1, db1)
//   dh2 = dz3 + dG W1
//   dz2 = rstd2 (g - mean g - xh2 mean(g xh2)),  g = dh2 g2        LN2'
//
// plus per-tile column sums of dY xh3, dY (the LN3 weight and bias gradients) and dh2 xh2, dh2
// (LN2).  A workgroup is 12 waves of 16 cells; the inputs of a cell are loaded in the order that
// two D blocks give (features {4 g .. + 3, 16 + 4 g .. + 3} of each 32-block), which serves both
// as B fragments and as the per-feature operands of the norms.  Weight stream per 32 hidden
// units: W1' (units x features), W2^T (units x features), both with permuted feature columns,
// then W1^T (features x the chunk's units, permuted unit columns).
__global__ void k_mlp_bwd_stream(const float* __restrict__ w1, const float* __restrict__ g2,
                                 const float* __restrict__ w2, int E, int H,
                                 bf16* __restrict__ out) {
  const int NE = E / 16, NK = E / 32, FPS = 4 * NK + NE;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)(H / 32) * FPS * 512;
  if (t >= total) return;
  const int j = (int)(t & 7), lane = (int)((t >> 3) & 63);
  const int64_t f = t >> 9;
  const int c = (int)(f / FPS), fi = (int)(f % FPS);
  const int g = lane >> 4, r = lane & 15;
  float v;
  if (fi < 4 * NK) {
    const int part = fi / (2 * NK), hb = (fi % (2 * NK)) / NK, ks = fi % NK;
    const int u = c * 32 + hb * 16 + r, k = ks * 32 + perm_k(g, j);
    v = part == 0 ? w1[(int64_t)u * E + k] * g2[k] : w2[(int64_t)k * H + u];
  } else {
    const int eb = fi - 4 * NK;
    const int e = eb * 16 + r, u = c * 32 + perm_k(g, j);
    v = w1[(int64_t)u * E + e];
  }
  out[t] = f2bf(v);
}

int64_t mlp_bwd_stream_elems(int E, int H) { return (int64_t)(H / 32) * (3 * E / 16) * 512; }

hipError_t launch_mlp_bwd_stream(const float* w1, const float* g2, const float* w2, int E, int H,
                                 bf16* out, hipStream_t s) {
  const int64_t n = mlp_bwd_stream_elems(E, H);
  k_mlp_bwd_stream<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(w1, g2, w2, E, H, out);
  return hipGetLastError();
}

constexpr int MB_NW = 12, MB_TILE = MB_NW * 16;

int64_t mlp_bwd_tiles(int64_t M) { return (M + MB_TILE - 1) / MB_TILE; }

template <int E, int H>
__global__ __launch_bounds__(MB_NW * 64, 3) void k_mlp_bwd(MlpBwdArgs a) {
  constexpr int NW = MB_NW, NT = NW * 64;
  constexpr int NE = E / 16, NK = E / 32;
  constexpr int FPS = 4 * NK + NE;         // fragments per stage (one 32-unit chunk)
  constexpr int SEL = FPS * 512;
  constexpr int NST = H / 32;
  constexpr int DPT = FPS * 64 / NT;
  static_assert(H % 32 == 0 && DPT >= 1 && FPS * 64 % NT == 0, "shape");
  __shared__ __attribute__((aligned(16))) bf16 ring[3 * SEL];  // three stages: two in flight
  __shared__ __attribute__((aligned(16))) float pe[2][E];   // g3, g2
  __shared__ __attribute__((aligned(16))) float pfb[H];     // b1'

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int c = lane & 15, g = lane >> 4;
  const int64_t tile = blockIdx.x;
  const int64_t cell = tile * MB_TILE + w * 16 + c;
  const bool valid = cell < a.M;
  const int64_t crow = valid ? cell : a.M - 1;

  auto issue = [&](int st) {
    const bf16* src = a.ws + (int64_t)st * SEL;
    bf16* dst = ring + (st % 3) * SEL;
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int piece = i * NT + w * 64;
      lds_dma16_s(src + piece * 8, (uint32_t)lane * 16, dst + piece * 8);
    }
  };
  issue(0);
  issue(1);

  // the cell's inputs, features {32 ks + 4 g .. + 3} (h = 0) and {32 ks + 16 + 4 g .. + 3}
  uint2 dyl[NK][2], x3l[NK][2];
  {
    const bf16* dyr = a.dy + native_cell(a.g, crow) * E;
    const bf16* x3r = a.xh3 + crow * E;
#pragma unroll
    for (int ks = 0; ks < NK; ++ks)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e0 = ks * 32 + h * 16 + 4 * g;
        dyl[ks][h] = *reinterpret_cast<const uint2*>(dyr + e0);
        x3l[ks][h] = *reinterpret_cast<const uint2*>(x3r + e0);
      }
  }
  const float rs3 = valid ? a.rs3[crow] : 0.f, rs2 = valid ? a.rs2[crow] : 0.f;
  for (int i = tid; i < E; i += NT) {
    pe[0][i] = a.g3[i];
    pe[1][i] = a.g2[i];
  }
  for (int i = tid; i < H; i += NT) pfb[i] = a.fb1[i];
  __syncthreads();

  // column sums over the wave's 16 cells into red[w][which]: every lane of a 16-lane row ends
  // with the same sums and stores them (same address, same value)
  // [NW][2][E] per-wave sums: LN3's in the ring's third slot (free until the first stage
  // begins), LN2's in its first slot (after the last stage)
  float* red = reinterpret_cast<float*>(ring + 2 * SEL);
  float* red2 = reinterpret_cast<float*>(ring);
  static_assert(NW * 2 * E * 4 <= SEL * 2, "column sums fit a ring slot");
  auto colsum = [&](int which, int eb, f32x4 v) {
    f32x4 t;
#pragma unroll
    for (int q = 0; q < 4; ++q) t[q] = row16_sum(v[q]);
    float* dst = which < 2 ? red + (w * 2 + which) * E : red2 + (w * 2 + which - 2) * E;
    *reinterpret_cast<f32x4*>(dst + eb * 16 + 4 * g) = t;
  };
  // the tile's sums of one norm (waves added in order) -> part[tile][off .. off + 2E)
  auto flush = [&](const float* src, int off) {
    __syncthreads();
    for (int i = tid; i < 2 * E; i += NT) {
      float sm = 0.f;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) sm += src[ww * 2 * E + i];
      a.part[tile * 4 * E + off + i] = sm;
    }
  };

  // LN3': dz3 = rs3 (dY g3 - mean(dY g3) - xh3 mean(dY g3 xh3)); invalid cells contribute 0
  // (their dY is scaled by 0, without a branch)
  const float vmask = valid ? 1.f : 0.f;
  bf16x8 dzf[NK];
  {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const int ks = eb >> 1, h = eb & 1;
      const f32x4 dy = unpack4(dyl[ks][h].x, dyl[ks][h].y) * vmask;
      const f32x4 x3 = unpack4(x3l[ks][h].x, x3l[ks][h].y);
      const f32x4 gy = dy * lds4(&pe[0][eb * 16 + 4 * g]);
      s1 += sum4(gy);
      s2 += sum4(gy * x3);
      colsum(0, eb, dy * x3);
      colsum(1, eb, dy);
    }
    const float m1 = rows4_sum(s1) * (1.0f / E), m2 = rows4_sum(s2) * (1.0f / E);
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) {
      uint32_t pk[4];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int eb = 2 * ks + h;
        const f32x4 dy = unpack4(dyl[ks][h].x, dyl[ks][h].y) * vmask;
        const f32x4 x3 = unpack4(x3l[ks][h].x, x3l[ks][h].y);
        const f32x4 dz = rs3 * (dy * lds4(&pe[0][eb * 16 + 4 * g]) - m1 - x3 * m2);
        pk[2 * h] = pack2(dz[0], dz[1]);
        pk[2 * h + 1] = pack2(dz[2], dz[3]);
        if (valid)
          *reinterpret_cast<uint2*>(a.dz3 + cell * E + ks * 32 + h * 16 + 4 * g) =
              make_uint2(pk[2 * h], pk[2 * h + 1]);
      }
      uint4 u = make_uint4(pk[0], pk[1], pk[2], pk[3]);
      dzf[ks] = *reinterpret_cast<bf16x8*>(&u);
    }
  }
  flush(red, 0);
  // x-hat2 as B fragments (loaded once LN3' no longer holds its inputs)
  bf16x8 xf[NK];
#pragma unroll
  for (int ks = 0; ks < NK; ++ks) {
    const bf16* x2r = a.xh2 + crow * E + ks * 32 + 4 * g;
    const uint2 lo = *reinterpret_cast<const uint2*>(x2r);
    const uint2 hi = *reinterpret_cast<const uint2*>(x2r + 16);
    uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
    xf[ks] = *reinterpret_cast<bf16x8*>(&u);
  }

  // Stage st waits for its own pieces only: loads complete in issue order, so with the DPT
  // pieces of stage st + 1 issued after them, at most DPT outstanding vector-memory operations
  // means stage st has landed (stores in flight do not change that).  The barrier publishes
  // every wave's pieces and frees the slot of stage st - 1, which stage st + 2 then refills.
  auto stage_begin = [&](int st) -> const bf16* {
    if (st + 1 < NST)
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(DPT) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + 2 < NST) issue(st + 2);
    return ring + (st % 3) * SEL + lane * 8;
  };

  // dh2 = dz3 (as rounded to bf16) + dG W1, features 16 eb + 4 g .. + 3 of the lane's cell:
  // seeded with dz3 so that the fragments of dz3 are dead after the loop
  f32x4 acc[NE];
#pragma unroll
  for (int eb = 0; eb < NE; ++eb) {
    const uint4 dzu = *reinterpret_cast<const uint4*>(&dzf[eb >> 1]);
    acc[eb] = (eb & 1) ? unpack4(dzu.z, dzu.w) : unpack4(dzu.x, dzu.y);
  }
#pragma unroll 1
  for (int hc = 0; hc < NST; ++hc) {
    const bf16* sl = stage_begin(hc);
    f32x4 gacc[2] = {zero4(), zero4()}, dacc[2] = {zero4(), zero4()};
#pragma unroll
    for (int ks = 0; ks < NK; ++ks)
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        gacc[hb] = mfma16(ld8(sl + (hb * NK + ks) * 512), xf[ks], gacc[hb]);
        dacc[hb] = mfma16(ld8(sl + ((2 + hb) * NK + ks) * 512), dzf[ks], dacc[hb]);
      }
    uint32_t dp[4];
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const int u0 = hc * 32 + hb * 16 + 4 * g;
      const f32x4 gv = gacc[hb] + lds4(&pfb[u0]);
      f32x4 uv, dv;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float e;
        const float cdf = norm_cdf(gv[q], &e);
        uv[q] = gv[q] * cdf;
        dv[q] = dacc[hb][q] * fmaf(gv[q] * 0.39894228040143268f, e, cdf);
      }
      dp[2 * hb] = pack2(dv[0], dv[1]);
      dp[2 * hb + 1] = pack2(dv[2], dv[3]);
      if (valid) {
        *reinterpret_cast<uint2*>(a.u + cell * H + u0) =
            make_uint2(pack2(uv[0], uv[1]), pack2(uv[2], uv[3]));
        *reinterpret_cast<uint2*>(a.dg + cell * H + u0) = make_uint2(dp[2 * hb], dp[2 * hb + 1]);
      }
    }
    uint4 du = make_uint4(dp[0], dp[1], dp[2], dp[3]);
    const bf16x8 dgf = *reinterpret_cast<bf16x8*>(&du);
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) acc[eb] = mfma16(ld8(sl + (4 * NK + eb) * 512), dgf, acc[eb]);
  }

  // LN2': dz2 = rs2 (g - mean g - xh2 mean(g xh2)), g = dh2 g2
  __syncthreads();  // every wave is done with the ring
  {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const uint4 xu = *reinterpret_cast<const uint4*>(&xf[eb >> 1]);
      const f32x4 x2 = (eb & 1) ? unpack4(xu.z, xu.w) : unpack4(xu.x, xu.y);
      const f32x4 dh = valid ? acc[eb] : zero4();
      const f32x4 gg = acc[eb] * lds4(&pe[1][eb * 16 + 4 * g]);
      s1 += sum4(gg);
      s2 += sum4(gg * x2);
      colsum(2, eb, dh * x2);
      colsum(3, eb, dh);
    }
    const float m1 = rows4_sum(s1) * (1.0f / E), m2 = rows4_sum(s2) * (1.0f / E);
#pragma unroll
    for (int eb = 0; eb < NE; ++eb) {
      const uint4 xu = *reinterpret_cast<const uint4*>(&xf[eb >> 1]);
      const f32x4 x2 = (eb & 1) ? unpack4(xu.z, xu.w) : unpack4(xu.x, xu.y);
      const f32x4 dz = rs2 * (acc[eb] * lds4(&pe[1][eb * 16 + 4 * g]) - m1 - x2 * m2);
      if (valid)
        *reinterpret_cast<uint2*>(a.dz2 + cell * E + eb * 16 + 4 * g) =
            make_uint2(pack2(dz[0], dz[1]), pack2(dz[2], dz[3]));
    }
  }
  flush(red2, 2 * E);
}

hipError_t launch_mlp_bwd(const MlpBwdArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const unsigned grid = (unsigned)mlp_bwd_tiles(a.M);
  if (a.g.E == 192 && a.g.H == 384)
    k_mlp_bwd<192, 384><<<grid, MB_NW * 64, 0, s>>>(a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

bool mlp_fused_ok(int E, int H) { return E == 192 && H == 384; }

hipError_t launch_mlp_fwd(const MlpFwdArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((a.M + MLP_TILE - 1) / MLP_TILE);
  if (a.g.E == 192 && a.g.H == 384)
    k_mlp_fwd<192, 384><<<grid, MLP_NW * 64, 0, s>>>(a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tfm
