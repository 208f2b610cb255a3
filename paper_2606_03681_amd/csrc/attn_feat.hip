// Feature-axis attention on bf16 MFMA: within each row (b, r), every active cell attends to
// every active cell of that row, per head.  S_b <= 128 active cells per row.
//
// One wave owns one (row, head) pair.  The cells of row (b, r) are the compact cells
// p = (col0 + k) * R + r, so they are R * 3E elements apart in the Q|K|V buffer; a buffer
// resource based at the row's first cell with S_b cells in range returns zeros past the last
// active cell, which pads the cell count to whole 16-cell MFMA blocks.  Every operand fragment
// of the pair is loaded once, at the start (a single memory round trip per wave); the operands
// whose contraction runs over cells are written from those registers into row-major LDS tiles
// and read back transposed.
//
// Forward, per 16-query block: S^T = K Q^T (keys x queries), a softmax over all keys at once
// (no online rescaling: the row fits), and O^T = V^T P^T with V in the wave's LDS.
//
// Backward, two sweeps (probabilities recomputed from the saved log-sum-exp):
//   query-major:  dS^T = P^T (dP^T - D),  dQ^T = K^T dS^T             (K in LDS)
//   key-major:    dS = P (dP - D),  dV^T += dO^T P,  dK^T += Q^T dS    (Q, dO in LDS)
// so that every product's fragment comes from the lane's own registers or a transposed LDS
// read.
#include <math.h>

#include "attn.h"
#include "attn_frag.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr float LOG2E = 1.4426950408889634f;

// Makes this wave's LDS writes visible to its own later LDS reads (no workgroup barrier: each
// wave owns its LDS region).
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ bf16x8 pack8(const f32x4& a, const f32x4& b) {
  uint4 u = make_uint4(pack2(a[0], a[1]), pack2(a[2], a[3]), pack2(b[0], b[1]),
                       pack2(b[2], b[3]));
  return *reinterpret_cast<bf16x8*>(&u);
}

// Row (b, r) and head of the pair handled by this wave; false if past the last pair.
struct Pair {
  int64_t cell0;   // compact cell of the row's first active column
  int S;           // active cells of the row
  int head;
};

__device__ __forceinline__ bool pair_of(const Geo& g, int64_t t, Pair& p) {
  if (t >= (int64_t)g.B * g.R * g.heads) return false;
  p.head = (int)(t % g.heads);
  const int64_t rho = t / g.heads;
  const int b = (int)(rho / g.R), r = (int)(rho % g.R);
  const DsInfo di = g.ds[b];
  p.S = di.S;
  p.cell0 = (int64_t)di.col0 * g.R + r;
  return true;
}

// Row-major [cell][d] LDS tiles, read back transposed by ds_read_b64_tr_b16 (lds_read_tr16).
// A transposed read lets every lane of a 32-lane half name 8 bytes of rows r .. r + 7 at one
// 32-byte column chunk; rows are d * 2 bytes long with no padding, and the 32-byte chunks of
// row r are XOR-rotated so that those 8 rows land on 8 distinct groups of 8 banks:
//   d = 16: one chunk per row, rows 8 apart already distinct;
//   d = 32: chunk ^ ((r >> 2) & 1)   (rows r and r + 4 share banks otherwise);
//   d = 64: chunk ^ ((r >> 1) & 3)   (rows r, r + 2, r + 4, r + 6 share banks otherwise).
template <int D>
__device__ __forceinline__ int chunk_swz(int r) {
  return D == 16 ? 0 : (D == 32 ? (r >> 2) & 1 : (r >> 1) & 3);
}

// Store the row-role fragments fr[kb] (lane (lg, c): cell kb*16 + c, the HF<D> dims of lg) of
// the first nks 16-cell blocks into the row-major tile.
template <int D, int NKB>
__device__ __forceinline__ void put_rows(const typename HF<D>::frag* fr, int nks, int c, int lg,
                                         bf16* tile) {
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
    if (kb < nks) {
      const int r = kb * 16 + c;
      bf16* row = tile + r * D;
      const int z = chunk_swz<D>(r);
      if constexpr (D == 16) {
        *reinterpret_cast<uint2*>(row + 4 * lg) = *reinterpret_cast<const uint2*>(&fr[kb]);
      } else if constexpr (D == 32) {
        *reinterpret_cast<uint4*>(row + ((lg >> 1) ^ z) * 16 + (lg & 1) * 8) =
            *reinterpret_cast<const uint4*>(&fr[kb]);
      } else {
        *reinterpret_cast<uint4*>(row + ((lg >> 1) ^ z) * 16 + (lg & 1) * 8) =
            *reinterpret_cast<const uint4*>(&fr[kb].lo);
        *reinterpret_cast<uint4*>(row + ((2 + (lg >> 1)) ^ z) * 16 + (lg & 1) * 8) =
            *reinterpret_cast<const uint4*>(&fr[kb].hi);
      }
    }
}

// MFMA operand whose k positions run down the tile's cells: lane (g, c) receives dim
// db*16 + c of cells 32 ks + {4g .. 4g+3} (slots 0-3) and 32 ks + 16 + {4g .. 4g+3} (slots
// 4-7), the k order of two packed 16-cell score blocks (pack8).
template <int D>
__device__ __forceinline__ bf16x8 get_cols(const bf16* tile, int ks, int db, int lane) {
  const int r = ks * 32 + (lane >> 2);
  const bf16* p = tile + r * D + ((db ^ chunk_swz<D>(r)) * 16) + 4 * (lane & 3);
  const bf16x4 lo = lds_read_tr16(p), hi = lds_read_tr16(p + 16 * D);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

}  // namespace

// ================================================================================ forward
template <int D, int SM>
__global__ __launch_bounds__(256, D <= 32 ? 4 : 1) void k_feat_attn_fwd(Geo g, const bf16* __restrict__ qkv,
                                                       bf16* __restrict__ o,
                                                       float* __restrict__ lse) {
  constexpr int DB = D / 16;
  constexpr int NKB = SM / 16;   // 16-cell blocks of the longest row handled
  __shared__ __attribute__((aligned(16))) bf16 Vs[4][SM * D];  // per wave: V, [cell][d]
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = lane & 15, lg = lane >> 4;
  Pair pr;
  if (!pair_of(g, (int64_t)blockIdx.x * 4 + w, pr)) return;
  const int E = g.E, S = pr.S;
  const int nkb = (S + 15) / 16;
  const uint32_t cs = (uint32_t)g.R * 3 * E * 2;  // bytes between cells of the row
  const rsrc_t rq = make_rsrc(qkv + pr.cell0 * 3 * E, (uint32_t)(S - 1) * cs + 3 * E * 2);
  const uint32_t oq = pr.head * D * 2, ok = (E + pr.head * D) * 2, ov = (2 * E + pr.head * D) * 2;
  const float c2 = LOG2E / sqrtf((float)D);

  bf16* vt = Vs[w];
  const int nks = (nkb + 1) & ~1;  // staged blocks: whole pairs of 16-cell blocks
  typedef typename HF<D>::frag frag;
  frag kf[NKB], qf[NKB];
  {
    frag vf[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
      if (kb < nks) {
        const uint32_t row = (uint32_t)(kb * 16 + c) * cs;
        kf[kb] = HF<D>::buf(rq, row + ok, lg);
        vf[kb] = HF<D>::buf(rq, row + ov, lg);
        qf[kb] = HF<D>::buf(rq, row + oq, lg);
      }
    put_rows<D, NKB>(vf, nks, c, lg, vt);
  }
  wave_lds_sync();

  const uint32_t ocs = (uint32_t)g.R * E * 2;  // bytes between cells in O
  bf16* orow = o + pr.cell0 * E + pr.head * D;
  float* lrow = lse + pr.cell0 * g.heads + pr.head;
#pragma unroll
  for (int qb = 0; qb < NKB; ++qb) {
    if (qb >= nkb) break;
    f32x4 s[NKB];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      if (kb < nkb) {
        s[kb] = HF<D>::mma(kf[kb], qf[qb]);
        if (kb == nkb - 1) {  // keys past the row's last cell (only the last block has any)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (kb * 16 + lg * 4 + i >= S) s[kb][i] = -INFINITY;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[kb][i]);
      }
    }
    mx = rows4_max(mx);
    const float mb = -mx * c2;
    float l = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
      if (kb < nkb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s[kb][i] = exp2_hw(fmaf(s[kb][i], c2, mb));
          l += s[kb][i];
        }
      } else {
        s[kb] = zero4();
      }
    l = rows4_sum(l);
    f32x4 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = zero4();
#pragma unroll
    for (int ks = 0; ks < NKB / 2; ++ks) {
      if (2 * ks < nkb) {
        const bf16x8 pf = pack8(s[2 * ks], s[2 * ks + 1]);
#pragma unroll
        for (int db = 0; db < DB; ++db)
          oacc[db] = mfma16(get_cols<D>(vt, ks, db, lane), pf, oacc[db]);
      }
    }
    const int qq = qb * 16 + c;
    if (qq < S) {
      const float inv = 1.0f / l;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint2 u = make_uint2(pack2(oacc[db][0] * inv, oacc[db][1] * inv),
                                   pack2(oacc[db][2] * inv, oacc[db][3] * inv));
        *reinterpret_cast<uint2*>((char*)orow + (uint64_t)qq * ocs + (db * 16 + lg * 4) * 2) = u;
      }
      if (lg == 0) lrow[(int64_t)qq * g.R * g.heads] = mx / sqrtf((float)D) + logf(l);
    }
  }
}

// ================================================================================ backward
template <int D, int SM>
__global__ __launch_bounds__(256) void k_feat_attn_bwd(Geo g, const bf16* __restrict__ qkv,
                                                       const bf16* __restrict__ o,
                                                       const bf16* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       bf16* __restrict__ dqkv) {
  constexpr int DB = D / 16;
  constexpr int NKB = SM / 16;   // 16-cell blocks of the longest row handled
  // per wave, [cell][d] tiles: sweep 1 uses the first for K; sweep 2 holds Q and dO
  __shared__ __attribute__((aligned(16))) bf16 T[4][2 * SM * D];
  __shared__ __attribute__((aligned(16))) float Lr[4][SM];
  __shared__ __attribute__((aligned(16))) float Dr[4][SM];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = lane & 15, lg = lane >> 4;
  Pair pr;
  if (!pair_of(g, (int64_t)blockIdx.x * 4 + w, pr)) return;
  const int E = g.E, S = pr.S;
  const int nkb = (S + 15) / 16;
  const uint32_t cs = (uint32_t)g.R * 3 * E * 2;  // Q|K|V cell stride (bytes)
  const uint32_t ecs = (uint32_t)g.R * E * 2;     // O / dO cell stride (bytes)
  const rsrc_t rq = make_rsrc(qkv + pr.cell0 * 3 * E, (uint32_t)(S - 1) * cs + 3 * E * 2);
  const rsrc_t ro = make_rsrc(o + pr.cell0 * E, (uint32_t)(S - 1) * ecs + E * 2);
  const rsrc_t rdo = make_rsrc(dout + pr.cell0 * E, (uint32_t)(S - 1) * ecs + E * 2);
  const uint32_t hq = pr.head * D * 2, hk = (E + pr.head * D) * 2, hv = (2 * E + pr.head * D) * 2;
  const float c2 = LOG2E / sqrtf((float)D);
  const float tau = 1.0f / sqrtf((float)D);
  bf16* t0 = T[w];
  bf16* t1 = T[w] + SM * D;
  bf16* drow = dqkv + pr.cell0 * 3 * E + pr.head * D;
  const uint64_t dcs = (uint64_t)g.R * 3 * E;  // elements between cells in dQKV

  // every fragment of the pair in the row role (lane: cell kb*16 + c), loaded up front
  typedef typename HF<D>::frag frag;
  const int nks = (nkb + 1) & ~1;  // staged blocks: whole pairs of 16-cell blocks
  frag kf[NKB], vf[NKB], qf[NKB], df[NKB];
  float nbq[NKB], dq[NKB];  // per query kb*16 + c: -lse * log2(e) and D = rowsum(dO * O)
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
    if (kb < nks) {
      const uint32_t rr = (uint32_t)(kb * 16 + c);
      kf[kb] = HF<D>::buf(rq, rr * cs + hk, lg);
      vf[kb] = HF<D>::buf(rq, rr * cs + hv, lg);
      qf[kb] = HF<D>::buf(rq, rr * cs + hq, lg);
      df[kb] = HF<D>::buf(rdo, rr * ecs + hq, lg);
      dq[kb] = hf_dot<D>(df[kb], HF<D>::buf(ro, rr * ecs + hq, lg));
      nbq[kb] = (int)rr < S ? -lse[(pr.cell0 + (int64_t)rr * g.R) * g.heads + pr.head] * LOG2E
                            : 0.f;
    }
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
    if (kb < nks) {
      dq[kb] = rows4_sum(dq[kb]);
      if (lg == 0) {
        Lr[w][kb * 16 + c] = nbq[kb];
        Dr[w][kb * 16 + c] = dq[kb];
      }
    }
  put_rows<D, NKB>(kf, nks, c, lg, t0);  // K
  wave_lds_sync();

  // ---- sweep 1 (query-major): dQ^T = K^T dS^T, one pair of key blocks (32 keys) at a time
#pragma unroll
  for (int qb = 0; qb < NKB; ++qb) {
    if (qb >= nkb) break;
    const int qq = qb * 16 + c;
    f32x4 acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = zero4();
#pragma unroll
    for (int ks = 0; ks < NKB / 2; ++ks) {
      if (2 * ks >= nkb) break;
      f32x4 ds[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int kb = 2 * ks + h;
        if (kb < nkb) {
          const f32x4 s = HF<D>::mma(kf[kb], qf[qb]);
          const f32x4 dp = HF<D>::mma(vf[kb], df[qb]);
          f32x4 p;
#pragma unroll
          for (int i = 0; i < 4; ++i) p[i] = exp2_hw(fmaf(s[i], c2, nbq[qb]));
          if (kb == nkb - 1) {  // keys past the row's last cell
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (kb * 16 + lg * 4 + i >= S) p[i] = 0.f;
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) ds[h][i] = p[i] * (dp[i] - dq[qb]);
        } else {
          ds[h] = zero4();
        }
      }
      const bf16x8 sf = pack8(ds[0], ds[1]);
#pragma unroll
      for (int db = 0; db < DB; ++db)
        acc[db] = mfma16(get_cols<D>(t0, ks, db, lane), sf, acc[db]);
    }
    if (qq < S) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint2 u = make_uint2(pack2(acc[db][0] * tau, acc[db][1] * tau),
                                   pack2(acc[db][2] * tau, acc[db][3] * tau));
        *reinterpret_cast<uint2*>(drow + qq * dcs + db * 16 + lg * 4) = u;
      }
    }
  }
  wave_lds_sync();
  // ---- sweep 2 (key-major): dV^T += dO^T P, dK^T += Q^T dS over all query blocks
  put_rows<D, NKB>(qf, nks, c, lg, t0);  // Q
  put_rows<D, NKB>(df, nks, c, lg, t1);  // dO
  wave_lds_sync();
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb) {
    if (kb >= nkb) break;
    f32x4 dvt[DB], dkt[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) dvt[db] = dkt[db] = zero4();
#pragma unroll
    for (int ks = 0; ks < NKB / 2; ++ks) {
      if (2 * ks < nkb) {
        f32x4 p[2], dsv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int qb = 2 * ks + h;
          const f32x4 s = HF<D>::mma(qf[qb], kf[kb]);
          const f32x4 dp = HF<D>::mma(df[qb], vf[kb]);
          const float4 l4 = *reinterpret_cast<const float4*>(&Lr[w][qb * 16 + lg * 4]);
          const float4 d4 = *reinterpret_cast<const float4*>(&Dr[w][qb * 16 + lg * 4]);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) p[h][i] = exp2_hw(fmaf(s[i], c2, lv[i]));
          if (qb >= nkb - 1) {  // queries past the row's last cell (and the zero block after)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (qb * 16 + lg * 4 + i >= S) p[h][i] = 0.f;
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) dsv[h][i] = p[h][i] * (dp[i] - dv4[i]);
        }
        const bf16x8 pf = pack8(p[0], p[1]);
        const bf16x8 sf = pack8(dsv[0], dsv[1]);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dvt[db] = mfma16(get_cols<D>(t1, ks, db, lane), pf, dvt[db]);
          dkt[db] = mfma16(get_cols<D>(t0, ks, db, lane), sf, dkt[db]);
        }
      }
    }
    const int kk = kb * 16 + c;
    if (kk < S) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint2 uk = make_uint2(pack2(dkt[db][0] * tau, dkt[db][1] * tau),
                                    pack2(dkt[db][2] * tau, dkt[db][3] * tau));
        const uint2 uv = make_uint2(pack2(dvt[db][0], dvt[db][1]), pack2(dvt[db][2], dvt[db][3]));
        *reinterpret_cast<uint2*>(drow + kk * dcs + E + db * 16 + lg * 4) = uk;
        *reinterpret_cast<uint2*>(drow + kk * dcs + 2 * E + db * 16 + lg * 4) = uv;
      }
    }
  }
}

// Longest row (cells) handled by the MFMA kernels for head dim d: all of a pair's fragments
// stay in registers, four arrays of them in the backward pass.
static int feat_attn_smax(int d) { return d == 64 ? 64 : 128; }

bool feat_attn_mfma_ok(const Geo& g) {
  return (g.d == 16 || g.d == 32 || g.d == 64) && g.S <= feat_attn_smax(g.d) &&
         (int64_t)g.R * g.S * 3 * g.E * 2 < (int64_t(1) << 31);
}

template <int D>
static hipError_t feat_fwd_d(const Geo& g, unsigned grid, const bf16* qkv, bf16* o, float* lse,
                             hipStream_t s) {
  if (g.S <= 32)
    k_feat_attn_fwd<D, 32><<<grid, 256, 0, s>>>(g, qkv, o, lse);
  else if (g.S <= 64)
    k_feat_attn_fwd<D, 64><<<grid, 256, 0, s>>>(g, qkv, o, lse);
  else if (D < 64)
    k_feat_attn_fwd<D, (D < 64 ? 128 : 64)><<<grid, 256, 0, s>>>(g, qkv, o, lse);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int D>
static hipError_t feat_bwd_d(const Geo& g, unsigned grid, const bf16* qkv, const bf16* o,
                             const bf16* dout, const float* lse, bf16* dqkv, hipStream_t s) {
  if (g.S <= 32)
    k_feat_attn_bwd<D, 32><<<grid, 256, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  else if (g.S <= 64)
    k_feat_attn_bwd<D, 64><<<grid, 256, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  else if (D < 64)
    k_feat_attn_bwd<D, (D < 64 ? 128 : 64)><<<grid, 256, 0, s>>>(g, qkv, o, dout, lse, dqkv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_feat_attn_fwd(const Geo& g, const bf16* qkv, bf16* o, float* lse,
                                hipStream_t s) {
  if (!feat_attn_mfma_ok(g)) return hipErrorInvalidValue;
  const int64_t pairs = (int64_t)g.B * g.R * g.heads;
  const unsigned grid = (unsigned)((pairs + 3) / 4);
  if (g.d == 16) return feat_fwd_d<16>(g, grid, qkv, o, lse, s);
  if (g.d == 32) return feat_fwd_d<32>(g, grid, qkv, o, lse, s);
  return feat_fwd_d<64>(g, grid, qkv, o, lse, s);
}

hipError_t launch_feat_attn_bwd(const Geo& g, const bf16* qkv, const bf16* o, const bf16* dout,
                                const float* lse, bf16* dqkv, hipStream_t s) {
  if (!feat_attn_mfma_ok(g)) return hipErrorInvalidValue;
  const int64_t pairs = (int64_t)g.B * g.R * g.heads;
  const unsigned grid = (unsigned)((pairs + 3) / 4);
  if (g.d == 16) return feat_bwd_d<16>(g, grid, qkv, o, dout, lse, dqkv, s);
  if (g.d == 32) return feat_bwd_d<32>(g, grid, qkv, o, dout, lse, dqkv, s);
  return feat_bwd_d<64>(g, grid, qkv, o, dout, lse, dqkv, s);
}

}  // namespace tfm
