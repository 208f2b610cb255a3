// Item-axis flash attention on bf16 MFMA, backward pass, as two kernels that each recompute
// the probabilities from the saved log-sum-exp:
//
//   dQ kernel first (query-major, shaped like the forward pass): a workgroup owns 128 query
//     rows (4 waves x 32) and streams the train prefix in key tiles of 64 through LDS:
//       S^T = K Q^T, dP^T = V dO^T        (a lane holds 4 keys of one query)
//       dS^T = P^T (dP^T - D),  dQ^T += K^T dS^T,  D = rowsum(dO o O) also written out
//
//   dK/dV kernel (key-major): a workgroup owns 128 train rows (4 waves x 32 keys) of one
//     problem and streams all query rows (Q, dO, D, lse) in chunks of 64 through LDS:
//       S = Q K^T, dP = dO V^T            (D tiles: a lane holds 4 queries of one key)
//       P = exp2(S tau log2e - lse log2e),  dS = P (dP - D)
//       dV^T += dO^T P,  dK^T += Q^T dS   (the S-layout tiles are used directly as B operands)
//
// K arrives pre-multiplied by log2(e)/sqrt(d) (see the item Q|K|V projection), so Q K^T is in
// the exp2 domain.  The S accumulators start at -lse log2(e) and the dP accumulators at -D, so
// the MFMA returns the exponent of P and dP - D directly: P = exp2(acc), dS = P (dP - D).
//
// Both accumulate in registers only, so each output element is summed in a fixed order
// (bitwise reproducible), and neither needs more than ~30 KB of LDS, which keeps several
// workgroups resident per CU.  Tiles are staged row-major with 16-byte stores; the
// transposed operands (Q^T, dO^T, K^T) come from LDS transpose reads.  Workgroups of one
// problem are numbered onto the same XCD.
#include <math.h>

#include <type_traits>

#include "attn.h"
#include "attn_frag.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr float LOG2E = 1.4426950408889634f;
__device__ __forceinline__ bf16x8 cat8(uint2 lo, uint2 hi) {
  uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  return *reinterpret_cast<bf16x8*>(&u);
}

// Makes this wave's LDS writes visible to its own later LDS reads (and its reads complete before
// it overwrites what they read); no workgroup barrier.
__device__ __forceinline__ void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ bf16x8 pack8(const f32x4& a, const f32x4& b) {
  uint4 u = make_uint4(pack2(a[0], a[1]), pack2(a[2], a[3]), pack2(b[0], b[1]),
                       pack2(b[2], b[3]));
  return *reinterpret_cast<bf16x8*>(&u);
}

}  // namespace

// =============================================================================== dK / dV
template <int D>
__global__ __launch_bounds__(256) void k_item_attn_dkdv(Geo g, const bf16* __restrict__ q,
                                                        const bf16* __restrict__ k,
                                                        const bf16* __restrict__ v,
                                                        const bf16* __restrict__ o,
                                                        const bf16* __restrict__ dout,
                                                        const float* __restrict__ lse,
                                                        const float* __restrict__ Dbuf,
                                                        bf16* __restrict__ dk,
                                                        bf16* __restrict__ dv, int KT,
                                                        ColList cl) {
  constexpr int QC = 64;          // queries per chunk
  constexpr int KW = 32;          // keys per wave (two 16-key blocks)
  constexpr int DB = D / 16;
  constexpr int CPR = D / 8;      // 16-byte chunks per row of d values
  constexpr int NIT = QC * CPR / 128;  // staging items per thread (128 threads per tensor)
  constexpr int RS = tr_stride<D>();  // LDS row stride of Q / dO (see ld_tr8)
  __shared__ __attribute__((aligned(16))) bf16 Qs[2][QC * RS];
  __shared__ __attribute__((aligned(16))) bf16 dOs[2][QC * RS];
  __shared__ __attribute__((aligned(16))) float Dq[2][QC];
  __shared__ __attribute__((aligned(16))) float Lq[2][QC];

  const int bid = blockIdx.x;
  const int64_t pi = (int64_t)((bid >> 3) / KT) * 8 + (bid & 7);  // problem of the list
  const int kt = (bid >> 3) % KT;
  if (pi >= (int64_t)cl.count * g.heads) return;
  const int64_t ci = pi / g.heads;
  const int head = (int)(pi - ci * g.heads);
  const int64_t col = cl.cols ? cl.cols[ci] : ci;
  const int64_t prob = col * g.heads + head;
  const int n = g.col_ntr[col];
  const int t0 = kt * 4 * KW;
  if (t0 >= n) return;
  const int R = g.R, E = g.E;

  const uint32_t rowQ = D * 2, rowO = (uint32_t)E * 2;
  const rsrc_t rQ = make_rsrc(q + prob * R * D, (uint32_t)R * rowQ);
  const rsrc_t rK = make_rsrc(k + prob * R * D, (uint32_t)n * rowQ);
  const rsrc_t rV = make_rsrc(v + prob * R * D, (uint32_t)n * rowQ);
  const uint32_t obytes = (uint32_t)(R - 1) * rowO + rowQ;
  const rsrc_t rO = make_rsrc(o + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rdO = make_rsrc(dout + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rL = make_rsrc(lse + prob * R, (uint32_t)R * 4);
  const rsrc_t rD = make_rsrc(Dbuf + prob * R, (uint32_t)R * 4);

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int c = lane & 15, lg = lane >> 4;
  const float tau = 1.0f / sqrtf((float)D);

  // this lane's key column of key block kb in the S layout: t0 + w*32 + kb*16 + c; keys past
  // n read K = V = 0 here and their dK, dV are never written, so no key masking is needed
  const int kw0 = t0 + w * KW;
  typename HF<D>::frag kf[2], vf[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const uint32_t key = (uint32_t)(kw0 + kb * 16 + c);
    kf[kb] = HF<D>::buf(rK, key * rowQ, lg);
    vf[kb] = HF<D>::buf(rV, key * rowQ, lg);
  }

  // staging: threads 0-127 move Q, threads 128-255 move dO (and D and the LSE); each handles
  // NIT (query, 16-byte chunk) items; item it -> query it / CPR, dims (it % CPR) * 8.  Queries
  // past R read Q = dO = D = lse = 0: their P is 1 but dO and dS vanish.
  const int half = tid >> 7, st = tid & 127;
  uint4 ru[NIT];
  float rd[NIT], rl[NIT];
  auto gload = [&](int qc0) {
#pragma unroll
    for (int h = 0; h < NIT; ++h) {
      const int it = st + h * 128;
      const uint32_t qg = (uint32_t)(qc0 + it / CPR), d0 = (it % CPR) * 8;
      if (half == 0) {
        ru[h] = bload16(rQ, qg * rowQ + d0 * 2);
      } else {
        ru[h] = bload16(rdO, qg * rowO + d0 * 2);
        if ((it % CPR) == 0) {
          rd[h] = bloadf(rD, qg * 4);
          rl[h] = bloadf(rL, qg * 4);
        }
      }
    }
  };
  auto sstore = [&](int b) {
#pragma unroll
    for (int h = 0; h < NIT; ++h) {
      const int it = st + h * 128;
      const int qq = it / CPR, d0 = (it % CPR) * 8;
      stu4(&(half == 0 ? Qs[b] : dOs[b])[qq * RS + d0], ru[h]);
      if (half == 1 && (it % CPR) == 0) {
        Dq[b][qq] = -rd[h];
        Lq[b][qq] = -rl[h] * LOG2E;
      }
    }
  };

  f32x4 dkt[2][DB], dvt[2][DB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int db = 0; db < DB; ++db) dkt[kb][db] = dvt[kb][db] = zero4();

  const int NCH = (R + QC - 1) / QC;
  gload(0);
  sstore(0);
  lds_barrier();
  // one query chunk into LDS buffer b (a constant when bc is an integral_constant)
  auto step = [&](int ic, auto bc) __attribute__((always_inline)) {
    const int b = (int)bc;
    if (ic + 1 < NCH) gload((ic + 1) * QC);
    // S = Q K^T, dP = dO V^T per (query block, key block); lane: queries qb*16 + 4*lg + i
    uint32_t pw[2][4][2], sw[2][4][2];
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      const typename HF<D>::frag qa = HF<D>::lds(&Qs[b][(qb * 16 + c) * RS], lg);
      const typename HF<D>::frag da = HF<D>::lds(&dOs[b][(qb * 16 + c) * RS], lg);
      // seeds: -lse log2(e) and -D of the lane's 4 query rows
      const f32x4 nl = *reinterpret_cast<const f32x4*>(&Lq[b][qb * 16 + lg * 4]);
      const f32x4 nd = *reinterpret_cast<const f32x4*>(&Dq[b][qb * 16 + lg * 4]);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const f32x4 s = HF<D>::mma(qa, kf[kb], nl);     // S log2(e) - lse log2(e)
        const f32x4 dp = HF<D>::mma(da, vf[kb], nd);    // dP - D
        const float p0 = exp2_hw(s[0]), p1 = exp2_hw(s[1]);
        const float p2 = exp2_hw(s[2]), p3 = exp2_hw(s[3]);
        pw[kb][qb][0] = pack2(p0, p1);
        pw[kb][qb][1] = pack2(p2, p3);
        sw[kb][qb][0] = pack2(p0 * dp[0], p1 * dp[1]);
        sw[kb][qb][1] = pack2(p2 * dp[2], p3 * dp[3]);
      }
    }
    // dV^T += dO^T P, dK^T += Q^T dS over the chunk's 64 queries (two k steps of 32)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 dot_ = ld_tr8(&dOs[b][ks * 32 * RS], RS, db * 16, lane);
        const bf16x8 qt_ = ld_tr8(&Qs[b][ks * 32 * RS], RS, db * 16, lane);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 pf = cat8(make_uint2(pw[kb][2 * ks][0], pw[kb][2 * ks][1]),
                                 make_uint2(pw[kb][2 * ks + 1][0], pw[kb][2 * ks + 1][1]));
          const bf16x8 sf = cat8(make_uint2(sw[kb][2 * ks][0], sw[kb][2 * ks][1]),
                                 make_uint2(sw[kb][2 * ks + 1][0], sw[kb][2 * ks + 1][1]));
          dvt[kb][db] = mfma16(dot_, pf, dvt[kb][db]);
          dkt[kb][db] = mfma16(qt_, sf, dkt[kb][db]);
        }
      }
    }
    if (ic + 1 < NCH) sstore(b ^ 1);
    lds_barrier();
  };
  if constexpr (D <= 32) {
    // two chunks per iteration, so every LDS buffer offset is a constant
    for (int ic = 0; ic < NCH; ic += 2) {
      step(ic, std::integral_constant<int, 0>{});
      if (ic + 1 >= NCH) break;
      step(ic + 1, std::integral_constant<int, 1>{});
    }
  } else {
    // at d = 64 a doubled body needs more than 256 VGPRs (one wave per SIMD): keep one
    for (int ic = 0; ic < NCH; ++ic) step(ic, ic & 1);
  }
  // lane: dims db*16 + 4*lg + i of key kw0 + kb*16 + c
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int key = kw0 + kb * 16 + c;
    if (key >= n) continue;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint2 a = make_uint2(pack2(dkt[kb][db][0] * tau, dkt[kb][db][1] * tau),
                                 pack2(dkt[kb][db][2] * tau, dkt[kb][db][3] * tau));
      const uint2 bb = make_uint2(pack2(dvt[kb][db][0], dvt[kb][db][1]),
                                  pack2(dvt[kb][db][2], dvt[kb][db][3]));
      *reinterpret_cast<uint2*>(dk + (prob * R + key) * D + db * 16 + lg * 4) = a;
      *reinterpret_cast<uint2*>(dv + (prob * R + key) * D + db * 16 + lg * 4) = bb;
    }
  }
}

// =============================================================================== dQ
template <int D>
__global__ __launch_bounds__(256) void k_item_attn_dq(Geo g, const bf16* __restrict__ q,
                                                      const bf16* __restrict__ k,
                                                      const bf16* __restrict__ v,
                                                      const bf16* __restrict__ o,
                                                      const bf16* __restrict__ dout,
                                                      const float* __restrict__ lse,
                                                      float* __restrict__ Dbuf,
                                                      bf16* __restrict__ dq, int QT,
                                                      ColList cl) {
  constexpr int KTL = 64;         // keys per tile
  constexpr int DB = D / 16;
  constexpr int CPR = D / 8;
  constexpr int KS = tr_stride<D>();  // LDS row stride of K ([key][d]; see ld_tr8)
  constexpr int VS = D + 8;       // LDS row stride of V (conflict-free 16-byte row reads)
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][KTL * KS];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][KTL * VS];

  const int bid = blockIdx.x;
  const int64_t pi = (int64_t)((bid >> 3) / QT) * 8 + (bid & 7);  // problem of the list
  const int qt = (bid >> 3) % QT;
  if (pi >= (int64_t)cl.count * g.heads) return;
  const int64_t ci = pi / g.heads;
  const int head = (int)(pi - ci * g.heads);
  const int64_t col = cl.cols ? cl.cols[ci] : ci;
  const int64_t prob = col * g.heads + head;
  const int n = g.col_ntr[col];
  const int R = g.R, E = g.E;

  const uint32_t rowQ = D * 2, rowO = (uint32_t)E * 2;
  const rsrc_t rQ = make_rsrc(q + prob * R * D, (uint32_t)R * rowQ);
  const rsrc_t rK = make_rsrc(k + prob * R * D, (uint32_t)n * rowQ);
  const rsrc_t rV = make_rsrc(v + prob * R * D, (uint32_t)n * rowQ);
  const uint32_t obytes = (uint32_t)(R - 1) * rowO + rowQ;
  const rsrc_t rO = make_rsrc(o + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rdO = make_rsrc(dout + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rL = make_rsrc(lse + prob * R, (uint32_t)R * 4);

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int c = lane & 15, lg = lane >> 4;
  const int qw0 = qt * 128 + w * 32;
  // per query block: Q^T and dO^T fragments (B operands), D = rowsum(dO o O), -lse log2(e);
  // queries past R read as zero (their results are not written)
  typename HF<D>::frag qf[2], df[2];
  float Dv[2], nb[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const uint32_t qq = (uint32_t)(qw0 + qb * 16 + c);
    qf[qb] = HF<D>::buf(rQ, qq * rowQ, lg);
    df[qb] = HF<D>::buf(rdO, qq * rowO, lg);
    const typename HF<D>::frag of = HF<D>::buf(rO, qq * rowO, lg);
    float dot = hf_dot<D>(df[qb], of);
    dot = rows4_sum(dot);
    Dv[qb] = dot;
    nb[qb] = -bloadf(rL, qq * 4) * LOG2E;
    if (lg == 0 && (int)qq < R) Dbuf[prob * R + qq] = dot;
  }

  // key tile staging: item it = tid + 256 i -> (key it / CPR, 16-byte chunk of its d values);
  // keys past n read 0
  constexpr int NSI = (KTL * CPR + 255) / 256;  // staging items per thread
  uint4 rk[NSI], rv[NSI];
  auto gload = [&](int t0) {
#pragma unroll
    for (int i = 0; i < NSI; ++i) {
      const int it = tid + 256 * i;
      const uint32_t key = (uint32_t)(t0 + it / CPR), ch = (it % CPR) * 8;
      const bool ok = it < KTL * CPR;
      rk[i] = ok ? bload16(rK, key * rowQ + ch * 2) : make_uint4(0, 0, 0, 0);
      rv[i] = ok ? bload16(rV, key * rowQ + ch * 2) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int b) {
#pragma unroll
    for (int i = 0; i < NSI; ++i) {
      const int it = tid + 256 * i;
      if (it >= KTL * CPR) break;
      const int key = it / CPR, ch = (it % CPR) * 8;
      stu4(&Ks[b][key * KS + ch], rk[i]);
      stu4(&Vs[b][key * VS + ch], rv[i]);
    }
  };

  f32x4 acc[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db][0] = acc[db][1] = zero4();

  // seeds: -lse log2(e) and -D of the lane's query (one query per lane in the S^T layout)
  f32x4 snl[2], snd[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    snl[qb][0] = snl[qb][1] = snl[qb][2] = snl[qb][3] = nb[qb];
    snd[qb][0] = snd[qb][1] = snd[qb][2] = snd[qb][3] = -Dv[qb];
  }
  auto tile = [&](const int b, const int t0, const bool tail) {
    f32x4 dsv[4][2];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const typename HF<D>::frag kfr = HF<D>::lds(&Ks[b][(kb * 16 + c) * KS], lg);
      const typename HF<D>::frag vfr = HF<D>::lds(&Vs[b][(kb * 16 + c) * VS], lg);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const f32x4 s = HF<D>::mma(kfr, qf[qb], snl[qb]);    // exponent of P^T
        const f32x4 dp = HF<D>::mma(vfr, df[qb], snd[qb]);   // dP^T - D
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float p = exp2_hw(s[i]);
          if (tail && t0 + kb * 16 + lg * 4 + i >= n) p = 0.f;
          dsv[kb][qb][i] = p * dp[i];
        }
      }
    }
    // dQ^T += K^T dS^T  (k = keys, in the S^T tile order)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 kt_ = ld_tr8(&Ks[b][ks * 32 * KS], KS, db * 16, lane);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
          acc[db][qb] = mfma16(kt_, pack8(dsv[2 * ks][qb], dsv[2 * ks + 1][qb]), acc[db][qb]);
      }
  };

  const int NT = (n + KTL - 1) / KTL;
  const int NF = n / KTL;
  gload(0);
  sstore(0);
  lds_barrier();
  for (int it = 0; it < NF; ++it) {
    const int b = it & 1;
    if (it + 1 < NT) gload((it + 1) * KTL);
    tile(b, it * KTL, false);
    if (it + 1 < NT) sstore(b ^ 1);
    lds_barrier();
  }
  if (NF < NT) tile(NF & 1, NF * KTL, true);

  // lane: dims db*16 + 4*lg + i of query qw0 + qb*16 + c.  dQ = tau dS K, and the staged K
  // is log2(e) tau K, so the factor left is 1 / log2(e) = ln 2.
  constexpr float kLn2 = 0.69314718055994531f;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int qq = qw0 + qb * 16 + c;
    if (qq >= R) continue;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint2 u = make_uint2(pack2(acc[db][qb][0] * kLn2, acc[db][qb][1] * kLn2),
                                 pack2(acc[db][qb][2] * kLn2, acc[db][qb][3] * kLn2));
      *reinterpret_cast<uint2*>(dq + (prob * R + qq) * D + db * 16 + lg * 4) = u;
    }
  }
}

// The dS tile holds, in row `key`, the 32 queries of a chunk in the lane order of the score
// blocks: byte 16 g + 8 qb holds queries qb*16 + 4g .. + 3, so the 8 values of one lane (its
// two 16-query blocks) are one 16-byte write.  Transposed read (ds_read_b64_tr_b16) of key
// rows kr0 + {4g .. 4g+3, 16 + 4g .. 16 + 4g+3} (kr0 a multiple of 32): lane (g, c) receives
// query qb*16 + c.  off is the lane's byte offset for kr0 = 0 (ds_tile_off), which the swizzle
// leaves unchanged by multiples of 8 rows.
__device__ __forceinline__ int ds_tile_off(int lane, int qb) {
  const int r = lane >> 2;
  return r * 64 + row64_swz(r, 16 * (lane & 3) + 8 * qb);
}
__device__ __forceinline__ bf16x8 ds_tile_tr(const bf16* T, int kr0, int off) {
  return tr8_row64(T + kr0 * 32, off);
}

// =============================================================================== fused
// One workgroup per (column, head) problem whose train prefix has at most 8 * 16 * NKB rows
// (NKB <= 6):
// 8 waves, wave w owns the keys [w KW, (w + 1) KW), KW = 16 NKB, and every wave walks all query
// rows in chunks of 32 (Q, dO, D and the LSE of a chunk staged once in LDS for all waves).  Per
// chunk and wave, in the key-major layout of the dK/dV kernel above:
//   S = Q K^T, dP = dO V^T  (seeded with -lse log2 e and -D),  P = exp2(S),  dS = P (dP - D)
//   dV^T += dO^T P,  dK^T += Q^T dS                     (registers, across every chunk)
//   dQ_w^T = K^T dS^T over the wave's own keys: dS goes through the wave's LDS tile
//          [key][query] (one 16-byte row write per key block), read back transposed as the B
//          operand; K^T fragments are built once from an LDS copy of the wave's keys
// then the eight dQ_w of the chunk are added in wave order through LDS and stored.  P and dS
// are computed once per score (the two-kernel form computes them in both kernels), and every
// output element is summed in a fixed order, so results are bitwise reproducible.
template <int D, int NKB>
__global__ __launch_bounds__(512) void k_item_attn_bwd_fused(Geo g, const bf16* __restrict__ q,
                                                             const bf16* __restrict__ k,
                                                             const bf16* __restrict__ v,
                                                             const bf16* __restrict__ o,
                                                             const bf16* __restrict__ dout,
                                                             const float* __restrict__ lse,
                                                             bf16* __restrict__ dq,
                                                             bf16* __restrict__ dk,
                                                             bf16* __restrict__ dv, int per_xcd,
                                                             ColList cl) {
  constexpr int W = 8;                 // waves
  constexpr int QC = 32;               // queries per chunk (two 16-query blocks)
  constexpr int KW = 16 * NKB;         // keys per wave
  constexpr int DB = D / 16;
  constexpr int CPR = D / 8;           // 16-byte chunks per row of d values
  constexpr int RS = tr_stride<D>();   // LDS row stride of Q / dO and of the key copy
  constexpr int PQS = D + 4;           // dQ partial [query][d] floats: rows of 16 mod 32 bytes
  constexpr int T1 = KW * 64, T2 = QC * PQS * 4, T3 = KW * RS * 2;  // dS tile: 64-byte rows
  constexpr int REG = (T1 > T2 ? (T1 > T3 ? T1 : T3) : (T2 > T3 ? T2 : T3));
  // the wave's value rows: 64-byte swizzled rows at d = 32 (row64_swz), padded at d = 16
  constexpr int VS = D == 32 ? 32 : D + 8;
  static_assert(NKB % 2 == 0, "keys per wave must fill 32-key steps");
  __shared__ __attribute__((aligned(16))) bf16 Qs[2][QC * RS];
  __shared__ __attribute__((aligned(16))) bf16 dOs[2][QC * RS];
  __shared__ __attribute__((aligned(16))) float Lq[2][QC];
  __shared__ __attribute__((aligned(16))) float Dq[2][QC];
  __shared__ __attribute__((aligned(16))) char wreg[W][REG];
  __shared__ __attribute__((aligned(16))) bf16 Vw[W][KW * VS];

  // problems of one XCD are consecutive in the list (the heads of a column share their O / dO
  // rows in L2)
  const int bid = blockIdx.x;
  const int64_t pi = (int64_t)(bid & 7) * per_xcd + (bid >> 3);
  if (pi >= (int64_t)cl.count * g.heads) return;
  const int64_t ci = pi / g.heads;
  const int head = (int)(pi - ci * g.heads);
  const int64_t col = cl.cols ? cl.cols[ci] : ci;
  const int64_t prob = col * g.heads + head;
  const int n = g.col_ntr[col];
  const int R = g.R, E = g.E;
  const int nact = (n + KW - 1) / KW < W ? (n + KW - 1) / KW : W;  // waves that own keys

  const uint32_t rowQ = D * 2, rowO = (uint32_t)E * 2;
  const rsrc_t rQ = make_rsrc(q + prob * R * D, (uint32_t)R * rowQ);
  const rsrc_t rK = make_rsrc(k + prob * R * D, (uint32_t)n * rowQ);
  const rsrc_t rV = make_rsrc(v + prob * R * D, (uint32_t)n * rowQ);
  const uint32_t obytes = (uint32_t)(R - 1) * rowO + rowQ;
  const rsrc_t rO = make_rsrc(o + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rdO = make_rsrc(dout + col * R * (int64_t)E + head * D, obytes);
  const rsrc_t rL = make_rsrc(lse + prob * R, (uint32_t)R * 4);

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int c = lane & 15, lg = lane >> 4;
  const float tau = 1.0f / sqrtf((float)D);
  const bool active = w < nact;
  const int kw0 = w * KW;
  typedef typename HF<D>::frag frag;

  // the wave's keys (lane: key kw0 + kb*16 + c) in registers, its values in LDS; keys past n
  // read K = V = 0: their dK, dV are never stored and they add K = 0 to dQ, so no key masking
  // is needed
  frag kf[NKB];
  bf16x8 ktf[NKB / 2][DB];  // K^T as the A operand of K^T dS^T: dims db*16 + c, 32-key steps
  f32x4 dkt[NKB][DB], dvt[NKB][DB];
  bf16* vw = Vw[w];
  // the lane's byte offsets in 64-byte swizzled rows: its 16-byte piece of row c (+ 16 kb rows)
  // and its transposed-read addresses in the dS tile
  const int roff = c * 64 + row64_swz(c, 16 * lg);
  const int toff0 = ds_tile_off(lane, 0), toff1 = ds_tile_off(lane, 1);
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
    for (int db = 0; db < DB; ++db) dkt[kb][db] = dvt[kb][db] = zero4();
    const uint32_t key = (uint32_t)(kw0 + kb * 16 + c);
    kf[kb] = HF<D>::buf(rK, key * rowQ, lg);
    const frag vv = HF<D>::buf(rV, key * rowQ, lg);
    const int vr = kb * 16 + c;
    if constexpr (D == 32)
      *reinterpret_cast<frag*>(&vw[kb * 16 * 32 + roff / 2]) = vv;
    else
      *reinterpret_cast<frag*>(&vw[vr * VS + lg * HF<D>::EPL]) = vv;
  }
  {
    bf16* kst = reinterpret_cast<bf16*>(wreg[w]);  // [KW][RS] row-major copy of the keys
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
      *reinterpret_cast<frag*>(&kst[(kb * 16 + c) * RS + lg * HF<D>::EPL]) = kf[kb];
    wave_lds_sync();
#pragma unroll
    for (int ks = 0; ks < NKB / 2; ++ks)
#pragma unroll
      for (int db = 0; db < DB; ++db) ktf[ks][db] = ld_tr8(&kst[ks * 32 * RS], RS, db * 16, lane);
    wave_lds_sync();
  }

  // staging of a query chunk: threads [0, 128) move Q, threads [128, 256) move dO and read O
  // for D = rowsum(dO o O) (the CPR threads of a query are adjacent lanes); queries past R read
  // Q = dO = O = lse = 0 (P = 1 there, but dO and dS vanish and their dQ is not stored)
  constexpr int NIT = QC * CPR;  // items per tensor (<= 128)
  const bool qthr = tid < NIT, othr = tid >= 128 && tid < 128 + NIT;
  const int it = qthr ? tid : tid - 128;
  const int iq = it / CPR, id0 = (it % CPR) * 8;
  uint4 rq = make_uint4(0, 0, 0, 0), rdo = rq, ro = rq;
  float rl = 0.f;
  auto gload = [&](int q0) {
    const uint32_t qg = (uint32_t)(q0 + iq);
    if (qthr) rq = bload16(rQ, qg * rowQ + id0 * 2);
    if (othr) {
      rdo = bload16(rdO, qg * rowO + id0 * 2);
      ro = bload16(rO, qg * rowO + id0 * 2);
      if (id0 == 0) rl = bloadf(rL, qg * 4);
    }
  };
  auto sstore = [&](int b) {
    if (qthr) stu4(&Qs[b][iq * RS + id0], rq);
    if (tid >= 128 && tid < 256) {  // whole waves: the lane sums below see only their own
      float dd = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) dd = fmaf(bf2f(u4_elem(rdo, j)), bf2f(u4_elem(ro, j)), dd);
      dd += dpp_mov<0xB1>(dd);                  // lanes of a query: 4 (d = 32) or 2 (d = 16)
      if (CPR == 4) dd += dpp_mov<0x4E>(dd);
      if (othr) {
        stu4(&dOs[b][iq * RS + id0], rdo);
        if (id0 == 0) {
          Dq[b][iq] = -dd;
          Lq[b][iq] = -rl * LOG2E;
        }
      }
    }
  };

  const int NCH = (R + QC - 1) / QC;
  gload(0);
  sstore(0);
  lds_barrier();
  constexpr float kLn2 = 0.69314718055994531f;
  for (int ic = 0; ic < NCH; ++ic) {
    const int b = ic & 1;
    if (ic + 1 < NCH) gload((ic + 1) * QC);
    if (active) {
      frag qa[2], da[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        qa[qb] = HF<D>::lds(&Qs[b][(qb * 16 + c) * RS], lg);
        da[qb] = HF<D>::lds(&dOs[b][(qb * 16 + c) * RS], lg);
      }
      bf16x8 qt[DB], dot[DB];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        qt[db] = ld_tr8(Qs[b], RS, db * 16, lane);
        dot[db] = ld_tr8(dOs[b], RS, db * 16, lane);
      }
      bf16* dst = reinterpret_cast<bf16*>(wreg[w]);  // dS tile [KW][32 queries]
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int vr = kb * 16 + c;
        frag vfk;
        if constexpr (D == 32)
          vfk = *reinterpret_cast<const frag*>(&vw[kb * 16 * 32 + roff / 2]);
        else
          vfk = HF<D>::lds(&vw[vr * VS], lg);
        uint32_t pw[2][2], sw[2][2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const f32x4 nl = *reinterpret_cast<const f32x4*>(&Lq[b][qb * 16 + lg * 4]);
          const f32x4 nd = *reinterpret_cast<const f32x4*>(&Dq[b][qb * 16 + lg * 4]);
          const f32x4 sc = HF<D>::mma(qa[qb], kf[kb], nl);   // S log2(e) - lse log2(e)
          const f32x4 dp = HF<D>::mma(da[qb], vfk, nd);      // dP - D
          const float p0 = exp2_hw(sc[0]), p1 = exp2_hw(sc[1]);
          const float p2 = exp2_hw(sc[2]), p3 = exp2_hw(sc[3]);
          pw[qb][0] = pack2(p0, p1);
          pw[qb][1] = pack2(p2, p3);
          sw[qb][0] = pack2(p0 * dp[0], p1 * dp[1]);
          sw[qb][1] = pack2(p2 * dp[2], p3 * dp[3]);
        }
        const bf16x8 pf = cat8(make_uint2(pw[0][0], pw[0][1]), make_uint2(pw[1][0], pw[1][1]));
        const bf16x8 sf = cat8(make_uint2(sw[0][0], sw[0][1]), make_uint2(sw[1][0], sw[1][1]));
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dvt[kb][db] = mfma16(dot[db], pf, dvt[kb][db]);
          dkt[kb][db] = mfma16(qt[db], sf, dkt[kb][db]);
        }
        // dS row of key kb*16 + c: the lane's queries 4 lg .. + 3 of both 16-query blocks
        *reinterpret_cast<bf16x8*>(&dst[kb * 16 * 32 + roff / 2]) = sf;
      }
      wave_lds_sync();
      // dQ_w^T[d][q] = sum over the wave's keys of K[key][d] dS[q][key]
      f32x4 dqp[2][DB];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < DB; ++db) dqp[qb][db] = zero4();
#pragma unroll
      for (int ks = 0; ks < NKB / 2; ++ks)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
          const bf16x8 bq = ds_tile_tr(dst, ks * 32, qb ? toff1 : toff0);
#pragma unroll
          for (int db = 0; db < DB; ++db) dqp[qb][db] = mfma16(ktf[ks][db], bq, dqp[qb][db]);
        }
      wave_lds_sync();  // the tile is read before the partial overwrites it
      // lane: dQ_w[q = qb*16 + c][d = db*16 + 4 lg + i] -> partial [q][d]
      float* pq = reinterpret_cast<float*>(wreg[w]);
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < DB; ++db)
          *reinterpret_cast<f32x4*>(&pq[(qb * 16 + c) * PQS + db * 16 + 4 * lg]) = dqp[qb][db];
    }
    if (ic + 1 < NCH) sstore(b ^ 1);
    lds_barrier();
    // dQ of the chunk: the partials of the active waves added in wave order, two dims a thread
    if (tid < QC * D / 2) {
      const int qq = tid / (D / 2), d0 = 2 * (tid % (D / 2));
      float s0 = 0.f, s1 = 0.f;
      for (int w2 = 0; w2 < nact; ++w2) {
        const float2 pv =
            *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(wreg[w2]) + qq * PQS + d0);
        s0 += pv.x;
        s1 += pv.y;
      }
      const int qg = ic * QC + qq;
      if (qg < R)
        *reinterpret_cast<uint32_t*>(dq + (prob * R + qg) * D + d0) = pack2(s0 * kLn2, s1 * kLn2);
    }
    lds_barrier();
  }
  // lane: dims db*16 + 4*lg + i of key kw0 + kb*16 + c
  if (!active) return;
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb) {
    const int key = kw0 + kb * 16 + c;
    if (key >= n) continue;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint2 a = make_uint2(pack2(dkt[kb][db][0] * tau, dkt[kb][db][1] * tau),
                                 pack2(dkt[kb][db][2] * tau, dkt[kb][db][3] * tau));
      const uint2 bb = make_uint2(pack2(dvt[kb][db][0], dvt[kb][db][1]),
                                  pack2(dvt[kb][db][2], dvt[kb][db][3]));
      *reinterpret_cast<uint2*>(dk + (prob * R + key) * D + db * 16 + lg * 4) = a;
      *reinterpret_cast<uint2*>(dv + (prob * R + key) * D + db * 16 + lg * 4) = bb;
    }
  }
}

// Key blocks of 16 per wave of the fused backward for train prefixes of at most nmax rows;
// 0 where it does not apply (d = 64, or more than 768 train rows: the keys' dK / dV
// accumulators and fragments would not fit the registers of two waves per SIMD).
static int fused_nkb(int d, int nmax) {
  if (d != 16 && d != 32) return 0;
  if (nmax <= 256) return 2;
  if (nmax <= 512) return 4;
  if (nmax <= 768) return 6;
  return 0;
}

bool item_attn_bwd_fused_ok(const Geo& g, int nmax) { return fused_nkb(g.d, nmax) > 0; }

int item_attn_bwd_fused_max_rows(int d) { return fused_nkb(d, 1) > 0 ? 768 : 0; }

template <int D>
static hipError_t fused_d(const Geo& g, const ColList& cl, int nkb, unsigned grid, int per,
                          const bf16* q, const bf16* k, const bf16* v, const bf16* o,
                          const bf16* dout, const float* lse, bf16* dq, bf16* dk, bf16* dv,
                          hipStream_t s) {
  switch (nkb) {
    case 2:
      k_item_attn_bwd_fused<D, 2><<<grid, 512, 0, s>>>(g, q, k, v, o, dout, lse, dq, dk, dv,
                                                         per, cl);
      break;
    case 4:
      k_item_attn_bwd_fused<D, 4><<<grid, 512, 0, s>>>(g, q, k, v, o, dout, lse, dq, dk, dv,
                                                         per, cl);
      break;
    case 6:
      k_item_attn_bwd_fused<D, 6><<<grid, 512, 0, s>>>(g, q, k, v, o, dout, lse, dq, dk, dv,
                                                         per, cl);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_item_attn_bwd_fused(const Geo& g, const ColList& cl, int nmax, const bf16* q,
                                      const bf16* k, const bf16* v, const bf16* o,
                                      const bf16* dout, const float* lse, bf16* dq, bf16* dk,
                                      bf16* dv, hipStream_t s) {
  const int nkb = fused_nkb(g.d, nmax);
  if (nkb == 0) return hipErrorInvalidValue;
  const int64_t P = (int64_t)cl.count * g.heads;
  if (P == 0) return hipSuccess;
  const int per = (int)((P + 7) / 8);
  const unsigned grid = (unsigned)(8 * per);
  if (g.d == 16) return fused_d<16>(g, cl, nkb, grid, per, q, k, v, o, dout, lse, dq, dk, dv, s);
  return fused_d<32>(g, cl, nkb, grid, per, q, k, v, o, dout, lse, dq, dk, dv, s);
}

hipError_t launch_item_attn_dq(const Geo& g, const ColList& cl, const bf16* q, const bf16* k,
                               const bf16* v, const bf16* o, const bf16* dout, const float* lse,
                               float* Dbuf, bf16* dq, hipStream_t s) {
  const int64_t P = (int64_t)cl.count * g.heads;
  if (P == 0) return hipSuccess;
  const int QT = (g.R + 127) / 128;
  const unsigned grid = (unsigned)((P + 7) / 8 * 8 * QT);
  if (g.d == 16)
    k_item_attn_dq<16><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dq, QT, cl);
  else if (g.d == 32)
    k_item_attn_dq<32><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dq, QT, cl);
  else if (g.d == 64)
    k_item_attn_dq<64><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dq, QT, cl);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_item_attn_dkdv(const Geo& g, const ColList& cl, const bf16* q, const bf16* k,
                                 const bf16* v, const bf16* o, const bf16* dout,
                                 const float* lse, const float* Dbuf, bf16* dk, bf16* dv,
                                 hipStream_t s) {
  const int64_t P = (int64_t)cl.count * g.heads;
  if (P == 0) return hipSuccess;
  const int KT = (g.R + 127) / 128;
  const unsigned grid = (unsigned)((P + 7) / 8 * 8 * KT);
  if (g.d == 16)
    k_item_attn_dkdv<16><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dk, dv, KT, cl);
  else if (g.d == 32)
    k_item_attn_dkdv<32><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dk, dv, KT, cl);
  else if (g.d == 64)
    k_item_attn_dkdv<64><<<grid, 256, 0, s>>>(g, q, k, v, o, dout, lse, Dbuf, dk, dv, KT, cl);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tfm
