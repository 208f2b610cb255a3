// Item-axis (down each column) flash attention on bf16 MFMA, forward pass.
//
// Problem (column g, head h): queries are all R rows of the column, keys and values are the
// first n_train rows (the train prefix).  The prefix is a loop bound over key tiles — scores
// are never materialised and the only masking is inside the last, partial key tile.
//
// One workgroup = 4 waves of one problem; each wave owns 64 queries (four 16-query MFMA blocks)
// at d <= 32 and 32 at d = 64.  Key tiles of 64 keys are staged in LDS (K and V as [key][d]; V
// is read back transposed) with double buffering and shared by the 4 waves.  Per tile a wave computes S^T = K Q^T
// (keys x queries, so that a lane holds 4 keys of one query), the online softmax in the exp2
// domain with the scale folded into one FMA, and O^T += V^T P^T where the D tile of S^T is
// reused directly as the B operand (the k positions of V^T are permuted to match).
//
// Workgroups are numbered so that all query tiles of one problem land on the same XCD (the
// hardware deals consecutive workgroup ids round-robin over the 8 XCDs), keeping the problem's
// keys and values in that XCD's L2.
#include <math.h>

#include "attn.h"
#include "attn_frag.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr int KT = 64;   // keys per tile
// 16-query blocks per wave: four at d <= 32 (every K and V fragment read from LDS serves 64
// queries; 163 VGPRs, three waves per SIMD), two at d = 64 (its fragments are twice as wide)
template <int D>
constexpr int qblocks() { return D == 64 ? 2 : 4; }
template <int D>
constexpr int qwave() { return 16 * qblocks<D>(); }   // queries per wave
template <int D>
constexpr int qgroup() { return 4 * qwave<D>(); }     // queries per workgroup (4 waves)

__device__ __forceinline__ uint32_t pk_bf16(float a, float b) { return pack2(a, b); }

}  // namespace

template <int D>
__global__ __launch_bounds__(256, 3) void k_item_attn_fwd(Geo g, const bf16* __restrict__ q,
                                                       const bf16* __restrict__ k,
                                                       const bf16* __restrict__ v,
                                                       bf16* __restrict__ o,
                                                       float* __restrict__ lse, int QT,
                                                       int kR) {
  // d = 32: K and V rows of 64 bytes, swizzled (row64_swz); otherwise padded rows
  constexpr bool SW = D == 32;
  // LDS row stride of K (elements): 16-byte row reads are conflict-free at strides of an odd
  // multiple of 32 bytes (d = 64: 160 bytes)
  constexpr int KS = SW ? 32 : (D == 64 ? tr_stride<D>() : D + 8);
  constexpr int VS = SW ? 32 : tr_stride<D>();     // LDS row stride of V
  constexpr int DB = D / 16;  // 16-wide dim blocks
  constexpr int QB = qblocks<D>();
  constexpr int CPR = D / 8;  // 16-byte chunks per key row
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][KT * KS];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][KT * VS];

  const int bid = blockIdx.x;
  const int64_t prob = (int64_t)((bid >> 3) / QT) * 8 + (bid & 7);
  const int qt = (bid >> 3) % QT;
  if (prob >= (int64_t)g.NC * g.heads) return;
  const int64_t col = prob / g.heads;
  const int head = (int)(prob - col * g.heads);
  const int n = g.col_ntr[col];
  const int R = g.R;
  const bf16* Qp = q + prob * R * D;
  const bf16* Kp = k + prob * kR * D;  // keys and values: kR rows per problem
  const bf16* Vp = v + prob * kR * D;

  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int c = lane & 15, lg = lane >> 4;
  const int qw0 = qt * qgroup<D>() + wave * qwave<D>();

  // Buffer resources of the problem: loads past the end (queries past R, keys past n) return 0
  // without an exec-masked branch, so the compiler's wait counts stay exact and the prefetch of
  // the next key tile is not waited for before the current tile's products.
  const rsrc_t rQ = make_rsrc(Qp, (uint32_t)R * D * 2);
  const rsrc_t rK = make_rsrc(Kp, (uint32_t)n * D * 2);
  const rsrc_t rV = make_rsrc(Vp, (uint32_t)n * D * 2);

  // Q^T fragments (B operand): lane holds query qw0 + qb*16 + c
  typename HF<D>::frag qf[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) qf[qb] = HF<D>::buf(rQ, (uint32_t)(qw0 + qb * 16 + c) * D * 2, lg);

  // staging: item it = tid + 256 i -> (key, 16-byte chunk of its dims): key it / CPR, chunk
  // it % CPR; at d = 32 key (it % 16) + 16 (it / 64), chunk (it / 16) % 4, so that each store
  // instruction names one chunk of 16 rows (the conflict-free access of the swizzled rows)
  constexpr int NSI = (KT * CPR + 255) / 256;  // staging items per thread
  uint4 rk[NSI], rv[NSI];
  auto item_key = [&](int it) { return SW ? (it & 15) + 16 * (it >> 6) : it / CPR; };
  auto item_ch = [&](int it) { return SW ? (it >> 4) & 3 : it % CPR; };
  auto gload = [&](int t0) {
#pragma unroll
    for (int i = 0; i < NSI; ++i) {
      const int it = tid + 256 * i;
      const int t = t0 + item_key(it), ch = item_ch(it) * 8;
      // items past the tile (d = 16) name an offset past the range and read 0
      const uint32_t off = it < KT * CPR ? (uint32_t)(t * D + ch) * 2 : 0xfffffff0u;
      rk[i] = bload16(rK, off);
      rv[i] = bload16(rV, off);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NSI; ++i) {
      const int it = tid + 256 * i;
      if (it >= KT * CPR) break;
      const int key = item_key(it), ch = item_ch(it);
      if constexpr (SW) {
        stu4(&Ks[buf][key * 32 + row64_swz(key, 16 * ch) / 2], rk[i]);
        stu4(&Vs[buf][key * 32 + row64_swz(key, 16 * ch) / 2], rv[i]);
      } else {
        stu4(&Ks[buf][key * KS + ch * 8], rk[i]);
        stu4(&Vs[buf][key * VS + ch * 8], rv[i]);
      }
    }
  };
  // d = 32: the lane's byte offsets in the swizzled rows: its K fragment piece of row c, and
  // its transposed-read addresses of V (dims db*16 + c)
  const int roff = c * 64 + row64_swz(c, 16 * lg);
  int voff[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
    voff[db] = (lane >> 2) * 64 + row64_swz(lane >> 2, 32 * db + 8 * (lane & 3));

  // K arrives pre-multiplied by log2(e)/sqrt(d), so S^T = K Q^T is in the exp2 domain.  The MFMA
  // accumulators start at -ref, a running reference of the exponent per query, so they return
  // S^T - ref and p = exp2(acc) needs no further arithmetic.  The reference is set by the first
  // tile and raised only when a tile's maximum exceeds it by more than 8, which keeps every p
  // below 2^8 and makes the shift-and-rescale rare.
  float ref[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) ref[qb] = -INFINITY;
  constexpr float slack = 8.0f;
  // O^T accumulators: DB blocks of V^T rows plus one block whose first row is all ones, so
  // that row accumulates the softmax denominator with the same rescaling as O.
  f32x4 oacc[DB + 1][QB];
#pragma unroll
  for (int db = 0; db <= DB; ++db)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) oacc[db][qb] = zero4();
  bf16x8 ones;
  {
    const uint32_t w = c == 0 ? 0x3f803f80u : 0u;  // bf16 1.0 pairs in row 0 only
    uint4 u = make_uint4(w, w, w, w);
    ones = *reinterpret_cast<bf16x8*>(&u);
  }

  auto tile = [&](const int cur, const int t0, const bool tail) {
    // S^T - ref for 4 key blocks x 2 query blocks
    f32x4 sc[4][QB];
    f32x4 init[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float r0 = ref[qb] == -INFINITY ? 0.f : -ref[qb];
      init[qb][0] = init[qb][1] = init[qb][2] = init[qb][3] = r0;
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      typename HF<D>::frag kf;
      if constexpr (SW)
        kf = *reinterpret_cast<const typename HF<D>::frag*>(&Ks[cur][kb * 16 * 32 + roff / 2]);
      else
        kf = HF<D>::lds(&Ks[cur][(kb * 16 + c) * KS], lg);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) sc[kb][qb] = HF<D>::mma(kf, qf[qb], init[qb]);
    }
    if (tail) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (t0 + kb * 16 + lg * 4 + i >= n) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) sc[kb][qb][i] = -INFINITY;
          }
    }
    bf16x8 pf[QB][2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = fmaxf(fmaxf(sc[0][qb][0], sc[0][qb][1]), fmaxf(sc[0][qb][2], sc[0][qb][3]));
#pragma unroll
      for (int kb = 1; kb < 4; ++kb)
        mx = fmaxf(mx, fmaxf(fmaxf(sc[kb][qb][0], sc[kb][qb][1]),
                             fmaxf(sc[kb][qb][2], sc[kb][qb][3])));
      mx = rows4_max(mx);
      // first tile: ref = the tile maximum; later: raise ref by the excess when it is large
      const bool first = ref[qb] == -INFINITY;
      if (__any(first || mx > slack)) {
        const float delta = first ? mx : fmaxf(mx, 0.f);
        ref[qb] = first ? mx : ref[qb] + delta;
        const float corr = exp2_hw(-delta);
#pragma unroll
        for (int db = 0; db <= DB; ++db) oacc[db][qb] *= corr;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) sc[kb][qb] -= delta;
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        f32x4 a0 = sc[2 * ks][qb], a1 = sc[2 * ks + 1][qb];
        uint4 u;
        u.x = pk_bf16(exp2_hw(a0[0]), exp2_hw(a0[1]));
        u.y = pk_bf16(exp2_hw(a0[2]), exp2_hw(a0[3]));
        u.z = pk_bf16(exp2_hw(a1[0]), exp2_hw(a1[1]));
        u.w = pk_bf16(exp2_hw(a1[2]), exp2_hw(a1[3]));
        pf[qb][ks] = *reinterpret_cast<bf16x8*>(&u);
      }
    }
    // O^T += V^T P^T (and the ones row += sum of P)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16x8 vf = SW ? tr8_row64(&Vs[cur][ks * 32 * 32], voff[db])
                             : ld_tr8(&Vs[cur][ks * 32 * VS], VS, db * 16, lane);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) oacc[db][qb] = mfma16(vf, pf[qb][ks], oacc[db][qb]);
      }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) oacc[DB][qb] = mfma16(ones, pf[qb][ks], oacc[DB][qb]);
    }
  };

  const int NT = (n + KT - 1) / KT;
  const int NF = n / KT;  // full tiles; a partial tail tile follows if NT > NF
  gload(0);
  sstore(0);
  // the Q fragments have arrived before the loop (no load is pending at its head)
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) hf_touch<D>(qf[qb]);
  lds_barrier();
  for (int it = 0; it < NF; ++it) {
    const int cur = it & 1;
    if (it + 1 < NT) gload((it + 1) * KT);
    tile(cur, it * KT, false);
    if (it + 1 < NT) sstore(cur ^ 1);
    lds_barrier();
  }
  if (NF < NT) tile(NF & 1, NF * KT, true);

  // normalise and write O (cell-major) and the natural-log LSE = ln 2 * (ref + log2 l)
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = __shfl(oacc[DB][qb][0], c, 64);  // row 0 of the ones block, lane (0, c)
    const int qq = qw0 + qb * 16 + c;
    if (qq >= R) continue;
    const float inv = 1.0f / lt;
    bf16* orow = o + (col * R + qq) * (int64_t)g.E + head * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      uint2 u;
      u.x = pk_bf16(oacc[db][qb][0] * inv, oacc[db][qb][1] * inv);
      u.y = pk_bf16(oacc[db][qb][2] * inv, oacc[db][qb][3] * inv);
      *reinterpret_cast<uint2*>(orow + db * 16 + lg * 4) = u;
    }
    if (lg == 0) lse[prob * R + qq] = (ref[qb] + log2f(lt)) * 0.69314718055994531f;
  }
}

hipError_t launch_item_attn_fwd(const Geo& g, const bf16* q, const bf16* k, const bf16* v,
                                bf16* o, float* lse, hipStream_t s, int kR) {
  if (kR <= 0) kR = g.R;
  const int64_t P = (int64_t)g.NC * g.heads;
  auto grid = [&](int QT) { return (unsigned)((P + 7) / 8 * 8 * QT); };
  if (g.d == 16) {
    const int QT = (g.R + qgroup<16>() - 1) / qgroup<16>();
    k_item_attn_fwd<16><<<grid(QT), 256, 0, s>>>(g, q, k, v, o, lse, QT, kR);
  } else if (g.d == 32) {
    const int QT = (g.R + qgroup<32>() - 1) / qgroup<32>();
    k_item_attn_fwd<32><<<grid(QT), 256, 0, s>>>(g, q, k, v, o, lse, QT, kR);
  } else if (g.d == 64) {
    const int QT = (g.R + qgroup<64>() - 1) / qgroup<64>();
    k_item_attn_fwd<64><<<grid(QT), 256, 0, s>>>(g, q, k, v, o, lse, QT, kR);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tfm
