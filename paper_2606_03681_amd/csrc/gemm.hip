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
#include "gelu.h"
#include "mfma.h"

namespace tfm {

namespace {

constexpr int BK = 32;       // k per pipeline stage: one 64-byte LDS row per operand row

// Source of the 16-byte loads of rows that do not exist (past M, or K/V rows of test cells).
__device__ __attribute__((aligned(16))) const uint4 kZeroChunk = {0u, 0u, 0u, 0u};

// Slot of 16-byte k chunk kc (0..3) in LDS row r (64-byte rows).  A 16-byte fragment read
// names the same kc in 16 consecutive rows; XOR-rotating the chunks by bits 1 and 2 of the row
// makes those reads free of bank conflicts on this LDS (measured: rotating by bits 2 and 3
// instead costs about 3 conflict cycles per read).
__device__ __forceinline__ int kslot(int r, int kc) { return kc ^ ((r >> 1) & 3); }

__device__ __forceinline__ int64_t row_addr(const Geo& g, int mode, int64_t m, int64_t ld) {
  return mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
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

// The single-output epilogues without row reductions (bias, head-major Q|K|V) pass their
// output tile through LDS in two halves of BM/2 rows and keep one stage in flight ahead of the
// MFMAs: 44 KB of LDS at E = 192, three workgroups per CU instead of two, so that one
// workgroup's stores overlap more of the others' loads (their K loops are short: K = E); 8-9 %
// faster per launch.  The GELU epilogue (two outputs, four barriers per half) was 17 % slower
// that way, and wider tiles (E = 256) would need more registers than three workgroups per CU
// leave: both keep the full tile.
template <int EPI, int BN>
constexpr bool gemm_half_tile() {
  return (EPI == EPI_BIAS || EPI == EPI_ITEM_QKV) && BN <= 192;
}

template <int BN, int EPI, int BM>
__global__ __launch_bounds__(256, (gemm_half_tile<EPI, BN>() ? 3 : 2)) void k_gemm(GemmArgs a) {
  constexpr int MI = BM / 32;          // 16-row blocks per wave (2 x 2 waves, each BM/2 rows)
  constexpr int NBA = BM / 64;         // 1 KB blocks of A per wave and stage
  constexpr int NB = BN / 32;          // 16-wide column blocks per wave
  constexpr int TS = BN + 8;           // epilogue tile row stride (elements)
  constexpr bool HALF = gemm_half_tile<EPI, BN>();
  // pipeline stages in the LDS ring (60 KB at E = 192 and 128 rows: 2 workgroups per CU; 40 KB
  // with two stages)
  constexpr int S = HALF ? 2 : 3;
  constexpr int A_EL = BM * BK;        // elements of one stage's A rows
  constexpr int STAGE_EL = (BM + BN) * BK;
  constexpr int NBB = BN / 64;         // 1 KB blocks of B per wave and stage
  constexpr int RING_BYTES = S * STAGE_EL * 2;
  constexpr int TILE_BYTES = (HALF ? BM / 2 : BM) * TS * 2;
  // The epilogue's tile and its row / column reduction arrays reuse the ring once it drains.
  constexpr int RED_BYTES = 2 * BM * 4, CRED_BYTES = 4 * BN * 4;
  constexpr int EPI_BYTES = TILE_BYTES + RED_BYTES + CRED_BYTES;
  __shared__ __attribute__((aligned(16))) char smem[RING_BYTES > EPI_BYTES ? RING_BYTES : EPI_BYTES];
  bf16* ring = reinterpret_cast<bf16*>(smem);  // stage slot s: A at s*STAGE_EL, B after A
  bf16* tile = reinterpret_cast<bf16*>(smem);  // epilogue: [BM][TS], after the main loop
  float (*red)[BM] = reinterpret_cast<float (*)[BM]>(smem + TILE_BYTES);          // [2][BM]
  float (*cred)[2][BN] =
      reinterpret_cast<float (*)[2][BN]>(smem + TILE_BYTES + RED_BYTES);        // [2][2][BN]
  // bias, gamma, beta of the tile; residual affine (EPI_LN)
  __shared__ __attribute__((aligned(16))) float cpar[5][BN];
  __shared__ int64_t rbase[BM];  // epilogue: per-row element offset for the current mode

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lg = lane >> 4;
  // Workgroup -> (row tile bx, column tile by).  The hardware deals consecutive workgroups
  // round-robin over the 8 XCDs; all column tiles of a row tile are given consecutive slots
  // of one XCD so that the row tile's A rows are fetched from memory once and then hit that
  // XCD's L2.
  const int NY = a.N / BN;
  const int idx = (int)(blockIdx.x >> 3), xcd = (int)(blockIdx.x & 7);
  const int64_t bx = (int64_t)(idx / NY) * 8 + xcd;
  const int by = idx % NY;
  const int64_t m0 = bx * BM;
  if (m0 >= a.M) return;
  const int n0 = by * BN;
  const Geo& g = a.g;
  // item Q|K|V: which of the three this column tile is (BN divides E), and its first column
  // within that part
  const int part = EPI == EPI_ITEM_QKV ? n0 / g.E : 0;
  const int pc0 = n0 - part * g.E;

  if (EPI == EPI_ITEM_QKV && part > 0) {
    // K and V exist for train rows only: skip tiles made of test rows alone
    int64_t last = m0 + BM - 1 < a.M ? m0 + BM - 1 : a.M - 1;
    int64_t c0 = m0 / g.R, c1 = last / g.R;
    bool any = false;
    for (int64_t c = c0; c <= c1 && !any; ++c) {
      int64_t rlo = c == c0 ? m0 - c0 * g.R : 0;
      any = rlo < g.col_ntr[c];
    }
    if (!any) return;
  }

  // ---- operand streaming.  Every stage moves A rows [m0, m0+64) and B rows [n0, n0+BN), k in
  // [k0, k0+32), straight from memory into the stage's LDS slot (global_load_lds: lane L of a
  // wave fills bytes 16L..16L+15 of the wave's 1 KB block).  LDS position p (16-byte units)
  // holds row p / 4, k chunk kslot^-1(p % 4); this lane's A position is wave*64 + lane.
  // This lane's A positions: block t covers rows 16 (wave + 4 t) .. + 15.
  const bf16* zero = reinterpret_cast<const bf16*>(&kZeroChunk);
  int akc[NBA];
  bool arow_ok[NBA];
  const bf16* aptr[NBA];  // row address + chunk, for compact / native rows
  int64_t hcol[NBA];
  int hr[NBA], hntr[NBA];
#pragma unroll
  for (int t = 0; t < NBA; ++t) {
    const int ar = ((wave + 4 * t) * 64 + lane) >> 2;
    akc[t] = kslot(ar, lane & 3);
    const int64_t am = m0 + ar;
    arow_ok[t] = am < a.M;
    aptr[t] = zero;
    hcol[t] = 0;
    hr[t] = 0;
    hntr[t] = 0;
    if (a.amode == ROWS_ITEM_HM) {
      if (arow_ok[t]) {
        hcol[t] = am / g.R;
        hr[t] = (int)(am - hcol[t] * g.R);
        hntr[t] = g.col_ntr[hcol[t]];
      }
    } else if (arow_ok[t]) {
      aptr[t] = a.A + row_addr(g, a.amode, am, a.lda) + akc[t] * 8;
    }
  }
  const bf16* bptr[NBB];
#pragma unroll
  for (int t = 0; t < NBB; ++t) {
    const int p = (wave + 4 * t) * 64 + lane;
    const int n = p >> 2;
    bptr[t] = a.Bt + (int64_t)(n0 + n) * a.K + kslot(n, p & 3) * 8;
  }
  auto issue = [&](int st) {
    bf16* sa = ring + (st % S) * STAGE_EL;
    const int k0 = st * BK;
#pragma unroll
    for (int t = 0; t < NBA; ++t) {
      const bf16* src = arow_ok[t] ? aptr[t] + k0 : zero;
      if (a.amode == ROWS_ITEM_HM) {
        // k -> part (Q, K, V), head, offset in head; K and V rows exist for train rows only.
        // A stage never straddles two parts (BK divides BN), so the part follows from k0
        // alone and the base pointer is chosen by a scalar branch.
        const int part = k0 / BN;
        const int within = k0 - part * BN + akc[t] * 8;
        const int head = within / g.d, jj = within - head * g.d;
        const bf16* base = part == 0 ? a.A : (part == 1 ? a.A2 : a.A3);
        src = arow_ok[t] && (part == 0 || hr[t] < hntr[t])
                  ? base + ((hcol[t] * g.heads + head) * g.R + hr[t]) * (int64_t)g.d + jj
                  : zero;
      }
      lds_dma16(src, sa + (wave + 4 * t) * 512);
    }
#pragma unroll
    for (int t = 0; t < NBB; ++t) lds_dma16(bptr[t] + k0, sa + A_EL + (wave + 4 * t) * 512);
  };

  // per-column epilogue parameters of this column tile, staged once
  if (tid < BN) {
    cpar[0][tid] = a.bias ? a.bias[n0 + tid] : 0.f;
    if (EPI == EPI_LN || EPI == EPI_LN_BWD || EPI == EPI_RMS || EPI == EPI_RMS_BWD)
      cpar[1][tid] = a.gamma[tid];
    if (EPI == EPI_LN) cpar[2][tid] = a.beta[tid];
    if (EPI == EPI_LN && a.rgamma) {
      cpar[3][tid] = a.rgamma[tid];
      cpar[4][tid] = a.rbeta[tid];
    }
  }

  // ---- epilogue inputs (residual, x-hat, pre-activation) do not depend on the product: their
  // rows are fetched into registers now, so that they travel with the first stages instead of
  // costing a memory round trip after the main loop.
  constexpr int CPRW = BN / 8;              // 16-byte chunks per tile row
  constexpr int NCH = BM * CPRW / 256;      // chunks per thread of one tile
  constexpr bool IN0 = EPI == EPI_GELU_BWD || EPI == EPI_DX || EPI == EPI_LN ||
                      EPI == EPI_LN_BWD || EPI == EPI_RMS || EPI == EPI_RMS_BWD;
  constexpr bool IN1 = EPI == EPI_LN_BWD || EPI == EPI_RMS_BWD;
  // Input tiles are prefetched at 64 rows; at 128 rows the second one (and at BN = 256 the
  // first too) is loaded when the main loop ends: prefetched, they would not fit in registers
  // next to the accumulators.
  constexpr bool IN0_PRE = IN0 && (BM == 64 || BN <= 192);
  constexpr bool IN1_PRE = IN1 && BM == 64;
  uint4 pin0[IN0 ? NCH : 1], pin1[IN1 ? NCH : 1];
  if (IN0) {
    if (tid < BM) {
      const int64_t m = m0 + tid;
      int64_t off = -1;
      if (m < a.M) {
        if (EPI == EPI_GELU_BWD) off = m * a.ldo;
        else if (EPI == EPI_LN || EPI == EPI_RMS || EPI == EPI_RMS_BWD)
          off = row_addr(g, a.rmode, m, BN);
        else off = m * BN;
      }
      rbase[tid] = off;
    }
    lds_barrier();
    const bf16* src0 = EPI == EPI_GELU_BWD ? a.aux + n0 : a.resid;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 256 * c;
      const int64_t off = rbase[ch / CPRW];
      const int cc = (ch % CPRW) * 8;
      if (IN0_PRE) pin0[c] = off >= 0 ? ldu4(src0 + off + cc) : make_uint4(0, 0, 0, 0);
      // The second input is always compact rows (x-hat, or h).  Rows past M read row M - 1
      // instead of zeros (no select on the loaded value): their accumulators and first input
      // are zero, so they add nothing to the column sums and are never stored.
      const int64_t m1 = m0 + ch / CPRW < a.M ? m0 + ch / CPRW : a.M - 1;
      if (IN1_PRE) pin1[c] = ldu4(a.aux + m1 * BN + cc);
    }
  }

  f32x4 acc[MI][NB];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = zero4();

  // Stage kt is consumed at iteration kt; S - 1 stages are in flight ahead of it.  Each wave
  // waits for its own loads of stage kt (vmcnt counts in issue order; a stage is 1 + NBB
  // loads), then the barrier makes every wave's part visible and frees the slot of stage
  // kt - 1, which stage kt + S - 1 refills.
  const int KT = a.K / BK;
#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < KT) issue(st);
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + S - 2 < KT) {
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((S - 2) * (NBA + NBB)) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    }
    if (kt + S - 1 < KT) issue(kt + S - 1);
    const bf16* sa = ring + (kt % S) * STAGE_EL;
    const bf16* sb = sa + A_EL;
    bf16x8 af[MI], bfr[NB];
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int r = wm * (BM / 2) + i * 16 + lr;
      af[i] = ld8(&sa[r * BK + kslot(r, lg) * 8]);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int n = wn * (BN / 2) + j * 16 + lr;
      bfr[j] = ld8(&sb[n * BK + kslot(n, lg) * 8]);
    }
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = mfma16(bfr[j], af[i], acc[i][j]);
  }
  lds_barrier();  // every wave is done with the ring before the epilogue tile reuses it
  if ((IN0 && !IN0_PRE) || (IN1 && !IN1_PRE)) {
    const bf16* src0 = EPI == EPI_GELU_BWD ? a.aux + n0 : a.resid;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 256 * c;
      const int64_t off = rbase[ch / CPRW];
      const int cc = (ch % CPRW) * 8;
      if (IN0 && !IN0_PRE) pin0[c] = off >= 0 ? ldu4(src0 + off + cc) : make_uint4(0, 0, 0, 0);
      const int64_t m1 = m0 + ch / CPRW < a.M ? m0 + ch / CPRW : a.M - 1;  // (as above)
      if (IN1 && !IN1_PRE) pin1[c] = ldu4(a.aux + m1 * BN + cc);
    }
  }

  // ---- epilogues.  acc[i][j][q] is C[row, col] with
  //   row = m0 + wm*BM/2 + i*16 + lr,  col = n0 + wn*BN/2 + j*16 + lg*4 + q
  // Global traffic goes through the LDS tile [BM][TS] in 16-byte row chunks: residual / x-hat
  // inputs are loaded into it, outputs are written into it and copied out row by row.
  const int cb0 = wn * (BN / 2) + lg * 4;  // tile column of q = 0 for j = 0
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
          if (hm_part == 0 || r < g.col_ntr[col])
            off = (col * g.heads * g.R + r) * (int64_t)g.d;
        } else {
          off = mode == ROWS_NATIVE ? native_cell(g, m) * g.E : m * ld;
        }
      }
      rbase[tid] = off;
    }
  };
  // tile <- prefetched rows
  auto fill_tile = [&](const uint4* pin) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 256 * c;
      stu4(&tile[(ch / CPRW) * TS + (ch % CPRW) * 8], pin[c]);
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
        const int head = (pc0 + cc) / g.d, jj = pc0 + cc - head * g.d;
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

  if (HALF) {
    if (EPI == EPI_ITEM_QKV)
      set_rows(ROWS_COMPACT, 0, part);
    else
      set_rows(ROWS_COMPACT, a.ldo, -1);
    // item K is stored pre-multiplied by log2(e)/sqrt(d) (in fp32, before the bf16 rounding):
    // the attention kernels then get scores in the exp2 domain straight from the MFMA
    const float ksc =
        EPI == EPI_ITEM_QKV && part == 1 ? 1.4426950408889634f / sqrtf((float)g.d) : 1.0f;
    bf16* dst = EPI == EPI_ITEM_QKV ? (part == 0 ? a.out : (part == 1 ? a.out2 : a.out3))
                                    : a.out;
    // half h holds tile rows [h BM/2, (h + 1) BM/2): the rows of the waves with wm == h
    for (int h = 0; h < 2; ++h) {
      if (wm == h) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const f32x4 b = par4(0, j);
#pragma unroll
          for (int i = 0; i < MI; ++i) {
            const f32x4 v = (acc[i][j] + b) * ksc;
            *reinterpret_cast<uint2*>(&tile[(i * 16 + lr) * TS + cb0 + j * 16]) =
                make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
          }
        }
      }
      lds_barrier();
      for (int ch = tid; ch < (BM / 2) * CPRW; ch += 256) {
        const int rl = ch / CPRW, cc = (ch % CPRW) * 8;
        const int64_t off = rbase[h * (BM / 2) + rl];
        if (off < 0) continue;
        int64_t o = off + (EPI == EPI_ITEM_QKV ? 0 : n0) + cc;
        if (EPI == EPI_ITEM_QKV) {
          const int head = (pc0 + cc) / g.d, jj = pc0 + cc - head * g.d;
          o = off + (int64_t)head * g.R * g.d + jj;
        }
        stu4(dst + o, ldu4(&tile[rl * TS + cc]));
      }
      lds_barrier();  // the next half overwrites the tile
    }
    return;
  }
  if (EPI == EPI_BIAS || EPI == EPI_GELU_FWD || EPI == EPI_ITEM_QKV) {
    if (EPI == EPI_ITEM_QKV)
      set_rows(ROWS_COMPACT, 0, part);
    else
      set_rows(ROWS_COMPACT, a.ldo, -1);
    // item K is stored pre-multiplied by log2(e)/sqrt(d) (in fp32, before the bf16 rounding):
    // the attention kernels then get scores in the exp2 domain straight from the MFMA
    const float ksc =
        EPI == EPI_ITEM_QKV && part == 1 ? 1.4426950408889634f / sqrtf((float)g.d) : 1.0f;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f32x4 b = par4(0, j);
#pragma unroll
      for (int i = 0; i < MI; ++i) put4(i, j, (acc[i][j] + b) * ksc);
    }
    lds_barrier();
    if (EPI == EPI_ITEM_QKV) {
      bf16* dst = part == 0 ? a.out : (part == 1 ? a.out2 : a.out3);
      store_tile(dst, 0, true);
      return;
    }
    // the GELU epilogue may skip the pre-activation store (out == nullptr: forward-only calls)
    if (EPI != EPI_GELU_FWD || a.out) store_tile(a.out, n0, false);
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
    fill_tile(pin0);  // rbase still holds the compact rows (leading dimension ldo)
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
    fill_tile(pin0);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] += tile4(i, j) + par4(0, j);
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
      sm = rows4_sum(sm);
      if (lg == 0) red[wn][rloc(i)] = sm;
    }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i) out[i] = (red[0][rloc(i)] + red[1][rloc(i)]) * (1.0f / BN);
    lds_barrier();
  };

  if (EPI == EPI_LN) {
    fill_tile(pin0);
    lds_barrier();
    if (a.rgamma) {  // the residual arrives as x-hat of the previous norm: rgamma x-hat + rbeta
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4 b = par4(0, j), rg = par4(3, j), rb = par4(4, j);
#pragma unroll
        for (int i = 0; i < MI; ++i) val[i][j] = acc[i][j] + b + (rg * tile4(i, j) + rb);
      }
    } else {
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4 b = par4(0, j);
#pragma unroll
        for (int i = 0; i < MI; ++i) val[i][j] = acc[i][j] + b + tile4(i, j);
      }
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
      if (a.rstd && wn == 0 && lg == 0 && m0 + rloc(i) < a.M) a.rstd[m0 + rloc(i)] = rs;
    }
    // h = gamma * x-hat + beta -> out (omode), or x-hat itself when xhat_out; x-hat -> xhat
    // (compact) unless xhat is null
    if (a.xhat_out) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) put4(i, j, val[i][j]);
    } else {
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const f32x4 gm = par4(1, j), bt = par4(2, j);
#pragma unroll
        for (int i = 0; i < MI; ++i) put4(i, j, gm * val[i][j] + bt);
      }
    }
    set_rows(a.omode, BN, -1);
    lds_barrier();
    store_tile(a.out, 0, false);
    if (!a.xhat) return;
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
    fill_tile(pin0);  // rbase still holds the compact rows
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) val[i][j] = acc[i][j] + tile4(i, j);
    lds_barrier();
    fill_tile(pin1);  // x-hat stays in the tile for the rest of the epilogue
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
        const float t1 = row16_sum(s1[q]), t2 = row16_sum(s2[q]);
        if (lr == 0) {
          cred[0][wm][cb0 + j * 16 + q] = t1;
          cred[1][wm][cb0 + j * 16 + q] = t2;
        }
      }
    }
    float m1[MI], m2[MI];
    row_sum([&](int i, int j) { return val[i][j] * par4(1, j); }, m1);
    if (tid < BN) {
      float* pg = a.part + bx * 2 * BN;
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

  // ---- pre-norm RMSNorm epilogues (BN == E, n0 == 0)
  if (EPI == EPI_RMS) {
    // h = C + bias + rscale * resid -> out; r = gamma h / sqrt(mean(h^2) + eps) -> out2
    fill_tile(pin0);
    lds_barrier();
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const f32x4 b = par4(0, j);
#pragma unroll
      for (int i = 0; i < MI; ++i) val[i][j] = acc[i][j] + b + a.rscale * tile4(i, j);
    }
    float ms[MI];
    row_sum([&](int i, int j) { return val[i][j] * val[i][j]; }, ms);
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, val[i][j]);
    set_rows(ROWS_COMPACT, BN, -1);
    lds_barrier();
    store_tile(a.out, 0, false);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const float rs = 1.0f / sqrtf(ms[i] + a.eps);
      if (a.rstd && wn == 0 && lg == 0 && m0 + rloc(i) < a.M) a.rstd[m0 + rloc(i)] = rs;
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, par4(1, j) * val[i][j] * rs);
    }
    lds_barrier();
    store_tile(a.out2, 0, false);
    return;
  }

  if (EPI == EPI_RMS_BWD) {
    // dr = C, uhat = h rstd_in:  out = oscale (resid + rstd_in (gamma dr - uhat mean(gamma dr
    // uhat))); column partials of dr uhat per workgroup
    fill_tile(pin1);  // h
    lds_barrier();
    float rsi[MI];
#pragma unroll
    for (int i = 0; i < MI; ++i) rsi[i] = m0 + rloc(i) < a.M ? a.rstd_in[m0 + rloc(i)] : 0.f;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      f32x4 s1 = zero4();
#pragma unroll
      for (int i = 0; i < MI; ++i) s1 += acc[i][j] * tile4(i, j) * rsi[i];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float t1 = row16_sum(s1[q]);
        if (lr == 0) cred[0][wm][cb0 + j * 16 + q] = t1;
      }
    }
    float m1[MI];
    row_sum([&](int i, int j) { return par4(1, j) * acc[i][j] * tile4(i, j) * rsi[i]; }, m1);
    if (tid < BN) a.part[bx * BN + tid] = cred[0][0][tid] + cred[0][1][tid];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        val[i][j] = rsi[i] * (par4(1, j) * acc[i][j] - tile4(i, j) * (rsi[i] * m1[i]));
    lds_barrier();
    fill_tile(pin0);  // resid
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) val[i][j] = a.oscale * (val[i][j] + tile4(i, j));
    lds_barrier();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) put4(i, j, val[i][j]);
    set_rows(a.omode, BN, -1);
    lds_barrier();
    store_tile(a.out, 0, false);
    return;
  }
}


// ============================================================== weight-resident persistent GEMM
// For the bias-only products whose contraction is the embedding width (K = E = BN): the
// workgroup's weight column tile (BN x K, at most 72 KB) lives in registers for the whole
// launch, split over 8 waves (2 row groups x 4 column groups), and the workgroup walks a
// sequence of 128-row tiles, streaming only A through an LDS ring of 8 KB stages that runs
// across tile boundaries: the next tile's rows are in flight during this tile's epilogue, and
// no LDS traffic is spent on B.  One workgroup per CU.  With several column tiles (N = 3E) the
// workgroups of one row-tile sequence are placed on one XCD, so that A comes from HBM once and
// then from that XCD's L2.  Epilogues: bias (EPI_BIAS) and head-major item Q|K|V
// (EPI_ITEM_QKV).  The products and the epilogue arithmetic are those of k_gemm (same MFMA
// order), so both kernels give identical results.  (The GELU epilogues stay on k_gemm: their
// VALU work needs the overlap of several workgroups per CU.)
// 16-byte store marked non-temporal (streamed past the caches' retention), for outputs that
// no later access of the same kernel reads
__device__ __forceinline__ void stu4_nt(bf16* p, uint4 v) {
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  const u32x4_t x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
}

template <int BN>
struct WrShape {
  static constexpr int WN = 4;                  // column waves
  static constexpr int WM = 2;                  // row waves
  static constexpr int BM = 128;
  static constexpr int MI = BM / WM / 16;       // 16-row blocks per wave
  static constexpr int NB = BN / WN / 16;       // 16-column blocks per wave
  static constexpr int KT = BN / BK;            // k steps (K = BN)
  static constexpr int NS = 8;                  // A stages in the ring (8 KB each)
  static constexpr int TS = BN + 8;             // epilogue tile row stride (elements)
  static constexpr int CPRW = BN / 8;           // 16-byte chunks per tile row
  static constexpr int NCH = BM * CPRW / 512;   // chunks of one tile per thread
};

template <int BN, int EPI>
__global__ __launch_bounds__(512, 1) void k_gemm_wr(GemmArgs a) {
  typedef WrShape<BN> Sh;
  constexpr int WN = Sh::WN, WM = Sh::WM, BM = Sh::BM, MI = Sh::MI, NB = Sh::NB, KT = Sh::KT;
  constexpr int NS = Sh::NS, TS = Sh::TS, CPRW = Sh::CPRW, NCH = Sh::NCH;
  constexpr int STAGE = BM * BK;
  __shared__ __attribute__((aligned(16))) bf16 ring[NS * STAGE];
  __shared__ __attribute__((aligned(16))) bf16 tile[BM * TS];
  __shared__ __attribute__((aligned(16))) float cb[BN];
  __shared__ int64_t rbase[BM];

  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 15, lg = lane >> 4;
  const Geo& g = a.g;
  // workgroup -> (column tile, row-tile sequence); the NY column tiles of a sequence share an XCD
  const int NY = a.N / BN;
  const int xcd = (int)(blockIdx.x & 7), li = (int)(blockIdx.x >> 3);
  const int gpx = (int)(gridDim.x >> 3) / NY;  // sequences per XCD
  if (li >= gpx * NY) return;
  const int by = li % NY;
  const int64_t grp = (int64_t)xcd * gpx + li / NY, NG = 8 * (int64_t)gpx;
  const int n0 = by * BN;
  const int64_t MT = (a.M + BM - 1) / BM;
  const int64_t ntile = grp < MT ? (MT - 1 - grp) / NG + 1 : 0;
  if (ntile == 0) return;
  const int64_t nst = ntile * KT;
  const int part = EPI == EPI_ITEM_QKV ? n0 / g.E : 0;
  const int pc0 = n0 - part * g.E;

  // this wave's weight slice: output columns n0 + wn * BN / WN + j * 16 + lr, k 8 lg (+ 32 ks)
  bf16x8 bfr[KT][NB];
#pragma unroll
  for (int ks = 0; ks < KT; ++ks)
#pragma unroll
    for (int j = 0; j < NB; ++j)
      bfr[ks][j] = ld8(a.Bt + (int64_t)(n0 + wn * (BN / WN) + j * 16 + lr) * a.K + ks * BK + 8 * lg);
  if (tid < BN) cb[tid] = a.bias ? a.bias[n0 + tid] : 0.f;

  // A streaming: every thread moves one 16-byte piece per stage: row tid / 4 of the tile, k
  // chunk kslot(row, tid % 4) (the layout k_gemm reads); a stage is one load of each thread,
  // so that its completion can be awaited by count
  const bf16* zero = reinterpret_cast<const bf16*>(&kZeroChunk);
  const int ar = tid >> 2;
  const int akc = kslot(ar, tid & 3);
  int64_t iss_tile = -1;
  const bf16* iss_row = zero;
  auto issue = [&](int64_t st) {
    const int64_t j = st / KT;
    const int kt = (int)(st - j * KT);
    if (j != iss_tile) {
      iss_tile = j;
      const int64_t am = (grp + j * NG) * BM + ar;
      iss_row = am < a.M ? a.A + row_addr(g, a.amode, am, a.lda) + akc * 8 : nullptr;
    }
    lds_dma16(iss_row ? iss_row + kt * BK : zero, ring + (st % NS) * STAGE + wave * 512);
  };
  // NS - 1 stages ahead; past the last stage, loads of zeros into the free slots keep the
  // count of younger loads that the waits below rely on
#pragma unroll
  for (int st = 0; st < NS - 1; ++st) {
    if (st < nst) issue(st);
    else lds_dma16(zero, ring + st * STAGE + wave * 512);
  }

  auto rloc = [&](int i) { return wm * (BM / WM) + i * 16 + lr; };
  const int cb0 = wn * (BN / WN) + lg * 4;
  // item K is stored pre-multiplied by log2(e)/sqrt(d), as k_gemm does
  const float ksc =
      EPI == EPI_ITEM_QKV && part == 1 ? 1.4426950408889634f / sqrtf((float)g.d) : 1.0f;

  for (int64_t j = 0; j < ntile; ++j) {
    const int64_t m0 = (grp + j * NG) * BM;
    f32x4 acc[MI][NB];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int jj = 0; jj < NB; ++jj) acc[i][jj] = zero4();
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      const int64_t st = j * KT + kt;
      // stage st has landed once at most the NS - 2 stage loads issued after it are
      // outstanding (loads complete in order; stores issued since only add younger ops)
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(NS - 2) : "memory");
      if (st + NS - 1 < nst) issue(st + NS - 1);
      else  // a load into the free slot keeps the count of younger loads
        lds_dma16(zero, ring + ((st + NS - 1) % NS) * STAGE + wave * 512);
      const bf16* sa = ring + (st % NS) * STAGE;
      bf16x8 af[MI];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int r = rloc(i);
        af[i] = ld8(&sa[r * BK + kslot(r, lg) * 8]);
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int jj = 0; jj < NB; ++jj) acc[i][jj] = mfma16(bfr[kt][jj], af[i], acc[i][jj]);
    }

    // ---- epilogue: per-row destinations, then the tile through LDS in 16-byte row chunks
    if (tid < BM) {
      const int64_t m = m0 + tid;
      int64_t off = -1;
      if (m < a.M) {
        if (EPI == EPI_ITEM_QKV) {
          const int64_t col = m / g.R;
          const int r = (int)(m - col * g.R);
          if (part == 0 || r < g.col_ntr[col]) off = (col * g.heads * g.R + r) * (int64_t)g.d;
        } else {
          off = m * a.ldo + n0;
        }
      }
      rbase[tid] = off;
    }
#pragma unroll
    for (int jj = 0; jj < NB; ++jj) {
      const float4 bb = *reinterpret_cast<const float4*>(&cb[cb0 + jj * 16]);
      f32x4 b4;
      b4[0] = bb.x; b4[1] = bb.y; b4[2] = bb.z; b4[3] = bb.w;
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const f32x4 v = (acc[i][jj] + b4) * ksc;
        *reinterpret_cast<uint2*>(&tile[rloc(i) * TS + cb0 + jj * 16]) =
            make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
      }
    }
    lds_barrier();
    bf16* dst = EPI == EPI_ITEM_QKV ? (part == 0 ? a.out : (part == 1 ? a.out2 : a.out3)) : a.out;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int ch = tid + 512 * c;
      const int row = ch / CPRW, cc = (ch % CPRW) * 8;
      const int64_t off = rbase[row];
      if (off < 0) continue;
      int64_t o = off + cc;
      if (EPI == EPI_ITEM_QKV) {
        const int head = (pc0 + cc) / g.d, jd = pc0 + cc - head * g.d;
        o = off + (int64_t)head * g.R * g.d + jd;
      }
      // saved tensors read only by later kernels (the Q|K|V projections) stream past the caches;
      // the single-tile products' outputs, which the next kernel reads, do not
      if (EPI == EPI_ITEM_QKV || NY > 1)
        stu4_nt(dst + o, ldu4(&tile[row * TS + cc]));
      else
        stu4(dst + o, ldu4(&tile[row * TS + cc]));
    }
  }
}

// The weight-resident kernel applies to K = E = BN <= 192 products with the bias or item
// Q|K|V epilogue, A rows compact or native (at BN = 256 the weight slice leaves too few
// registers); grid: one workgroup per CU.
static bool gemm_wr_ok(const GemmArgs& a) {
  const bool epi = a.epi == EPI_BIAS || a.epi == EPI_ITEM_QKV;
  const bool mode = a.amode == ROWS_COMPACT || a.amode == ROWS_NATIVE;
  return epi && mode && a.K == a.BN && a.N % a.BN == 0 && a.N / a.BN <= 32 &&
         (a.BN == 64 || a.BN == 128 || a.BN == 192);
}

template <int BN>
static hipError_t gemm_wr_dispatch(const GemmArgs& a, hipStream_t s) {
  const unsigned grid = 256;
  if (a.epi == EPI_BIAS)
    k_gemm_wr<BN, EPI_BIAS><<<grid, 512, 0, s>>>(a);
  else
    k_gemm_wr<BN, EPI_ITEM_QKV><<<grid, 512, 0, s>>>(a);
  return hipGetLastError();
}

template <int BN>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t s) {
  // 128-row tiles (each weight tile staged through LDS serves twice the rows), except for the
  // two-input epilogues at BN = 256, which would spill.  gemm_tiles() gives the row-tile count
  // (the partial-sum rows of LN_BWD / RMS_BWD).
  const bool in0 = a.epi == EPI_GELU_BWD || a.epi == EPI_LN || a.epi == EPI_DX ||
                   a.epi == EPI_RMS;
  const bool wide = !(BN > 192 && (a.epi == EPI_LN_BWD || a.epi == EPI_RMS_BWD));
  const int bm = wide ? 128 : GEMM_BM;
  const int64_t mt = (a.M + bm - 1) / bm;
  const dim3 grid((unsigned)((mt + 7) / 8 * 8 * (a.N / BN)));
  if (wide) {
    switch (a.epi) {
      case EPI_BIAS: k_gemm<BN, EPI_BIAS, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_GELU_FWD: k_gemm<BN, EPI_GELU_FWD, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_ITEM_QKV: k_gemm<BN, EPI_ITEM_QKV, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_GELU_BWD: k_gemm<BN, EPI_GELU_BWD, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_LN: k_gemm<BN, EPI_LN, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_DX: k_gemm<BN, EPI_DX, 128><<<grid, 256, 0, s>>>(a); break;
      case EPI_RMS: k_gemm<BN, EPI_RMS, 128><<<grid, 256, 0, s>>>(a); break;
      default:
        if constexpr (BN <= 192) {
          if (a.epi == EPI_LN_BWD) k_gemm<BN, EPI_LN_BWD, 128><<<grid, 256, 0, s>>>(a);
          else if (a.epi == EPI_RMS_BWD) k_gemm<BN, EPI_RMS_BWD, 128><<<grid, 256, 0, s>>>(a);
          else return hipErrorInvalidValue;
        } else {
          return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
  }
  switch (a.epi) {
    case EPI_BIAS: k_gemm<BN, EPI_BIAS, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_GELU_FWD: k_gemm<BN, EPI_GELU_FWD, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_GELU_BWD: k_gemm<BN, EPI_GELU_BWD, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_ITEM_QKV: k_gemm<BN, EPI_ITEM_QKV, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_LN: k_gemm<BN, EPI_LN, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_LN_BWD: k_gemm<BN, EPI_LN_BWD, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_DX: k_gemm<BN, EPI_DX, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_RMS: k_gemm<BN, EPI_RMS, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    case EPI_RMS_BWD: k_gemm<BN, EPI_RMS_BWD, GEMM_BM><<<grid, 256, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int64_t gemm_tiles(int epi, int BN, int64_t M) {
  const int bm = BN > 192 && (epi == EPI_LN_BWD || epi == EPI_RMS_BWD) ? GEMM_BM : 128;
  return (M + bm - 1) / bm;
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.K % BK || a.N % a.BN) return hipErrorInvalidValue;
  if (gemm_wr_ok(a)) {
    switch (a.BN) {
      case 64: return gemm_wr_dispatch<64>(a, s);
      case 128: return gemm_wr_dispatch<128>(a, s);
      default: return gemm_wr_dispatch<192>(a, s);
    }
  }
  switch (a.BN) {
    case 64: return gemm_dispatch<64>(a, s);
    case 128: return gemm_dispatch<128>(a, s);
    case 192: return gemm_dispatch<192>(a, s);
    case 256: return gemm_dispatch<256>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tfm
