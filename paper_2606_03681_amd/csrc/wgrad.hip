// Weight gradients on bf16 MFMA: dW[n][k] = sum over active cells m of dY[m][n] X[m][k], with
// the bias gradient db[n] = sum_m dY[m][n] formed from the same staged data.
//
// The reduction runs over the cells (1.6 M at eval scale) while the output is one E x E tile
// of the weight, so the cells are split into chunks (split-K): workgroup (n-tile, k-tile, z)
// sums chunk z into a float32 partial, and a second kernel adds the partials in a fixed order
// (bitwise reproducible).  The MFMA contraction index is the cell, the slow index in memory
// for both operands: 32-cell slices of dY and X are copied row-major into LDS with 16-byte
// stores and read back transposed with ds_read_b64_tr_b16.  Slot t of a lane's 8-element
// fragment (lane group g = lane / 16) holds cell 16 (t / 4) + 4 g + t % 4 of the slice, for A
// and B alike, so each half-wave transpose read touches 8 consecutive rows; with a row stride
// of an odd multiple of 32 bytes those rows fall on disjoint LDS banks.
#include "fast.h"
#include "mfma.h"

namespace tfm {

namespace {
constexpr int MS = 32;  // cells per step

// One staged 16-byte chunk of an operand: features [f, f + 8) of the cell `off` rows into each
// slice.  The cursor moves one slice (MS cells) per load without division; the layout MODE
// (compact, native, head-major item gradients) selects which fields are used.
struct Cursor {
  int64_t addr;  // element offset of the chunk for the next slice to load
  int rem;       // cells left in the workgroup's range from this chunk's cell (<= 0: done)
  int col, r;    // active column and row of that cell (ROWS_NATIVE, ROWS_ITEM_HM)
  int ntr;       // train-prefix length of the column (ROWS_ITEM_HM)
  int hmo;       // ROWS_ITEM_HM: head * R * d + offset in head
  int part;      // ROWS_ITEM_HM: 0, 1, 2 for Q, K, V
};

template <int MODE>
__device__ __forceinline__ void cur_init(Cursor& c, const Geo& g, int64_t m, int64_t me, int f,
                                         int64_t ld) {
  c.rem = (int)(me - m);
  c.col = (int)(m / g.R);
  c.r = (int)(m - (int64_t)c.col * g.R);
  c.ntr = 0;
  c.part = 0;
  c.hmo = 0;
  if (MODE == ROWS_COMPACT) {
    c.addr = m * ld + f;
  } else if (MODE == ROWS_NATIVE) {
    c.addr = c.rem > 0 ? native_cell(g, m) * g.E + f : 0;
  } else {
    c.part = f / g.E;
    const int within = f - c.part * g.E;
    const int head = within / g.d;
    c.hmo = head * g.R * g.d + (within - head * g.d);
    c.addr = 0;
    if (c.rem > 0) {
      c.ntr = g.col_ntr[c.col];
      c.addr = ((int64_t)c.col * g.heads * g.R + c.r) * g.d + c.hmo;
    }
  }
}

// The load is always issued (a row that does not exist reads the operand's first chunk, and
// *ok tells the consumer to use zeros instead): with no branch around it and no use of the
// value until the slice is stored to LDS, the number of loads in flight is fixed and each wait
// counts exactly the older loads instead of draining all of them.
template <int MODE>
__device__ __forceinline__ uint4 cur_load(const Cursor& c, const bf16* p0, const bf16* p1,
                                          const bf16* p2, bool* ok) {
  bool v = c.rem > 0;
  const bf16* base = p0;
  if (MODE == ROWS_ITEM_HM) {
    base = c.part == 0 ? p0 : (c.part == 1 ? p1 : p2);
    v = v && (c.part == 0 || c.r < c.ntr);
  }
  *ok = v;
  return ldu4(base + (v ? c.addr : 0));
}

// cell0 / ntr: the column metadata (entry col - lo for column col); the workgroup's own copy
// in LDS where it has one, so that crossing into the next column costs no global load (whose
// wait would also wait for every data load in flight).
template <int MODE>
__device__ __forceinline__ void cur_advance(Cursor& c, const Geo& g, int64_t ld, int f,
                                            const int64_t* cell0, const int32_t* ntr, int lo) {
  c.rem -= MS;
  if (MODE == ROWS_COMPACT) {
    c.addr += MS * ld;
    return;
  }
  c.r += MS;
  if (c.r < g.R) {
    c.addr += (MODE == ROWS_NATIVE ? (int64_t)g.S * g.E : (int64_t)g.d) * MS;
    return;
  }
  while (c.r >= g.R) {
    c.r -= g.R;
    ++c.col;
  }
  if (c.rem <= 0) return;
  if (MODE == ROWS_NATIVE) {
    c.addr = (cell0[c.col - lo] + (int64_t)c.r * g.S) * g.E + f;
  } else {
    c.ntr = ntr[c.col - lo];
    c.addr = ((int64_t)c.col * g.heads * g.R + c.r) * g.d + c.hmo;
  }
}
}  // namespace

// 512 threads = 8 waves in a 2 (n) x 4 (k) arrangement; tile BN x BK.  dY is in layout YM
// (compact, native or head-major item gradients), X in layout XM (compact or native).  TBL: the
// workgroup copies the metadata of the columns its chunk spans into LDS (requires R >= MS, so
// that a chunk spans at most WGRAD_CHUNK_MAX / MS + 1 columns).
template <int BN, int BK, int YM, int XM, bool TBL>
__global__ __launch_bounds__(512) void k_wgrad(WgradArgs a) {
  constexpr int NBW = BN / 32;      // 16-row blocks per wave along n (BN/2 rows)
  constexpr int KBW = BK / 64;      // 16-col blocks per wave along k (BK/4 cols)
  constexpr int LSA = BN + 16;      // LDS row strides (elements): odd multiples of 32 bytes
  constexpr int LSB = BK + 16;
  constexpr int CPA = BN / 64;      // 16-byte chunks per staging thread and slice (dY)
  constexpr int CPB = BK / 64;      // (X)
  __shared__ __attribute__((aligned(16))) bf16 As[2][MS * LSA];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][MS * LSB];

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int lg = lane >> 4, c = lane & 15;
  const int wn = w >> 2, wk = w & 3;
  // Workgroup -> (cell chunk z, n-tile, k-tile).  The hardware deals consecutive workgroups
  // round-robin over the 8 XCDs; all tiles of one chunk get consecutive slots of one XCD, so
  // the chunk's rows come from memory once and are then served by that XCD's L2.
  const int NX = a.N / BN, NT = NX * (a.K / BK);
  const int idx = (int)(blockIdx.x >> 3), xcd = (int)(blockIdx.x & 7);
  const int64_t zb = (int64_t)(idx / NT) * 8 + xcd;
  const int tl = idx % NT;
  const int tx = tl % NX, ty = tl / NX;
  const int64_t mb = zb * a.chunk;
  if (mb >= a.M) return;
  const int n0 = tx * BN, k0 = ty * BK;
  const int64_t me = mb + a.chunk < a.M ? mb + a.chunk : a.M;
  const Geo& g = a.g;

  constexpr int CT = WGRAD_CHUNK_MAX / MS + 2;
  __shared__ int64_t tcell[TBL ? CT : 1];
  __shared__ int32_t tntr[TBL ? CT : 1];
  const int lo = TBL ? (int)(mb / g.R) : 0;
  if (TBL) {
    const int ncol = (int)((me - 1) / g.R) - lo + 1;
    for (int i = tid; i < ncol && i < CT; i += 512) {
      tcell[i] = g.col_cell0[lo + i];
      tntr[i] = g.col_ntr[lo + i];
    }
    __syncthreads();
  }
  const int64_t* cell0 = TBL ? tcell : g.col_cell0;
  const int32_t* ntrp = TBL ? tntr : g.col_ntr;

  // staging: threads 0-255 stage dY features [n0, n0+BN), threads 256-511 X features
  // [k0, k0+BK); chunk ch -> cell ch / (width/8) of the slice, features (ch % (width/8)) * 8
  // role of the wave (uniform across it: scalar branches, so the two roles' loads are never
  // taken for one instruction stream)
  const bool opa = __builtin_amdgcn_readfirstlane(w) < 4;
  const int st = tid & 255;
  constexpr int CPM = CPA > CPB ? CPA : CPB;
  Cursor cu[CPM];  // one array for both roles (a select between two arrays would not stay in
                   // registers)
#pragma unroll
  for (int i = 0; i < CPM; ++i) {
    const int ch = st + 256 * i;
    if (opa) {
      if (i < CPA) cur_init<YM>(cu[i], g, mb + ch / (BN / 8), me, n0 + (ch % (BN / 8)) * 8, a.ldy);
    } else {
      if (i < CPB) cur_init<XM>(cu[i], g, mb + ch / (BK / 8), me, k0 + (ch % (BK / 8)) * 8, a.ldx);
    }
  }
  // One role branch around all of a thread's loads (not one per load), so that the other
  // role's loads never precede them on any path; the zeroing of missing rows is deferred to
  // the LDS store (okm: bit i set when chunk i of the slice exists).
  static_assert(CPA == CPB, "square tiles: with unequal chunk counts the compiler merges the "
                            "two role branches with non-constant indices (scratch arrays)");
  auto gload = [&](uint4* r, uint32_t& okm) __attribute__((always_inline)) {
    okm = 0u;
    if (opa) {
#pragma unroll
      for (int i = 0; i < CPA; ++i) {
        const int ch = st + 256 * i;
        bool ok;
        r[i] = cur_load<YM>(cu[i], a.dY, a.dY2, a.dY3, &ok);
        okm |= ok ? 1u << i : 0u;
        cur_advance<YM>(cu[i], g, a.ldy, n0 + (ch % (BN / 8)) * 8, cell0, ntrp, lo);
      }
    } else {
#pragma unroll
      for (int i = 0; i < CPB; ++i) {
        const int ch = st + 256 * i;
        bool ok;
        r[i] = cur_load<XM>(cu[i], a.X, nullptr, nullptr, &ok);
        okm |= ok ? 1u << i : 0u;
        cur_advance<XM>(cu[i], g, a.ldx, k0 + (ch % (BK / 8)) * 8, cell0, ntrp, lo);
      }
    }
  };
  const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
  auto sstore = [&](const uint4* r, uint32_t okm, int b) __attribute__((always_inline)) {
    if (opa) {
#pragma unroll
      for (int i = 0; i < CPA; ++i) {
        const int ch = st + 256 * i;
        stu4(&As[b][(ch / (BN / 8)) * LSA + (ch % (BN / 8)) * 8], (okm >> i) & 1u ? r[i] : z4);
      }
    } else {
#pragma unroll
      for (int i = 0; i < CPB; ++i) {
        const int ch = st + 256 * i;
        stu4(&Bs[b][(ch / (BK / 8)) * LSB + (ch % (BK / 8)) * 8], (okm >> i) & 1u ? r[i] : z4);
      }
    }
  };
  // fragment of the 16 columns starting at c0 (k positions: the slice's 32 cells)
  auto frag = [&](const bf16* T, int ls, int c0) -> bf16x8 { return ld_tr8(T, ls, c0, lane); };

  f32x4 acc[NBW][KBW];
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int j = 0; j < KBW; ++j) acc[i][j] = zero4();
  // bias gradient: the k-tile-0 waves with wk == 0 sum the dY fragments they already hold
  const bool bsum = a.bpart && ty == 0 && wk == 0;  // wave-uniform
  float bacc[NBW];
#pragma unroll
  for (int i = 0; i < NBW; ++i) bacc[i] = 0.f;

  auto compute = [&](int b) __attribute__((always_inline)) {
    bf16x8 af[NBW], bfr[KBW];
#pragma unroll
    for (int i = 0; i < NBW; ++i) af[i] = frag(As[b], LSA, wn * (BN / 2) + i * 16);
#pragma unroll
    for (int j = 0; j < KBW; ++j) bfr[j] = frag(Bs[b], LSB, wk * (BK / 4) + j * 16);
#pragma unroll
    for (int i = 0; i < NBW; ++i)
#pragma unroll
      for (int j = 0; j < KBW; ++j) acc[i][j] = mfma16(af[i], bfr[j], acc[i][j]);
    if (bsum) {
#pragma unroll
      for (int i = 0; i < NBW; ++i) {
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) t += (float)af[i][e];
        bacc[i] += t;
      }
    }
  };

  // Two register sets: slice s + 2 is loaded while slice s is multiplied, and slice s + 1
  // (loaded one step earlier) goes to LDS at the end of step s.  Loads and stores run
  // unconditionally (slices past the end are zero and never multiplied), so the loads in
  // flight are always the same ones.
  const int64_t steps = (me - mb + MS - 1) / MS;
  uint4 r0[CPM], r1[CPM];
  uint32_t ok0, ok1;
  gload(r0, ok0);
  gload(r1, ok1);
  sstore(r0, ok0, 0);
  lds_barrier();
  for (int64_t s = 0; s < steps; s += 2) {
    // even step s: compute buffer 0; r0 refills with slice s + 2; r1 (slice s + 1) -> buffer 1
    gload(r0, ok0);
    compute(0);
    sstore(r1, ok1, 1);
    lds_barrier();
    if (s + 1 >= steps) break;
    // odd step s + 1: compute buffer 1; r1 refills with slice s + 3; r0 (slice s + 2) -> 0
    gload(r1, ok1);
    compute(1);
    sstore(r0, ok0, 0);
    lds_barrier();
  }

  // partial tile: lane holds rows n = wn*BN/2 + i*16 + 4*lg + q, column k = wk*BK/4 + j*16 + c
  float* out = a.part + zb * a.N * a.K;
#pragma unroll
  for (int i = 0; i < NBW; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + wn * (BN / 2) + i * 16 + lg * 4 + q;
#pragma unroll
      for (int j = 0; j < KBW; ++j)
        out[(int64_t)n * a.K + k0 + wk * (BK / 4) + j * 16 + c] = acc[i][j][q];
    }
  if (bsum) {
    // lane (lg, c) summed 8 cells of feature n = wn*BN/2 + i*16 + c; add the four lane groups
#pragma unroll
    for (int i = 0; i < NBW; ++i) {
      float t = bacc[i];
      t = rows4_sum(t);
      if (lg == 0) a.bpart[zb * a.N + n0 + wn * (BN / 2) + i * 16 + c] = t;
    }
  }
}

// out[i] = (accumulate ? out[i] : 0) + sum over z in [z0, z1) of part[z * stride + i], with
// z0 = blockIdx.y * zc, z1 = min(Z, z0 + zc), and out advanced by blockIdx.y * out_ystride.  A
// block owns 32 groups of four consecutive outputs; 8 z-groups of threads each sum z = z0 + zg,
// z0 + zg + 8, ... with four independent accumulators, combined in a fixed order (bitwise
// reproducible).  out may be the first partial row of the block's own range (the first pass of
// a two-pass sum): every read of the range precedes the barrier, every write follows it, and no
// other block touches the range.  With fg given, output i = n K + k receives
// sum * fg[k] + sb[n] * fb[k] instead of the sum (the folded LayerNorm affine of the product's
// input; sb holds the bias-gradient sums).
__global__ __launch_bounds__(256) void k_reduce_z(int Z, int zc, int64_t count, int64_t stride,
                                                  const float* part, float* out,
                                                  int64_t out_ystride, int accumulate,
                                                  const float* fg, const float* fb,
                                                  const float* sb, int fK) {
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
    float tv[4] = {t.x, t.y, t.z, t.w};
    if (fg) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t i = i4 + k;
        const int n = (int)(i / fK), kk = (int)(i - (int64_t)n * fK);
        if (i < count) tv[k] = fmaf(tv[k], fg[kk], sb[n] * fb[kk]);
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (i4 + k < count) out[i4 + k] = (accumulate ? out[i4 + k] : 0.f) + tv[k];
  }
}

int64_t wgrad_chunk(int64_t M) {
  int64_t c = (M + WGRAD_SLOTS - 1) / WGRAD_SLOTS;
  c = (c + MS - 1) / MS * MS;
  if (c < MS) c = MS;
  return c < WGRAD_CHUNK_MAX ? c : WGRAD_CHUNK_MAX;
}

int wgrad_chunks(int64_t M) {
  const int64_t c = wgrad_chunk(M);
  const int64_t z = (M + c - 1) / c;
  return (int)(z < 1 ? 1 : z);
}

int64_t wgrad_max_chunks(int64_t Mmax) {
  const int64_t big = (Mmax + WGRAD_CHUNK_MAX - 1) / WGRAD_CHUNK_MAX;
  return big > WGRAD_SLOTS ? big : WGRAD_SLOTS;
}

template <int BN, int BK>
static hipError_t wgrad_modes(const WgradArgs& b, dim3 grid, hipStream_t s) {
  const bool yhm = b.ymode == ROWS_ITEM_HM, xnat = b.xmode == ROWS_NATIVE;
  const bool ynat = b.ymode == ROWS_NATIVE;
  if (b.ymode != ROWS_COMPACT && !yhm && !ynat) return hipErrorInvalidValue;
  if (b.xmode != ROWS_COMPACT && !xnat) return hipErrorInvalidValue;
  if (ynat && xnat) return hipErrorInvalidValue;
  const bool tbl = b.g.R >= MS;
  if (ynat) {
    if (tbl) k_wgrad<BN, BK, ROWS_NATIVE, ROWS_COMPACT, true><<<grid, 512, 0, s>>>(b);
    else k_wgrad<BN, BK, ROWS_NATIVE, ROWS_COMPACT, false><<<grid, 512, 0, s>>>(b);
  } else if (yhm && xnat) {
    if (tbl) k_wgrad<BN, BK, ROWS_ITEM_HM, ROWS_NATIVE, true><<<grid, 512, 0, s>>>(b);
    else k_wgrad<BN, BK, ROWS_ITEM_HM, ROWS_NATIVE, false><<<grid, 512, 0, s>>>(b);
  } else if (yhm) {
    if (tbl) k_wgrad<BN, BK, ROWS_ITEM_HM, ROWS_COMPACT, true><<<grid, 512, 0, s>>>(b);
    else k_wgrad<BN, BK, ROWS_ITEM_HM, ROWS_COMPACT, false><<<grid, 512, 0, s>>>(b);
  } else if (xnat) {
    if (tbl) k_wgrad<BN, BK, ROWS_COMPACT, ROWS_NATIVE, true><<<grid, 512, 0, s>>>(b);
    else k_wgrad<BN, BK, ROWS_COMPACT, ROWS_NATIVE, false><<<grid, 512, 0, s>>>(b);
  } else {
    k_wgrad<BN, BK, ROWS_COMPACT, ROWS_COMPACT, false><<<grid, 512, 0, s>>>(b);
  }
  return hipGetLastError();
}

hipError_t launch_wgrad_mfma(const WgradArgs& a, hipStream_t s) {
  const int Z = wgrad_chunks(a.M);
  // Square tiles (the two staging roles then move equal chunk counts); E = 256 takes 128 x 128
  // tiles, whose accumulators fit the registers of a 512-thread workgroup.
  const int BN = a.g.E > 192 ? 128 : a.g.E, BK = BN;
  if (a.N % BN || a.K % BK) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(((int64_t)Z + 7) / 8 * 8 * (a.N / BN) * (a.K / BK)));
  WgradArgs b = a;
  b.chunk = wgrad_chunk(a.M);
  switch (BN) {
    case 64: return wgrad_modes<64, 64>(b, grid, s);
    case 128: return wgrad_modes<128, 128>(b, grid, s);
    case 192: return wgrad_modes<192, 192>(b, grid, s);
    default: return hipErrorInvalidValue;
  }
}

static hipError_t reduce_z(int Z, int64_t count, int64_t stride, float* part, float* out,
                           int accumulate, const float* fg, const float* fb, const float* sb,
                           int fK, hipStream_t s) {
  if (Z <= 0 || count <= 0) return hipSuccess;
  const unsigned bx = (unsigned)((count + 127) / 128);
  // Few output blocks and many partials: first fold groups of ZC partials into the first row
  // of each group, leaving ceil(Z / ZC) partials ZC rows apart.
  constexpr int ZC = 64;
  if (bx < 512 && Z > 2 * ZC) {
    const unsigned groups = (unsigned)((Z + ZC - 1) / ZC);
    k_reduce_z<<<dim3(bx, groups), 256, 0, s>>>(Z, ZC, count, stride, part, part,
                                                 (int64_t)ZC * stride, 0, nullptr, nullptr,
                                                 nullptr, 1);
    Z = (int)groups;
    stride *= ZC;
  }
  k_reduce_z<<<dim3(bx, 1), 256, 0, s>>>(Z, Z, count, stride, part, out, 0, accumulate, fg, fb,
                                         sb, fK);
  return hipGetLastError();
}

hipError_t launch_reduce_z(int Z, int64_t count, int64_t stride, float* part, float* out,
                           int accumulate, hipStream_t s) {
  return reduce_z(Z, count, stride, part, out, accumulate, nullptr, nullptr, nullptr, 1, s);
}

hipError_t launch_reduce_wfold(int Z, int N, int K, float* wpart, float* bpart,
                               const float* gamma, const float* beta, float* grad,
                               int accumulate, hipStream_t s) {
  if (Z <= 0 || N <= 0 || K <= 0) return hipSuccess;
  // the bias sums first, into the first partial row of bpart (in place), which the folded
  // weight sums then read
  hipError_t e = reduce_z(Z, N, N, bpart, bpart, 0, nullptr, nullptr, nullptr, 1, s);
  if (e != hipSuccess) return e;
  return reduce_z(Z, (int64_t)N * K, (int64_t)N * K, wpart, grad, accumulate, gamma, beta, bpart,
                  K, s);
}

}  // namespace tfm
