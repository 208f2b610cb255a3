// Host side of the C ABI declared in include/tfm_layer.h: argument validation, the
// active-cell plan, buffer layouts and the launch sequences of the forward and backward pass.
#include "tfm_layer.h"
#include "tfm_prof.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <numeric>
#include <string>
#include <vector>

#include "kernels.h"
#include "attn.h"
#include "fast.h"
#include "prof.h"
#include "static_scratch.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

constexpr size_t kAlign = 256;
constexpr int64_t kChunk = 8192;  // rows per partial sum of the parameter-gradient reductions
constexpr int64_t kMaxCells = int64_t(1) << 26;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Dims {
  int B, R, C, S, E, heads, d, H, dtype;
  int block;       // TFM_BLOCK_POSTNORM or TFM_BLOCK_PRENORM
  float decay;     // pre-norm block: factor on the block input
  size_t tsz;      // bytes per stored element
  int64_t Nmax;    // B * R * S
  int words;       // 32-bit mask words per dataset
};

int check_dims(const tfm_dims* p, Dims& d) {
  if (!p) return fail(TFM_ERR_POINTER, "dims is null");
  d.B = p->B; d.R = p->R; d.C = p->C; d.E = p->E; d.heads = p->heads; d.H = p->H;
  d.dtype = p->dtype;
  if (d.dtype != TFM_F32 && d.dtype != TFM_BF16)
    return fail(TFM_ERR_DIMS, "dtype %d is neither TFM_F32 nor TFM_BF16", d.dtype);
  if (d.B < 1 || d.R < 1) return fail(TFM_ERR_DIMS, "B=%d and R=%d must be >= 1", d.B, d.R);
  if (d.C < 0 || d.C > 255) return fail(TFM_ERR_DIMS, "C=%d outside [0, 255]", d.C);
  if (d.E < 32 || d.E > 256 || d.E % 32)
    return fail(TFM_ERR_DIMS, "E=%d must be a multiple of 32 in [32, 256]", d.E);
  if (d.H < 32 || d.H > 1024 || d.H % 32)
    return fail(TFM_ERR_DIMS, "H=%d must be a multiple of 32 in [32, 1024]", d.H);
  if (d.heads < 1 || d.E % d.heads)
    return fail(TFM_ERR_HEAD_DIM, "E=%d is not a multiple of heads=%d", d.E, d.heads);
  d.d = d.E / d.heads;
  if (d.d != 16 && d.d != 32 && d.d != 64)
    return fail(TFM_ERR_HEAD_DIM, "head dim E/heads=%d not supported (16, 32 or 64)", d.d);
  d.S = d.C + 1;
  d.Nmax = (int64_t)d.B * d.R * d.S;
  if (d.Nmax > kMaxCells)
    return fail(TFM_ERR_DIMS, "B*R*(C+1)=%lld cells exceeds %lld", (long long)d.Nmax,
                (long long)kMaxCells);
  // the attention kernels address one dataset's bf16 Q|K|V [C+1][R][3E] through 32-bit
  // buffer offsets
  if ((int64_t)d.R * d.S * 3 * d.E * 2 > (int64_t)UINT32_MAX)
    return fail(TFM_ERR_DIMS, "R*(C+1)*E=%lld: one dataset's Q|K|V would exceed 4 GiB",
                (long long)d.R * d.S * d.E);
  d.tsz = d.dtype == TFM_F32 ? 4 : 2;
  d.words = (d.S + 31) / 32;
  d.block = p->block;
  d.decay = p->decay;
  if (d.block != TFM_BLOCK_POSTNORM && d.block != TFM_BLOCK_PRENORM)
    return fail(TFM_ERR_DIMS, "block %d is neither TFM_BLOCK_POSTNORM nor TFM_BLOCK_PRENORM",
                d.block);
  if (d.block == TFM_BLOCK_PRENORM) {
    if (d.dtype != TFM_BF16 || !(d.E == 64 || d.E == 128 || d.E == 192 || d.E == 256) ||
        d.H % d.E)
      return fail(TFM_ERR_DIMS, "the pre-norm block needs TFM_BF16, E in {64, 128, 192, 256} "
                                "and H a multiple of E");
    if (!std::isfinite(d.decay)) return fail(TFM_ERR_DIMS, "decay must be finite");
  }
  return TFM_OK;
}

// ---- parameter offsets (floats) -------------------------------------------------------------
struct POff {
  size_t Wqkv_f, bqkv_f, Wo_f, bo_f, Wqkv_i, bqkv_i, Wo_i, bo_i, W1, b1, W2, b2;
  size_t g1, be1, g2, be2, g3, be3, total;
};

// Packed order of include/tfm_layer.h; the pre-norm block has RMSNorm weights g1, g2, g3 only
// (its be* offsets are unused).
POff param_offsets(int E, int H, int block = TFM_BLOCK_POSTNORM) {
  POff o;
  size_t x = 0;
  auto take = [&](size_t n) { size_t r = x; x += n; return r; };
  o.Wqkv_f = take((size_t)3 * E * E); o.bqkv_f = take(3 * E);
  o.Wo_f = take((size_t)E * E); o.bo_f = take(E);
  o.Wqkv_i = take((size_t)3 * E * E); o.bqkv_i = take(3 * E);
  o.Wo_i = take((size_t)E * E); o.bo_i = take(E);
  o.W1 = take((size_t)H * E); o.b1 = take(H);
  o.W2 = take((size_t)E * H); o.b2 = take(E);
  if (block == TFM_BLOCK_PRENORM) {
    o.g1 = take(E); o.g2 = take(E); o.g3 = take(E);
    o.be1 = o.be2 = o.be3 = 0;
  } else {
    o.g1 = take(E); o.be1 = take(E); o.g2 = take(E); o.be2 = take(E);
    o.g3 = take(E); o.be3 = take(E);
  }
  o.total = x;
  return o;
}

// ---- buffer layouts --------------------------------------------------------------------------
struct Arena {
  size_t off = 0;
  size_t take(size_t bytes) { size_t r = off; off = align_up(off + bytes); return r; }
};

// Offsets of the device copy of the plan inside a workspace.
struct MetaOff {
  size_t blob, ds, col_ds, col_c, colmap, col_cell0, col_ntr, cord;
};

MetaOff take_meta(const Dims& d, Arena& a) {
  MetaOff L;
  L.blob = a.take((size_t)d.B * (3 + d.words) * 4);
  L.ds = a.take((size_t)d.B * sizeof(tfm::DsInfo));
  L.col_ds = a.take((size_t)d.B * d.S * 4);
  L.col_c = a.take((size_t)d.B * d.S * 4);
  L.colmap = a.take((size_t)d.B * d.S * 4);
  L.col_cell0 = a.take((size_t)d.B * d.S * 8);
  L.col_ntr = a.take((size_t)d.B * d.S * 4);
  L.cord = a.take((size_t)d.B * d.S * 4);
  return L;
}

struct SavedLayout {
  size_t qkvf, of, lsef, h1, xh1, rs1, qi, ki, vi, oi, lsei, h2, xh2, rs2, g, u, xh3, rs3;
  size_t total;
};

SavedLayout saved_layout(const Dims& d) {
  SavedLayout L;
  Arena a;
  const size_t N = (size_t)d.Nmax, t = d.tsz, E = d.E;
  L.qkvf = a.take(N * 3 * E * t);
  L.of = a.take(N * E * t);
  L.lsef = a.take(N * d.heads * 4);
  // the float32 path keeps H and x-hat of LN1 and LN2; the MFMA path keeps x-hat only, in the
  // H slots (its LN1 / LN2 affines are folded into the consumers)
  const size_t xhn = d.dtype == TFM_F32 ? N * E * t : 0;
  L.h1 = a.take(N * E * t);
  L.xh1 = a.take(xhn);
  L.rs1 = a.take(N * 4);
  L.qi = a.take(N * E * t);
  L.ki = a.take(N * E * t);
  L.vi = a.take(N * E * t);
  L.oi = a.take(N * E * t);
  L.lsei = a.take(N * d.heads * 4);
  L.h2 = a.take(N * E * t);
  L.xh2 = a.take(xhn);
  L.rs2 = a.take(N * 4);
  // the fused MLP backward recomputes G and U: no saved copies
  const size_t gun = d.dtype == TFM_BF16 && tfm::mlp_fused_ok(d.E, d.H) ? 0 : N * d.H * t;
  L.g = a.take(gun);
  L.u = a.take(gun);
  L.xh3 = a.take(N * E * t);
  L.rs3 = a.take(N * 4);
  L.total = a.off;
  return L;
}

// Saved state of the pre-norm block: x' = decay X, r1 = RMS1(x'), the residual stream h1, h2
// and the norm outputs r2, r3 (the GEMM inputs), rstd of each norm, the attention state and
// the MLP pre-activation and activation.
struct PreSaved {
  size_t xs, r1, rs1, qkvf, of, lsef, h1, r2, rs2, qi, ki, vi, oi, lsei, h2, r3, rs3, g, u;
  size_t total;
};

PreSaved pre_saved_layout(const Dims& d) {
  PreSaved L;
  Arena a;
  const size_t N = (size_t)d.Nmax, t = d.tsz, E = d.E;
  L.xs = a.take(N * E * t);
  L.r1 = a.take(N * E * t);
  L.rs1 = a.take(N * 4);
  L.qkvf = a.take(N * 3 * E * t);
  L.of = a.take(N * E * t);
  L.lsef = a.take(N * d.heads * 4);
  L.h1 = a.take(N * E * t);
  L.r2 = a.take(N * E * t);
  L.rs2 = a.take(N * 4);
  L.qi = a.take(N * E * t);
  L.ki = a.take(N * E * t);
  L.vi = a.take(N * E * t);
  L.oi = a.take(N * E * t);
  L.lsei = a.take(N * d.heads * 4);
  L.h2 = a.take(N * E * t);
  L.r3 = a.take(N * E * t);
  L.rs3 = a.take(N * 4);
  L.g = a.take(N * d.H * t);
  L.u = a.take(N * d.H * t);
  L.total = a.off;
  return L;
}

size_t saved_total(const Dims& d) {
  return d.block == TFM_BLOCK_PRENORM ? pre_saved_layout(d).total : saved_layout(d).total;
}

struct WsLayout {
  MetaOff meta;
  size_t xc, ta, tb, tc, td, te, tf, th1, th2, tq, tk, tv, tqkv, D, part, cpart, cpart2;
  size_t fast;  // region owned by the MFMA path
  size_t total;
  int64_t Z;    // partial-sum chunks
};

WsLayout ws_layout(const Dims& d) {
  WsLayout L;
  Arena a;
  const size_t N = (size_t)d.Nmax, t = d.tsz, E = d.E;
  L.meta = take_meta(d, a);
  L.xc = a.take(N * E * t);
  L.ta = a.take(N * E * t);
  L.tb = a.take(N * E * t);
  L.tc = a.take(N * E * t);
  L.td = a.take(N * E * t);
  L.te = a.take(N * E * t);
  L.tf = a.take(N * E * t);
  L.th1 = a.take(N * d.H * t);
  L.th2 = a.take(N * d.H * t);
  L.tq = a.take(N * E * t);
  L.tk = a.take(N * E * t);
  L.tv = a.take(N * E * t);
  L.tqkv = a.take(N * 3 * E * t);
  L.D = a.take(N * d.heads * 4);
  L.Z = (d.Nmax + kChunk - 1) / kChunk;
  size_t maxw = (size_t)3 * E * E;
  if ((size_t)d.H * E > maxw) maxw = (size_t)d.H * E;
  L.part = a.take((size_t)L.Z * maxw * 4);
  size_t maxc = 3 * E > (size_t)d.H ? 3 * E : (size_t)d.H;
  L.cpart = a.take((size_t)L.Z * maxc * 4);
  L.cpart2 = a.take((size_t)L.Z * maxc * 4);
  L.fast = a.take(tfm::fast_workspace_bytes(d.B, d.R, d.S, d.E, d.heads, d.H,
                                            d.dtype == TFM_BF16));
  L.total = a.off;
  return L;
}

bool aligned(const void* p) { return p && ((uintptr_t)p % 16) == 0; }

// ---- per-call plan ---------------------------------------------------------------------------
struct Plan {
  int NC = 0;
  int nmax = 0;  // longest train prefix
  std::vector<int32_t> blob;
};

// nt_max: the largest allowed n_train (R, or the context rows of a query call).
int make_plan(const Dims& d, const int32_t* n_train, const uint8_t* mask, Plan& P,
              int nt_max = -1) {
  if (nt_max < 0) nt_max = d.R;
  if (!n_train || !mask) return fail(TFM_ERR_POINTER, "n_train or cell_mask is null");
  P.blob.assign((size_t)d.B * (3 + d.words), 0);
  int col = 0;
  for (int b = 0; b < d.B; ++b) {
    if (n_train[b] < 1 || n_train[b] > nt_max)
      return fail(TFM_ERR_NTRAIN, "n_train[%d]=%d outside [1, %d]", b, n_train[b], nt_max);
    const uint8_t* m = mask + (size_t)b * d.S;
    if (!m[d.C]) return fail(TFM_ERR_MASK, "target cell (index C=%d) of dataset %d inactive",
                             d.C, b);
    int32_t* e = &P.blob[(size_t)b * (3 + d.words)];
    int cnt = 0;
    for (int c = 0; c < d.S; ++c)
      if (m[c]) {
        ++cnt;
        e[3 + (c >> 5)] |= (int32_t)(1u << (c & 31));
      }
    e[0] = n_train[b];
    if (n_train[b] > P.nmax) P.nmax = n_train[b];
    e[1] = col;
    e[2] = cnt;
    col += cnt;
  }
  P.NC = col;
  return TFM_OK;
}

#define HIPCHK(...)                                                                     \
  do {                                                                                  \
    hipError_t e_ = (__VA_ARGS__);                                                      \
    if (e_ != hipSuccess)                                                               \
      return fail(TFM_ERR_HIP, "%s failed: %s", #__VA_ARGS__, hipGetErrorString(e_));   \
  } while (0)

#define STEP(name, ...)              \
  do {                               \
    tfm::prof_begin(name, s);        \
    HIPCHK(__VA_ARGS__);             \
    tfm::prof_end(s);                \
  } while (0)

#define STEP_ERR(...)                \
  do {                               \
    const int rc_ = (__VA_ARGS__);   \
    if (rc_ != TFM_OK) return rc_;   \
  } while (0)

int setup_geo(const Dims& d, const Plan& P, char* ws, const MetaOff& W, tfm::Geo& g,
              hipStream_t s) {
  int32_t* blob = (int32_t*)(ws + W.blob);
  g.B = d.B; g.R = d.R; g.S = d.S; g.E = d.E; g.heads = d.heads; g.d = d.d; g.H = d.H;
  g.NC = P.NC;
  g.nmax = P.nmax;
  g.N = (int64_t)P.NC * d.R;
  g.ds = (const tfm::DsInfo*)(ws + W.ds);
  g.col_ds = (const int32_t*)(ws + W.col_ds);
  g.col_c = (const int32_t*)(ws + W.col_c);
  g.colmap = (const int32_t*)(ws + W.colmap);
  g.col_cell0 = (const int64_t*)(ws + W.col_cell0);
  g.col_ntr = (const int32_t*)(ws + W.col_ntr);
  HIPCHK(tfm::launch_upload(P.blob.data(), (int64_t)P.blob.size(), blob, s));
  HIPCHK(tfm::launch_expand_meta(blob, d.B, d.R, d.S, d.words, (tfm::DsInfo*)(ws + W.ds),
                                 (int32_t*)(ws + W.col_ds), (int32_t*)(ws + W.col_c),
                                 (int32_t*)(ws + W.colmap), (int64_t*)(ws + W.col_cell0),
                                 (int32_t*)(ws + W.col_ntr), s));
  return TFM_OK;
}

// Item-attention backward on the MFMA path.  The columns of datasets whose train prefix fits
// the one-kernel form go through it, the others through the dQ and dK/dV kernels; within each
// group the columns of longer prefixes come first, so the largest problems start earliest and
// the launches end evenly.  The column order is uploaded only when it is not the natural one.
int item_attn_bwd(const Dims& d, const tfm::Geo& g, const Plan& P, char* ws, const MetaOff& M,
                  const tfm::bf16* qi, const tfm::bf16* ki, const tfm::bf16* vi,
                  const tfm::bf16* oi, const tfm::bf16* doi, const float* lsei, float* Dq,
                  tfm::bf16* dq, tfm::bf16* dk, tfm::bf16* dv, hipStream_t s) {
  using namespace tfm;
  const int fmax = item_attn_bwd_fused_max_rows(d.d);
  const int stride = 3 + d.words;
  std::vector<int> order(d.B);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
    return P.blob[(size_t)x * stride] > P.blob[(size_t)y * stride];
  });
  std::vector<int32_t> cols;
  cols.reserve(P.NC);
  int nF = 0, nmaxF = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (int b : order) {
      const int32_t* e = &P.blob[(size_t)b * stride];
      const bool fused = e[0] <= fmax;
      if (fused != (pass == 0)) continue;
      for (int k = 0; k < e[2]; ++k) cols.push_back(e[1] + k);
      if (fused) {
        nF += e[2];
        nmaxF = std::max(nmaxF, e[0]);
      }
    }
  bool natural = nF == 0 || nF == P.NC;  // a single group in the natural column order
  for (int i = 0; i < P.NC && natural; ++i) natural = cols[i] == i;
  int32_t* dcols = nullptr;
  if (!natural) {
    dcols = (int32_t*)(ws + M.cord);
    HIPCHK(launch_upload(cols.data(), P.NC, dcols, s));
  }
  const ColList F{dcols, nF};
  const ColList T{dcols ? dcols + nF : nullptr, P.NC - nF};
  if (nF > 0)
    STEP("item_attn_bwd/mfma",
         launch_item_attn_bwd_fused(g, F, nmaxF, qi, ki, vi, oi, doi, lsei, dq, dk, dv, s));
  if (nF < P.NC) {
    STEP("item_attn_dq/mfma", launch_item_attn_dq(g, T, qi, ki, vi, oi, doi, lsei, Dq, dq, s));
    STEP("item_attn_dkdv/mfma",
         launch_item_attn_dkdv(g, T, qi, ki, vi, oi, doi, lsei, Dq, dk, dv, s));
  }
  return TFM_OK;
}

// ---- forward ---------------------------------------------------------------------------------
template <class T>
int fwd_simple(const Dims& d, const tfm::Geo& g, const T* X, const float* prm, T* Y, char* sv,
               const SavedLayout& S, char* ws, const WsLayout& W, hipStream_t s) {
  using namespace tfm;
  const POff o = param_offsets(d.E, d.H);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  T* xc = (T*)(ws + W.xc);
  T* ta = (T*)(ws + W.ta);
  T* tu = (T*)(ws + W.th1);
  T* qkvf = (T*)(sv + S.qkvf);
  T* of = (T*)(sv + S.of);
  T* h1 = (T*)(sv + S.h1);
  T* h2 = (T*)(sv + S.h2);
  T* oi = (T*)(sv + S.oi);
  T* gp = (T*)(sv + S.g);
  T* yc = (T*)(ws + W.tb);
  STEP("gather/hbm", launch_gather<T>(g, X, xc, s));
  STEP("feat_qkv/valu", launch_linear<T, T>(N, 3 * E, E, xc, E, prm + o.Wqkv_f, E, 1, prm + o.bqkv_f, qkvf,
                             3 * E, s));
  STEP("feat_attn_fwd/valu", launch_feat_attn_fwd_simple<T>(g, qkvf, of, (float*)(sv + S.lsef), s));
  STEP("feat_out/valu", launch_linear<T, T>(N, E, E, of, E, prm + o.Wo_f, E, 1, prm + o.bo_f, ta, E, s));
  STEP("ln1/hbm", launch_add_ln<T>(N, E, xc, ta, prm + o.g1, prm + o.be1, h1, (T*)(sv + S.xh1),
                          (float*)(sv + S.rs1), s));
  STEP("item_qkv/valu", launch_linear_item_qkv<T>(g, h1, prm + o.Wqkv_i, prm + o.bqkv_i, (T*)(sv + S.qi),
                                   (T*)(sv + S.ki), (T*)(sv + S.vi), s));
  STEP("item_attn_fwd/valu", launch_item_attn_fwd_simple<T>(g, (T*)(sv + S.qi), (T*)(sv + S.ki), (T*)(sv + S.vi),
                                        oi, (float*)(sv + S.lsei), s));
  STEP("item_out/valu", launch_linear<T, T>(N, E, E, oi, E, prm + o.Wo_i, E, 1, prm + o.bo_i, ta, E, s));
  STEP("ln2/hbm", launch_add_ln<T>(N, E, h1, ta, prm + o.g2, prm + o.be2, h2, (T*)(sv + S.xh2),
                          (float*)(sv + S.rs2), s));
  STEP("mlp_up/valu", launch_linear<T, T>(N, H, E, h2, E, prm + o.W1, E, 1, prm + o.b1, gp, H, s));
  STEP("gelu/hbm", launch_gelu<T>(N * H, gp, tu, s));
  STEP("mlp_down/valu", launch_linear<T, T>(N, E, H, tu, H, prm + o.W2, H, 1, prm + o.b2, ta, E, s));
  STEP("ln3/hbm", launch_add_ln<T>(N, E, h2, ta, prm + o.g3, prm + o.be3, yc, (T*)(sv + S.xh3),
                          (float*)(sv + S.rs3), s));
  STEP("scatter/hbm", launch_scatter<T>(g, yc, (const T*)nullptr, Y, s));
  return TFM_OK;
}

// ---- backward --------------------------------------------------------------------------------
template <class T>
struct GradSink {
  const WsLayout& W;
  char* ws;
  float* grads;
  int accumulate;
  int64_t M;
  hipStream_t s;
  // dW[j][i] = sum_m dY[m][j] X[m][i]
  int wgrad(const T* dY, int Nj, const T* X, int Ki, size_t off) {
    float* part = (float*)(ws + W.part);
    int64_t Z = (M + kChunk - 1) / kChunk;
    if (Z < 1) Z = 1;
    STEP("wgrad/valu", tfm::launch_wgrad<T>(M, Nj, Ki, dY, Nj, X, Ki, kChunk, part, s));
    STEP("reduce/hbm", tfm::launch_reduce_partials((int)Z, (int64_t)Nj * Ki, part, grads + off,
                                               accumulate, s));
    return TFM_OK;
  }
  // g[j] = sum_m A[m][j] (* B[m][j])
  int colsum(const T* A, const T* B, int Nj, size_t off) {
    float* part = (float*)(ws + W.cpart);
    int64_t Z = (M + kChunk - 1) / kChunk;
    if (Z < 1) Z = 1;
    STEP("colsum/hbm", tfm::launch_colsum<T>(M, Nj, A, Nj, B, Nj, kChunk, part, s));
    STEP("reduce/hbm", tfm::launch_reduce_partials((int)Z, Nj, part, grads + off, accumulate, s));
    return TFM_OK;
  }
};

#define CHK(...)                 \
  do {                           \
    int c_ = (__VA_ARGS__);      \
    if (c_ != TFM_OK) return c_; \
  } while (0)

template <class T>
int bwd_simple(const Dims& d, const tfm::Geo& g, const T* X, const float* prm, const char* sv,
               const SavedLayout& S, const T* dY, T* dX, float* grads, int accumulate,
               char* ws, const WsLayout& W, hipStream_t s) {
  using namespace tfm;
  const POff o = param_offsets(d.E, d.H);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  GradSink<T> G{W, ws, grads, accumulate, N, s};
  T* xc = (T*)(ws + W.xc);
  T* dyc = (T*)(ws + W.ta);
  T* dz3 = (T*)(ws + W.tb);
  T* tmp = (T*)(ws + W.tc);
  T* dh = (T*)(ws + W.td);
  T* dz2 = (T*)(ws + W.te);
  T* dz1 = (T*)(ws + W.tf);
  T* du = (T*)(ws + W.th1);
  T* uu = (T*)(ws + W.th2);
  T* dqkv = (T*)(ws + W.tqkv);
  const T* h1 = (const T*)(sv + S.h1);
  const T* h2 = (const T*)(sv + S.h2);
  const T* gp = (const T*)(sv + S.g);
  STEP("gather/hbm", launch_gather<T>(g, dY, dyc, s));
  STEP("gather/hbm", launch_gather<T>(g, X, xc, s));
  // LN3
  STEP("ln3_bwd/hbm", launch_ln_bwd<T>(N, E, dyc, (const T*)nullptr, (const T*)(sv + S.xh3),
                          (const float*)(sv + S.rs3), prm + o.g3, dz3, (T*)nullptr, s));
  CHK(G.colsum(dyc, (const T*)(sv + S.xh3), E, o.g3));
  CHK(G.colsum(dyc, (const T*)nullptr, E, o.be3));
  // MLP
  STEP("mlp_down_dx/valu", launch_linear<T, T>(N, H, E, dz3, E, prm + o.W2, 1, H, nullptr, du, H, s));
  STEP("gelu/hbm", launch_gelu<T>(N * H, gp, uu, s));
  CHK(G.wgrad(dz3, E, uu, H, o.W2));
  CHK(G.colsum(dz3, (const T*)nullptr, E, o.b2));
  STEP("gelu_bwd/hbm", launch_gelu_bwd<T>(N * H, gp, du, s));
  CHK(G.wgrad(du, H, h2, E, o.W1));
  CHK(G.colsum(du, (const T*)nullptr, H, o.b1));
  STEP("mlp_up_dx/valu", launch_linear<T, T>(N, E, H, du, H, prm + o.W1, 1, E, nullptr, tmp, E, s));
  // LN2
  STEP("ln2_bwd/hbm", launch_ln_bwd<T>(N, E, dz3, tmp, (const T*)(sv + S.xh2), (const float*)(sv + S.rs2),
                          prm + o.g2, dz2, dh, s));
  CHK(G.colsum(dh, (const T*)(sv + S.xh2), E, o.g2));
  CHK(G.colsum(dh, (const T*)nullptr, E, o.be2));
  // item attention
  T* doi = (T*)(ws + W.tc);
  STEP("item_out_dx/valu", launch_linear<T, T>(N, E, E, dz2, E, prm + o.Wo_i, 1, E, nullptr, doi, E, s));
  CHK(G.wgrad(dz2, E, (const T*)(sv + S.oi), E, o.Wo_i));
  CHK(G.colsum(dz2, (const T*)nullptr, E, o.bo_i));
  T* dq = (T*)(ws + W.tq);
  T* dk = (T*)(ws + W.tk);
  T* dv = (T*)(ws + W.tv);
  STEP("item_attn_bwd/valu", launch_item_attn_bwd_simple<T>(g, (const T*)(sv + S.qi), (const T*)(sv + S.ki),
                                        (const T*)(sv + S.vi), (const T*)(sv + S.oi), doi,
                                        (const float*)(sv + S.lsei), (float*)(ws + W.D), dq, dk,
                                        dv, s));
  STEP("item_dqkv_cells/hbm", launch_item_dqkv_to_cells<T>(g, dq, dk, dv, dqkv, s));
  CHK(G.wgrad(dqkv, 3 * E, h1, E, o.Wqkv_i));
  CHK(G.colsum(dqkv, (const T*)nullptr, 3 * E, o.bqkv_i));
  STEP("item_qkv_dx/valu", launch_linear<T, T>(N, E, 3 * E, dqkv, 3 * E, prm + o.Wqkv_i, 1, E, nullptr, tmp, E,
                             s));
  // LN1
  STEP("ln1_bwd/hbm", launch_ln_bwd<T>(N, E, dz2, tmp, (const T*)(sv + S.xh1), (const float*)(sv + S.rs1),
                          prm + o.g1, dz1, dh, s));
  CHK(G.colsum(dh, (const T*)(sv + S.xh1), E, o.g1));
  CHK(G.colsum(dh, (const T*)nullptr, E, o.be1));
  // feature attention
  T* dof = (T*)(ws + W.tc);
  STEP("feat_out_dx/valu", launch_linear<T, T>(N, E, E, dz1, E, prm + o.Wo_f, 1, E, nullptr, dof, E, s));
  CHK(G.wgrad(dz1, E, (const T*)(sv + S.of), E, o.Wo_f));
  CHK(G.colsum(dz1, (const T*)nullptr, E, o.bo_f));
  STEP("feat_attn_bwd/valu", launch_feat_attn_bwd_simple<T>(g, (const T*)(sv + S.qkvf), (const T*)(sv + S.of), dof,
                                        (const float*)(sv + S.lsef), dqkv, s));
  CHK(G.wgrad(dqkv, 3 * E, xc, E, o.Wqkv_f));
  CHK(G.colsum(dqkv, (const T*)nullptr, 3 * E, o.bqkv_f));
  STEP("feat_qkv_dx/valu", launch_linear<T, T>(N, E, 3 * E, dqkv, 3 * E, prm + o.Wqkv_f, 1, E, nullptr, tmp, E,
                             s));
  STEP("scatter/hbm", launch_scatter<T>(g, dz1, tmp, dX, s));
  return TFM_OK;
}

// ---- MFMA path (bfloat16) -------------------------------------------------------------------
bool fast_eligible(const Dims& d) {
  return d.dtype == TFM_BF16 && (d.E == 64 || d.E == 128 || d.E == 192 || d.E == 256) &&
         d.H % d.E == 0;
}

struct FastWs {
  tfm::bf16* w;
  tfm::bf16* wt;
  float* lnpart;
  float* wpart;
  float* bpart;
  tfm::WOff wo;
};

FastWs fast_ws(const Dims& d, char* ws, const WsLayout& W) {
  FastWs f;
  f.wo = tfm::weight_offsets(d.E, d.H);
  char* p = ws + W.fast;
  f.w = (tfm::bf16*)p;
  p += align_up((size_t)f.wo.total * 2);
  f.wt = (tfm::bf16*)p;
  p += align_up((size_t)f.wo.total * 2);
  f.lnpart = (float*)p;
  p += align_up(tfm::ln_partial_bytes(d.Nmax, d.E));
  const int64_t zw = tfm::wgrad_max_chunks(d.Nmax);
  const int64_t maxw = 3LL * d.E * d.E > (int64_t)d.H * d.E ? 3LL * d.E * d.E : (int64_t)d.H * d.E;
  f.wpart = (float*)p;
  p += align_up((size_t)zw * maxw * 4 + 256);
  f.bpart = (float*)p;
  return f;
}

tfm::GemmArgs gemm_base(const tfm::Geo& g, int64_t M, int N, int K, int epi) {
  tfm::GemmArgs a{};
  a.M = M;
  a.N = N;
  a.K = K;
  a.BN = g.E;
  a.epi = epi;
  a.g = g;
  return a;
}

// Buffers of one forward pass on the MFMA path.  The training forward points them into the
// saved state; the forward-only calls point them into the workspace (reused where lifetimes
// allow; the optional ones null) and into the caller's key/value cache.  h1, h2: in the
// post-norm block the x-hat of LN1 and LN2 (their affines are folded into the consumers); in
// the pre-norm block the residual stream.
struct FwdBufs {
  tfm::bf16 *qkvf = nullptr, *of = nullptr, *h1 = nullptr, *qi = nullptr, *ki = nullptr,
            *vi = nullptr, *oi = nullptr, *h2 = nullptr, *u = nullptr;
  tfm::bf16 *xh3 = nullptr, *g = nullptr;  // optional
  tfm::bf16 *xs = nullptr, *r1 = nullptr, *r2 = nullptr, *r3 = nullptr;    // pre-norm block
  float *lsef = nullptr, *lsei = nullptr, *rs1 = nullptr, *rs2 = nullptr, *rs3 = nullptr;
  bool query = false;  // ki / vi hold the keys and values of a context call: project Q only
  int kR = 0;          // rows per (column, head) of ki / vi; 0: R
  bool save = true;    // the forward keeps what its backward reads (false: forward-only calls)
};

FwdBufs bufs_from_saved(char* sv, const SavedLayout& S) {
  typedef tfm::bf16 T;
  FwdBufs b;
  b.qkvf = (T*)(sv + S.qkvf); b.of = (T*)(sv + S.of); b.lsef = (float*)(sv + S.lsef);
  b.h1 = (T*)(sv + S.h1); b.rs1 = (float*)(sv + S.rs1);
  b.qi = (T*)(sv + S.qi); b.ki = (T*)(sv + S.ki); b.vi = (T*)(sv + S.vi);
  b.oi = (T*)(sv + S.oi); b.lsei = (float*)(sv + S.lsei);
  b.h2 = (T*)(sv + S.h2); b.rs2 = (float*)(sv + S.rs2);
  b.g = (T*)(sv + S.g); b.u = (T*)(sv + S.u); b.xh3 = (T*)(sv + S.xh3);
  b.rs3 = (float*)(sv + S.rs3);
  return b;
}

// Feature Q|K|V (projection of the layer input x, rows per xmode), then the feature attention.
int feat_fwd(const tfm::Geo& g, const tfm::bf16* x, int xmode, const float* bqkv,
             const FwdBufs& b, const FastWs& f, hipStream_t s) {
  using namespace tfm;
  GemmArgs a = gemm_base(g, g.N, 3 * g.E, g.E, EPI_BIAS);
  a.A = x; a.amode = xmode; a.lda = g.E;
  a.Bt = f.w + f.wo.qkv_f; a.bias = bqkv; a.out = b.qkvf; a.ldo = 3 * g.E;
  STEP("feat_qkv/mfma", launch_gemm(a, s));
  if (feat_attn_mfma_ok(g))
    STEP("feat_attn_fwd/mfma", launch_feat_attn_fwd(g, b.qkvf, b.of, b.lsef, s));
  else
    STEP("feat_attn_fwd/valu", launch_feat_attn_fwd_simple<bf16>(g, b.qkvf, b.of, b.lsef, s));
  return TFM_OK;
}

int fwd_fast(const Dims& d, const tfm::Geo& g, const tfm::bf16* X, const float* prm,
             tfm::bf16* Y, const FwdBufs& b, const FastWs& f, hipStream_t s) {
  using namespace tfm;
  const POff o = param_offsets(d.E, d.H);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  // H1 and H2 are kept as their x-hat only: the affines of LN1 and LN2 are folded into the
  // products that read them (weights and biases) and into the residual reads
  const WFold fold{prm + o.g1, prm + o.be1, prm + o.bqkv_i, prm + o.g2, prm + o.be2, prm + o.b1};
  STEP("weight_prep/hbm", launch_weight_prep(prm, E, H, f.w, f.wt, &fold, s));
  const float* fb = reinterpret_cast<const float*>(f.w + f.wo.fb);
  // feature Q|K|V from the native cells, and the feature attention
  STEP_ERR(feat_fwd(g, X, ROWS_NATIVE, prm + o.bqkv_f, b, f, s));
  // x-hat1 of H1 = LN1(X + O_f Wo_f^T + bo_f)
  GemmArgs a = gemm_base(g, N, E, E, EPI_LN);
  a.A = b.of; a.lda = E; a.Bt = f.w + f.wo.o_f; a.bias = prm + o.bo_f;
  a.resid = X; a.rmode = ROWS_NATIVE; a.gamma = prm + o.g1; a.beta = prm + o.be1;
  a.out = b.h1; a.omode = ROWS_COMPACT; a.xhat_out = 1; a.rstd = b.rs1;
  STEP("feat_out_ln1/mfma", launch_gemm(a, s));
  // item Q (all rows), K, V (train rows), head-major, from x-hat1 with the folded weights;
  // Q only when K/V come from a context call
  a = gemm_base(g, N, b.query ? E : 3 * E, E, EPI_ITEM_QKV);
  a.A = b.h1; a.lda = E; a.Bt = f.w + f.wo.qkv_i; a.bias = fb;
  a.out = b.qi; a.out2 = b.ki; a.out3 = b.vi;
  STEP("item_qkv/mfma", launch_gemm(a, s));
  STEP("item_attn_fwd/mfma",
       launch_item_attn_fwd(g, b.qi, b.ki, b.vi, b.oi, b.lsei, s, b.kR));
  if (mlp_fused_ok(E, H)) {
    // out-projection + LN2, MLP and LN3 in one kernel, the hidden layer in registers
    bf16* ms = f.w + f.wo.ms;
    STEP("mlp_stream/hbm",
         launch_mlp_fwd_stream(prm + o.Wo_i, prm + o.W1, prm + o.g2, prm + o.W2, E, H, ms, s));
    MlpFwdArgs m{};
    m.M = N; m.oi = b.oi; m.xh1 = b.h1; m.ws = ms;
    m.bo = prm + o.bo_i; m.g1 = prm + o.g1; m.be1 = prm + o.be1; m.g2 = prm + o.g2;
    m.be2 = prm + o.be2; m.b2 = prm + o.b2; m.g3 = prm + o.g3; m.be3 = prm + o.be3;
    m.fb1 = fb + 3 * E;
    // saved for the backward only (G and U are recomputed by the fused backward)
    m.xh2 = b.save ? b.h2 : nullptr; m.rs2 = b.save ? b.rs2 : nullptr;
    m.y = Y; m.xh3 = b.save ? b.xh3 : nullptr; m.rs3 = b.save ? b.rs3 : nullptr; m.g = g;
    STEP("mlp_fused/mfma", launch_mlp_fwd(m, s));
    STEP("zero_inactive/hbm", launch_zero_inactive(g, Y, s));
    return TFM_OK;
  }
  // x-hat2 of H2 = LN2(H1 + O_i Wo_i^T + bo_i), H1 = g1 x-hat1 + be1
  a = gemm_base(g, N, E, E, EPI_LN);
  a.A = b.oi; a.lda = E; a.Bt = f.w + f.wo.o_i; a.bias = prm + o.bo_i;
  a.resid = b.h1; a.rmode = ROWS_COMPACT; a.rgamma = prm + o.g1; a.rbeta = prm + o.be1;
  a.gamma = prm + o.g2; a.beta = prm + o.be2;
  a.out = b.h2; a.omode = ROWS_COMPACT; a.xhat_out = 1; a.rstd = b.rs2;
  STEP("item_out_ln2/mfma", launch_gemm(a, s));
  // G = H2 W1^T + b1 (from x-hat2, folded), U = GELU(G)
  a = gemm_base(g, N, H, E, EPI_GELU_FWD);
  a.A = b.h2; a.lda = E; a.Bt = f.w + f.wo.w1; a.bias = fb + 3 * E;
  a.out = b.g; a.out2 = b.u; a.ldo = H;
  STEP("mlp_up/mfma", launch_gemm(a, s));
  // Y = LN3(H2 + U W2^T + b2), written to the native layout
  a = gemm_base(g, N, E, H, EPI_LN);
  a.A = b.u; a.lda = H; a.Bt = f.w + f.wo.w2; a.bias = prm + o.b2;
  a.resid = b.h2; a.rmode = ROWS_COMPACT; a.rgamma = prm + o.g2; a.rbeta = prm + o.be2;
  a.gamma = prm + o.g3; a.beta = prm + o.be3;
  a.out = Y; a.omode = ROWS_NATIVE; a.xhat = b.xh3; a.rstd = b.rs3;
  STEP("mlp_down_ln3/mfma", launch_gemm(a, s));
  STEP("zero_inactive/hbm", launch_zero_inactive(g, Y, s));
  return TFM_OK;
}

// Weight and bias gradients of one linear on the MFMA path (split over cells, fixed-order sums).
struct FastGrads {
  const FastWs& f;
  const tfm::Geo& g;
  float* grads;
  int accumulate;
  hipStream_t s;
  // ymode: layout of dY (compact, native; head-major item gradients when dY2 is given)
  // xg, xb: X is the x-hat of a norm with affine (xg, xb): the weight gradient is formed for
  // h = xg o X + xb (launch_reduce_wfold)
  int run(const tfm::bf16* dY, int N, const tfm::bf16* X, int K, int xmode, size_t offW,
          size_t offb, const tfm::bf16* dY2 = nullptr, const tfm::bf16* dY3 = nullptr,
          int ymode = tfm::ROWS_COMPACT, const float* xg = nullptr, const float* xb = nullptr) {
    tfm::WgradArgs a{};
    a.M = g.N; a.N = N; a.K = K; a.dY = dY; a.ldy = N; a.X = X; a.ldx = K; a.xmode = xmode;
    a.dY2 = dY2; a.dY3 = dY3; a.ymode = dY2 ? tfm::ROWS_ITEM_HM : ymode;
    a.part = f.wpart; a.bpart = f.bpart; a.g = g;
    const int Z = tfm::wgrad_chunks(g.N);
    STEP("wgrad/mfma", tfm::launch_wgrad_mfma(a, s));
    if (xg) {
      // leaves the bias sums in the first row of bpart
      STEP("reduce/hbm", tfm::launch_reduce_wfold(Z, N, K, f.wpart, f.bpart, xg, xb,
                                                  grads + offW, accumulate, s));
      STEP("reduce/hbm", tfm::launch_reduce_z(1, N, N, f.bpart, grads + offb, accumulate, s));
    } else {
      STEP("reduce/hbm", tfm::launch_reduce_z(Z, (int64_t)N * K, (int64_t)N * K, f.wpart,
                                              grads + offW, accumulate, s));
      STEP("reduce/hbm", tfm::launch_reduce_z(Z, N, N, f.bpart, grads + offb, accumulate, s));
    }
    return TFM_OK;
  }
};

int bwd_fast(const Dims& d, const tfm::Geo& g, const Plan& P, const tfm::bf16* X,
             const float* prm, const char* sv, const SavedLayout& S, const tfm::bf16* dY,
             tfm::bf16* dX, float* grads, int accumulate, char* ws, const WsLayout& W,
             hipStream_t s) {
  using namespace tfm;
  typedef tfm::bf16 T;
  const POff o = param_offsets(d.E, d.H);
  const FastWs f = fast_ws(d, ws, W);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  const int tiles = (int)tfm::gemm_tiles(tfm::EPI_LN_BWD, E, N);
  FastGrads G{f, g, grads, accumulate, s};
  const bool fused_mlp = mlp_fused_ok(E, H);
  // the backward reads the transposed copies only; the fold (x-hat2's affine in W1 and b1)
  // gives the fused MLP backward the folded up-projection bias it recomputes G with
  const WFold fold{prm + o.g1, prm + o.be1, prm + o.bqkv_i, prm + o.g2, prm + o.be2, prm + o.b1};
  STEP("weight_prep/hbm", launch_weight_prep(prm, E, H, f.w, f.wt, fused_mlp ? &fold : nullptr, s));
  T* dz3 = (T*)(ws + W.tb);
  T* dz2 = (T*)(ws + W.te);
  T* dz1 = (T*)(ws + W.tf);
  T* dgb = (T*)(ws + W.th1);
  T* dqkv = (T*)(ws + W.tqkv);
  const T* xh1 = (const T*)(sv + S.h1);  // the forward keeps x-hat1 and x-hat2 only
  const T* xh2 = (const T*)(sv + S.h2);
  if (fused_mlp) {
    // LN3', the MLP backward with G recomputed, LN2' in one kernel; its column sums give the
    // LN3 and LN2 weight and bias gradients (each pair adjacent in the packed order)
    T* ub = (T*)(ws + W.th2);
    bf16* ms = f.w + f.wo.ms;
    STEP("mlp_stream/hbm",
         launch_mlp_bwd_stream(prm + o.W1, prm + o.g2, prm + o.W2, E, H, ms, s));
    MlpBwdArgs m{};
    m.M = N; m.dy = dY; m.xh3 = (const T*)(sv + S.xh3); m.rs3 = (const float*)(sv + S.rs3);
    m.xh2 = xh2; m.rs2 = (const float*)(sv + S.rs2); m.ws = ms;
    m.g3 = prm + o.g3; m.g2 = prm + o.g2;
    m.fb1 = reinterpret_cast<const float*>(f.w + f.wo.fb) + 3 * E;
    m.dz3 = dz3; m.dz2 = dz2; m.dg = dgb; m.u = ub; m.part = f.lnpart; m.g = g;
    STEP("mlp_bwd_fused/mfma", launch_mlp_bwd(m, s));
    const int nt = (int)mlp_bwd_tiles(N);
    STEP("reduce/hbm", launch_reduce_z(nt, 2 * E, 4 * E, f.lnpart, grads + o.g3, accumulate, s));
    STEP("reduce/hbm",
         launch_reduce_z(nt, 2 * E, 4 * E, f.lnpart + 2 * E, grads + o.g2, accumulate, s));
    CHK(G.run(dz3, E, ub, H, ROWS_COMPACT, o.W2, o.b2));
    CHK(G.run(dgb, H, xh2, E, ROWS_COMPACT, o.W1, o.b1, nullptr, nullptr, ROWS_COMPACT,
              prm + o.g2, prm + o.be2));
  } else {
    // LN3 (from the native dY), with its gamma/beta column sums
    int nb = 0;
    STEP("ln3_bwd/hbm", launch_ln_out_bwd(g, dY, (const T*)(sv + S.xh3),
                                          (const float*)(sv + S.rs3), prm + o.g3, dz3, f.lnpart,
                                          &nb, s));
    // gamma and beta gradients are adjacent in the packed order: one sum over 2E columns
    STEP("reduce/hbm", launch_reduce_z(nb, 2 * E, 2 * E, f.lnpart, grads + o.g3, accumulate, s));
    // MLP: dG = (dZ3 W2) * GELU'(G)
    GemmArgs a = gemm_base(g, N, H, E, EPI_GELU_BWD);
    a.A = dz3; a.lda = E; a.Bt = f.wt + f.wo.w2; a.out = dgb; a.ldo = H;
    a.aux = (const T*)(sv + S.g);
    STEP("mlp_down_dx/mfma", launch_gemm(a, s));
    CHK(G.run(dz3, E, (const T*)(sv + S.u), H, ROWS_COMPACT, o.W2, o.b2));
    CHK(G.run(dgb, H, xh2, E, ROWS_COMPACT, o.W1, o.b1, nullptr, nullptr, ROWS_COMPACT,
              prm + o.g2, prm + o.be2));
    // dZ2 = LN2'(dZ3 + dG W1)
    a = gemm_base(g, N, E, H, EPI_LN_BWD);
    a.A = dgb; a.lda = H; a.Bt = f.wt + f.wo.w1; a.resid = dz3; a.aux = xh2;
    a.rstd_in = (const float*)(sv + S.rs2); a.gamma = prm + o.g2; a.out = dz2; a.part = f.lnpart;
    STEP("mlp_up_dx_ln2/mfma", launch_gemm(a, s));
    STEP("reduce/hbm", launch_reduce_z(tiles, 2 * E, 2 * E, f.lnpart, grads + o.g2, accumulate, s));
  }
  GemmArgs a;
  // item attention
  T* doi = (T*)(ws + W.tc);
  a = gemm_base(g, N, E, E, EPI_BIAS);
  a.A = dz2; a.lda = E; a.Bt = f.wt + f.wo.o_i; a.out = doi; a.ldo = E;
  STEP("item_out_dx/mfma", launch_gemm(a, s));
  CHK(G.run(dz2, E, (const T*)(sv + S.oi), E, ROWS_COMPACT, o.Wo_i, o.bo_i));
  T* dq = (T*)(ws + W.tq);
  T* dk = (T*)(ws + W.tk);
  T* dv = (T*)(ws + W.tv);
  const T* qi = (const T*)(sv + S.qi);
  const T* ki = (const T*)(sv + S.ki);
  const T* vi = (const T*)(sv + S.vi);
  const T* oi = (const T*)(sv + S.oi);
  const float* lsei = (const float*)(sv + S.lsei);
  float* Dq = (float*)(ws + W.D);
  CHK(item_attn_bwd(d, g, P, ws, W.meta, qi, ki, vi, oi, doi, lsei, Dq, dq, dk, dv, s));
  CHK(G.run(dq, 3 * E, xh1, E, ROWS_COMPACT, o.Wqkv_i, o.bqkv_i, dk, dv, ROWS_COMPACT,
            prm + o.g1, prm + o.be1));
  // dZ1 = LN1'(dZ2 + dQKV_i Wqkv_i), the gradients read head-major in place
  a = gemm_base(g, N, E, 3 * E, EPI_LN_BWD);
  a.A = dq; a.A2 = dk; a.A3 = dv; a.amode = ROWS_ITEM_HM; a.lda = 3 * E;
  a.Bt = f.wt + f.wo.qkv_i; a.resid = dz2;
  a.aux = xh1; a.rstd_in = (const float*)(sv + S.rs1); a.gamma = prm + o.g1;
  a.out = dz1; a.part = f.lnpart;
  STEP("item_qkv_dx_ln1/mfma", launch_gemm(a, s));
  STEP("reduce/hbm", launch_reduce_z(tiles, 2 * E, 2 * E, f.lnpart, grads + o.g1, accumulate, s));
  // feature attention
  T* dof = (T*)(ws + W.tc);
  a = gemm_base(g, N, E, E, EPI_BIAS);
  a.A = dz1; a.lda = E; a.Bt = f.wt + f.wo.o_f; a.out = dof; a.ldo = E;
  STEP("feat_out_dx/mfma", launch_gemm(a, s));
  CHK(G.run(dz1, E, (const T*)(sv + S.of), E, ROWS_COMPACT, o.Wo_f, o.bo_f));
  if (feat_attn_mfma_ok(g))
    STEP("feat_attn_bwd/mfma",
         launch_feat_attn_bwd(g, (const T*)(sv + S.qkvf), (const T*)(sv + S.of), dof,
                              (const float*)(sv + S.lsef), dqkv, s));
  else
    STEP("feat_attn_bwd/valu",
         launch_feat_attn_bwd_simple<T>(g, (const T*)(sv + S.qkvf), (const T*)(sv + S.of), dof,
                                        (const float*)(sv + S.lsef), dqkv, s));
  CHK(G.run(dqkv, 3 * E, X, E, ROWS_NATIVE, o.Wqkv_f, o.bqkv_f));
  // dX = dZ1 + dQKV_f Wqkv_f, native layout
  a = gemm_base(g, N, E, 3 * E, EPI_DX);
  a.A = dqkv; a.lda = 3 * E; a.Bt = f.wt + f.wo.qkv_f; a.resid = dz1; a.out = dX;
  STEP("feat_qkv_dx/mfma", launch_gemm(a, s));
  STEP("zero_inactive/hbm", launch_zero_inactive(g, dX, s));
  return TFM_OK;
}

// ---- pre-norm RMSNorm block (bfloat16, MFMA path) --------------------------------------------
constexpr float kRmsEps = 1e-6f;

FwdBufs bufs_from_pre_saved(char* sv, const PreSaved& S) {
  typedef tfm::bf16 T;
  FwdBufs b;
  b.xs = (T*)(sv + S.xs); b.r1 = (T*)(sv + S.r1); b.rs1 = (float*)(sv + S.rs1);
  b.qkvf = (T*)(sv + S.qkvf); b.of = (T*)(sv + S.of); b.lsef = (float*)(sv + S.lsef);
  b.h1 = (T*)(sv + S.h1); b.r2 = (T*)(sv + S.r2); b.rs2 = (float*)(sv + S.rs2);
  b.qi = (T*)(sv + S.qi); b.ki = (T*)(sv + S.ki); b.vi = (T*)(sv + S.vi);
  b.oi = (T*)(sv + S.oi); b.lsei = (float*)(sv + S.lsei);
  b.h2 = (T*)(sv + S.h2); b.r3 = (T*)(sv + S.r3); b.rs3 = (float*)(sv + S.rs3);
  b.g = (T*)(sv + S.g); b.u = (T*)(sv + S.u);
  return b;
}

int fwd_pre(const Dims& d, const tfm::Geo& g, const tfm::bf16* X, const float* prm,
            tfm::bf16* Y, const FwdBufs& b, const FastWs& f, hipStream_t s) {
  using namespace tfm;
  const POff o = param_offsets(d.E, d.H, d.block);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  STEP("weight_prep/hbm", launch_weight_prep(prm, E, H, f.w, f.wt, nullptr, s));
  // x' = decay X, r1 = RMS1(x')
  STEP("rms_in/hbm", launch_rms_in(g, X, d.decay, prm + o.g1, kRmsEps, b.xs, b.r1, b.rs1, s));
  STEP_ERR(feat_fwd(g, b.r1, ROWS_COMPACT, prm + o.bqkv_f, b, f, s));
  // h1 = x' + O_f Wo_f^T + bo_f, r2 = RMS2(h1)
  GemmArgs a = gemm_base(g, N, E, E, EPI_RMS);
  a.A = b.of; a.lda = E; a.Bt = f.w + f.wo.o_f; a.bias = prm + o.bo_f;
  a.resid = b.xs; a.rmode = ROWS_COMPACT; a.rscale = 1.0f; a.gamma = prm + o.g2;
  a.eps = kRmsEps; a.out = b.h1; a.out2 = b.r2; a.rstd = b.rs2;
  STEP("feat_out_rms2/mfma", launch_gemm(a, s));
  // item Q (all rows), K and V (train rows), head-major; Q only when K/V come from a context
  // call
  a = gemm_base(g, N, b.query ? E : 3 * E, E, EPI_ITEM_QKV);
  a.A = b.r2; a.lda = E; a.Bt = f.w + f.wo.qkv_i; a.bias = prm + o.bqkv_i;
  a.out = b.qi; a.out2 = b.ki; a.out3 = b.vi;
  STEP("item_qkv/mfma", launch_gemm(a, s));
  STEP("item_attn_fwd/mfma",
       launch_item_attn_fwd(g, b.qi, b.ki, b.vi, b.oi, b.lsei, s, b.kR));
  // h2 = h1 + O_i Wo_i^T + bo_i, r3 = RMS3(h2)
  a = gemm_base(g, N, E, E, EPI_RMS);
  a.A = b.oi; a.lda = E; a.Bt = f.w + f.wo.o_i; a.bias = prm + o.bo_i;
  a.resid = b.h1; a.rmode = ROWS_COMPACT; a.rscale = 1.0f; a.gamma = prm + o.g3;
  a.eps = kRmsEps; a.out = b.h2; a.out2 = b.r3; a.rstd = b.rs3;
  STEP("item_out_rms3/mfma", launch_gemm(a, s));
  // G = r3 W1^T + b1, U = GELU(G)
  a = gemm_base(g, N, H, E, EPI_GELU_FWD);
  a.A = b.r3; a.lda = E; a.Bt = f.w + f.wo.w1; a.bias = prm + o.b1;
  a.out = b.g; a.out2 = b.u; a.ldo = H;
  STEP("mlp_up/mfma", launch_gemm(a, s));
  // Y = h2 + U W2^T + b2, native
  a = gemm_base(g, N, E, H, EPI_DX);
  a.A = b.u; a.lda = H; a.Bt = f.w + f.wo.w2; a.bias = prm + o.b2; a.resid = b.h2;
  a.out = Y;
  STEP("mlp_down_res/mfma", launch_gemm(a, s));
  STEP("zero_inactive/hbm", launch_zero_inactive(g, Y, s));
  return TFM_OK;
}

int bwd_pre(const Dims& d, const tfm::Geo& g, const Plan& P, const float* prm, const char* sv,
            const PreSaved& S, const tfm::bf16* dY, tfm::bf16* dX, float* grads, int accumulate,
            char* ws, const WsLayout& W, hipStream_t s) {
  using namespace tfm;
  typedef tfm::bf16 T;
  const POff o = param_offsets(d.E, d.H, d.block);
  const FastWs f = fast_ws(d, ws, W);
  const int E = d.E, H = d.H;
  const int64_t N = g.N;
  const int tiles = (int)tfm::gemm_tiles(tfm::EPI_RMS_BWD, E, N);
  FastGrads G{f, g, grads, accumulate, s};
  STEP("weight_prep/hbm", launch_weight_prep(prm, E, H, f.w, f.wt, nullptr, s));
  T* dh2 = (T*)(ws + W.te);
  T* dh1 = (T*)(ws + W.tf);
  T* dgb = (T*)(ws + W.th1);
  T* dqkv = (T*)(ws + W.tqkv);
  // dY is read in its native layout by the three steps that need it (no compact copy)
  // dG = (dY W2) * GELU'(G)
  GemmArgs a = gemm_base(g, N, H, E, EPI_GELU_BWD);
  a.A = dY; a.amode = ROWS_NATIVE; a.lda = E; a.Bt = f.wt + f.wo.w2; a.out = dgb; a.ldo = H;
  a.aux = (const T*)(sv + S.g);
  STEP("mlp_down_dx/mfma", launch_gemm(a, s));
  CHK(G.run(dY, E, (const T*)(sv + S.u), H, ROWS_COMPACT, o.W2, o.b2, nullptr, nullptr,
            ROWS_NATIVE));
  CHK(G.run(dgb, H, (const T*)(sv + S.r3), E, ROWS_COMPACT, o.W1, o.b1));
  // dh2 = dY + RMS3'(dG W1)
  a = gemm_base(g, N, E, H, EPI_RMS_BWD);
  a.A = dgb; a.lda = H; a.Bt = f.wt + f.wo.w1; a.resid = dY; a.rmode = ROWS_NATIVE;
  a.aux = (const T*)(sv + S.h2);
  a.rstd_in = (const float*)(sv + S.rs3); a.gamma = prm + o.g3; a.eps = kRmsEps;
  a.oscale = 1.0f; a.omode = ROWS_COMPACT; a.out = dh2; a.part = f.lnpart;
  STEP("mlp_up_dx_rms3/mfma", launch_gemm(a, s));
  STEP("reduce/hbm", launch_reduce_z(tiles, E, E, f.lnpart, grads + o.g3, accumulate, s));
  // item attention
  T* doi = (T*)(ws + W.tc);
  a = gemm_base(g, N, E, E, EPI_BIAS);
  a.A = dh2; a.lda = E; a.Bt = f.wt + f.wo.o_i; a.out = doi; a.ldo = E;
  STEP("item_out_dx/mfma", launch_gemm(a, s));
  CHK(G.run(dh2, E, (const T*)(sv + S.oi), E, ROWS_COMPACT, o.Wo_i, o.bo_i));
  T* dq = (T*)(ws + W.tq);
  T* dk = (T*)(ws + W.tk);
  T* dv = (T*)(ws + W.tv);
  const T* qi = (const T*)(sv + S.qi);
  const T* ki = (const T*)(sv + S.ki);
  const T* vi = (const T*)(sv + S.vi);
  const T* oi = (const T*)(sv + S.oi);
  const float* lsei = (const float*)(sv + S.lsei);
  float* Dq = (float*)(ws + W.D);
  CHK(item_attn_bwd(d, g, P, ws, W.meta, qi, ki, vi, oi, doi, lsei, Dq, dq, dk, dv, s));
  CHK(G.run(dq, 3 * E, (const T*)(sv + S.r2), E, ROWS_COMPACT, o.Wqkv_i, o.bqkv_i, dk, dv));
  // dh1 = dh2 + RMS2'(dQKV_i Wqkv_i), the gradients read head-major in place
  a = gemm_base(g, N, E, 3 * E, EPI_RMS_BWD);
  a.A = dq; a.A2 = dk; a.A3 = dv; a.amode = ROWS_ITEM_HM; a.lda = 3 * E;
  a.Bt = f.wt + f.wo.qkv_i; a.resid = dh2; a.aux = (const T*)(sv + S.h1);
  a.rstd_in = (const float*)(sv + S.rs2); a.gamma = prm + o.g2; a.eps = kRmsEps;
  a.oscale = 1.0f; a.omode = ROWS_COMPACT; a.out = dh1; a.part = f.lnpart;
  STEP("item_qkv_dx_rms2/mfma", launch_gemm(a, s));
  STEP("reduce/hbm", launch_reduce_z(tiles, E, E, f.lnpart, grads + o.g2, accumulate, s));
  // feature attention
  T* dof = (T*)(ws + W.tc);
  a = gemm_base(g, N, E, E, EPI_BIAS);
  a.A = dh1; a.lda = E; a.Bt = f.wt + f.wo.o_f; a.out = dof; a.ldo = E;
  STEP("feat_out_dx/mfma", launch_gemm(a, s));
  CHK(G.run(dh1, E, (const T*)(sv + S.of), E, ROWS_COMPACT, o.Wo_f, o.bo_f));
  if (feat_attn_mfma_ok(g))
    STEP("feat_attn_bwd/mfma",
         launch_feat_attn_bwd(g, (const T*)(sv + S.qkvf), (const T*)(sv + S.of), dof,
                              (const float*)(sv + S.lsef), dqkv, s));
  else
    STEP("feat_attn_bwd/valu",
         launch_feat_attn_bwd_simple<T>(g, (const T*)(sv + S.qkvf), (const T*)(sv + S.of), dof,
                                        (const float*)(sv + S.lsef), dqkv, s));
  CHK(G.run(dqkv, 3 * E, (const T*)(sv + S.r1), E, ROWS_COMPACT, o.Wqkv_f, o.bqkv_f));
  // dX = decay (dh1 + RMS1'(dQKV_f Wqkv_f)), native
  a = gemm_base(g, N, E, 3 * E, EPI_RMS_BWD);
  a.A = dqkv; a.lda = 3 * E; a.Bt = f.wt + f.wo.qkv_f; a.resid = dh1;
  a.aux = (const T*)(sv + S.xs); a.rstd_in = (const float*)(sv + S.rs1); a.gamma = prm + o.g1;
  a.eps = kRmsEps; a.oscale = d.decay; a.omode = ROWS_NATIVE; a.out = dX; a.part = f.lnpart;
  STEP("feat_qkv_dx_rms1/mfma", launch_gemm(a, s));
  STEP("reduce/hbm", launch_reduce_z(tiles, E, E, f.lnpart, grads + o.g1, accumulate, s));
  STEP("zero_inactive/hbm", launch_zero_inactive(g, dX, s));
  return TFM_OK;
}

// ---- forward-only calls ----------------------------------------------------------------------
// Workspace of a forward-only call: the plan, the bf16 weights, and the activations of one
// pass with lifetimes overlapped (p1: feature Q|K|V, then GELU output; p2: feature attention
// output, then item attention output; p3: h1; p4: item Q, then h2 (post-norm); pre-norm adds
// p5: x', then h2, and p6: r1, then r2, then r3), one rstd and one log-sum-exp scratch.
struct InferLayout {
  MetaOff meta;
  size_t w, wt, p1, p2, p3, p4, p5, p6, rs, lse, total;
};

bool infer_eligible(const Dims& d) {
  return d.dtype == TFM_BF16 && (d.E == 64 || d.E == 128 || d.E == 192 || d.E == 256) &&
         d.H % d.E == 0;
}

InferLayout infer_layout(const Dims& d) {
  InferLayout L;
  Arena a;
  const size_t N = (size_t)d.Nmax, E = d.E;
  const tfm::WOff wo = tfm::weight_offsets(d.E, d.H);
  L.meta = take_meta(d, a);
  L.w = a.take((size_t)wo.total * 2);
  L.wt = a.take((size_t)wo.total * 2);
  L.p1 = a.take(N * (3 * E > (size_t)d.H ? 3 * E : (size_t)d.H) * 2);
  L.p2 = a.take(N * E * 2);
  L.p3 = a.take(N * E * 2);
  L.p4 = a.take(N * E * 2);
  const bool pre = d.block == TFM_BLOCK_PRENORM;
  L.p5 = pre ? a.take(N * E * 2) : 0;
  L.p6 = pre ? a.take(N * E * 2) : 0;
  L.rs = a.take(N * 4);
  L.lse = a.take(N * d.heads * 4);
  L.total = a.off;
  return L;
}

// Key/value cache of one layer: K then V, head-major [column][head][R][d] over every possible
// active column (B * (C + 1)), R = the context rows.
size_t cache_half(const Dims& d) { return align_up((size_t)d.B * d.S * d.R * d.E * 2); }

FwdBufs infer_bufs(const Dims& d, char* ws, const InferLayout& L, tfm::bf16* kc, tfm::bf16* vc,
                   bool query, int kR) {
  typedef tfm::bf16 T;
  FwdBufs b;
  T* p1 = (T*)(ws + L.p1);
  T* p2 = (T*)(ws + L.p2);
  T* p3 = (T*)(ws + L.p3);
  T* p4 = (T*)(ws + L.p4);
  float* rs = (float*)(ws + L.rs);
  float* lse = (float*)(ws + L.lse);
  b.qkvf = p1; b.u = p1;
  b.of = p2; b.oi = p2;
  b.h1 = p3;
  b.qi = p4;
  b.ki = kc; b.vi = vc;
  b.lsef = lse; b.lsei = lse;
  b.rs1 = b.rs2 = b.rs3 = rs;
  if (d.block == TFM_BLOCK_PRENORM) {
    T* p5 = (T*)(ws + L.p5);
    T* p6 = (T*)(ws + L.p6);
    b.xs = p5; b.h2 = p5;
    b.r1 = b.r2 = b.r3 = p6;
  } else {
    b.h2 = p4;
  }
  b.query = query;
  b.kR = kR;
  b.save = false;
  return b;
}

FastWs infer_fast_ws(const Dims& d, char* ws, const InferLayout& L) {
  FastWs f{};
  f.wo = tfm::weight_offsets(d.E, d.H);
  f.w = (tfm::bf16*)(ws + L.w);
  f.wt = (tfm::bf16*)(ws + L.wt);
  return f;
}

// Shared part of the two forward-only calls.  ctx_rows < 0: a context call (dims->R rows, the
// cache written); otherwise a query call whose cache came from a context call with ctx_rows
// rows.
int infer_call(const tfm_dims* dims, int ctx_rows, const int32_t* n_train,
               const uint8_t* cell_mask, const void* X, const float* params, void* Y,
               void* cache, size_t cache_bytes, void* workspace, size_t workspace_bytes,
               hipStream_t s) {
  Dims d;
  int rc = check_dims(dims, d);
  if (rc) return rc;
  if (!infer_eligible(d))
    return fail(TFM_ERR_DIMS, "forward-only calls need TFM_BF16, E in {64, 128, 192, 256} and H "
                              "a multiple of E");
  const bool query = ctx_rows >= 0;
  Dims dc = d;  // the dims the cache was laid out for
  if (query) {
    if (ctx_rows < 1) return fail(TFM_ERR_DIMS, "context_rows=%d must be >= 1", ctx_rows);
    tfm_dims pc = *dims;
    pc.R = ctx_rows;
    rc = check_dims(&pc, dc);
    if (rc) return rc;
  }
  if (!aligned(X) || !aligned(params) || !aligned(Y) || !aligned(cache) || !aligned(workspace))
    return fail(TFM_ERR_POINTER, "X, params, Y, kv_cache and workspace must be non-null and "
                                 "16-byte aligned");
  const InferLayout L = infer_layout(d);
  if (workspace_bytes < L.total)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes,
                L.total);
  if (cache_bytes < 2 * cache_half(dc))
    return fail(TFM_ERR_BUFFER, "kv_cache has %zu bytes, %zu required", cache_bytes,
                2 * cache_half(dc));
  Plan P;
  rc = make_plan(d, n_train, cell_mask, P, query ? ctx_rows : d.R);
  if (rc) return rc;
  char* ws = (char*)workspace;
  tfm::Geo g;
  rc = setup_geo(d, P, ws, L.meta, g, s);
  if (rc) return rc;
  tfm::bf16* kc = (tfm::bf16*)cache;
  tfm::bf16* vc = (tfm::bf16*)((char*)cache + cache_half(dc));
  const FwdBufs b = infer_bufs(d, ws, L, kc, vc, query, query ? ctx_rows : d.R);
  const FastWs f = infer_fast_ws(d, ws, L);
  if (d.block == TFM_BLOCK_PRENORM)
    return fwd_pre(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y, b, f, s);
  return fwd_fast(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y, b, f, s);
}

}  // namespace

// ============================================================================ C ABI
namespace tfm {
int abi_fail(int code, const char* msg) { return fail(code, "%s", msg); }
int abi_check_dims(const void* dims) {
  Dims d;
  return check_dims((const tfm_dims*)dims, d);
}
}  // namespace tfm

extern "C" {

size_t tfm_layer_param_count(const tfm_dims* dims) {
  Dims d;
  if (check_dims(dims, d) != TFM_OK) return 0;
  return param_offsets(d.E, d.H, d.block).total;
}

size_t tfm_layer_saved_bytes(const tfm_dims* dims) {
  Dims d;
  if (check_dims(dims, d) != TFM_OK) return 0;
  return saved_total(d);
}

size_t tfm_layer_workspace_bytes(const tfm_dims* dims) {
  Dims d;
  if (check_dims(dims, d) != TFM_OK) return 0;
  return ws_layout(d).total;
}

const char* tfm_last_error(void) { return g_err.c_str(); }

int tfm_prof_item_bwd_fused_rows(int head_dim) {
  return tfm::item_attn_bwd_fused_max_rows(head_dim);
}

int tfm_layer_fwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                  const void* X, const float* params, void* Y, void* saved, size_t saved_bytes,
                  void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  int rc = check_dims(dims, d);
  if (rc) return rc;
  if (!aligned(X) || !aligned(params) || !aligned(Y) || !aligned(saved) || !aligned(workspace))
    return fail(TFM_ERR_POINTER, "X, params, Y, saved and workspace must be non-null and "
                                 "16-byte aligned");
  const SavedLayout S = saved_layout(d);
  const WsLayout W = ws_layout(d);
  if (saved_bytes < saved_total(d))
    return fail(TFM_ERR_BUFFER, "saved buffer has %zu bytes, %zu required", saved_bytes,
                saved_total(d));
  if (workspace_bytes < W.total)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes,
                W.total);
  Plan P;
  rc = make_plan(d, n_train, cell_mask, P);
  if (rc) return rc;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  char* sv = (char*)saved;
  tfm::Geo g;
  rc = setup_geo(d, P, ws, W.meta, g, s);
  if (rc) return rc;
  if (d.block == TFM_BLOCK_PRENORM)
    return fwd_pre(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y,
                   bufs_from_pre_saved(sv, pre_saved_layout(d)), fast_ws(d, ws, W), s);
  if (d.dtype == TFM_F32)
    return fwd_simple<float>(d, g, (const float*)X, params, (float*)Y, sv, S, ws, W, s);
  if (fast_eligible(d))
    return fwd_fast(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y, bufs_from_saved(sv, S),
                    fast_ws(d, ws, W), s);
  return fwd_simple<tfm::bf16>(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y, sv, S, ws, W,
                               s);
}

int tfm_layer_bwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                  const void* X, const float* params, const void* saved, size_t saved_bytes,
                  const void* dY, void* dX, float* grads, int accumulate, void* workspace,
                  size_t workspace_bytes, void* stream) {
  Dims d;
  int rc = check_dims(dims, d);
  if (rc) return rc;
  if (!aligned(X) || !aligned(params) || !aligned(saved) || !aligned(dY) || !aligned(dX) ||
      !aligned(grads) || !aligned(workspace))
    return fail(TFM_ERR_POINTER, "X, params, saved, dY, dX, grads and workspace must be "
                                 "non-null and 16-byte aligned");
  const SavedLayout S = saved_layout(d);
  const WsLayout W = ws_layout(d);
  if (saved_bytes < saved_total(d))
    return fail(TFM_ERR_BUFFER, "saved buffer has %zu bytes, %zu required", saved_bytes,
                saved_total(d));
  if (workspace_bytes < W.total)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes,
                W.total);
  Plan P;
  rc = make_plan(d, n_train, cell_mask, P);
  if (rc) return rc;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  tfm::Geo g;
  rc = setup_geo(d, P, ws, W.meta, g, s);
  if (rc) return rc;
  if (d.block == TFM_BLOCK_PRENORM)
    return bwd_pre(d, g, P, params, (const char*)saved, pre_saved_layout(d),
                   (const tfm::bf16*)dY, (tfm::bf16*)dX, grads, accumulate, ws, W, s);
  if (d.dtype == TFM_F32)
    return bwd_simple<float>(d, g, (const float*)X, params, (const char*)saved, S,
                             (const float*)dY, (float*)dX, grads, accumulate, ws, W, s);
  if (fast_eligible(d))
    return bwd_fast(d, g, P, (const tfm::bf16*)X, params, (const char*)saved, S,
                    (const tfm::bf16*)dY, (tfm::bf16*)dX, grads, accumulate, ws, W, s);
  return bwd_simple<tfm::bf16>(d, g, (const tfm::bf16*)X, params, (const char*)saved, S,
                               (const tfm::bf16*)dY, (tfm::bf16*)dX, grads, accumulate, ws, W,
                               s);
}

// Allocation-free forward: the plan and the bf16 weights in the library's static scratch.
int tfm_layer_fwd_noalloc(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          const void* X, const float* params, void* Y, void* saved,
                          size_t saved_bytes, void* stream) {
  Dims d;
  int rc = check_dims(dims, d);
  if (rc) return rc;
  if (!infer_eligible(d))
    return fail(TFM_ERR_DIMS, "tfm_layer_fwd_noalloc needs TFM_BF16, E in {64, 128, 192, 256} "
                              "and H a multiple of E");
  if (!aligned(X) || !aligned(params) || !aligned(Y) || !aligned(saved))
    return fail(TFM_ERR_POINTER, "X, params, Y and saved must be non-null and 16-byte aligned");
  Arena a;
  const MetaOff M = take_meta(d, a);
  const tfm::WOff wo = tfm::weight_offsets(d.E, d.H);
  const size_t w_off = a.take((size_t)wo.total * 2);
  const size_t wt_off = a.take((size_t)wo.total * 2);
  if (a.off > tfm::kStaticScratchBytes)
    return fail(TFM_ERR_BUFFER, "these dims need %zu bytes of library scratch; the maximum is "
                                "%zu (TFM_NOALLOC_SCRATCH_BYTES)", a.off,
                tfm::kStaticScratchBytes);
  if (saved_bytes < saved_total(d))
    return fail(TFM_ERR_BUFFER, "saved buffer has %zu bytes, %zu required", saved_bytes,
                saved_total(d));
  Plan P;
  rc = make_plan(d, n_train, cell_mask, P);
  if (rc) return rc;
  hipStream_t s = (hipStream_t)stream;
  void* base = nullptr;
  HIPCHK(tfm::static_scratch(s, &base));
  char* ws = (char*)base;
  tfm::Geo g;
  rc = setup_geo(d, P, ws, M, g, s);
  if (rc) return rc;
  FastWs f{};
  f.wo = wo;
  f.w = (tfm::bf16*)(ws + w_off);
  f.wt = (tfm::bf16*)(ws + wt_off);
  char* sv = (char*)saved;
  if (d.block == TFM_BLOCK_PRENORM)
    return fwd_pre(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y,
                   bufs_from_pre_saved(sv, pre_saved_layout(d)), f, s);
  return fwd_fast(d, g, (const tfm::bf16*)X, params, (tfm::bf16*)Y,
                  bufs_from_saved(sv, saved_layout(d)), f, s);
}

// Shared checks of the thinking-row calls (the dims, the workspace that holds the column map,
// the plan from n_train and the mask, 1 <= T <= every n_train), then the column map upload.
static int thinking_setup(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          int T, void* workspace, size_t workspace_bytes, Dims& d, tfm::Geo& g,
                          hipStream_t s) {
  int rc = check_dims(dims, d);
  if (rc) return rc;
  if (!aligned(workspace)) return fail(TFM_ERR_POINTER, "workspace must be 16-byte aligned");
  // only the column map is used: it leads both the training and the forward-only workspaces
  Arena a;
  const MetaOff M = take_meta(d, a);
  if (workspace_bytes < a.off)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes, a.off);
  Plan P;
  rc = make_plan(d, n_train, cell_mask, P);
  if (rc) return rc;
  for (int b = 0; b < d.B; ++b)
    if (T < 1 || T > n_train[b])
      return fail(TFM_ERR_DIMS, "T=%d thinking rows outside [1, n_train[%d]=%d]", T, b,
                  n_train[b]);
  return setup_geo(d, P, (char*)workspace, M, g, s);
}

int tfm_thinking_rows_fwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          int T, const float* table, void* X, void* workspace,
                          size_t workspace_bytes, void* stream) {
  Dims d;
  tfm::Geo g;
  hipStream_t s = (hipStream_t)stream;
  if (!aligned(table) || !aligned(X))
    return fail(TFM_ERR_POINTER, "table and X must be non-null and 16-byte aligned");
  int rc = thinking_setup(dims, n_train, cell_mask, T, workspace, workspace_bytes, d, g, s);
  if (rc) return rc;
  if (d.dtype == TFM_F32) HIPCHK(tfm::launch_thinking_fwd<float>(g, T, table, (float*)X, s));
  else HIPCHK(tfm::launch_thinking_fwd<tfm::bf16>(g, T, table, (tfm::bf16*)X, s));
  return TFM_OK;
}

int tfm_thinking_rows_bwd(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          int T, const void* dX, float* dtable, int accumulate, void* workspace,
                          size_t workspace_bytes, void* stream) {
  Dims d;
  tfm::Geo g;
  hipStream_t s = (hipStream_t)stream;
  if (!aligned(dX) || !aligned(dtable))
    return fail(TFM_ERR_POINTER, "dX and dtable must be non-null and 16-byte aligned");
  int rc = thinking_setup(dims, n_train, cell_mask, T, workspace, workspace_bytes, d, g, s);
  if (rc) return rc;
  if (d.dtype == TFM_F32)
    HIPCHK(tfm::launch_thinking_bwd<float>(g, T, (const float*)dX, dtable, accumulate, s));
  else
    HIPCHK(tfm::launch_thinking_bwd<tfm::bf16>(g, T, (const tfm::bf16*)dX, dtable, accumulate,
                                               s));
  return TFM_OK;
}

size_t tfm_infer_workspace_bytes(const tfm_dims* dims) {
  Dims d;
  if (check_dims(dims, d) != TFM_OK) return 0;
  if (!infer_eligible(d)) {
    fail(TFM_ERR_DIMS, "forward-only calls need TFM_BF16, E in {64, 128, 192, 256} and H a "
                       "multiple of E");
    return 0;
  }
  return infer_layout(d).total;
}

size_t tfm_infer_cache_bytes(const tfm_dims* dims) {
  Dims d;
  if (check_dims(dims, d) != TFM_OK) return 0;
  return 2 * cache_half(d);
}

int tfm_layer_fwd_context(const tfm_dims* dims, const int32_t* n_train, const uint8_t* cell_mask,
                          const void* X, const float* params, void* Y, void* kv_cache,
                          size_t cache_bytes, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return infer_call(dims, -1, n_train, cell_mask, X, params, Y, kv_cache, cache_bytes,
                    workspace, workspace_bytes, (hipStream_t)stream);
}

int tfm_layer_fwd_query(const tfm_dims* dims, int32_t context_rows, const int32_t* n_train,
                        const uint8_t* cell_mask, const void* X, const float* params,
                        const void* kv_cache, size_t cache_bytes, void* Y, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (context_rows < 0) return fail(TFM_ERR_DIMS, "context_rows=%d must be >= 1", context_rows);
  return infer_call(dims, context_rows, n_train, cell_mask, X, params, Y,
                    const_cast<void*>(kv_cache), cache_bytes, workspace, workspace_bytes,
                    (hipStream_t)stream);
}

}  // extern "C"
