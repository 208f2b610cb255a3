// Host side of the C ABI declared in include/tfm_ends.h: argument validation, the per-dataset
// metadata, the workspace layout and the launch sequences of the encoders and the decoder.
#include "tfm_ends.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <vector>

#include "ends.h"
#include "fast.h"
#include "kernels.h"
#include "prof.h"

namespace {

using tfm::EndsDs;
using tfm::EndsGeo;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return tfm::abi_fail(code, buf);
}

constexpr size_t kAlign = 256;
constexpr int kRowChunk = 256;  // decoder rows per partial product of the weight gradients
constexpr int kColChunk = 32;   // decoder rows per partial column sum of the bias gradients
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
bool aligned(const void* p) { return p && ((uintptr_t)p % 16) == 0; }

struct Shape {
  int B, R, C, S, E, dtype;
  int G, F, T, Hd, K, mean;
  int off[8];
};

int check(const tfm_dims* dims, const tfm_ends* ends, Shape& s) {
  int rc = tfm::abi_check_dims(dims);
  if (rc) return rc;
  if (!ends) return fail(TFM_ERR_POINTER, "ends is null");
  s.B = dims->B; s.R = dims->R; s.C = dims->C; s.S = dims->C + 1; s.E = dims->E;
  s.dtype = dims->dtype;
  s.G = ends->G; s.F = ends->F; s.T = ends->T; s.Hd = ends->Hd; s.K = ends->K;
  s.mean = ends->decode_mean;
  if (s.C < 1) return fail(TFM_ERR_DIMS, "C=%d: the ends need at least one feature cell", s.C);
  if (s.G < 1 || s.G > tfm::ENDS_GMAX)
    return fail(TFM_ERR_DIMS, "group size G=%d outside [1, %d]", s.G, tfm::ENDS_GMAX);
  for (int k = 0; k < 8; ++k) {
    s.off[k] = k < s.G ? ends->offsets[k] : 0;
    if (k < s.G && (s.off[k] < 0 || s.off[k] > (1 << 20)))
      return fail(TFM_ERR_DIMS, "offsets[%d]=%d outside [0, 2^20]", k, s.off[k]);
  }
  if (s.F < 1) return fail(TFM_ERR_DIMS, "F=%d must be >= 1", s.F);
  if (s.T < 0 || s.T >= s.R) return fail(TFM_ERR_DIMS, "T=%d outside [0, R-1=%d]", s.T, s.R - 1);
  if (s.Hd < 1 || s.Hd > 4096) return fail(TFM_ERR_DIMS, "Hd=%d outside [1, 4096]", s.Hd);
  if (s.K < 1 || s.K > tfm::ENDS_KMAX)
    return fail(TFM_ERR_DIMS, "K=%d outside [1, %d]", s.K, tfm::ENDS_KMAX);
  if (s.mean != 0 && s.mean != 1) return fail(TFM_ERR_DIMS, "decode_mean=%d is not 0 or 1", s.mean);
  return TFM_OK;
}

struct Offsets {
  size_t Wfe, bfe, Wte, bte, Wd1, bd1, Wd2, bd2, total;
};
Offsets param_offsets(const Shape& s) {
  Offsets o;
  o.Wfe = 0;
  o.bfe = o.Wfe + (size_t)s.E * s.G;
  o.Wte = o.bfe + s.E;
  o.bte = o.Wte + s.E;
  o.Wd1 = o.bte + s.E;
  o.bd1 = o.Wd1 + (size_t)s.Hd * s.E;
  o.Wd2 = o.bd1 + s.Hd;
  o.bd2 = o.Wd2 + (size_t)s.K * s.Hd;
  o.total = o.bd2 + s.K;
  return o;
}

// Workspace, sized for the most decoder rows the dims allow (every row of every dataset: the
// forward-only decoder call takes tables without labelled rows).
struct Ws {
  size_t meta, epart, Z, H1, A1, LG, DL, LROW, DH1, DZ, wpart, bpart, total;
};
Ws ws_layout(const Shape& s) {
  const int64_t Tmax = (int64_t)s.B * s.R;
  const int64_t nz = (Tmax + kRowChunk - 1) / kRowChunk;
  const int64_t nzc = (Tmax + kColChunk - 1) / kColChunk;
  const int64_t slabs = (int64_t)s.B * ((s.R - s.T + tfm::ENC_ROWS - 1) / tfm::ENC_ROWS);
  const size_t wmax = (size_t)s.Hd * (s.E > s.K ? s.E : s.K);
  Ws w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align_up(bytes > 0 ? bytes : 1);
    return at;
  };
  w.meta = take((size_t)s.B * sizeof(EndsDs));
  w.epart = take((size_t)slabs * s.E * (s.G + 3) * 4);
  w.Z = take((size_t)Tmax * s.E * 4);
  w.H1 = take((size_t)Tmax * s.Hd * 4);
  w.A1 = take((size_t)Tmax * s.Hd * 4);
  w.LG = take((size_t)Tmax * s.K * 4);
  w.DL = take((size_t)Tmax * s.K * 4);
  w.LROW = take((size_t)Tmax * 4);
  w.DH1 = take((size_t)Tmax * s.Hd * 4);
  w.DZ = take((size_t)Tmax * s.E * 4);
  w.wpart = take((size_t)nz * wmax * 4);
  w.bpart = take((size_t)nzc * (s.Hd > s.K ? s.Hd : s.K) * 4);
  w.total = off;
  return w;
}

// Per-dataset metadata: validates the host arrays, fills the device-side table through kernel
// arguments and returns the geometry (n_class may be null for the calls that do not need it).
// n_train[b] must lie in [nt_min, R]: T + 1 for the calls that need a labelled row, 0 for the
// forward-only decoder.
int setup(const Shape& s, const int32_t* n_train, const int32_t* n_feat, const int32_t* n_class,
          char* ws, const Ws& W, EndsGeo& g, hipStream_t st, int nt_min = -1) {
  if (nt_min < 0) nt_min = s.T + 1;
  if (!n_train || !n_feat) return fail(TFM_ERR_POINTER, "n_train or n_feat is null");
  std::vector<int32_t> blob((size_t)s.B * 4);
  int64_t test0 = 0;
  const int mmax = s.C < s.F ? s.C : s.F;
  for (int b = 0; b < s.B; ++b) {
    if (n_train[b] < nt_min || n_train[b] > s.R)
      return fail(TFM_ERR_NTRAIN, "n_train[%d]=%d outside [%d, R=%d]", b, n_train[b], nt_min,
                  s.R);
    if (n_feat[b] < 1 || n_feat[b] > mmax)
      return fail(TFM_ERR_DIMS, "n_feat[%d]=%d outside [1, min(C, F)=%d]", b, n_feat[b], mmax);
    if (n_class && (n_class[b] < 1 || n_class[b] > s.K))
      return fail(TFM_ERR_DIMS, "n_class[%d]=%d outside [1, K=%d]", b, n_class[b], s.K);
    blob[4 * b + 0] = n_train[b];
    blob[4 * b + 1] = n_feat[b];
    blob[4 * b + 2] = n_class ? n_class[b] : 1;
    blob[4 * b + 3] = (int32_t)test0;
    test0 += s.R - n_train[b];
  }
  g.B = s.B; g.R = s.R; g.S = s.S; g.E = s.E; g.T = s.T; g.F = s.F; g.G = s.G;
  for (int k = 0; k < 8; ++k) g.off[k] = s.off[k];
  g.Hd = s.Hd; g.K = s.K; g.mean = s.mean;
  g.Ttot = test0;
  g.ds = (const EndsDs*)(ws + W.meta);
  hipError_t e = tfm::launch_upload(blob.data(), (int64_t)blob.size(), (int32_t*)(ws + W.meta), st);
  if (e != hipSuccess)
    return fail(TFM_ERR_HIP, "metadata upload failed: %s", hipGetErrorString(e));
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
    tfm::prof_begin(name, st);       \
    HIPCHK(__VA_ARGS__);             \
    tfm::prof_end(st);               \
  } while (0)

int common(const tfm_dims* dims, const tfm_ends* ends, void* workspace, size_t workspace_bytes,
           Shape& s, Ws& W) {
  int rc = check(dims, ends, s);
  if (rc) return rc;
  W = ws_layout(s);
  if (!aligned(workspace)) return fail(TFM_ERR_POINTER, "workspace null or not 16-byte aligned");
  if (workspace_bytes < W.total)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes,
                W.total);
  return TFM_OK;
}

// Decoder forward: Z, H1 = Z W1^T + b1, A1 = GELU(H1), logits = A1 W2^T + b2.
int decoder_forward(const Shape& s, const EndsGeo& g, const void* Y, const float* prm,
                    float* logits, char* ws, const Ws& W, hipStream_t st) {
  const Offsets o = param_offsets(s);
  float* Z = (float*)(ws + W.Z);
  if (s.dtype == TFM_BF16)
    STEP("dec_gather/hbm", tfm::launch_decode_gather(g, (const tfm::bf16*)Y, Z, st));
  else
    STEP("dec_gather/hbm", tfm::launch_decode_gather(g, (const float*)Y, Z, st));
  tfm::SgemmArgs a{};
  a.A = Z; a.lda = s.E;
  a.B = prm + o.Wd1; a.ldb = s.E;
  a.C = (float*)(ws + W.H1); a.C2 = (float*)(ws + W.A1); a.ldc = s.Hd;
  a.bias = prm + o.bd1;
  a.M = (int)g.Ttot; a.N = s.Hd; a.K = s.E;
  STEP("dec_hidden/mfma", tfm::launch_sgemm(a, false, true, tfm::SG_GELU, st));
  tfm::SgemmArgs b{};
  b.A = (const float*)(ws + W.A1); b.lda = s.Hd;
  b.B = prm + o.Wd2; b.ldb = s.Hd;
  b.C = logits; b.ldc = s.K;
  b.bias = prm + o.bd2;
  b.M = (int)g.Ttot; b.N = s.K; b.K = s.Hd;
  STEP("dec_logits/mfma", tfm::launch_sgemm(b, false, true, tfm::SG_BIAS, st));
  return TFM_OK;
}

// grads[off .. off + M*N) (+)= sum over decoder rows of op(A)^T B, reduced over row chunks in a
// fixed order.
int row_contraction(const float* A, int64_t lda, const float* B, int64_t ldb, int M, int N,
                    int64_t rows, float* part, float* out, int accumulate, hipStream_t st) {
  const int nz = (int)((rows + kRowChunk - 1) / kRowChunk);
  tfm::SgemmArgs a{};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb;
  a.C = part; a.ldc = N; a.zstride = (int64_t)M * N;
  a.M = M; a.N = N; a.K = (int)rows; a.kchunk = kRowChunk;
  STEP("dec_wgrad/mfma", tfm::launch_sgemm(a, true, false, tfm::SG_BIAS, st));
  STEP("dec_wgrad_reduce/hbm", tfm::launch_reduce_z(nz, (int64_t)M * N, (int64_t)M * N, part, out,
                                                 accumulate, st));
  return TFM_OK;
}

int column_sums(const float* A, int64_t lda, int N, int64_t rows, float* part, float* out,
                int accumulate, hipStream_t st) {
  const int nz = (int)((rows + kColChunk - 1) / kColChunk);
  STEP("dec_bgrad/hbm", tfm::launch_colsum<float>(rows, N, A, lda, nullptr, 0, kColChunk, part, st));
  STEP("dec_bgrad_reduce/hbm", tfm::launch_reduce_z(nz, N, N, part, out, accumulate, st));
  return TFM_OK;
}

}  // namespace

extern "C" {

size_t tfm_ends_param_count(const tfm_dims* dims, const tfm_ends* ends) {
  Shape s;
  if (check(dims, ends, s)) return 0;
  return param_offsets(s).total;
}

size_t tfm_ends_workspace_bytes(const tfm_dims* dims, const tfm_ends* ends) {
  Shape s;
  if (check(dims, ends, s)) return 0;
  return ws_layout(s).total;
}

int tfm_encode_fwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const float* x, const int32_t* labels,
                   const float* params, void* X, void* workspace, size_t workspace_bytes,
                   void* stream) {
  Shape s;
  Ws W;
  int rc = common(dims, ends, workspace, workspace_bytes, s, W);
  if (rc) return rc;
  if (!aligned(x) || !aligned(labels) || !aligned(params) || !aligned(X))
    return fail(TFM_ERR_POINTER, "x, labels, params and X must be non-null and 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  EndsGeo g;
  rc = setup(s, n_train, n_feat, nullptr, ws, W, g, st);
  if (rc) return rc;
  if (s.dtype == TFM_BF16)
    STEP("encode_fwd/hbm", tfm::launch_encode_fwd(g, x, labels, params, (tfm::bf16*)X, st));
  else
    STEP("encode_fwd/hbm", tfm::launch_encode_fwd(g, x, labels, params, (float*)X, st));
  return TFM_OK;
}

int tfm_encode_bwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const float* x, const int32_t* labels, const void* dX,
                   float* grads, int accumulate, void* workspace, size_t workspace_bytes,
                   void* stream) {
  Shape s;
  Ws W;
  int rc = common(dims, ends, workspace, workspace_bytes, s, W);
  if (rc) return rc;
  if (!aligned(x) || !aligned(labels) || !aligned(dX) || !aligned(grads))
    return fail(TFM_ERR_POINTER, "x, labels, dX and grads must be non-null and 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  EndsGeo g;
  rc = setup(s, n_train, n_feat, nullptr, ws, W, g, st);
  if (rc) return rc;
  float* part = (float*)(ws + W.epart);
  if (s.dtype == TFM_BF16)
    STEP("encode_bwd/hbm", tfm::launch_encode_bwd(g, x, labels, (const tfm::bf16*)dX, part, st));
  else
    STEP("encode_bwd/hbm", tfm::launch_encode_bwd(g, x, labels, (const float*)dX, part, st));
  const int64_t cnt = (int64_t)s.E * (s.G + 3);
  STEP("encode_bwd_reduce/hbm", tfm::launch_reduce_z((int)tfm::encode_bwd_parts(g), cnt, cnt, part,
                                                  grads, accumulate, st));
  return TFM_OK;
}

int tfm_decode_fwd(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                   const int32_t* n_feat, const void* Y, const float* params, float* logits,
                   void* workspace, size_t workspace_bytes, void* stream) {
  Shape s;
  Ws W;
  int rc = common(dims, ends, workspace, workspace_bytes, s, W);
  if (rc) return rc;
  if (!aligned(Y) || !aligned(params) || !aligned(logits))
    return fail(TFM_ERR_POINTER, "Y, params and logits must be non-null and 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  EndsGeo g;
  rc = setup(s, n_train, n_feat, nullptr, ws, W, g, st, 0);
  if (rc) return rc;
  return decoder_forward(s, g, Y, params, logits, ws, W, st);
}

int tfm_decode_loss(const tfm_dims* dims, const tfm_ends* ends, const int32_t* n_train,
                    const int32_t* n_feat, const int32_t* n_class, const int32_t* labels,
                    const void* Y, const float* params, float* loss, float* logits, void* dY,
                    float* grads, int accumulate, void* workspace, size_t workspace_bytes,
                    void* stream) {
  Shape s;
  Ws W;
  int rc = common(dims, ends, workspace, workspace_bytes, s, W);
  if (rc) return rc;
  if (!aligned(labels) || !aligned(Y) || !aligned(params) || !aligned(loss) || !aligned(dY) ||
      !aligned(grads) || (logits && !aligned(logits)))
    return fail(TFM_ERR_POINTER, "labels, Y, params, loss, dY and grads must be non-null and "
                                 "16-byte aligned (logits too when given)");
  if (!n_class) return fail(TFM_ERR_POINTER, "n_class is null");
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  EndsGeo g;
  rc = setup(s, n_train, n_feat, n_class, ws, W, g, st);
  if (rc) return rc;
  const Offsets o = param_offsets(s);
  const int64_t T = g.Ttot;
  float* DZ = (float*)(ws + W.DZ);
  if (T == 0) {
    // No unlabelled rows: zero loss, zero dY, zero decoder gradients.
    STEP("dec_loss/hbm", tfm::launch_fill_f32(loss, 1, 0.f, st));
    if (s.dtype == TFM_BF16)
      STEP("dec_scatter/hbm", tfm::launch_decode_scatter(g, DZ, (tfm::bf16*)dY, st));
    else
      STEP("dec_scatter/hbm", tfm::launch_decode_scatter(g, DZ, (float*)dY, st));
    if (!accumulate)
      STEP("dec_zero/hbm", tfm::launch_fill_f32(grads + o.Wd1, (int64_t)(o.total - o.Wd1), 0.f, st));
    return TFM_OK;
  }
  float* LG = logits ? logits : (float*)(ws + W.LG);
  rc = decoder_forward(s, g, Y, params, LG, ws, W, st);
  if (rc) return rc;
  float* DL = (float*)(ws + W.DL);
  float* LROW = (float*)(ws + W.LROW);
  STEP("dec_xent/valu", tfm::launch_cross_entropy(g, LG, labels, LROW, DL, st));
  STEP("dec_loss/hbm", tfm::launch_reduce_z((int)T, 1, 1, LROW, loss, 0, st));
  // dH1 = (dL W2) * GELU'(H1)
  tfm::SgemmArgs a{};
  a.A = DL; a.lda = s.K;
  a.B = params + o.Wd2; a.ldb = s.Hd;
  a.C = (float*)(ws + W.DH1); a.ldc = s.Hd;
  a.aux = (const float*)(ws + W.H1);
  a.M = (int)T; a.N = s.Hd; a.K = s.K;
  STEP("dec_dhidden/mfma", tfm::launch_sgemm(a, false, false, tfm::SG_GELU_GRAD, st));
  // dZ = dH1 W1
  tfm::SgemmArgs b{};
  b.A = (const float*)(ws + W.DH1); b.lda = s.Hd;
  b.B = params + o.Wd1; b.ldb = s.E;
  b.C = DZ; b.ldc = s.E;
  b.M = (int)T; b.N = s.E; b.K = s.Hd;
  STEP("dec_dinput/mfma", tfm::launch_sgemm(b, false, false, tfm::SG_BIAS, st));
  if (s.dtype == TFM_BF16)
    STEP("dec_scatter/hbm", tfm::launch_decode_scatter(g, DZ, (tfm::bf16*)dY, st));
  else
    STEP("dec_scatter/hbm", tfm::launch_decode_scatter(g, DZ, (float*)dY, st));
  float* wpart = (float*)(ws + W.wpart);
  float* bpart = (float*)(ws + W.bpart);
  rc = row_contraction((const float*)(ws + W.DH1), s.Hd, (const float*)(ws + W.Z), s.E, s.Hd,
                       s.E, T, wpart, grads + o.Wd1, accumulate, st);
  if (rc) return rc;
  rc = column_sums((const float*)(ws + W.DH1), s.Hd, s.Hd, T, bpart, grads + o.bd1, accumulate,
                   st);
  if (rc) return rc;
  rc = row_contraction(DL, s.K, (const float*)(ws + W.A1), s.Hd, s.K, s.Hd, T, wpart,
                       grads + o.Wd2, accumulate, st);
  if (rc) return rc;
  return column_sums(DL, s.K, s.K, T, bpart, grads + o.bd2, accumulate, st);
}

}  // extern "C"
