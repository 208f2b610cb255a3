// Host side of the C ABI declared in include/tfm_optim.h: argument validation, the step
// scalars of schedule-free AdamW, and the launch sequences of clipping and Muon.
#include "tfm_optim.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <utility>
#include <vector>

#include "ends.h"
#include "kernels.h"
#include "optim.h"
#include "prof.h"

namespace {

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return tfm::abi_fail(code, buf);
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
bool aligned16(const void* p) { return p && ((uintptr_t)p % 16) == 0; }
bool aligned4(const void* p) { return p && ((uintptr_t)p % 4) == 0; }
bool finite_nonneg(float x) { return std::isfinite(x) && x >= 0.f; }

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

int64_t clip_parts(int32_t nvec, const int64_t* counts) {
  int64_t p = 0;
  for (int i = 0; i < nvec; ++i) p += tfm::opt_blocks(counts[i]);
  return p;
}

struct MuonWs {
  size_t ptr, part, X0, X1, A, Bm, total;
};
MuonWs muon_layout(int32_t count, int32_t rows, int32_t cols) {
  const int64_t n = std::min(rows, cols), m = std::max(rows, cols);
  MuonWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += align_up(bytes > 0 ? bytes : 1);
    return at;
  };
  w.ptr = take((size_t)count * 3 * 8);
  w.part = take((size_t)count * tfm::opt_blocks((int64_t)rows * cols) * 4);
  w.X0 = take((size_t)count * n * m * 4);
  w.X1 = take((size_t)count * n * m * 4);
  w.A = take((size_t)count * n * n * 4);
  w.Bm = take((size_t)count * n * n * 4);
  w.total = off;
  return w;
}

bool muon_shape_ok(int32_t count, int32_t rows, int32_t cols) {
  return count >= 1 && count <= 1024 && rows >= 1 && rows <= 8192 && cols >= 1 && cols <= 8192;
}

}  // namespace

extern "C" {

size_t tfm_clip_workspace_bytes(int32_t nvec, const int64_t* counts) {
  if (nvec < 1 || nvec > 1024 || !counts) return 0;
  for (int i = 0; i < nvec; ++i)
    if (counts[i] < 0) return 0;
  return align_up((size_t)std::max<int64_t>(clip_parts(nvec, counts), 1) * 4);
}

int tfm_clip_scale(int32_t nvec, const float* const* grads, const int64_t* counts, float max_norm,
                   float* scale, float* norm, void* workspace, size_t workspace_bytes,
                   void* stream) {
  if (nvec < 1 || nvec > 1024) return fail(TFM_ERR_DIMS, "nvec=%d outside [1, 1024]", nvec);
  if (!grads || !counts) return fail(TFM_ERR_POINTER, "grads or counts is null");
  for (int i = 0; i < nvec; ++i) {
    if (counts[i] < 0) return fail(TFM_ERR_DIMS, "counts[%d]=%lld is negative", i,
                                   (long long)counts[i]);
    if (counts[i] > 0 && !aligned4(grads[i]))
      return fail(TFM_ERR_POINTER, "grads[%d] is null or not 4-byte aligned", i);
  }
  if (!(std::isfinite(max_norm) && max_norm > 0.f))
    return fail(TFM_ERR_DIMS, "max_norm must be finite and > 0");
  if (!aligned16(scale) || (norm && !aligned16(norm)) || !aligned16(workspace))
    return fail(TFM_ERR_POINTER, "scale, norm and workspace must be 16-byte aligned");
  const size_t need = tfm_clip_workspace_bytes(nvec, counts);
  if (workspace_bytes < need)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  float* part = (float*)workspace;
  int64_t off = 0;
  for (int i = 0; i < nvec; ++i) {
    STEP("clip_sumsq/hbm", tfm::launch_sumsq(grads[i], counts[i], part + off, st));
    off += tfm::opt_blocks(counts[i]);
  }
  STEP("clip_final/hbm", tfm::launch_clip_final(part, off, max_norm, scale, norm, st));
  return TFM_OK;
}

int tfm_sfadamw_step(const tfm_sfadamw* hp, int64_t t, int32_t nseg, const int64_t* seg_off,
                     const int64_t* seg_len, float* y, float* z, float* v, const float* grad,
                     const float* grad_scale, void* stream) {
  if (!hp) return fail(TFM_ERR_POINTER, "hp is null");
  if (!finite_nonneg(hp->lr) || !(hp->beta1 >= 0.f && hp->beta1 <= 1.f) ||
      !(hp->beta2 >= 0.f && hp->beta2 < 1.f) || !finite_nonneg(hp->eps) ||
      !finite_nonneg(hp->weight_decay) || hp->warmup < 0)
    return fail(TFM_ERR_DIMS, "schedule-free AdamW needs lr, eps, weight_decay >= 0, beta1 in "
                              "[0, 1], beta2 in [0, 1) and warmup >= 0");
  if (t < 1) return fail(TFM_ERR_DIMS, "step t=%lld must be >= 1", (long long)t);
  if (nseg < 1 || nseg > tfm::SF_MAXSEG)
    return fail(TFM_ERR_DIMS, "nseg=%d outside [1, %d]", nseg, tfm::SF_MAXSEG);
  if (!seg_off || !seg_len) return fail(TFM_ERR_POINTER, "seg_off or seg_len is null");
  std::vector<std::pair<int64_t, int64_t>> segs;
  for (int k = 0; k < nseg; ++k) {
    if (seg_off[k] < 0 || seg_len[k] < 0)
      return fail(TFM_ERR_DIMS, "segment %d has a negative offset or length", k);
    segs.emplace_back(seg_off[k], seg_len[k]);
  }
  std::sort(segs.begin(), segs.end());
  for (size_t k = 1; k < segs.size(); ++k)
    if (segs[k - 1].first + segs[k - 1].second > segs[k].first)
      return fail(TFM_ERR_DIMS, "segments overlap");
  if (!aligned4(y) || !aligned4(z) || !aligned4(v) || !aligned4(grad) ||
      (grad_scale && !aligned4(grad_scale)))
    return fail(TFM_ERR_POINTER, "y, z, v and grad must be non-null and 4-byte aligned");
  tfm::SfSegs sg{};
  sg.nseg = nseg;
  sg.start[0] = 0;
  for (int k = 0; k < nseg; ++k) {
    sg.off[k] = seg_off[k];
    sg.start[k + 1] = sg.start[k] + seg_len[k];
  }
  // step scalars in double: the scheduled rate s_t, the step rate gamma_t = s_t sqrt(1 - b2^t),
  // the averaging weight c = gamma_t^2 / sum_{i<=t} gamma_i^2 and the y coefficient.  The sum
  // runs term by term over the warm-up steps; past them s_i = lr and the tail is
  // lr^2 ((t - w) - sum_{i=w+1}^{t} b2^i), the geometric part in closed form.
  const double lr = hp->lr, b2 = hp->beta2;
  const int64_t w = hp->warmup;
  const double st_rate = w > 0 ? lr * std::min(1.0, (double)t / (double)w) : lr;
  const int64_t kw = w > 0 ? std::min<int64_t>(t, w) : 0;
  double gsum = 0.0;
  for (int64_t i = 1; i <= kw; ++i) {
    const double si = lr * (double)i / (double)w;
    gsum += si * si * (1.0 - std::pow(b2, (double)i));
  }
  if (t > kw) {
    const double geo = b2 == 1.0 ? 0.0 : std::pow(b2, (double)(kw + 1)) *
                                             (1.0 - std::pow(b2, (double)(t - kw))) / (1.0 - b2);
    gsum += lr * lr * ((double)(t - kw) - (b2 == 1.0 ? (double)(t - kw) : geo));
  }
  const double gamma = st_rate * std::sqrt(1.0 - std::pow(b2, (double)t));
  const double c = gsum > 0.0 ? gamma * gamma / gsum : 1.0;
  tfm::SfScalars sc;
  sc.beta2 = hp->beta2;
  sc.eps = hp->eps;
  sc.wd = hp->weight_decay;
  sc.c = (float)c;
  sc.gamma = (float)gamma;
  sc.ycoef = (float)(gamma * ((double)hp->beta1 * (1.0 - c) - 1.0));
  hipStream_t st = (hipStream_t)stream;
  STEP("sfadamw/hbm", tfm::launch_sfadamw(sg, sc, y, z, v, grad, grad_scale, st));
  return TFM_OK;
}

size_t tfm_muon_workspace_bytes(int32_t count, int32_t rows, int32_t cols) {
  if (!muon_shape_ok(count, rows, cols)) return 0;
  return muon_layout(count, rows, cols).total;
}

int tfm_muon_step(const tfm_muon* hp, int32_t count, int32_t rows, int32_t cols, float* const* W,
                  const float* const* G, float* const* buf, const float* grad_scale,
                  void* workspace, size_t workspace_bytes, void* stream) {
  if (!hp) return fail(TFM_ERR_POINTER, "hp is null");
  if (!finite_nonneg(hp->lr) || !(hp->momentum >= 0.f && hp->momentum < 1.f) ||
      !finite_nonneg(hp->weight_decay) || hp->ns_steps < 1 || hp->ns_steps > 16)
    return fail(TFM_ERR_DIMS, "Muon needs lr, weight_decay >= 0, momentum in [0, 1) and "
                              "ns_steps in [1, 16]");
  if (!muon_shape_ok(count, rows, cols))
    return fail(TFM_ERR_DIMS, "count=%d rows=%d cols=%d outside [1, 1024] x [1, 8192]^2", count,
                rows, cols);
  if (!W || !G || !buf) return fail(TFM_ERR_POINTER, "W, G or buf is null");
  for (int i = 0; i < count; ++i)
    if (!aligned4(W[i]) || !aligned4(G[i]) || !aligned4(buf[i]))
      return fail(TFM_ERR_POINTER, "matrix %d: W, G and buf must be non-null and 4-byte aligned",
                  i);
  if ((grad_scale && !aligned4(grad_scale)) || !aligned16(workspace))
    return fail(TFM_ERR_POINTER, "grad_scale must be 4-byte and workspace 16-byte aligned");
  const MuonWs L = muon_layout(count, rows, cols);
  if (workspace_bytes < L.total)
    return fail(TFM_ERR_BUFFER, "workspace has %zu bytes, %zu required", workspace_bytes,
                L.total);
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  // the pointer table goes to the device through kernel arguments (as int32 halves)
  std::vector<int32_t> tab((size_t)count * 6);
  for (int i = 0; i < count; ++i) {
    const uintptr_t p[3] = {(uintptr_t)W[i], (uintptr_t)G[i], (uintptr_t)buf[i]};
    for (int j = 0; j < 3; ++j) {
      tab[(size_t)6 * i + 2 * j] = (int32_t)(uint32_t)(p[j] & 0xffffffffu);
      tab[(size_t)6 * i + 2 * j + 1] = (int32_t)(uint32_t)(p[j] >> 32);
    }
  }
  STEP("muon_upload/hbm", tfm::launch_upload(tab.data(), (int64_t)tab.size(),
                                             (int32_t*)(ws + L.ptr), st));
  const int64_t* ptr = (const int64_t*)(ws + L.ptr);
  tfm::MuonGeo mg;
  mg.count = count;
  mg.rows = rows;
  mg.cols = cols;
  mg.tall = rows > cols;
  mg.nesterov = hp->nesterov != 0;
  mg.momentum = hp->momentum;
  mg.eps = 1e-7f;
  mg.shrink = (float)(1.0 - (double)hp->lr * hp->weight_decay);
  mg.step = (float)(hp->lr * std::sqrt(std::max(1.0, (double)rows / (double)cols)));
  const int n = std::min(rows, cols), m = std::max(rows, cols);
  float* X = (float*)(ws + L.X0);
  float* Xn = (float*)(ws + L.X1);
  float* A = (float*)(ws + L.A);
  float* Bm = (float*)(ws + L.Bm);
  float* part = (float*)(ws + L.part);
  STEP("muon_prep/hbm", tfm::launch_muon_prep(mg, ptr, grad_scale, X, part, st));
  STEP("muon_norm/hbm", tfm::launch_muon_norm(mg, part, X, st));
  const float a = 3.4445f, b = -4.7750f, c = 2.0315f;
  for (int s = 0; s < hp->ns_steps; ++s) {
    tfm::SgemmArgs g1{};  // A = X X^T
    g1.A = X; g1.lda = m; g1.B = X; g1.ldb = m; g1.C = A; g1.ldc = n;
    g1.M = n; g1.N = n; g1.K = m;
    g1.batch = count; g1.bsa = (int64_t)n * m; g1.bsb = (int64_t)n * m;
    g1.zstride = (int64_t)n * n;
    STEP("muon_ns/mfma", tfm::launch_sgemm(g1, false, true, tfm::SG_BIAS, st));
    tfm::SgemmArgs g2{};  // Bm = b A + c A A
    g2.A = A; g2.lda = n; g2.B = A; g2.ldb = n; g2.C = Bm; g2.ldc = n;
    g2.aux = A; g2.alpha = c; g2.beta = b;
    g2.M = n; g2.N = n; g2.K = n;
    g2.batch = count; g2.bsa = (int64_t)n * n; g2.bsb = (int64_t)n * n;
    g2.bsaux = (int64_t)n * n; g2.zstride = (int64_t)n * n;
    STEP("muon_ns/mfma", tfm::launch_sgemm(g2, false, false, tfm::SG_AXPBY, st));
    tfm::SgemmArgs g3{};  // X' = a X + Bm X
    g3.A = Bm; g3.lda = n; g3.B = X; g3.ldb = m; g3.C = Xn; g3.ldc = m;
    g3.aux = X; g3.alpha = 1.f; g3.beta = a;
    g3.M = n; g3.N = m; g3.K = n;
    g3.batch = count; g3.bsa = (int64_t)n * n; g3.bsb = (int64_t)n * m;
    g3.bsaux = (int64_t)n * m; g3.zstride = (int64_t)n * m;
    STEP("muon_ns/mfma", tfm::launch_sgemm(g3, false, false, tfm::SG_AXPBY, st));
    std::swap(X, Xn);
  }
  STEP("muon_apply/hbm", tfm::launch_muon_apply(mg, ptr, X, st));
  return TFM_OK;
}

}  // extern "C"
