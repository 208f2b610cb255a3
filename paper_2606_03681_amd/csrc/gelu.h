// Exact-erf GELU and its derivative on the VALU, shared by the MFMA kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace tfm {

// Normal CDF Phi(x) = (1 + erf(x / sqrt 2)) / 2 with erf from Abramowitz & Stegun 7.1.26
// (|error| <= 1.5e-7): erf(z) = 1 - t (a1 + t (a2 + ... + t a5)) exp(-z^2), t = 1 / (1 + p z)
// for z >= 0, odd in z.  *e returns exp(-x^2 / 2), which the normal density shares.
__device__ __forceinline__ float norm_cdf(float x, float* e) {
  const float az = fabsf(x) * 0.70710678118654752f;
  *e = __builtin_amdgcn_exp2f(-0.72134752044448170f * x * x);  // exp(-x^2/2) = 2^(-x^2 log2e / 2)
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, az, 1.0f));
  float poly = fmaf(t, 1.061405429f, -1.453152027f);
  poly = fmaf(t, poly, 1.421413741f);
  poly = fmaf(t, poly, -0.284496736f);
  poly = fmaf(t, poly, 0.254829592f);
  const float h = 0.5f * t * poly * *e;  // (1 - erf(|z|)) / 2
  return x >= 0.f ? 1.0f - h : h;
}
// GELU(x) = x Phi(x)
__device__ __forceinline__ float gelu_f(float x) {
  float e;
  return x * norm_cdf(x, &e);
}
// GELU'(x) = Phi(x) + x phi(x), phi(x) = exp(-x^2 / 2) / sqrt(2 pi)
__device__ __forceinline__ float gelu_grad_f(float x) {
  float e;
  const float cdf = norm_cdf(x, &e);
  return fmaf(x * 0.39894228040143268f, e, cdf);
}

}  // namespace tfm
