// Device-side scalar math shared by the HIP kernels (not by the host code).
#pragma once

namespace partir {

// GELU with the exact (erf) form, GELU(x) = x * Phi(x) = x/2 * (1 + erf(x/sqrt2)).
// erfc(z) for z >= 0 uses Abramowitz & Stegun, Handbook of Mathematical
// Functions, formula 7.1.26: erfc(z) ~ t (a1 + t (a2 + t (a3 + t (a4 + t a5))))
// e^{-z^2}, t = 1 / (1 + p z), absolute error <= 1.5e-7.  Writing the negative
// half as x/2 * erfc(|x|/sqrt2) avoids the cancellation of 1 + erf(x) for
// x << 0.  Cost: one reciprocal, one exp2 and seven FMA-class operations.
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = __builtin_fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, z, 1.0f));
  float q = __builtin_fmaf(t, 1.061405429f, -1.453152027f);
  q = __builtin_fmaf(t, q, 1.421413741f);
  q = __builtin_fmaf(t, q, -0.284496736f);
  q = __builtin_fmaf(t, q, 0.254829592f);
  q *= t * __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);   // erfc(z)
  return 0.5f * x * (x >= 0.0f ? 2.0f - q : q);
}

// Phi(x) = (1 + erf(x / sqrt2)) / 2 from the same erfc approximation.
__device__ __forceinline__ float phi_cdf(float x) {
  const float z = __builtin_fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, z, 1.0f));
  float q = __builtin_fmaf(t, 1.061405429f, -1.453152027f);
  q = __builtin_fmaf(t, q, 1.421413741f);
  q = __builtin_fmaf(t, q, -0.284496736f);
  q = __builtin_fmaf(t, q, 0.254829592f);
  q *= t * __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);   // erfc(z)
  return x >= 0.0f ? 1.0f - 0.5f * q : 0.5f * q;
}

// GELU and its derivative together: gelu'(x) = Phi(x) + x phi(x), with
// phi(x) = exp(-x^2 / 2) / sqrt(2 pi) sharing the exponential of the erfc
// approximation above (z = |x| / sqrt2, so exp(-z^2) = exp(-x^2 / 2)).
__device__ __forceinline__ void gelu_erf_and_grad(float x, float& y, float& dy) {
  const float z = __builtin_fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, z, 1.0f));
  float q = __builtin_fmaf(t, 1.061405429f, -1.453152027f);
  q = __builtin_fmaf(t, q, 1.421413741f);
  q = __builtin_fmaf(t, q, -0.284496736f);
  q = __builtin_fmaf(t, q, 0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);
  q *= t * e;                                       // erfc(z)
  const float phi_cdf = x >= 0.0f ? 1.0f - 0.5f * q : 0.5f * q;
  y = x * phi_cdf;
  dy = __builtin_fmaf(x * e, 0.39894228040143268f, phi_cdf);
}

}  // namespace partir
