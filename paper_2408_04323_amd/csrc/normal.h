// Normal partial expectation and distribution function on the device, shared
// by the acquisition kernels (Sec. 4.4.1, Eq. 7-8; Sec. 4.4.2, Eq. 9).
//
// G(c) = E[(c - Y)^+] for Y ~ N(mu, sd^2) is sd * h(u), u = (c - mu) / sd,
// h(u) = u Phi(u) + phi(u), and max(0, c - mu) when sd = 0.  h(u) - h(-u) = u,
// so h(u) = max(u, 0) + h(-|u|), and for x >= 0, h(-x) = phi(x) g(x) with
// g(x) = 1 - x M(x), M the Mills ratio P(Z > x) / phi(x).
// * float: g is a rational function P4 / Q6 of s = x / 4 fitted on [0, 14]
//   (coefficients from gen_normal_tail.py: relative error 1e-8 in exact
//   arithmetic, 4e-7 evaluated in float), phi from one exp2; no branches, and
//   1 / sd is formed once per candidate;
// * double: Phi from erfc for u >= -5; below, where the two terms of h cancel,
//   g from the continued fraction of the Mills ratio (Laplace):
//   M(x) = 1 / F_1 with F_k = x + k / F_{k+1}, so g(x) = 1 / (x F_2 + 1).
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>

namespace scoot {

// ---- double ---------------------------------------------------------------
// h(u) for u >= -5 from erfc; below, x = -u: with F_2 = x + 2/(x + 3/(x + ...)),
// h(-x) = phi(x) / (x F_2 + 1); F_2 = P/Q from the forward recurrence of its
// convergents, P_k = x P_{k-1} + (k+1) P_{k-2} (same for Q), 24 terms, one
// division; 0 beyond x = 38.6 where phi underflows.
__device__ inline double h_normal(double u) {
  const double inv_sqrt2pi = 0.39894228040143267794;
  if (u >= -5.0) return u * 0.5 * erfc(u * -0.70710678118654752440) + inv_sqrt2pi * exp(-0.5 * u * u);
  const double x = -u;
  if (x > 38.6) return 0.0;
  double pm = 1.0, p0 = x, qm = 0.0, q0 = 1.0;
#pragma unroll
  for (int k = 1; k <= 24; ++k) {
    const double p1 = x * p0 + (double)(k + 1) * pm;
    const double q1 = x * q0 + (double)(k + 1) * qm;
    pm = p0;
    p0 = p1;
    qm = q0;
    q0 = q1;
  }
  return inv_sqrt2pi * exp(-0.5 * x * x) * q0 / (x * p0 + q0);
}

// ---- float ------------------------------------------------------------------
// h(u) = max(u, 0) + phi(x) P4(s) / Q6(s), x = min(|u|, 16), s = x / 4.  Past
// x = 14 phi has underflowed to 0 in float (the clamp keeps P and Q finite).
__device__ inline float h_normal(float u) {
  const float x = fminf(fabsf(u), 16.0f);
  const float s = x * 0.25f;
  const float P = fmaf(fmaf(fmaf(fmaf(1.168936206e+00f, s, 3.086232540e+00f), s, 3.946713647e+00f), s,
                            2.790141401e+00f),
                       s, 9.999999897e-01f);
  const float Q =
      fmaf(fmaf(fmaf(fmaf(fmaf(fmaf(1.870267853e+01f, s, 4.938444122e+01f), s, 6.662181372e+01f), s, 5.403020981e+01f),
                     s, 2.706728781e+01f),
                s, 7.803394828e+00f),
           s, 1.0f);
  // phi(x) = exp(-x^2 / 2) / sqrt(2 pi) = 2^(-x^2 log2(e) / 2) / sqrt(2 pi)
  const float phi = 0.39894228040143267794f * __builtin_amdgcn_exp2f(x * x * -0.72134752044448170368f);
  return fmaxf(u, 0.0f) + phi * P * __builtin_amdgcn_rcpf(Q);
}

// G(c) given mu, sd and inv_sd = 1 / sd (inf when sd = 0, then unused).
template <typename T>
__device__ inline T partial_expectation(T c, T mu, T sd, T inv_sd) {
  const T g = sd * h_normal((c - mu) * inv_sd);
  return sd > T(0) ? g : (c - mu > T(0) ? c - mu : T(0));
}
template <typename T>
__device__ inline T reciprocal(T sd) {
  return T(1) / sd;
}

// Phi(u) = P(Z <= u) = erfc(-u / sqrt 2) / 2.
__device__ inline float normal_cdf(float u) { return 0.5f * erfcf(u * -0.70710678118654752440f); }
__device__ inline double normal_cdf(double u) { return 0.5 * erfc(u * -0.70710678118654752440); }

}  // namespace scoot
