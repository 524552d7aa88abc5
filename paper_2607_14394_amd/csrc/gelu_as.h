// Shared device GELU of the block epilogue kernels (included inside their
// anonymous namespace).
#pragma once

// GELU(v) = v Phi(v), Phi(v) = (1 + erf(v / sqrt 2)) / 2, with erf from the
// rational-exponential approximation of Abramowitz & Stegun, Handbook of
// Mathematical Functions, formula 7.1.26 (absolute error below 1.5e-7 for
// x >= 0; erf is odd): erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5))))
// exp(-x^2), t = 1 / (1 + p x).  Branch-free: with x = |v| / sqrt 2,
// q = (1 - erf(x)) / 2 = Phi(-|v|) (the halving folded into the a_k), and
// v Phi(v) = max(v, 0) - |v| q for either sign of v (v (1 - q) for v >= 0,
// v q for v < 0): a reciprocal, an exponential, five FMAs, four multiplies
// and a max.
__device__ __forceinline__ float gelu_as(float v) {
  const float av = fabsf(v);
  const float x = av * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  float p = fmaf(t, 0.5307027145f, -0.7265760135f);
  p = fmaf(t, p, 0.7107068705f);
  p = fmaf(t, p, -0.142248368f);
  p = fmaf(t, p, 0.127414796f);
  const float e = __builtin_amdgcn_exp2f(-1.44269504088896341f * x * x);
  const float q = (p * t) * e;
  return fmaf(-av, q, fmaxf(v, 0.f));
}
