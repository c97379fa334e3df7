// fp64 exponential, log(1 + x) and the logistic function for the task
// gradients (the logistic losses of Appendix C's KGE, word-vector and CTR
// tasks), written for the hot loops: a few dozen fused multiply-adds instead
// of the general-purpose library routines, accurate to a few units in the
// last place of fp64 over the ranges used here.
//
//   exp_nonpos(t), t <= 0: Cody-Waite range reduction t = k ln2 + r with
//     |r| <= ln2 / 2 (ln2 split into a 42-bit head, so k * head is exact for
//     |k| < 2^11, and a tail), e^r by its Taylor series through r^13 / 13!
//     (the next term is below 2^-57 relative), then scaled by 2^k.
//   log1p_unit(e), 0 <= e <= 1: log(1 + e) = 2 atanh(s) with s = e / (2 + e)
//     in [0, 1/3], atanh(s) = s (1 + z/3 + z^2/5 + ...), z = s^2 <= 1/9,
//     summed through z^17 / 35 (the next term is below 2^-56 relative).
// Both are plain host/device functions (no intrinsics) so that a host build
// can check them against the C library.
#pragma once

namespace adapm {

#ifndef ADAPM_HD
#define ADAPM_HD __host__ __device__
#endif

ADAPM_HD inline double exp_nonpos(double t) {
  if (t < -745.2) return 0.0;                         // below half the smallest subnormal
  constexpr double INV_LN2 = 1.4426950408889634;
  constexpr double LN2_HI = 0.6931471805598903;       // ln 2, low 11 mantissa bits cleared
  constexpr double LN2_LO = 5.497923018708371e-14;    // ln 2 - LN2_HI
  const double k = __builtin_rint(t * INV_LN2);
  const double r = __builtin_fma(-k, LN2_LO, __builtin_fma(-k, LN2_HI, t));
  double p = 1.6059043836821613e-10;                  // 1/13!
  p = __builtin_fma(p, r, 2.08767569878681e-09);      // 1/12!
  p = __builtin_fma(p, r, 2.505210838544172e-08);     // 1/11!
  p = __builtin_fma(p, r, 2.755731922398589e-07);     // 1/10!
  p = __builtin_fma(p, r, 2.7557319223985893e-06);    // 1/9!
  p = __builtin_fma(p, r, 2.48015873015873e-05);      // 1/8!
  p = __builtin_fma(p, r, 0.0001984126984126984);     // 1/7!
  p = __builtin_fma(p, r, 0.001388888888888889);      // 1/6!
  p = __builtin_fma(p, r, 0.008333333333333333);      // 1/5!
  p = __builtin_fma(p, r, 0.041666666666666664);      // 1/4!
  p = __builtin_fma(p, r, 0.16666666666666666);       // 1/3!
  p = __builtin_fma(p, r, 0.5);                       // 1/2!
  p = __builtin_fma(p, r, 1.0);
  p = __builtin_fma(p, r, 1.0);
  return __builtin_ldexp(p, (int)k);
}

ADAPM_HD inline double log1p_unit(double e) {
  const double s = e / (2.0 + e);
  const double z = s * s;
  double q = 0.02857142857142857;                     // 1/35
  q = __builtin_fma(q, z, 0.030303030303030304);      // 1/33
  q = __builtin_fma(q, z, 0.03225806451612903);       // 1/31
  q = __builtin_fma(q, z, 0.034482758620689655);      // 1/29
  q = __builtin_fma(q, z, 0.037037037037037035);      // 1/27
  q = __builtin_fma(q, z, 0.04);                      // 1/25
  q = __builtin_fma(q, z, 0.043478260869565216);      // 1/23
  q = __builtin_fma(q, z, 0.047619047619047616);      // 1/21
  q = __builtin_fma(q, z, 0.05263157894736842);       // 1/19
  q = __builtin_fma(q, z, 0.058823529411764705);      // 1/17
  q = __builtin_fma(q, z, 0.06666666666666667);       // 1/15
  q = __builtin_fma(q, z, 0.07692307692307693);       // 1/13
  q = __builtin_fma(q, z, 0.09090909090909091);       // 1/11
  q = __builtin_fma(q, z, 0.1111111111111111);        // 1/9
  q = __builtin_fma(q, z, 0.14285714285714285);       // 1/7
  q = __builtin_fma(q, z, 0.2);                       // 1/5
  q = __builtin_fma(q, z, 0.3333333333333333);        // 1/3
  q = __builtin_fma(q, z, 1.0);
  return 2.0 * s * q;
}

// sigmoid(x) = 1 / (1 + e^-x) and softplus(x) = log(1 + e^x) from one
// e = exp(-|x|): sigmoid = (x >= 0 ? 1 : e) / (1 + e), softplus =
// max(x, 0) + log(1 + e).
ADAPM_HD inline void sigmoid_softplus(double x, double* sig, double* sp) {
  const double e = exp_nonpos(-__builtin_fabs(x));
  *sig = (x >= 0.0 ? 1.0 : e) / (1.0 + e);
  const double l = log1p_unit(e);
  *sp = x > 0.0 ? x + l : l;
}

}  // namespace adapm
