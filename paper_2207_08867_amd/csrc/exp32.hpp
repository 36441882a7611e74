// exp32.hpp -- correctly rounded binary32 exponential on gfx950, the component
// exponential of Exp-MCN for binary32 components.
//
// Fast path: e^x evaluated in binary64 by HIP's exp (a few binary64 ulps of error)
// and rounded to binary32, accepted when a relative margin of 2^-48 on either side
// of it rounds to the same binary32 value -- the true e^x then rounds to that value
// too.  The few inputs whose e^x lies closer than that to a binary32 rounding
// boundary take a double-double evaluation (relative error below 2^-95), rounded to
// binary32 from the pair.
//
// Double-double arithmetic follows the error-free sums and products of Dekker
// (1971) and Knuth; the exponential uses e^x = 2^k e^r with k = rint(x / ln 2),
// r = x - k ln 2 taken with a three-part ln 2 (the first two parts have 44
// significant bits, so their products with |k| < 256 are exact), and e^r by its
// Taylor series to degree 24 (|r| < 0.35: the tail is below 2^-120).
#pragma once

#include <hip/hip_runtime.h>

namespace mcf {

struct DD {
  double hi, lo;
};

__device__ __forceinline__ DD dd_sum(double a, double b) {  // exact: a + b = hi + lo
  const double s = a + b;
  const double bv = s - a;
  const double av = s - bv;
  return {s, (a - av) + (b - bv)};
}

__device__ __forceinline__ DD dd_fast_sum(double a, double b) {  // exact when |a| >= |b|
  const double s = a + b;
  return {s, b - (s - a)};
}

__device__ __forceinline__ DD dd_add(DD x, DD y) {
  DD s = dd_sum(x.hi, y.hi);
  const DD t = dd_sum(x.lo, y.lo);
  s = dd_fast_sum(s.hi, s.lo + t.hi);
  return dd_fast_sum(s.hi, s.lo + t.lo);
}

__device__ __forceinline__ DD dd_mul(DD x, DD y) {
  const double p = x.hi * y.hi;
  double e = __builtin_fma(x.hi, y.hi, -p);  // exact error of p
  e = e + (x.hi * y.lo + x.lo * y.hi);
  return dd_fast_sum(p, e);
}

// x / n for a small positive integer n.
__device__ __forceinline__ DD dd_div_small(DD x, double n) {
  const double q = x.hi / n;
  const double r = __builtin_fma(-q, n, x.hi) + x.lo;  // fma: x.hi - q n exactly
  return dd_fast_sum(q, r / n);
}

// e^x as a double-double, for finite x with |x| < 128 (binary32 arguments whose
// exponential is neither 0 nor infinite after rounding).
__device__ __noinline__ DD exp_dd(double x) {
  // ln 2 = LN2_A + LN2_B + LN2_C (LN2_A, LN2_B: 44 significant bits)
  constexpr double LN2_A = 0x1.62e42fefa3800p-1;
  constexpr double LN2_B = 0x1.ef35793c76600p-45;
  constexpr double LN2_C = 0x1.3007e5ed5e81ep-89;
  constexpr double INV_LN2 = 0x1.71547652b82fep+0;
  const double k = __builtin_rint(x * INV_LN2);
  DD r = dd_sum(x, -(k * LN2_A));
  r = dd_add(r, DD{-(k * LN2_B), 0.0});
  r = dd_add(r, DD{-(k * LN2_C), 0.0});
  DD p = {1.0, 0.0};
  for (int n = 24; n >= 1; --n) p = dd_add(DD{1.0, 0.0}, dd_div_small(dd_mul(r, p), (double)n));
  const int ki = (int)k;
  return {__builtin_ldexp(p.hi, ki), __builtin_ldexp(p.lo, ki)};
}

// Round hi + lo (|lo| at most half an ulp of hi, hi > 0) to binary32, to nearest even.
__device__ __forceinline__ float dd_round_f32(DD v) {
  const float f = (float)v.hi;
  const double fd = __builtin_isinf(f) ? 0x1p128 : (double)f;  // infinity stands for 2^128 here
  const double d = v.hi - fd;
  if (d == 0.0) return f;  // hi is a binary32 value; |lo| cannot reach a rounding boundary
  unsigned bits = __builtin_bit_cast(unsigned, f);
  bits = d > 0 ? bits + 1u : bits - 1u;  // the binary32 neighbour on the side of hi
  const float g = __builtin_bit_cast(float, bits);
  const double mid = 0.5 * (fd + (double)g);  // exact
  if (v.hi != mid) return f;                  // hi + lo stays on f's side of the boundary
  if (v.lo == 0.0) return f;                  // an exact tie: (float)hi already rounded to even
  return ((v.lo > 0.0) == (d > 0.0)) ? g : f;
}

// Correctly rounded binary32 e^x.
__device__ __forceinline__ float exp32_cr(float x) {
  const double y = exp((double)x);
  const float a = (float)(y * (1.0 - 0x1p-48));
  const float b = (float)(y * (1.0 + 0x1p-48));
  if (__builtin_expect(a == b, 1)) return a;
  if (x != x) return x + x;  // NaN
  return dd_round_f32(exp_dd((double)x));
}

}  // namespace mcf
