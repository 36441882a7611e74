// mm_steps.hpp -- the two steps of one MM-MCN term (ScalingN, then Add-MCN into the
// accumulator) in the form the product kernels execute them, with the Simple-Renorm
// fast paths.  Shared by the sequential product (matmul.hip) and the K-split product
// (splitk.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "mcf_arith.hpp"

namespace mcf {

// ---------------------------------------------------------------------------------
// The two steps of one MM-MCN term, in the form the product kernel executes them.
//
// They compute exactly what scaling_n / add_mcn of mcf_arith.hpp compute on finite,
// non-overflowing data.  The shortcuts below change nothing but the sign of zero
// terms, and zero terms are all dropped by Simple-Renorm; the kernel writes every
// zero output component as +0, Simple-Renorm's padding, so the results are
// bit-identical:
//   * the first Two-Sum of each step adds the initial carry +0: Two-Sum(h, +0) =
//     (h + 0, +0), so h_0 is the first product (resp. sum) and the carry its error;
//   * Simple-Renorm of the nc+1 terms takes a fast path chosen by a policy (below);
//     lanes that miss it run the general compaction in a divergent block shared by
//     all the terms of a reduction step, so the arithmetic of the independent terms
//     stays in one straight-line block the compiler can interleave.
// ---------------------------------------------------------------------------------

// First R non-zero entries of v[0..M-1], in order; the remaining slots hold zeros
// of either sign.  Built back to front: after visiting v[i..M-1], out is the
// compaction of that suffix, and prepending a non-zero v[i] shifts it by one slot.
template <typename T, int M, int R>
__device__ __forceinline__ void compact_nz(const T (&v)[M], T (&out)[R]) {
  out[0] = v[M - 1];
#pragma unroll
  for (int r = 1; r < R; ++r) out[r] = T(0);
#pragma unroll
  for (int i = M - 2; i >= 0; --i) {
    const bool nz = v[i] != T(0);
    const int top = (M - 1 - i) < R - 1 ? (M - 1 - i) : R - 1;  // slots that can hold a value
#pragma unroll
    for (int r = top; r >= 1; --r) out[r] = nz ? out[r - 1] : out[r];
    out[0] = nz ? v[i] : out[0];
  }
}

// True when every one of v[0..K-1] is non-zero: min(|v_i|) != 0.  (A NaN is
// non-zero and min ignores it unless all are NaN, which is non-zero too.)
template <typename T, int K>
__device__ __forceinline__ bool all_nonzero(const T (&v)[K]) {
  static_assert(K >= 1 && K <= 4, "");
  if constexpr (K == 1) {
    return v[0] != T(0);
  } else if constexpr (sizeof(T) == 8) {  // binary64: a binary32 magnitude could underflow
    bool nz = true;
#pragma unroll
    for (int i = 0; i < K; ++i) nz = nz & (v[i] != T(0));
    return nz;
  } else if constexpr (K == 2) {
    return __builtin_fminf(__builtin_fabsf((float)v[0]), __builtin_fabsf((float)v[1])) != 0.0f;
  } else {
    T m = __builtin_fminf(__builtin_fminf(__builtin_fabsf((float)v[0]), __builtin_fabsf((float)v[1])),
                          __builtin_fabsf((float)v[2]));
    if constexpr (K == 4) return __builtin_fminf(m, __builtin_fabsf((float)v[3])) != 0.0f;
    return m != T(0);
  }
}

// Simple-Renorm fast paths for the nc+1 terms h of a step:
//   SR_FULL:   valid when h_0 .. h_{nc-1} are all non-zero: keep them; the dropped h_nc
//              is then never needed (binary32 data, where a zero term is rare);
//   SR_SELECT: valid when h_0 .. h_{nc-2} are non-zero: keep them and take the first
//              non-zero of h_{nc-1}, h_nc;
//   SR_HEAD:   valid when h_0 is non-zero: keep it and compact h_1 .. h_nc into the
//              other nc-1 slots without branching (binary16 data, where the low terms
//              of a step often fall below the subnormal grid);
//   SR_NET:    always valid: the general compaction without a branch.
// sr_try writes the fast-path result and returns true when the lane needs the general
// compaction instead.  `ok` marks lanes whose terms are known to be all zero: any
// fast-path result is then correct up to zero signs.
//   SR_SUFFIX: the kept-terms form below (scaling_kept / add_kept / kept_invalid); the
//              final carry is computed only by lanes that fail its test.
enum SrPolicy { SR_FULL = 0, SR_SELECT = 1, SR_HEAD = 2, SR_NET = 3, SR_SUFFIX = 4 };

template <typename T, int N, int POL>
__device__ __forceinline__ bool sr_try(const T (&h)[N + 1], T (&out)[N], bool ok = false) {
  if constexpr (N == 1 && POL == SR_FULL) {
    // keep h_0 when it is non-zero; the dropped h_1 is then never needed
    out[0] = h[0];
    return !(ok || h[0] != T(0));
  } else if constexpr (N == 1) {
    out[0] = (h[0] != T(0)) ? h[0] : h[1];
    return false;
  } else if constexpr (POL == SR_NET) {
    compact_nz<T, N + 1, N>(h, out);
    return false;
  } else if constexpr (POL == SR_HEAD) {
    out[0] = h[0];
    T tail_in[N], tail_out[N - 1];
#pragma unroll
    for (int i = 0; i < N; ++i) tail_in[i] = h[i + 1];
    compact_nz<T, N, N - 1>(tail_in, tail_out);
#pragma unroll
    for (int i = 1; i < N; ++i) out[i] = tail_out[i - 1];
    return !(ok || h[0] != T(0));
  } else {
    constexpr int NCHK = (POL == SR_FULL) ? N : N - 1;
    T lead[NCHK];
#pragma unroll
    for (int i = 0; i < NCHK; ++i) lead[i] = h[i];
#pragma unroll
    for (int i = 0; i < N - 1; ++i) out[i] = h[i];
    if constexpr (POL == SR_FULL)
      out[N - 1] = h[N - 1];
    else
      out[N - 1] = (h[N - 1] != T(0)) ? h[N - 1] : h[N];
    return !(ok || all_nonzero<T, NCHK>(lead));
  }
}

// The nc+1 terms of ScalingN(x, v) (before Simple-Renorm).
template <typename T, int N>
__device__ __forceinline__ void scaling_terms(const T (&x)[N], T v, T (&h)[N + 1]) {
  T e;
  two_prod(x[0], v, h[0], e);
#pragma unroll
  for (int i = 1; i < N; ++i) {
    T hp, e1, e2;
    two_prod(x[i], v, hp, e1);
    two_sum(hp, e, h[i], e2);
    e = e1 + e2;
  }
  h[N] = e;
}

// The nc+1 terms of Add-MCN(x, y) (before Simple-Renorm).
template <typename T, int N>
__device__ __forceinline__ void add_terms(const T (&x)[N], const T (&y)[N], T (&h)[N + 1]) {
  T e;
  two_sum(x[0], y[0], h[0], e);
#pragma unroll
  for (int i = 1; i < N; ++i) {
    T hp, e1, e2;
    two_sum(x[i], y[i], hp, e1);
    two_sum(hp, e, h[i], e2);
    e = e1 + e2;
  }
  h[N] = e;
}

// ---------------------------------------------------------------------------------
// Kept-terms form of a step (policy SR_SUFFIX, used for binary16).
//
// Simple-Renorm of the nc+1 terms h keeps h_0 .. h_{nc-1} unchanged (up to zero
// signs) exactly when
//   (a) the zero terms among h_0 .. h_{nc-1} form a suffix, and
//   (b) h_nc = 0 whenever one of them is zero.
// If h_{nc-1} = fl(hp + e) is zero, hp + e is exactly zero (a sum of two floats that
// is not zero is at least the smallest subnormal), so the last Two-Sum's error is
// zero and h_nc equals the error of the last component's own operation
// (fl(x_{nc-1} * v) for ScalingN, fl(x_{nc-1} + y_{nc-1}) for Add-MCN).  That error
// is zero when |hp| < 2^(emin+1): below that magnitude consecutive floats are one
// smallest subnormal apart, so a sum of two floats is exact and a product's error is
// at most half a subnormal spacing, which rounds to zero (a tie rounds to the even
// neighbour, zero).  The kernels therefore compute only the kept terms, test (a) and
// |hp| < 2^(emin+1), and run the general step for a lane that fails the test.
// ---------------------------------------------------------------------------------

// 2^(emin+1): below it the spacing of the format is its smallest subnormal.
template <typename T>
__device__ __forceinline__ constexpr double exact_limit();
template <>
__device__ __forceinline__ constexpr double exact_limit<_Float16>() {
  return 0x1p-13;
}
template <>
__device__ __forceinline__ constexpr double exact_limit<float>() {
  return 0x1p-125;
}
template <>
__device__ __forceinline__ constexpr double exact_limit<double>() {
  return 0x1p-1021;
}

// |x| < lim, compared in the component format (one compare with an abs modifier).
__device__ __forceinline__ bool abs_below(float x, float lim) { return __builtin_fabsf(x) < lim; }
__device__ __forceinline__ bool abs_below(_Float16 x, _Float16 lim) { return __builtin_fabsf16(x) < lim; }
__device__ __forceinline__ bool abs_below(double x, double lim) { return __builtin_fabs(x) < lim; }

// Magnitudes out of order: !(|b| <= |a|), true when |b| > |a| or either is a NaN (one
// compare with abs modifiers).
__device__ __forceinline__ bool out_of_order(float a, float b) { return !(__builtin_fabsf(b) <= __builtin_fabsf(a)); }
__device__ __forceinline__ bool out_of_order(_Float16 a, _Float16 b) {
  return !(__builtin_fabsf16(b) <= __builtin_fabsf16(a));
}
__device__ __forceinline__ bool out_of_order(double a, double b) { return !(__builtin_fabs(b) <= __builtin_fabs(a)); }

// h_0 .. h_{N-1} of ScalingN(x, v) and the last product hp = fl(x_{N-1} v).
// HEAD_EXACT: the error of x_0 v is known to be zero; TAIL_EXACT: so are the errors
// of x_i v, i >= 1 (both follow from |product| < exact_limit, established per tile).
// A carry known to be zero is not added (Two-Sum(hp, 0) = (hp, 0)).
template <typename T, int N, bool HEAD_EXACT, bool TAIL_EXACT>
__device__ __forceinline__ void scaling_kept(const T (&x)[N], T v, T (&h)[N], T &last) {
  h[0] = x[0] * v;
  last = h[0];
  if constexpr (N == 1) return;
  T e = HEAD_EXACT ? T(0) : fma_(x[0], v, -h[0]);
  bool carry_zero = HEAD_EXACT;
#pragma unroll
  for (int i = 1; i < N; ++i) {
    const T hp = x[i] * v;
    if (i == N - 1) {
      h[i] = carry_zero ? hp : hp + e;
      last = hp;
    } else if (carry_zero && TAIL_EXACT) {
      h[i] = hp;
    } else {
      T e2;
      two_sum(hp, e, h[i], e2);
      if constexpr (TAIL_EXACT) {
        e = e2;
      } else {
        e = fma_(x[i], v, -hp) + e2;
      }
      carry_zero = false;
    }
  }
}

// h_0 .. h_{N-1} of Add-MCN(x, y) and the last component sum hp = fl(x_{N-1} + y_{N-1}).
template <typename T, int N>
__device__ __forceinline__ void add_kept(const T (&x)[N], const T (&y)[N], T (&h)[N], T &last) {
  if constexpr (N == 1) {
    h[0] = x[0] + y[0];
    last = h[0];
  } else {
    T e;
    two_sum(x[0], y[0], h[0], e);
#pragma unroll
    for (int i = 1; i < N - 1; ++i) {
      T hp, e1, e2;
      two_sum(x[i], y[i], hp, e1);
      two_sum(hp, e, h[i], e2);
      e = e1 + e2;
    }
    last = x[N - 1] + y[N - 1];
    h[N - 1] = last + e;
  }
}

// Add-MCN(x, y) of two values whose component sums are all below exact_limit (the
// accumulators of the low components of B in an MC x MC product, whose products the
// tile flag shows to be below it): each sum x_i + y_i is then exact, every Two-Sum
// error and carry is zero, and the final carry is zero, so the terms are the N sums
// followed by zero.  Returns true when a lane may not meet that condition or when
// Simple-Renorm may move a term; such a lane runs the general step.  The test is the
// magnitude order of the sums (see kept_invalid) and |h_0| < exact_limit: sums in
// order are all at most |h_0|, so they are below the limit too.
template <typename T, int N>
__device__ __forceinline__ bool add_tiny(const T (&x)[N], const T (&y)[N], T (&h)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) h[i] = x[i] + y[i];
  bool bad = !abs_below(h[0], (T)exact_limit<T>());
#pragma unroll
  for (int i = 0; i + 1 < N; ++i) bad = bad | out_of_order(h[i], h[i + 1]);
  return bad;
}

// True when Simple-Renorm of the step's nc+1 terms could change h: a non-zero term
// follows a zero one, or a term is zero and the last operation may have been inexact
// (LAST_EXACT: known exact for the whole tile; else tested as |last| < exact_limit).
// ORDERED tests the first condition as magnitudes out of order, |h_{i+1}| > |h_i| for
// some i (or a NaN): a zero followed by a non-zero is out of order, so this flags a
// superset of those lanes with one compare per pair instead of three and a mask
// operation; the extra lanes run the general step, which gives the same result.  It
// suits ScalingN's terms, whose magnitudes decrease (a later term exceeds an earlier
// non-zero one only in the subnormal range), but not Add-MCN's: an accumulator's
// leading component passes near zero during a reduction while its second component
// still holds the errors gathered before, so there the zero pattern itself is tested.
// With N = 1 the single kept term is the result whenever it is non-zero, and when it
// is zero the dropped term is zero too (a zero product or sum is exact).
template <typename T, int N, bool LAST_EXACT, bool ORDERED = false>
__device__ __forceinline__ bool kept_invalid(const T (&h)[N], T last) {
  if constexpr (N == 1) {
    return false;
  } else {
    // bitwise operators, not short-circuit ones: the flags stay lane masks in
    // scalar registers instead of being materialized per lane
    bool z[N];
#pragma unroll
    for (int i = 0; i < N; ++i) z[i] = h[i] == T(0);
    bool bad = false;
#pragma unroll
    for (int i = 0; i + 1 < N; ++i) bad = bad | (ORDERED ? out_of_order(h[i], h[i + 1]) : (z[i] & !z[i + 1]));
    if constexpr (LAST_EXACT) return bad;
    return bad | (z[N - 1] & !abs_below(last, (T)exact_limit<T>()));
  }
}

// The same tests as wavefront lane masks (bit l for active lane l): the flags stay
// masks in scalar registers, combined there (a flag and the negation of another take
// one scalar and-not instead of a second compare), and the step that follows can
// branch once for the wavefront.  A lane whose kept terms are valid gets the same
// terms from the general step, so a wavefront may run the general step for all its
// lanes whenever one of them fails.
__device__ __forceinline__ uint64_t lane_mask(bool b) { return __builtin_amdgcn_ballot_w64(b); }

template <typename T, int N, bool LAST_EXACT, bool ORDERED = false>
__device__ __forceinline__ uint64_t kept_invalid_mask(const T (&h)[N], T last) {
  if constexpr (N == 1) {
    return 0;
  } else {
    uint64_t z[N];
#pragma unroll
    for (int i = 0; i < N; ++i) z[i] = lane_mask(h[i] == T(0));
    uint64_t bad = 0;
#pragma unroll
    for (int i = 0; i + 1 < N; ++i) bad |= ORDERED ? lane_mask(out_of_order(h[i], h[i + 1])) : (z[i] & ~z[i + 1]);
    if constexpr (LAST_EXACT) return bad;
    return bad | (z[N - 1] & lane_mask(!abs_below(last, (T)exact_limit<T>())));
  }
}

template <typename T, int N>
__device__ __forceinline__ uint64_t add_tiny_mask(const T (&x)[N], const T (&y)[N], T (&h)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) h[i] = x[i] + y[i];
  uint64_t bad = lane_mask(!abs_below(h[0], (T)exact_limit<T>()));
#pragma unroll
  for (int i = 0; i + 1 < N; ++i) bad |= lane_mask(out_of_order(h[i], h[i + 1]));
  return bad;
}

// ScalingN of (x, v) in kept-terms form into t; lanes failing the test run the
// general step (MASK: the whole wavefront runs it when one lane fails, see
// kept_invalid_mask).  HEAD / TAIL: the products' errors are known to be zero.
template <typename T, int N, bool HEAD, bool TAIL, bool MASK = false>
__device__ __forceinline__ void kept_scale(const T (&x)[N], T v, T (&t)[N]) {
  T last;
  scaling_kept<T, N, HEAD, TAIL>(x, v, t, last);
  bool bad;
  if constexpr (MASK)
    bad = kept_invalid_mask<T, N, TAIL, true>(t, last) != 0;
  else
    bad = kept_invalid<T, N, TAIL, true>(t, last);
  if (__builtin_expect(bad, 0)) {
    T h[N + 1];
    scaling_terms<T, N>(x, v, h);
    compact_nz<T, N + 1, N>(h, t);
  }
}

// a = Add-MCN(a, t) in kept-terms form (TINY: the add_tiny form; MASK as in
// kept_scale).
template <typename T, int N, bool TINY, bool MASK = false>
__device__ __forceinline__ void kept_add(T (&a)[N], const T (&t)[N]) {
  T s[N], last;
  bool bad;
  if constexpr (TINY) {
    bad = MASK ? add_tiny_mask<T, N>(a, t, s) != 0 : add_tiny<T, N>(a, t, s);
  } else {
    add_kept<T, N>(a, t, s, last);
    bad = MASK ? kept_invalid_mask<T, N, false>(s, last) != 0 : kept_invalid<T, N, false>(s, last);
  }
  if (__builtin_expect(bad, 0)) {
    T h[N + 1];
    add_terms<T, N>(a, t, h);
    compact_nz<T, N + 1, N>(h, s);
  }
#pragma unroll
  for (int c = 0; c < N; ++c) a[c] = s[c];
}

// The steps above elide the first Two-Sum of ScalingN with the +0 carry, which is
// exact for finite terms.  When a term is infinite or NaN that Two-Sum (and every one
// after it) leaves a NaN carry, so every later component of the algorithm's result is
// NaN; an Add-MCN that follows restores this by itself (its Two-Sums with a non-finite
// term have NaN errors), but a ScalingN result that is stored as it is -- the product
// of a single reduction step -- is patched here.
__device__ __forceinline__ bool finite_(float x) { return __builtin_isfinite(x); }
__device__ __forceinline__ bool finite_(double x) { return __builtin_isfinite(x); }
__device__ __forceinline__ bool finite_(_Float16 x) { return __builtin_isfinite((float)x); }

template <typename T, int N>
__device__ __forceinline__ void nonfinite_tail(T (&t)[N]) {
  bool nf = false;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i > 0) t[i] = nf ? T(__builtin_nanf("")) : t[i];
    nf = nf | !finite_(t[i]);
  }
}

// out = Add-MCN(x, y) for one value (the epilogue's combinations).
template <typename T, int N, int POL>
__device__ __forceinline__ void mm_add(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T h[N + 1];
  add_terms<T, N>(x, y, h);
  if (sr_try<T, N, POL>(h, out)) compact_nz<T, N + 1, N>(h, out);
}

}  // namespace mcf
