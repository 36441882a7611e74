// mcf_arith.hpp -- device-side multi-component floating-point arithmetic for gfx950.
//
// Each function below computes one algorithm of "MCTensor" (arXiv 2207.08867),
// Appendix A.2.1: every floating-point operation of the algorithm is one IEEE
// operation in the component type T (binary16 `_Float16`, binary32 `float` or
// binary64 `double`), with round to nearest even and gradual underflow, taken in the
// algorithm's order.  The library is compiled with -ffp-contract=off so no
// multiply-add is fused except the explicit FMA of Two-Prod.
//
// Components live in registers as small fixed-size arrays indexed by compile-time
// constants only (fully unrolled loops), so nothing spills to scratch memory.
#pragma once

#include <hip/hip_runtime.h>

namespace mcf {

template <typename T>
__device__ __forceinline__ T fma_(T a, T b, T c);
template <>
__device__ __forceinline__ float fma_<float>(float a, float b, float c) {
  return __builtin_fmaf(a, b, c);
}
template <>
__device__ __forceinline__ _Float16 fma_<_Float16>(_Float16 a, _Float16 b, _Float16 c) {
  return __builtin_fmaf16(a, b, c);
}
template <>
__device__ __forceinline__ double fma_<double>(double a, double b, double c) {
  return __builtin_fma(a, b, c);
}

// Correctly rounded component division.  binary32 and binary64: IEEE division (HIP's
// default division is correctly rounded).  binary16: the binary32 quotient of the exact
// binary16 operands, rounded to binary16; the double rounding is innocuous because
// 24 >= 2*11 + 2.
template <typename T>
__device__ __forceinline__ T div_(T a, T b);
template <>
__device__ __forceinline__ float div_<float>(float a, float b) {
  return a / b;
}
template <>
__device__ __forceinline__ _Float16 div_<_Float16>(_Float16 a, _Float16 b) {
  return (_Float16)((float)a / (float)b);
}
template <>
__device__ __forceinline__ double div_<double>(double a, double b) {
  return a / b;
}

// Knuth's error-free sum (Two-Sum, Appendix A.2.1): s = fl(a + b) together with the
// rounding error e = (a + b) - s, which is exactly representable.  With no ordering of
// |a| and |b| known, the error is recovered from the share of s that each operand
// accounts for: share_b = s - a, share_a = s - share_b; what rounding took from each
// operand is b - share_b and a - share_a, and their sum is the error.  The order of
// these six operations is part of the definition: it fixes the sign of a zero error.
template <typename T>
__device__ __forceinline__ void two_sum(T a, T b, T &s, T &e) {
  const T sum = a + b;
  const T share_b = sum - a;
  const T share_a = sum - share_b;
  const T lost_b = b - share_b;
  const T lost_a = a - share_a;
  s = sum;
  e = lost_a + lost_b;
}

// Two-Prod, FMA variant: p = fl(a * b), e = fl(a * b - p) with a single rounding.
template <typename T>
__device__ __forceinline__ void two_prod(T a, T b, T &p, T &e) {
  p = a * b;
  e = fma_(a, b, -p);
}

// Stable compaction: out[0..R-1] = the first R entries of v[0..M-1] whose flag is
// set, in order, +0 where fewer than R are flagged.  Built back to front: after
// visiting v[i..M-1], out holds the compaction of that suffix; prepending v[i]
// shifts it by one slot (the compaction of a suffix is a prefix-stable list).
template <typename T, int M, int R>
__device__ __forceinline__ void compact(const T (&v)[M], const bool (&keep)[M], T (&out)[R]) {
#pragma unroll
  for (int r = 0; r < R; ++r) out[r] = T(0);
#pragma unroll
  for (int i = M - 1; i >= 0; --i) {
#pragma unroll
    for (int r = R - 1; r >= 1; --r) out[r] = keep[i] ? out[r - 1] : out[r];
    out[0] = keep[i] ? v[i] : out[0];
  }
}

// Simple-Renorm: the first R non-zero components, in order, +0 padded.  Every one
// of the M inputs is scanned (the prose: all non-zero values are extracted).
template <typename T, int M, int R>
__device__ __forceinline__ void simple_renorm(const T (&h)[M], T (&b)[R]) {
  bool nz[M];
#pragma unroll
  for (int i = 0; i < M; ++i) nz[i] = (h[i] != T(0));
  compact<T, M, R>(h, nz, b);
}

// Renormalize (Priest variant).  First sweep s = x_0, (s, t_i) = Two-Sum(x_i, s) for
// the components that exist; t_0 = 0.  Second sweep (s, e) = Two-Sum(s, t_i),
// emitting s when e != 0 and continuing with e.  The s left at the end is emitted as
// well.  The first R emitted values are returned, +0 padded.
template <typename T, int N, int R>
__device__ __forceinline__ void renormalize(const T (&x)[N], T (&b)[R]) {
  T t[N];
  T s = x[0];
  t[0] = T(0);
#pragma unroll
  for (int i = 1; i < N; ++i) two_sum(x[i], s, s, t[i]);
  T cand[N + 1];
  bool emit[N + 1];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    T sn, e;
    two_sum(s, t[i], sn, e);
    emit[i] = (e != T(0));
    cand[i] = sn;
    s = emit[i] ? e : sn;
  }
  cand[N] = s;
  emit[N] = true;
  compact<T, N + 1, R>(cand, emit, b);
}

// Grow-ExpN: an N-component value plus a plain value v.
template <typename T, int N>
__device__ __forceinline__ void grow_expn(const T (&x)[N], T v, T (&out)[N]) {
  T h[N + 1];
  T Q = v;
#pragma unroll
  for (int k = N; k >= 1; --k) two_sum(x[k - 1], Q, Q, h[k]);
  h[0] = Q;
  simple_renorm<T, N + 1, N>(h, out);
}

// ScalingN: an M-component value times a plain value v; R = M (expand off) or M+1.
// The first Two-Sum adds the initial carry +0: Two-Sum(hp, +0) = (hp + 0, e2) with
// e2 = +0 for finite hp and NaN for infinite or NaN hp (its hp - hp step), so h_0 = hp
// up to the sign of a zero (Simple-Renorm drops zeros) and the carry e1 + e2 is
// e1 + (hp - hp): two operations in place of the Two-Sum, the same value in every
// case -- a product that overflows although both factors are finite leaves a NaN
// carry, not the infinite Two-Prod error.
template <typename T, int M, int R>
__device__ __forceinline__ void scaling_n(const T (&x)[M], T v, T (&out)[R]) {
  T h[M + 1];
  T e;
  two_prod(x[0], v, h[0], e);
  e = e + (h[0] - h[0]);
#pragma unroll
  for (int i = 1; i < M; ++i) {
    T hp, e1, e2;
    two_prod(x[i], v, hp, e1);
    two_sum(hp, e, h[i], e2);
    e = e1 + e2;
  }
  h[M] = e;
  simple_renorm<T, M + 1, R>(h, out);
}

// Add-MCN: sum of two N-component values.  The first Two-Sum with the +0 carry is
// elided: its error would be NaN only for infinite or NaN hp, and then the Two-Sum
// error e1 that forms hp is NaN already.
template <typename T, int N>
__device__ __forceinline__ void add_mcn(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T h[N + 1];
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
  simple_renorm<T, N + 1, N>(h, out);
}

// Div-MCN: long division with N+1 quotient digits.
template <typename T, int N>
__device__ __forceinline__ void div_mcn(const T (&x_in)[N], const T (&y)[N], T (&out)[N]) {
  T x[N];
#pragma unroll
  for (int c = 0; c < N; ++c) x[c] = x_in[c];
  T h[N + 1];
  T q = div_(x[0], y[0]);
  h[0] = q;
#pragma unroll
  for (int i = 1; i <= N; ++i) {
    T s[N], neg[N];
    scaling_n<T, N, N>(y, q, s);
#pragma unroll
    for (int c = 0; c < N; ++c) neg[c] = -s[c];
    add_mcn<T, N>(x, neg, x);
    q = div_(x[0], y[0]);
    h[i] = q;
  }
  simple_renorm<T, N + 1, N>(h, out);
}

// Mult-MCN, fast version: x / (1 / y), each quotient renormalized.
template <typename T, int N>
__device__ __forceinline__ void mult_mcn(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T one[N], q[N], yinv[N];
  one[0] = T(1);
#pragma unroll
  for (int c = 1; c < N; ++c) one[c] = T(0);
  div_mcn<T, N>(one, y, q);
  renormalize<T, N, N>(q, yinv);
  div_mcn<T, N>(x, yinv, q);
  renormalize<T, N, N>(q, out);
}

// Mult-MCN-Slow: product digits by repeated division.  p = fl(x_0 y_0) is the first
// digit; N times the remainder x = Add-MCN(x, -DivN(p, y)) is formed and its next
// digit p = fl(x_0 y_0) taken; the N+1 digits pass through Simple-Renorm.
template <typename T, int N>
__device__ __forceinline__ void mult_mcn_slow(const T (&x_in)[N], const T (&y)[N], T (&out)[N]) {
  T x[N];
#pragma unroll
  for (int c = 0; c < N; ++c) x[c] = x_in[c];
  T h[N + 1];
  T p = x[0] * y[0];
  h[0] = p;
#pragma unroll
  for (int i = 1; i <= N; ++i) {
    T pv[N], d[N], neg[N];
    pv[0] = p;
#pragma unroll
    for (int c = 1; c < N; ++c) pv[c] = T(0);
    div_mcn<T, N>(pv, y, d);  // DivN(p, y): the plain dividend padded with zeros
#pragma unroll
    for (int c = 0; c < N; ++c) neg[c] = -d[c];
    add_mcn<T, N>(x, neg, x);
    p = x[0] * y[0];
    h[i] = p;
  }
  simple_renorm<T, N + 1, N>(h, out);
}

// Square-MCN.  The printed first step fl(2^(x_0)) is read as fl(x_0 x_0), the
// square's leading term: h = (fl(x_0 x_0), 0, ..., 0), then h = Grow-ExpN(h,
// fl(2 x_0 x_1)) (2 x_0 is exact, so the addend is one rounding of the product).
// With N = 1 there is no x_1 and the addend is zero.
template <typename T, int N>
__device__ __forceinline__ void square_mcn(const T (&x)[N], T (&out)[N]) {
  T h[N];
  h[0] = x[0] * x[0];
#pragma unroll
  for (int c = 1; c < N; ++c) h[c] = T(0);
  T v = T(0);
  if constexpr (N > 1) v = (T(2) * x[0]) * x[1];
  grow_expn<T, N>(h, v, out);
}

}  // namespace mcf
