// div_steps.hpp -- Div-MCN and Mult-MCN (A.2.1) as the elementwise kernels run them.
//
// They return exactly what div_mcn / mult_mcn of mcf_arith.hpp return, bit for bit,
// with three shortcuts:
//   * each ScalingN(y, q) takes the kept-terms form of mm_steps.hpp (the nc terms
//     Simple-Renorm keeps, no final carry, and a per-lane test that Simple-Renorm
//     would not change them; failing lanes compute the full terms and compact them).
//     A zero term of either sign may then reach the next Add-MCN where the literal
//     step has +0; that only changes zero signs of that Add-MCN's Two-Sum errors,
//     which Simple-Renorm drops, and its outputs are the same;
//   * the last quotient digit q_nc is computed only by lanes where one of the digits
//     q_0 .. q_{nc-1} is zero.  Simple-Renorm of the nc+1 digits keeps the first nc
//     non-zero ones, so when those are all non-zero q_nc is never used;
//   * the remainder updates x - y q compact their terms by a shift (add_mcn_shift).
// Measured on 2^26 elements at nc = 3 against the literal algorithm: binary16 Div-MCN
// 514 -> 426 us and Mult-MCN 986 -> 824 us; binary32 562 -> 425 and 1112 -> 697 us.
// The remainder updates x - y q cancel the leading component, so their terms usually
// start with a zero and trail off in zeros; the shift compaction covers those
// patterns (a simulation of the binary16 nc = 3 workload found no other pattern in
// more than 99.99% of the updates).
#pragma once

#include "mcf_arith.hpp"
#include "mm_steps.hpp"

namespace mcf {

// ScalingN(y, q) with expand off, kept-terms form.
template <typename T, int N>
__device__ __forceinline__ void scaling_n_kept(const T (&y)[N], T q, T (&out)[N]) {
  T last;
  scaling_kept<T, N, false, false>(y, q, out, last);
  if (kept_invalid<T, N, false, true>(out, last)) {
    T h[N + 1];
    scaling_terms<T, N>(y, q, h);
    compact_nz<T, N + 1, N>(h, out);
  }
}

// Add-MCN(x, y) for the remainder updates x - y q, whose leading term usually cancels
// to zero and whose last terms are often zero (binary16).  Simple-Renorm of the nc+1
// terms is a shift by one slot when h_0 is zero and the identity otherwise, provided
// no zero precedes a non-zero among h_1 .. h_nc; lanes where one does take the
// general compaction.  (A zero output component may differ from the literal step in
// sign only; Div-MCN's zero remainders only ever yield zero quotient digits, which
// Simple-Renorm drops.)
template <typename T, int N>
__device__ __forceinline__ void add_mcn_shift(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T h[N + 1];
  add_terms<T, N>(x, y, h);
  bool z[N + 1];
#pragma unroll
  for (int i = 0; i <= N; ++i) z[i] = h[i] == T(0);
  bool bad = false;
#pragma unroll
  for (int i = 1; i < N; ++i) bad = bad | (z[i] & !z[i + 1]);
  if (__builtin_expect(bad, 0)) {
    compact_nz<T, N + 1, N>(h, out);
    return;
  }
#pragma unroll
  for (int i = 0; i < N; ++i) out[i] = z[0] ? h[i + 1] : h[i];
}

template <typename T, int N>
__device__ __forceinline__ void div_mcn_fast(const T (&x_in)[N], const T (&y)[N], T (&out)[N]) {
  T x[N];
#pragma unroll
  for (int c = 0; c < N; ++c) x[c] = x_in[c];
  T h[N + 1];
  T q = div_(x[0], y[0]);
  h[0] = q;
#pragma unroll
  for (int i = 1; i <= N; ++i) {
    if (i == N) {
      bool all = true;
#pragma unroll
      for (int c = 0; c < N; ++c) all = all & (h[c] != T(0));
      if (all) {
#pragma unroll
        for (int c = 0; c < N; ++c) out[c] = h[c];
        return;
      }
    }
    T s[N], neg[N];
    scaling_n_kept<T, N>(y, q, s);
#pragma unroll
    for (int c = 0; c < N; ++c) neg[c] = -s[c];
    add_mcn_shift<T, N>(x, neg, x);
    q = div_(x[0], y[0]);
    h[i] = q;
  }
  simple_renorm<T, N + 1, N>(h, out);
}

// Mult-MCN, fast version: Renormalize(Div-MCN(x, Renormalize(Div-MCN(1, y)))).
template <typename T, int N>
__device__ __forceinline__ void mult_mcn_fast(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T one[N], q[N], yinv[N];
  one[0] = T(1);
#pragma unroll
  for (int c = 1; c < N; ++c) one[c] = T(0);
  div_mcn_fast<T, N>(one, y, q);
  renormalize<T, N, N>(q, yinv);
  div_mcn_fast<T, N>(x, yinv, q);
  renormalize<T, N, N>(q, out);
}

// Mult-MCN-Slow (mcf_arith.hpp: mult_mcn_slow) with its DivN steps taken by
// div_mcn_fast: the same bits.
template <typename T, int N>
__device__ __forceinline__ void mult_mcn_slow_fast(const T (&x_in)[N], const T (&y)[N], T (&out)[N]) {
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
    div_mcn_fast<T, N>(pv, y, d);
#pragma unroll
    for (int c = 0; c < N; ++c) neg[c] = -d[c];
    add_mcn_shift<T, N>(x, neg, x);
    p = x[0] * y[0];
    h[i] = p;
  }
  simple_renorm<T, N + 1, N>(h, out);
}

}  // namespace mcf
