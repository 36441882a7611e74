// div_steps.hpp -- Div-MCN and Mult-MCN (A.2.1) as the elementwise kernels run them.
//
// They return exactly what div_mcn / mult_mcn of mcf_arith.hpp return, bit for bit,
// with two shortcuts:
//   * each ScalingN(y, q) takes the kept-terms form of mm_steps.hpp (the nc terms
//     Simple-Renorm keeps, no final carry, and a per-lane test that Simple-Renorm
//     would not change them; failing lanes compute the full terms and compact them).
//     A zero term of either sign may then reach the next Add-MCN where the literal
//     step has +0; that only changes zero signs of that Add-MCN's Two-Sum errors,
//     which Simple-Renorm drops, and its outputs are the same;
//   * the last quotient digit q_nc is computed only by lanes where one of the digits
//     q_0 .. q_{nc-1} is zero.  Simple-Renorm of the nc+1 digits keeps the first nc
//     non-zero ones, so when those are all non-zero q_nc is never used.
// Measured on 2^26 elements at nc = 3 against the literal algorithm: binary16 Div-MCN
// 514 -> 426 us and Mult-MCN 986 -> 824 us; binary32 562 -> 425 and 1112 -> 697 us.
// The Add-MCN steps stay literal: x - y q cancels the leading component, so their
// terms usually start with a zero and need the compaction.
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
    add_mcn<T, N>(x, neg, x);
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
    add_mcn<T, N>(x, neg, x);
    p = x[0] * y[0];
    h[i] = p;
  }
  simple_renorm<T, N + 1, N>(h, out);
}

}  // namespace mcf
