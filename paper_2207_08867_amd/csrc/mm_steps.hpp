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
enum SrPolicy { SR_FULL = 0, SR_SELECT = 1, SR_HEAD = 2, SR_NET = 3 };

template <typename T, int N, int POL>
__device__ __forceinline__ bool sr_try(const T (&h)[N + 1], T (&out)[N], bool ok = false) {
  if constexpr (N == 1) {
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

// out = Add-MCN(x, y) for one value (the epilogue's combinations).
template <typename T, int N, int POL>
__device__ __forceinline__ void mm_add(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
  T h[N + 1];
  add_terms<T, N>(x, y, h);
  if (sr_try<T, N, POL>(h, out)) compact_nz<T, N + 1, N>(h, out);
}

}  // namespace mcf
