// scaled.hip -- binary16 components with scaled low components (format MCF_F16S) on
// gfx950: elementwise Add-MCN and ScalingN, the MC matrix product and MC-Linear.
//
// The format reads the paper's remark that scaling the smaller components by a factor
// 2^-k captures errors below binary16's smallest subnormal (Section 2.4): component c
// is a binary16 number y_c standing for 2^(-11 c) y_c.  The algorithms are the paper's,
// with every quantity at a level and every rounding taken in the binary16 format of
// that level.  On the device a level-l quantity is held scaled by 2^(11 l), so:
//   * an operation whose operands share a level is one native binary16 operation on
//     the scaled values (scaling by a power of two commutes with the rounding), and a
//     product of a level-a by a level-b value is, scaled, at level a + b;
//   * the error of a level-l Two-Sum is exact at level l and moves to level l + 1 by
//     an exact multiplication by 2^11;
//   * the error of a level-l Two-Prod, a b - p, is exact in binary32 (a product of two
//     binary16 values and its distance to the rounded product both fit), and is scaled
//     by 2^11 and rounded once into level l + 1;
//   * a value that Simple-Renorm moves d slots forward is rescaled by 2^(-11 d) in
//     binary32 (exact) and rounded once into its new level.
// Step functions run the common case (every kept term non-zero: Simple-Renorm returns
// the kept terms unchanged and drops the final carry, so the carry is not formed) and
// report whether it applied; otherwise the lane runs the complete algorithm with the
// general compaction.  Both give the algorithm's result.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_arith.hpp"
#include "mcf_internal.hpp"

namespace mcf {
namespace {

using h16 = _Float16;

// Moves a level-l error to level l + 1 (exact: a power of two, and an error never
// exceeds the value it belongs to).
__device__ __forceinline__ h16 up1(h16 v) { return v * (h16)2048.0f; }

// Two-Prod (FMA variant) of two scaled values: p at the product's level, e at the next.
__device__ __forceinline__ void sc_two_prod(h16 a, h16 b, h16 &p, h16 &e) {
  p = a * b;
  const float r = __builtin_fmaf((float)a, (float)b, -(float)p);
  e = (h16)(r * 2048.0f);
}

// v moved d slots forward: rounded once into the level d above its own.
__device__ __forceinline__ h16 move_up(h16 v, int d) {
  if (d == 0) return v;
  const float s = d == 1 ? 0x1p-11f : (d == 2 ? 0x1p-22f : (d == 3 ? 0x1p-33f : 0x1p-44f));
  return (h16)((float)v * s);
}

// Simple-Renorm of h[0..MH-1] (h[k] at level k relative to the result) into R slots:
// the first R non-zero values in order, the one landing in slot j rounded into level
// j; +0 in the remaining slots.
template <int MH, int R>
__device__ __forceinline__ void sc_compact(const h16 (&h)[MH], h16 (&out)[R]) {
#pragma unroll
  for (int r = 0; r < R; ++r) out[r] = (h16)0.0f;
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < MH; ++k) {
    const bool nz = h[k] != (h16)0.0f;
#pragma unroll
    for (int j = 0; j < R && j <= k; ++j)
      if (nz && cnt == j) out[j] = move_up(h[k], k - j);
    cnt += nz ? 1 : 0;
  }
}

template <int M>
__device__ __forceinline__ bool all_nz(const h16 (&h)[M]) {
  bool ok = true;
#pragma unroll
  for (int i = 0; i < M; ++i) ok = ok & (h[i] != (h16)0.0f);
  return ok;
}

// ScalingN without expand of x (M components) by v, complete: M + 1 terms, the
// carry built at each next level, general Simple-Renorm.
template <int M>
__device__ __forceinline__ void sc_scaling_general(const h16 (&x)[M], h16 v, h16 (&out)[M]) {
  h16 h[M + 1];
  h16 e = (h16)0.0f;
#pragma unroll
  for (int i = 0; i < M; ++i) {
    h16 p, e1, e2;
    sc_two_prod(x[i], v, p, e1);
    two_sum(p, e, h[i], e2);
    e = e1 + up1(e2);
  }
  h[M] = e;
  sc_compact<M + 1, M>(h, out);
}

// ScalingN, kept terms only; false when a kept term is zero (the caller then runs the
// complete algorithm).  The Two-Sum of the first product p with the zero carry only
// changes the sign of a zero for finite p, and its error is NaN for infinite or NaN p:
// the carry is e1 + (p - p) in every case.
template <int M>
__device__ __forceinline__ bool sc_scaling_fast(const h16 (&x)[M], h16 v, h16 (&h)[M]) {
  h16 e;
  {
    h16 p, e1;
    sc_two_prod(x[0], v, p, e1);
    h[0] = p;
    e = e1 + (p - p);
  }
#pragma unroll
  for (int i = 1; i < M - 1; ++i) {
    h16 p, e1, e2;
    sc_two_prod(x[i], v, p, e1);
    two_sum(p, e, h[i], e2);
    e = e1 + up1(e2);
  }
  if constexpr (M >= 2) h[M - 1] = x[M - 1] * v + e;
  return all_nz(h);
}

template <int M>
__device__ __forceinline__ void sc_scaling(const h16 (&x)[M], h16 v, h16 (&out)[M]) {
  if (!sc_scaling_fast<M>(x, v, out)) sc_scaling_general<M>(x, v, out);
}

// Add-MCN of x and y (M components each, same levels), complete.
template <int M>
__device__ __forceinline__ void sc_add_general(const h16 (&x)[M], const h16 (&y)[M], h16 (&out)[M]) {
  h16 h[M + 1];
  h16 e = (h16)0.0f;
#pragma unroll
  for (int i = 0; i < M; ++i) {
    h16 hp, e1, e2;
    two_sum(x[i], y[i], hp, e1);
    two_sum(hp, e, h[i], e2);
    e = up1(e1) + up1(e2);
  }
  h[M] = e;
  sc_compact<M + 1, M>(h, out);
}

// Add-MCN, kept terms only (see sc_scaling_fast).
template <int M>
__device__ __forceinline__ bool sc_add_fast(const h16 (&x)[M], const h16 (&y)[M], h16 (&h)[M]) {
  h16 e;
  {
    h16 e1;
    two_sum(x[0], y[0], h[0], e1);
    e = up1(e1);
  }
#pragma unroll
  for (int i = 1; i < M - 1; ++i) {
    h16 hp, e1, e2;
    two_sum(x[i], y[i], hp, e1);
    two_sum(hp, e, h[i], e2);
    e = up1(e1) + up1(e2);
  }
  if constexpr (M >= 2) h[M - 1] = (x[M - 1] + y[M - 1]) + e;
  return all_nz(h);
}

template <int M>
__device__ __forceinline__ void sc_add(const h16 (&x)[M], const h16 (&y)[M], h16 (&out)[M]) {
  h16 t[M];
  if (sc_add_fast<M>(x, y, t)) {
#pragma unroll
    for (int i = 0; i < M; ++i) out[i] = t[i];
  } else {
    sc_add_general<M>(x, y, out);
  }
}

// ---------------------------------------------------------------------------------
// Elementwise kernels
// ---------------------------------------------------------------------------------

constexpr int SC_THREADS = 256;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct Pack8 {
  h16 v[8];
};

__device__ __forceinline__ Pack8 load8(const h16 *p) {
  Pack8 r;
  u32x4 raw = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
  __builtin_memcpy(&r, &raw, 16);
  return r;
}

__device__ __forceinline__ void store8(h16 *p, const Pack8 &r) {
  u32x4 raw;
  __builtin_memcpy(&raw, &r, 16);
  __builtin_nontemporal_store(raw, reinterpret_cast<u32x4 *>(p));
}

// One element: OP 0 = Add-MCN (both MC), OP 1 = ScalingN (x MC, y plain after the
// launcher puts the MC operand first).
template <int NC, int OP>
__device__ __forceinline__ void sc_elem(const h16 (&a)[NC], const h16 (&b)[NC], h16 (&r)[NC]) {
  if constexpr (OP == 0)
    sc_add<NC>(a, b, r);
  else
    sc_scaling<NC>(a, b[0], r);
}

template <int NC, int OP, int NY, int W>
__global__ __launch_bounds__(SC_THREADS) void sc_ew_kernel(const h16 *__restrict__ x, const h16 *__restrict__ y,
                                                         h16 *__restrict__ out, int64_t n) {
  const int64_t nchunk = n / W;
  const int64_t stride = (int64_t)gridDim.x * SC_THREADS;
  for (int64_t ch = (int64_t)blockIdx.x * SC_THREADS + threadIdx.x; ch < nchunk; ch += stride) {
    const int64_t e0 = ch * W;
    h16 xa[NC][W], ya[NY][W];
    if constexpr (W == 8) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const Pack8 p = load8(x + c * n + e0);
#pragma unroll
        for (int w = 0; w < W; ++w) xa[c][w] = p.v[w];
      }
#pragma unroll
      for (int c = 0; c < NY; ++c) {
        const Pack8 p = load8(y + c * n + e0);
#pragma unroll
        for (int w = 0; w < W; ++w) ya[c][w] = p.v[w];
      }
    } else {
#pragma unroll
      for (int c = 0; c < NC; ++c) xa[c][0] = x[c * n + e0];
#pragma unroll
      for (int c = 0; c < NY; ++c) ya[c][0] = y[c * n + e0];
    }
    h16 ra[NC][W];
#pragma unroll
    for (int w = 0; w < W; ++w) {
      h16 a[NC], b[NC], r[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        a[c] = xa[c][w];
        b[c] = c < NY ? ya[c][w] : (h16)0.0f;
      }
      sc_elem<NC, OP>(a, b, r);
#pragma unroll
      for (int c = 0; c < NC; ++c) ra[c][w] = r[c];
    }
    if constexpr (W == 8) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        Pack8 p;
#pragma unroll
        for (int w = 0; w < W; ++w) p.v[w] = ra[c][w];
        store8(out + c * n + e0, p);
      }
    } else {
#pragma unroll
      for (int c = 0; c < NC; ++c) out[c * n + e0] = ra[c][0];
    }
  }
}

template <int NC, int OP, int NY>
hipError_t sc_ew_launch(int64_t n, const void *x, const void *y, void *out, hipStream_t s) {
  const bool vec = (n % 8 == 0) && ((uintptr_t)x % 16 == 0) && ((uintptr_t)y % 16 == 0) && ((uintptr_t)out % 16 == 0);
  const int64_t work = vec ? n / 8 : n;
  int64_t blocks = (work + SC_THREADS - 1) / SC_THREADS;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  if (vec)
    hipLaunchKernelGGL((sc_ew_kernel<NC, OP, NY, 8>), dim3((unsigned)blocks), dim3(SC_THREADS), 0, s,
                       (const h16 *)x, (const h16 *)y, (h16 *)out, n);
  else
    hipLaunchKernelGGL((sc_ew_kernel<NC, OP, NY, 1>), dim3((unsigned)blocks), dim3(SC_THREADS), 0, s,
                       (const h16 *)x, (const h16 *)y, (h16 *)out, n);
  return hipGetLastError();
}

template <int NC>
hipError_t sc_ew_nc(int op, int64_t n, const void *x, const void *y, void *out, hipStream_t s) {
  if (op == EW_ADD) return sc_ew_launch<NC, 0, NC>(n, x, y, out, s);
  return sc_ew_launch<NC, 1, 1>(n, x, y, out, s);
}

// ---------------------------------------------------------------------------------
// Matrix product and MC-Linear
// ---------------------------------------------------------------------------------

constexpr int SC_BM = 16, SC_BN = 16, SC_KT = 32;

// The accumulators of one output: part p (p = 0 for one MC operand; p = 0 .. NC-1 for
// MC x MC) holds NC - p components at levels p .. NC-1.  Fixed arrays of NC entries;
// part p uses the first NC - p.
template <int NC, int NP>
struct ScAcc {
  h16 v[NP][NC];
};

// Reduction step of part P: ScalingN of the MC factor's first M = NC - P components by
// the plain factor, then Add-MCN into the accumulator (the first step initialises it).
template <int NC, int P>
__device__ __forceinline__ void sc_part_step(h16 (&acc)[NC], const h16 (&mc)[NC], h16 v, bool first) {
  constexpr int M = NC - P;
  h16 x[M], t[M];
#pragma unroll
  for (int i = 0; i < M; ++i) x[i] = mc[i];
  sc_scaling<M>(x, v, t);
  if (first) {
#pragma unroll
    for (int i = 0; i < M; ++i) acc[i] = t[i];
  } else {
    h16 a[M], r[M];
#pragma unroll
    for (int i = 0; i < M; ++i) a[i] = acc[i];
    sc_add<M>(a, t, r);
#pragma unroll
    for (int i = 0; i < M; ++i) acc[i] = r[i];
  }
}

template <int NC, int P, int NP>
__device__ __forceinline__ void sc_parts_step(ScAcc<NC, NP> &acc, const h16 (&a)[NC], const h16 (&b)[NC],
                                              bool first) {
  if constexpr (P < NP) {
    sc_part_step<NC, P>(acc.v[P], a, b[P], first);
    sc_parts_step<NC, P + 1, NP>(acc, a, b, first);
  }
}

// C = P_0 (+) (0, P_1) (+) (0, 0, P_2) ... : part P placed at its levels, Add-MCN left
// to right (complete algorithm: once per output).
template <int NC, int P, int NP>
__device__ __forceinline__ void sc_combine(const ScAcc<NC, NP> &acc, h16 (&c)[NC]) {
  if constexpr (P < NP) {
    h16 y[NC], r[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) y[i] = i < P ? (h16)0.0f : acc.v[P][i - P];
    sc_add_general<NC>(c, y, r);
#pragma unroll
    for (int i = 0; i < NC; ++i) c[i] = r[i];
    sc_combine<NC, P + 1, NP>(acc, c);
  }
}

// One 16 x 16 tile of C per 256-lane workgroup, one output per lane, k in order.
// AMC / BMC: operand kinds; BT: B stored [planes][N][K]; bias: [NC][N] or null.
template <int NC, bool AMC, bool BMC, bool BT>
__global__ __launch_bounds__(SC_BM *SC_BN) void sc_mm_kernel(const h16 *__restrict__ A, const h16 *__restrict__ B,
                                                              const h16 *__restrict__ bias, h16 *__restrict__ C,
                                                              int64_t M, int64_t N, int64_t K) {
  constexpr int NA = AMC ? NC : 1;
  constexpr int NB = BMC ? NC : 1;
  constexpr int NP = (AMC && BMC) ? NC : 1;
  __shared__ h16 As[NA][SC_KT][SC_BM + 2];
  __shared__ h16 Bs[NB][SC_KT][SC_BN + 2];
  const int tid = threadIdx.x;
  const int tx = tid % SC_BN, ty = tid / SC_BN;
  const int64_t tiles_n = (N + SC_BN - 1) / SC_BN;
  const int64_t row0 = ((int64_t)blockIdx.x / tiles_n) * SC_BM, col0 = ((int64_t)blockIdx.x % tiles_n) * SC_BN;
  const int64_t row = row0 + ty, col = col0 + tx;
  ScAcc<NC, NP> acc;
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int i = 0; i < NC; ++i) acc.v[p][i] = (h16)0.0f;
  for (int64_t k0 = 0; k0 < K; k0 += SC_KT) {
    __syncthreads();
#pragma unroll
    for (int idx = tid; idx < SC_BM * SC_KT; idx += SC_BM * SC_BN) {
      const int r = idx / SC_KT, kk = idx % SC_KT;
      const bool in = row0 + r < M && k0 + kk < K;
#pragma unroll
      for (int c = 0; c < NA; ++c) As[c][kk][r] = in ? A[c * M * K + (row0 + r) * K + k0 + kk] : (h16)0.0f;
    }
#pragma unroll
    for (int idx = tid; idx < SC_BN * SC_KT; idx += SC_BM * SC_BN) {
      int cc, kk;
      if constexpr (BT) {
        cc = idx / SC_KT;
        kk = idx % SC_KT;
      } else {
        kk = idx / SC_BN;
        cc = idx % SC_BN;
      }
      const bool in = col0 + cc < N && k0 + kk < K;
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const int64_t off = BT ? (col0 + cc) * K + k0 + kk : (k0 + kk) * N + col0 + cc;
        Bs[c][kk][cc] = in ? B[c * K * N + off] : (h16)0.0f;
      }
    }
    __syncthreads();
    const int kmax = K - k0 < SC_KT ? (int)(K - k0) : SC_KT;
    for (int kk = 0; kk < kmax; ++kk) {
      h16 a[NC], b[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        a[c] = c < NA ? As[c][kk][ty] : (h16)0.0f;
        b[c] = c < NB ? Bs[c][kk][tx] : (h16)0.0f;
      }
      const bool first = k0 + kk == 0;
      if constexpr (AMC && BMC) {
        sc_parts_step<NC, 0, NP>(acc, a, b, first);
      } else if constexpr (AMC) {
        sc_part_step<NC, 0>(acc.v[0], a, b[0], first);
      } else {
        sc_part_step<NC, 0>(acc.v[0], b, a[0], first);
      }
    }
  }
  if (row >= M || col >= N) return;
  h16 c[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) c[i] = acc.v[0][i];
  sc_combine<NC, 1, NP>(acc, c);
  if (bias != nullptr) {
    h16 bb[NC], r[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) bb[i] = bias[i * N + col];
    sc_add<NC>(c, bb, r);
#pragma unroll
    for (int i = 0; i < NC; ++i) c[i] = r[i];
  }
#pragma unroll
  for (int i = 0; i < NC; ++i) C[i * M * N + row * N + col] = c[i];
}

template <int NC>
hipError_t sc_mm_nc(int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B, int b_mc, int b_trans,
                    const void *bias, void *C, hipStream_t s) {
  // a 1-D grid of row-major tiles (the ABI keeps the tile count below 2^31)
  const dim3 grid((unsigned)(((N + SC_BN - 1) / SC_BN) * ((M + SC_BM - 1) / SC_BM)));
  const dim3 block(SC_BM * SC_BN);
  const h16 *a = (const h16 *)A, *b = (const h16 *)B, *bi = (const h16 *)bias;
  h16 *c = (h16 *)C;
  if (a_mc && b_mc)
    hipLaunchKernelGGL((sc_mm_kernel<NC, true, true, false>), grid, block, 0, s, a, b, bi, c, M, N, K);
  else if (a_mc)
    hipLaunchKernelGGL((sc_mm_kernel<NC, true, false, false>), grid, block, 0, s, a, b, bi, c, M, N, K);
  else if (b_trans)
    hipLaunchKernelGGL((sc_mm_kernel<NC, false, true, true>), grid, block, 0, s, a, b, bi, c, M, N, K);
  else
    hipLaunchKernelGGL((sc_mm_kernel<NC, false, true, false>), grid, block, 0, s, a, b, bi, c, M, N, K);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scaled_elementwise(int op, int nc, int64_t n, const void *x, const void *y, void *out,
                                     hipStream_t stream) {
  switch (nc) {
    case 1: return sc_ew_nc<1>(op, n, x, y, out, stream);
    case 2: return sc_ew_nc<2>(op, n, x, y, out, stream);
    case 3: return sc_ew_nc<3>(op, n, x, y, out, stream);
    case 4: return sc_ew_nc<4>(op, n, x, y, out, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_scaled_matmul(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                                int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream) {
  switch (nc) {
    case 1: return sc_mm_nc<1>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
    case 2: return sc_mm_nc<2>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
    case 3: return sc_mm_nc<3>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
    case 4: return sc_mm_nc<4>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace mcf
