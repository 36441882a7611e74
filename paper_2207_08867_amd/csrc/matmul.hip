// matmul.hip -- MC matrix product (MM-MCN) and MC-Linear forward on gfx950 VALU.
//
// Every output C[i][j] is owned by one lane, which walks k = 0 .. K-1 in order:
// acc = ScalingN(term 0), acc = Add-MCN(acc, ScalingN(term k)).  This is the
// sequential error propagation of MM-MCN, so the result does not depend on tiling
// or launch geometry and matches the reference order bit for bit.  The contraction
// cannot use the matrix cores: every product and partial sum needs its exact
// rounding error (Two-Prod / Two-Sum), which only the vector ALU's FMA and IEEE adds
// deliver.
//
// Tiling: a 256-lane workgroup owns a BM x BN block of C; each lane owns TM x TN
// outputs.  A and B tiles of KT reduction steps are staged through LDS, component
// planes kept separate, A transposed to [k][m] so a lane reads its TM rows with one
// vector LDS load.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_arith.hpp"
#include "mcf_internal.hpp"

namespace mcf {

constexpr int MM_THREADS = 256;

// ---------------------------------------------------------------------------------
// The two steps of one MM-MCN term, in the form the product kernel executes them.
//
// They compute exactly what scaling_n / add_mcn of mcf_arith.hpp compute on finite,
// non-overflowing data, with two shortcuts that change nothing but the sign of a
// zero term, and zero terms are all dropped by Simple-Renorm (which pads with +0):
//   * the first Two-Sum of each step adds the initial carry +0: Two-Sum(h, +0) =
//     (h + 0, +0), so h_0 is the first product (resp. sum) and the carry its error;
//   * Simple-Renorm of nc+1 terms keeps h_0 .. h_{nc-2} unchanged when they are all
//     non-zero and then only chooses between h_{nc-1} and h_nc; the general
//     compaction runs only in lanes where a leading term is zero.
// ---------------------------------------------------------------------------------

// True when every one of v[0..K-1] is non-zero: min(|v_i|) != 0.  (A NaN is
// non-zero and min ignores it unless all are NaN, which is non-zero too.)
template <typename T, int K>
__device__ __forceinline__ bool all_nonzero(const T (&v)[K]) {
  static_assert(K >= 1 && K <= 4, "");
  if constexpr (K == 1) {
    return v[0] != T(0);
  } else if constexpr (K == 2) {
    return __builtin_fminf((float)__builtin_fabsf((float)v[0]), __builtin_fabsf((float)v[1])) != 0.0f;
  } else {
    T m = __builtin_fminf(__builtin_fminf(__builtin_fabsf((float)v[0]), __builtin_fabsf((float)v[1])),
                          __builtin_fabsf((float)v[2]));
    if constexpr (K == 4) return __builtin_fminf(m, __builtin_fabsf((float)v[3])) != 0.0f;
    return m != T(0);
  }
}

// FULL = true: the fast path needs all of h_0 .. h_{nc-1} non-zero and then keeps
// them, so the dropped h_nc is never needed there (binary32 data, where a zero term
// is rare).  FULL = false: it needs only h_0 .. h_{nc-2} and selects the first
// non-zero of h_{nc-1}, h_nc (binary16 data, where the last component is often
// below the subnormal grid).  `ok` admits lanes whose h is known to be all zero: the
// fast path then returns zeros, which is Simple-Renorm's result up to zero signs.
template <typename T, int N, bool FULL>
__device__ __forceinline__ void sr_fast(const T (&h)[N + 1], T (&out)[N], bool ok = false) {
  if constexpr (N == 1) {
    out[0] = (h[0] != T(0)) ? h[0] : h[1];
  } else {
    constexpr int NCHK = FULL ? N : N - 1;
    T lead[NCHK];
#pragma unroll
    for (int i = 0; i < NCHK; ++i) lead[i] = h[i];
    const bool fast = ok || all_nonzero<T, NCHK>(lead);
#pragma unroll
    for (int i = 0; i < N - 1; ++i) out[i] = h[i];
    if constexpr (FULL)
      out[N - 1] = h[N - 1];
    else
      out[N - 1] = (h[N - 1] != T(0)) ? h[N - 1] : h[N];
    if (__builtin_expect(!fast, 0)) simple_renorm<T, N + 1, N>(h, out);
  }
}

// Full checks pay off for binary32, the select for binary16.
template <typename T>
constexpr bool sr_full() {
  return sizeof(T) == 4;
}

// ScalingN(x, v) without expand.  vzero: v is +-0, so every term is zero (finite x).
template <typename T, int N>
__device__ __forceinline__ void mm_scaling(const T (&x)[N], T v, T (&out)[N], bool vzero) {
  T h[N + 1];
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
  sr_fast<T, N, sr_full<T>()>(h, out, vzero);
}

// Add-MCN(x, y).
template <typename T, int N>
__device__ __forceinline__ void mm_add(const T (&x)[N], const T (&y)[N], T (&out)[N]) {
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
  sr_fast<T, N, sr_full<T>()>(h, out);
}

// acc = ScalingN(mc, v) (first term) or acc = Add-MCN(acc, ScalingN(mc, v)).
template <typename T, int NC, bool FIRST>
__device__ __forceinline__ void mac(T (&acc)[NC], const T (&mc)[NC], T v, bool vzero) {
  if constexpr (FIRST) {
    mm_scaling<T, NC>(mc, v, acc, vzero);
  } else {
    T term[NC];
    mm_scaling<T, NC>(mc, v, term, vzero);
    mm_add<T, NC>(acc, term, acc);
  }
}

// A term whose plain factor is +-0 in every active lane of the wave is skipped by the
// whole wave: ScalingN then returns (+0, ..., +0) and Add-MCN(acc, (+0, ..., +0))
// returns acc unchanged, because acc is already a Simple-Renorm output (non-zeros
// first, zeros after).  (binary16 MC operands often carry a last component that is
// zero everywhere.)
__device__ __forceinline__ bool wave_none(bool lane_flag) { return __builtin_amdgcn_ballot_w64(lane_flag) == 0; }

// One reduction step kk of the LDS tiles for the TM x TN outputs of a lane.
template <typename T, int NC, bool AMC, bool BMC, int TM, int TN, int KT, int BM, int BN, bool FIRST>
__device__ __forceinline__ void step(const T (*As)[KT][BM], const T (*Bs)[KT][BN], int kk, int tx, int ty,
                                     T (&acc)[(AMC && BMC) ? NC : 1][TM][TN][NC]) {
  constexpr int NA = AMC ? NC : 1;
  constexpr int NB = BMC ? NC : 1;
  constexpr int NP = (AMC && BMC) ? NC : 1;
  T a[TM][NA], b[TN][NB];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int c = 0; c < NA; ++c) a[i][c] = As[c][kk][ty * TM + i];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int c = 0; c < NB; ++c) b[j][c] = Bs[c][kk][tx * TN + j];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      if constexpr (AMC && BMC) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const bool vz = b[j][p] == T(0);
          if (FIRST || !wave_none(!vz)) mac<T, NC, FIRST>(acc[p][i][j], a[i], b[j][p], vz);
        }
      } else if constexpr (AMC) {
        const bool vz = b[j][0] == T(0);
        if (FIRST || !wave_none(!vz)) mac<T, NC, FIRST>(acc[0][i][j], a[i], b[j][0], vz);
      } else {
        const bool vz = a[i][0] == T(0);
        if (FIRST || !wave_none(!vz)) mac<T, NC, FIRST>(acc[0][i][j], b[j], a[i][0], vz);
      }
    }
}

// A: [NA][M][K] row-major planes.  B: [NB][K][N] (BT = false) or [NB][N][K] (BT =
// true).  NA = NC when A is MC else 1, likewise NB.
template <typename T, int NC, bool AMC, bool BMC, bool BT, int TM, int TN, int KT>
__global__ __launch_bounds__(MM_THREADS) void mm_kernel(const T *__restrict__ A, const T *__restrict__ B,
                                                        const T *__restrict__ bias, T *__restrict__ C, int64_t M,
                                                        int64_t N, int64_t K) {
  constexpr int NA = AMC ? NC : 1;
  constexpr int NB = BMC ? NC : 1;
  constexpr int TX = 16, TY = 16;  // lanes along N and along M
  constexpr int BM = TY * TM, BN = TX * TN;
  constexpr int NP = (AMC && BMC) ? NC : 1;  // plain components to sweep (MC x MC)
  __shared__ T As[NA][KT][BM];
  __shared__ T Bs[NB][KT][BN];

  const int tx = threadIdx.x % TX, ty = threadIdx.x / TX;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;

  T acc[NP][TM][TN][NC];

  for (int64_t k0 = 0; k0 < K; k0 += KT) {
    const int kt = (int)((K - k0) < KT ? (K - k0) : KT);
    // stage A tile: rows m0..m0+BM-1, reduction steps k0..k0+KT-1
    for (int idx = threadIdx.x; idx < BM * KT; idx += MM_THREADS) {
      const int r = idx / KT, kk = idx % KT;
      const int64_t gm = m0 + r, gk = k0 + kk;
      const bool ok = gm < M && gk < K;
#pragma unroll
      for (int c = 0; c < NA; ++c) As[c][kk][r] = ok ? A[c * M * K + gm * K + gk] : T(0);
    }
    for (int idx = threadIdx.x; idx < BN * KT; idx += MM_THREADS) {
      int col, kk;
      if constexpr (BT) {
        col = idx / KT;
        kk = idx % KT;
      } else {
        kk = idx / BN;
        col = idx % BN;
      }
      const int64_t gn = n0 + col, gk = k0 + kk;
      const bool ok = gn < N && gk < K;
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const int64_t off = BT ? (c * N * K + gn * K + gk) : (c * K * N + gk * N + gn);
        Bs[c][kk][col] = ok ? B[off] : T(0);
      }
    }
    __syncthreads();
    int kk0 = 0;
    if (k0 == 0) {  // term k = 0 initialises the accumulators
      step<T, NC, AMC, BMC, TM, TN, KT, BM, BN, true>(As, Bs, 0, tx, ty, acc);
      kk0 = 1;
    }
    for (int kk = kk0; kk < kt; ++kk) step<T, NC, AMC, BMC, TM, TN, KT, BM, BN, false>(As, Bs, kk, tx, ty, acc);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t gm = m0 + ty * TM + i, gn = n0 + tx * TN + j;
      T r[NC];
      if (K == 0) {
#pragma unroll
        for (int c = 0; c < NC; ++c) r[c] = T(0);
      } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) r[c] = acc[0][i][j][c];
        // MC x MC: combine the per-component products left to right
#pragma unroll
        for (int p = 1; p < NP; ++p) mm_add<T, NC>(r, acc[p][i][j], r);
      }
      if (gm < M && gn < N) {
        if (bias != nullptr) {
          T bv[NC];
#pragma unroll
          for (int c = 0; c < NC; ++c) bv[c] = bias[c * N + gn];
          mm_add<T, NC>(r, bv, r);
        }
        // Zero components leave as +0, the padding Simple-Renorm writes (a zero term
        // that was skipped or selected above may carry the sign of -0).
#pragma unroll
        for (int c = 0; c < NC; ++c) C[c * M * N + gm * N + gn] = (r[c] != T(0)) ? r[c] : T(0);
      }
    }
}

template <typename T, int NC, bool AMC, bool BMC, bool BT>
static hipError_t mm_launch(int64_t M, int64_t N, int64_t K, const void *A, const void *B, const void *bias,
                            void *C, hipStream_t s) {
  constexpr int TM = 2, TN = 2, KT = 16;
  constexpr int BM = 16 * TM, BN = 16 * TN;
  dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
  hipLaunchKernelGGL((mm_kernel<T, NC, AMC, BMC, BT, TM, TN, KT>), grid, dim3(MM_THREADS), 0, s, (const T *)A,
                     (const T *)B, (const T *)bias, (T *)C, M, N, K);
  return hipGetLastError();
}

template <typename T, int NC>
static hipError_t mm_kinds(int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B, int b_mc,
                           int b_trans, const void *bias, void *C, hipStream_t s) {
  if (b_trans) {
    // linear layer: plain input times MC weight stored [out][in]
    if (!a_mc && b_mc) return mm_launch<T, NC, false, true, true>(M, N, K, A, B, bias, C, s);
    return hipErrorInvalidValue;
  }
  if (a_mc && b_mc) return mm_launch<T, NC, true, true, false>(M, N, K, A, B, bias, C, s);
  if (a_mc) return mm_launch<T, NC, true, false, false>(M, N, K, A, B, bias, C, s);
  return mm_launch<T, NC, false, true, false>(M, N, K, A, B, bias, C, s);
}

template <typename T>
static hipError_t mm_dispatch(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                              int b_mc, int b_trans, const void *bias, void *C, hipStream_t s) {
  switch (nc) {
    case 1: return mm_kinds<T, 1>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, s);
    case 2: return mm_kinds<T, 2>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, s);
    case 3: return mm_kinds<T, 3>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, s);
    case 4: return mm_kinds<T, 4>(M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                         const void *B, int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream) {
  if (dtype == 0) return mm_dispatch<_Float16>(nc, M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
  return mm_dispatch<float>(nc, M, N, K, A, a_mc, B, b_mc, b_trans, bias, C, stream);
}

}  // namespace mcf
