// splitk.hip -- K-split MC matrix product on gfx950 VALU, for reductions that are
// long compared with the number of outputs (Dot-MCN, MV-MCN, small products).
//
// The function computed (fixed by the slice count S alone, not by the launch):
// the reduction steps are dealt round-robin to S slices, slice s taking
// k = s, s + S, s + 2S, ...; each slice is summed in MM-MCN order (ScalingN of its
// first term, then Add-MCN of each further ScalingN term); the S slice sums are then
// combined by a pairwise Add-MCN tree -- at each level entry q of the next level is
// Add-MCN(entry 2q, entry 2q+1) and an odd last entry moves up unchanged.  This is
// the log-depth accumulation that Section 2.2 of the paper names as the cost of an
// accurate N-term MC sum.  MC x MC products are taken by linearity over B's
// components, one K-split product per component, combined left to right.
//
// Launch: a 256-lane workgroup holds 256/KS outputs x KS consecutive slices (KS a
// power of two); lane (output o, slice s) reads A[i][k] and B[k][j] for its own k,
// so the lanes of a slice group read consecutive k.  The first log2(KS) tree levels
// run inside the workgroup (strides < 64 by lane exchange inside a wavefront, 64 and
// 128 through LDS); when S > KS the G = ceil(S/KS) group results go to a workspace
// and a second kernel runs all further levels in one launch: each of its lanes takes an
// aligned block of R consecutive roots (R = 1, 4 or 16, the smallest with G <= 256 R)
// and runs the first log2(R) of those levels in registers, and the lanes then run the
// last levels as in the first kernel.  Because every group and block is an aligned
// block of the level below, a pair of the tree never straddles two of them: the
// result equals the tree's definition for every launch shape.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "mcf_arith.hpp"
#include "mcf_internal.hpp"
#include "mm_steps.hpp"

namespace mcf {

constexpr int SK_THREADS = 256;
constexpr int SK_UNROLL = 4;

// Lane exchange inside a wavefront: the value of lane (l + d), for d < 64.  binary16
// values travel as binary32 (exact both ways).
__device__ __forceinline__ float lane_down(float v, int d) { return __shfl_down(v, (unsigned)d, 64); }
__device__ __forceinline__ _Float16 lane_down(_Float16 v, int d) {
  return (_Float16)__shfl_down((float)v, (unsigned)d, 64);
}
__device__ __forceinline__ double lane_down(double v, int d) { return __shfl_down(v, (unsigned)d, 64); }

// Pairwise Add-MCN tree over groups of W lanes (W a power of two, W <= 256): lane q
// of a group holds leaf q, and leaves q >= count are absent.  At stride d the entry of
// lane q (q a multiple of 2d) becomes Add-MCN(entry q, entry q + d) when q + d <
// count, and is unchanged otherwise.  Afterwards lane 0 of each group holds the root.
// Every lane of the workgroup must call this (it contains barriers and exchanges).
template <typename T, int NC, int NP, int APOL>
__device__ __forceinline__ void group_tree(T (&acc)[NP][NC], int q, int W, int count, T (*lds)[NP * NC]) {
  for (int d = 1; d < W; d <<= 1) {
    T other[NP][NC];
    if (d < 64) {
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int c = 0; c < NC; ++c) other[p][c] = lane_down(acc[p][c], d);
    } else {
      if ((q & (2 * d - 1)) == d) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int c = 0; c < NC; ++c) lds[threadIdx.x][p * NC + c] = acc[p][c];
      }
      __syncthreads();
      if ((q & (2 * d - 1)) == 0 && q + d < count) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int c = 0; c < NC; ++c) other[p][c] = lds[threadIdx.x + d][p * NC + c];
      }
      __syncthreads();
    }
    if ((q & (2 * d - 1)) == 0 && q + d < count) {
#pragma unroll
      for (int p = 0; p < NP; ++p) mm_add<T, NC, APOL>(acc[p], other[p], acc[p]);
    }
  }
}

// Combine the per-component products of B left to right and store one output
// (zero components as +0, Simple-Renorm's padding).
template <typename T, int NC, int NP, int APOL>
__device__ __forceinline__ void sk_store(const T (&acc)[NP][NC], T *__restrict__ C, int64_t MN, int64_t o) {
  T r[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) r[c] = acc[0][c];
#pragma unroll
  for (int p = 1; p < NP; ++p) mm_add<T, NC, APOL>(r, acc[p], r);
#pragma unroll
  for (int c = 0; c < NC; ++c) C[c * MN + o] = (r[c] != T(0)) ? r[c] : T(0);
}

// One MM-MCN term into the accumulators: acc[p] = Add-MCN(acc[p], ScalingN(mc, v_p)).
// FIRST: acc[p] = ScalingN(mc, v_p).
template <typename T, int NC, bool AMC, bool BMC, int SPOL, int APOL, bool FIRST>
__device__ __forceinline__ void sk_term(T (&acc)[(AMC && BMC) ? NC : 1][NC], const T (&a)[AMC ? NC : 1],
                                        const T (&b)[BMC ? NC : 1]) {
  constexpr int NP = (AMC && BMC) ? NC : 1;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const T v = AMC ? b[BMC ? p : 0] : a[0];
    T h[NC + 1];
    if constexpr (AMC)
      scaling_terms<T, NC>(a, v, h);
    else
      scaling_terms<T, NC>(b, v, h);
    if constexpr (FIRST) {
      if (__builtin_expect(sr_try<T, NC, SPOL>(h, acc[p], v == T(0)), 0)) compact_nz<T, NC + 1, NC>(h, acc[p]);
      nonfinite_tail<T, NC>(acc[p]);
    } else {
      T term[NC];
      if (__builtin_expect(sr_try<T, NC, SPOL>(h, term, v == T(0)), 0)) compact_nz<T, NC + 1, NC>(h, term);
      add_terms<T, NC>(acc[p], term, h);
      if (__builtin_expect(sr_try<T, NC, APOL>(h, acc[p]), 0)) compact_nz<T, NC + 1, NC>(h, acc[p]);
    }
  }
}

// Phase 1: slice sums and the in-workgroup tree levels.  A: [NA][M][K], B: [NB][K][N].
// G == 1: the result goes to C [NC][M*N].  G > 1: the group roots go to
// W [G][NP][NC][M*N].
template <typename T, int NC, bool AMC, bool BMC, int SPOL, int APOL>
__global__ __launch_bounds__(SK_THREADS) void sk_kernel(const T *__restrict__ A, const T *__restrict__ B,
                                                        T *__restrict__ C, T *__restrict__ W, int64_t M, int64_t N,
                                                        int64_t K, int64_t S, int KS, int G) {
  constexpr int NA = AMC ? NC : 1;
  constexpr int NB = BMC ? NC : 1;
  constexpr int NP = (AMC && BMC) ? NC : 1;
  __shared__ T lds[SK_THREADS][NP * NC];

  const int64_t MN = M * N;
  const int q = threadIdx.x & (KS - 1);
  const int64_t o = (int64_t)blockIdx.x * (SK_THREADS / KS) + threadIdx.x / KS;
  const int64_t s = (int64_t)blockIdx.y * KS + q;
  const int64_t i = o / N, j = o % N;

  T acc[NP][NC];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[p][c] = T(0);

  if (o < MN && s < S) {
    const T *Ai = A + i * K;
    const T *Bj = B + j;
    auto load = [&](int64_t k, T (&a)[NA], T (&b)[NB]) {
#pragma unroll
      for (int c = 0; c < NA; ++c) a[c] = Ai[c * M * K + k];
#pragma unroll
      for (int c = 0; c < NB; ++c) b[c] = Bj[c * K * N + k * N];
    };
    int64_t k = s;
    {
      T a[NA], b[NB];
      load(k, a, b);
      sk_term<T, NC, AMC, BMC, SPOL, APOL, true>(acc, a, b);
      k += S;
    }
    // Loads of SK_UNROLL steps are issued before their arithmetic.
    for (; k + (SK_UNROLL - 1) * S < K; k += SK_UNROLL * S) {
      T a[SK_UNROLL][NA], b[SK_UNROLL][NB];
#pragma unroll
      for (int u = 0; u < SK_UNROLL; ++u) load(k + u * S, a[u], b[u]);
#pragma unroll
      for (int u = 0; u < SK_UNROLL; ++u) sk_term<T, NC, AMC, BMC, SPOL, APOL, false>(acc, a[u], b[u]);
    }
    for (; k < K; k += S) {
      T a[NA], b[NB];
      load(k, a, b);
      sk_term<T, NC, AMC, BMC, SPOL, APOL, false>(acc, a, b);
    }
  }

  const int64_t left = S - (int64_t)blockIdx.y * KS;
  const int count = left < KS ? (int)left : KS;
  group_tree<T, NC, NP, APOL>(acc, q, KS, count, lds);

  if (q == 0 && o < MN) {
    if (G == 1) {
      sk_store<T, NC, NP, APOL>(acc, C, MN, o);
    } else {
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int c = 0; c < NC; ++c) W[(((int64_t)blockIdx.y * NP + p) * NC + c) * MN + o] = acc[p][c];
    }
  }
}

// Phase 2: the tree levels above the G group roots of each output in W, in one launch.
// Lane q of an output's GW-lane group takes roots q R .. q R + R - 1 (those below G)
// and folds them in tree order in registers: entry j is pushed after one Add-MCN with
// each completed left neighbour (one per trailing one bit of j), and what is left
// when fewer than R are present combines lowest level first -- an unpaired right
// entry moves up until it meets its left partner, as the tree's rule has it.  The
// lanes then run the last levels as a group tree over ceil(G / R) entries.
template <int R>
struct log2_of {
  static constexpr int value = R <= 1 ? 0 : 1 + log2_of<R / 2>::value;
};
template <>
struct log2_of<1> {
  static constexpr int value = 0;
};

template <typename T, int NC, int NP, int APOL, int R>
__global__ __launch_bounds__(SK_THREADS) void sk_reduce_kernel(const T *__restrict__ W, T *__restrict__ C, int64_t MN,
                                                               int G, int GW) {
  constexpr int L = log2_of<R>::value;
  __shared__ T lds[SK_THREADS][NP * NC];
  const int q = threadIdx.x & (GW - 1);
  const int64_t o = (int64_t)blockIdx.x * (SK_THREADS / GW) + threadIdx.x / GW;
  const int first = q * R;
  const int n = (o < MN && first < G) ? (G - first < R ? G - first : R) : 0;
  // Loads stay in bounds for absent entries (the last root of the last output) so that
  // they can all be issued before the arithmetic; absent entries are never used.
  const int64_t ol = o < MN ? o : MN - 1;
  T stk[L + 1][NP][NC];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const int64_t e = first + j < G ? first + j : G - 1;
    T v[NP][NC];
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int c = 0; c < NC; ++c) v[p][c] = W[((e * NP + p) * NC + c) * MN + ol];
    if (j < n) {
      int l = 0;
#pragma unroll
      for (; l < L && ((j >> l) & 1); ++l) {
#pragma unroll
        for (int p = 0; p < NP; ++p) mm_add<T, NC, APOL>(stk[l][p], v[p], v[p]);
      }
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int c = 0; c < NC; ++c) stk[l][p][c] = v[p][c];
    }
  }
  T acc[NP][NC];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[p][c] = T(0);
  bool have = false;
#pragma unroll
  for (int l = 0; l <= L; ++l) {
    if ((n >> l) & 1) {
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        if (have) {
          mm_add<T, NC, APOL>(stk[l][p], acc[p], acc[p]);
        } else {
#pragma unroll
          for (int c = 0; c < NC; ++c) acc[p][c] = stk[l][p][c];
        }
      }
      have = true;
    }
  }
  group_tree<T, NC, NP, APOL>(acc, q, GW, (G + R - 1) / R, lds);
  if (q == 0 && o < MN) sk_store<T, NC, NP, APOL>(acc, C, MN, o);
}

static int pow2_at_least(int64_t v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

int64_t splitk_default_slices(int64_t M, int64_t N, int64_t K) {
  const int64_t MN = M * N;
  if (MN <= 0 || K <= 0) return 1;
  int64_t s = ((int64_t)SPLITK_TARGET_LANES + MN - 1) / MN;
  const int64_t by_k = K / SPLITK_MIN_STEPS > 1 ? K / SPLITK_MIN_STEPS : 1;
  if (s > by_k) s = by_k;
  if (s > SPLITK_MAX_SLICES) s = SPLITK_MAX_SLICES;
  return s < 1 ? 1 : s;
}

void splitk_shape(int64_t S, int *KS, int *G) {
  const int ks = pow2_at_least(S < SK_THREADS ? S : SK_THREADS);
  *KS = ks;
  *G = (int)((S + ks - 1) / ks);
}

int64_t splitk_roots(int64_t S) {
  int KS, G;
  splitk_shape(S, &KS, &G);
  return G == 1 ? 0 : G;
}

template <typename T, int NC, int NP, int APOL, int R>
static void sk_reduce_launch(const T *W, T *C, int64_t MN, int G, hipStream_t s) {
  const int lanes = (G + R - 1) / R;
  const int GW = pow2_at_least(lanes);
  dim3 grid((unsigned)((MN + (SK_THREADS / GW) - 1) / (SK_THREADS / GW)));
  hipLaunchKernelGGL((sk_reduce_kernel<T, NC, NP, APOL, R>), grid, dim3(SK_THREADS), 0, s, W, C, MN, G, GW);
}

template <typename T, int NC, bool AMC, bool BMC>
static hipError_t sk_launch(int64_t M, int64_t N, int64_t K, const void *A, const void *B, int64_t S, void *W, void *C,
                            hipStream_t s) {
  constexpr int NP = (AMC && BMC) ? NC : 1;
  // Simple-Renorm fast-path policies as in the sequential product (they change speed only)
  constexpr int SPOL = sizeof(T) >= 4 ? SR_FULL : (NC == 2 ? SR_NET : SR_HEAD);
  constexpr int APOL = sizeof(T) >= 4 ? SR_FULL : SR_SELECT;
  const int64_t MN = M * N;
  int KS, G;
  splitk_shape(S, &KS, &G);
  // S <= SPLITK_MAX_SLICES = 2^20 gives G <= 4096 = 16 x 256 group roots.
  if (G > 16 * SK_THREADS) return hipErrorInvalidValue;
  dim3 grid((unsigned)((MN + (SK_THREADS / KS) - 1) / (SK_THREADS / KS)), (unsigned)G);
  hipLaunchKernelGGL((sk_kernel<T, NC, AMC, BMC, SPOL, APOL>), grid, dim3(SK_THREADS), 0, s, (const T *)A,
                     (const T *)B, (T *)C, (T *)W, M, N, K, S, KS, G);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || G == 1) return e;
  // W: the G group roots.
  if (G <= SK_THREADS)
    sk_reduce_launch<T, NC, NP, APOL, 1>((const T *)W, (T *)C, MN, G, s);
  else if (G <= 4 * SK_THREADS)
    sk_reduce_launch<T, NC, NP, APOL, 4>((const T *)W, (T *)C, MN, G, s);
  else
    sk_reduce_launch<T, NC, NP, APOL, 16>((const T *)W, (T *)C, MN, G, s);
  return hipGetLastError();
}

template <typename T, int NC>
static hipError_t sk_kinds(int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B, int b_mc,
                           int64_t S, void *W, void *C, hipStream_t s) {
  if (a_mc && b_mc) return sk_launch<T, NC, true, true>(M, N, K, A, B, S, W, C, s);
  if (a_mc) return sk_launch<T, NC, true, false>(M, N, K, A, B, S, W, C, s);
  return sk_launch<T, NC, false, true>(M, N, K, A, B, S, W, C, s);
}

template <typename T>
static hipError_t sk_dispatch(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                              int b_mc, int64_t S, void *W, void *C, hipStream_t s) {
  switch (nc) {
    case 1: return sk_kinds<T, 1>(M, N, K, A, a_mc, B, b_mc, S, W, C, s);
    case 2: return sk_kinds<T, 2>(M, N, K, A, a_mc, B, b_mc, S, W, C, s);
    case 3: return sk_kinds<T, 3>(M, N, K, A, a_mc, B, b_mc, S, W, C, s);
    case 4: return sk_kinds<T, 4>(M, N, K, A, a_mc, B, b_mc, S, W, C, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_matmul_splitk(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                                const void *B, int b_mc, int64_t S, void *W, void *C, hipStream_t stream) {
  if (dtype == 0) return sk_dispatch<_Float16>(nc, M, N, K, A, a_mc, B, b_mc, S, W, C, stream);
  if (dtype == 2) return sk_dispatch<double>(nc, M, N, K, A, a_mc, B, b_mc, S, W, C, stream);
  return sk_dispatch<float>(nc, M, N, K, A, a_mc, B, b_mc, S, W, C, stream);
}

// Static scratch of the allocation-free K-split entry point: the partial tree roots
// of one call live here instead of in a caller workspace.  Each device holds its own
// copy for the life of the process.  In host code `scratch` names a host-side
// stand-in, not device memory: the device address is looked up once per device with
// hipGetSymbolAddress and only that address is ever passed to a kernel.
__device__ __align__(256) unsigned char scratch[SPLITK_SCRATCH_BYTES];

namespace {
constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[SCRATCH_MAX_DEVICES] = {};
}  // namespace

// Device address of `scratch` on the device that runs `stream` (the current device
// for the null stream); the lookup runs with that device current, once per device.
hipError_t splitk_scratch(hipStream_t stream, void **ptr) {
  int dev = 0, cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  dev = cur;
  if (stream != nullptr) {
    e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
  }
  if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t r = hipSetDevice(cur);
      if (e == hipSuccess) e = r;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace mcf
