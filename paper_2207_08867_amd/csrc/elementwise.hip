// elementwise.hip -- elementwise MC kernels: Add-MCN / Grow-ExpN, ScalingN /
// Mult-MCN, Div-MCN / DivN, Renormalize / Simple-Renorm, and Exp-MCN (binary16 by
// table lookup, binary32 by a correctly rounded evaluation).
//
// Data are component-major planes; each thread moves 16 bytes per plane per step
// (8 binary16 or 4 binary32 elements) with dwordx4 loads and stores, so one wave
// reads 1 KiB contiguous per plane: fully coalesced HBM streams (the few longest
// per-element algorithms take one element per lane: see ew_one_per_lane).  The arithmetic of
// each element is the per-element algorithm of mcf_arith.hpp (Div-MCN and Mult-MCN
// through div_steps.hpp, which returns the same bits with fewer operations).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "div_steps.hpp"
#include "exp32.hpp"
#include "mcf_arith.hpp"
#include "mcf_internal.hpp"

namespace mcf {

constexpr int EW_THREADS = 256;

template <typename T, int W>
struct Pack {
  T v[W];
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte accesses are non-temporal: every byte is touched once, so keeping it out
// of the caches leaves them to the other streams (measured: 5.2 -> 6.1 TB/s for six
// input and three output planes).
template <typename T, int W>
__device__ __forceinline__ Pack<T, W> load_pack(const T *p) {
  Pack<T, W> r;
  if constexpr (W * sizeof(T) == 16) {
    u32x4 raw = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    __builtin_memcpy(&r, &raw, 16);
  } else {
#pragma unroll
    for (int w = 0; w < W; ++w) r.v[w] = p[w];
  }
  return r;
}

template <typename T, int W>
__device__ __forceinline__ void store_pack(T *p, const Pack<T, W> &r) {
  if constexpr (W * sizeof(T) == 16) {
    u32x4 raw;
    __builtin_memcpy(&raw, &r, 16);
    __builtin_nontemporal_store(raw, reinterpret_cast<u32x4 *>(p));
  } else {
#pragma unroll
    for (int w = 0; w < W; ++w) p[w] = r.v[w];
  }
}

// Exp-MCN for one element from the component exponentials ex[0..N-1]:
// h = (ex_0), then h = ScalingN(h, ex_i) with expand, one component longer per step.
template <typename T, int N, int M>
__device__ __forceinline__ void exp_chain(const T (&h)[M], const T (&ex)[N], T (&out)[N]) {
  if constexpr (M == N) {
#pragma unroll
    for (int c = 0; c < N; ++c) out[c] = h[c];
  } else {
    T g[M + 1];
    scaling_n<T, M, M + 1>(h, ex[M], g);
    exp_chain<T, N, M + 1>(g, ex, out);
  }
}

// The algorithm applied to one element.  Plain operands arrive in slot 0 with the
// other slots +0, which is exactly the zero padding DivN and (MC, T) division use.
template <typename T, int NC, int OP, bool XMC, bool YMC, int NCOUT>
__device__ __forceinline__ void elem(const T (&a)[NC], const T (&b)[NC], T (&r)[NCOUT]) {
  if constexpr (OP == EW_ADD) {
    if constexpr (XMC && YMC)
      add_mcn<T, NC>(a, b, r);
    else if constexpr (XMC)
      grow_expn<T, NC>(a, b[0], r);
    else
      grow_expn<T, NC>(b, a[0], r);
  } else if constexpr (OP == EW_MUL) {
    if constexpr (XMC && YMC)
      mult_mcn_fast<T, NC>(a, b, r);
    else if constexpr (XMC)
      scaling_n<T, NC, NC>(a, b[0], r);
    else
      scaling_n<T, NC, NC>(b, a[0], r);
  } else if constexpr (OP == EW_DIV) {
    div_mcn_fast<T, NC>(a, b, r);
  } else if constexpr (OP == EW_EXP) {
    static_assert(sizeof(T) == 4, "binary16 Exp-MCN has its own kernel");
    T ex[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) ex[c] = exp32_cr(a[c]);
    const T h0[1] = {ex[0]};
    exp_chain<T, NC, 1>(h0, ex, r);
  } else if constexpr (OP == EW_MUL_SLOW) {
    mult_mcn_slow_fast<T, NC>(a, b, r);
  } else if constexpr (OP == EW_SQUARE) {
    square_mcn<T, NC>(a, r);
  } else if constexpr (OP == EW_RENORM) {
    renormalize<T, NC, NCOUT>(a, r);
  } else {
    simple_renorm<T, NC, NCOUT>(a, r);
  }
}

// U chunks of W consecutive elements starting at element indices e0[u] (all in
// range): every load of every chunk is issued before any arithmetic or store, so a
// thread keeps (planes x U) 16-byte requests in flight; stores follow the arithmetic.
// (In place is safe: a chunk's stores come after its own loads.)
template <typename T, int NC, int OP, bool XMC, bool YMC, int NCOUT, int W, int U>
__device__ __forceinline__ void ew_chunks(const T *x, const T *y, T *out, int64_t n, const int64_t (&e0)[U]) {
  constexpr int XN = XMC ? NC : 1;
  constexpr int YN = (OP == EW_RENORM || OP == EW_SIMPLE_RENORM || OP == EW_EXP || OP == EW_SQUARE) ? 0
                                                                                               : (YMC ? NC : 1);
  Pack<T, W> xa[U][XN];
  Pack<T, W> ya[U][YN > 0 ? YN : 1];
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int c = 0; c < XN; ++c) xa[u][c] = load_pack<T, W>(x + c * n + e0[u]);
#pragma unroll
    for (int c = 0; c < YN; ++c) ya[u][c] = load_pack<T, W>(y + c * n + e0[u]);
  }
  Pack<T, W> res[U][NCOUT];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int w = 0; w < W; ++w) {
      T a[NC], b[NC], r[NCOUT];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        a[c] = c < XN ? xa[u][c < XN ? c : 0].v[w] : T(0);
        b[c] = c < YN ? ya[u][c < YN ? c : 0].v[w] : T(0);
      }
      elem<T, NC, OP, XMC, YMC, NCOUT>(a, b, r);
#pragma unroll
      for (int c = 0; c < NCOUT; ++c) res[u][c].v[w] = r[c];
    }
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int c = 0; c < NCOUT; ++c) store_pack<T, W>(out + c * n + e0[u], res[u][c]);
}

// Grid-stride over chunks of W elements, EW_UNROLL chunks per thread per step (a
// block covers EW_THREADS * EW_UNROLL consecutive chunks, lanes adjacent); the last
// n % W elements one per thread.  Inputs and output may alias exactly (in place):
// every element is read by the thread that writes it, before it writes.
constexpr int EW_UNROLL = 2;

template <typename T, int NC, int OP, bool XMC, bool YMC, int NCOUT, int W>
__global__ __launch_bounds__(EW_THREADS) void ew_kernel(const T *x, const T *y, T *out, int64_t n) {
  const int64_t nchunk = n / W;
  const int64_t step = (int64_t)gridDim.x * EW_THREADS * EW_UNROLL;
  int64_t base = (int64_t)blockIdx.x * EW_THREADS * EW_UNROLL + threadIdx.x;
  // full steps: all EW_UNROLL chunks of the thread are in range
  for (; base + (int64_t)(EW_UNROLL - 1) * EW_THREADS < nchunk; base += step) {
    int64_t e0[EW_UNROLL];
#pragma unroll
    for (int u = 0; u < EW_UNROLL; ++u) e0[u] = (base + (int64_t)u * EW_THREADS) * W;
    ew_chunks<T, NC, OP, XMC, YMC, NCOUT, W, EW_UNROLL>(x, y, out, n, e0);
  }
  // the last, partial step
  for (int u = 0; u < EW_UNROLL; ++u) {
    const int64_t ch = base + (int64_t)u * EW_THREADS;
    if (ch < nchunk) {
      const int64_t e1[1] = {ch * W};
      ew_chunks<T, NC, OP, XMC, YMC, NCOUT, W, 1>(x, y, out, n, e1);
    }
  }
  if constexpr (W > 1) {
    const int64_t tid = (int64_t)blockIdx.x * EW_THREADS + threadIdx.x;
    const int64_t tail = n - nchunk * W;
    if (tid < tail) {
      const int64_t e1[1] = {nchunk * W + tid};
      ew_chunks<T, NC, OP, XMC, YMC, NCOUT, 1, 1>(x, y, out, n, e1);
    }
  }
}

static int ew_blocks(int64_t work) {
  int64_t b = (work + EW_THREADS * EW_UNROLL - 1) / (EW_THREADS * EW_UNROLL);
  if (b < 1) b = 1;
  if (b > 16384) b = 16384;
  return (int)b;
}

// Instantiations whose per-element body is so long that the compiler does not unroll
// the loop over a 16-byte chunk's elements: their operand and result packs, indexed by
// the loop counter, would live in scratch memory (binary16 Mult-MCN-Slow at nc = 3
// moved 2.7 GB of it per 2^26 elements, mostly in cache: the steady-state time is 1%
// lower without it).  They take one element per lane and plane instead.
template <typename T, int NC, int OP, bool XMC, bool YMC>
constexpr bool ew_one_per_lane() {
  if constexpr (OP == EW_MUL_SLOW) return sizeof(T) == 2 ? NC >= 3 : (sizeof(T) == 4 && NC >= 4);
  if constexpr (OP == EW_MUL && XMC && YMC) return sizeof(T) == 2 && NC >= 4;
  return false;
}

template <typename T, int NC, int OP, bool XMC, bool YMC, int NCOUT>
static hipError_t ew_launch(int64_t n, const void *x, const void *y, void *out, hipStream_t s) {
  constexpr int W = ew_one_per_lane<T, NC, OP, XMC, YMC>() ? 1 : 16 / sizeof(T);
  constexpr int VB = W * (int)sizeof(T);
  const T *xp = (const T *)x;
  const T *yp = (const T *)y;
  T *op = (T *)out;
  // vector access of VB bytes needs every plane start aligned to VB bytes
  bool vec = ((n * (int64_t)sizeof(T)) % VB == 0) && ((uintptr_t)x % VB == 0) &&
             (y == nullptr || (uintptr_t)y % VB == 0) && ((uintptr_t)out % VB == 0);
  if (vec) {
    hipLaunchKernelGGL((ew_kernel<T, NC, OP, XMC, YMC, NCOUT, W>), dim3(ew_blocks(n / W)), dim3(EW_THREADS), 0, s,
                       xp, yp, op, n);
  } else {
    hipLaunchKernelGGL((ew_kernel<T, NC, OP, XMC, YMC, NCOUT, 1>), dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, xp,
                       yp, op, n);
  }
  return hipGetLastError();
}

template <typename T, int NC, int OP>
static hipError_t ew_kinds(int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out, hipStream_t s) {
  if (x_mc && y_mc) return ew_launch<T, NC, OP, true, true, NC>(n, x, y, out, s);
  if (x_mc) return ew_launch<T, NC, OP, true, false, NC>(n, x, y, out, s);
  return ew_launch<T, NC, OP, false, true, NC>(n, x, y, out, s);
}

template <typename T, int NC, int OP, int NCOUT>
static hipError_t renorm_out(int64_t n, const void *x, void *out, hipStream_t s) {
  return ew_launch<T, NC, OP, true, false, NCOUT>(n, x, nullptr, out, s);
}

template <typename T, int NC, int OP>
static hipError_t renorm_dispatch(int nc_out, int64_t n, const void *x, void *out, hipStream_t s) {
  switch (nc_out) {
    case 1: return renorm_out<T, NC, OP, 1>(n, x, out, s);
    case 2: if constexpr (NC >= 2) return renorm_out<T, NC, OP, 2>(n, x, out, s); break;
    case 3: if constexpr (NC >= 3) return renorm_out<T, NC, OP, 3>(n, x, out, s); break;
    case 4: if constexpr (NC >= 4) return renorm_out<T, NC, OP, 4>(n, x, out, s); break;
  }
  return hipErrorInvalidValue;
}

template <typename T, int NC>
static hipError_t ew_dispatch_nc(int op, int nc_out, int64_t n, const void *x, int x_mc, const void *y, int y_mc,
                                 void *out, hipStream_t s) {
  switch (op) {
    case EW_ADD: return ew_kinds<T, NC, EW_ADD>(n, x, x_mc, y, y_mc, out, s);
    case EW_MUL: return ew_kinds<T, NC, EW_MUL>(n, x, x_mc, y, y_mc, out, s);
    case EW_DIV: return ew_kinds<T, NC, EW_DIV>(n, x, x_mc, y, y_mc, out, s);
    case EW_MUL_SLOW: return ew_launch<T, NC, EW_MUL_SLOW, true, true, NC>(n, x, y, out, s);
    case EW_SQUARE: return ew_launch<T, NC, EW_SQUARE, true, false, NC>(n, x, nullptr, out, s);
    case EW_RENORM: return renorm_dispatch<T, NC, EW_RENORM>(nc_out, n, x, out, s);
    case EW_SIMPLE_RENORM: return renorm_dispatch<T, NC, EW_SIMPLE_RENORM>(nc_out, n, x, out, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t ew_dispatch(int op, int nc, int nc_out, int64_t n, const void *x, int x_mc, const void *y,
                              int y_mc, void *out, hipStream_t s) {
  switch (nc) {
    case 1: return ew_dispatch_nc<T, 1>(op, nc_out, n, x, x_mc, y, y_mc, out, s);
    case 2: return ew_dispatch_nc<T, 2>(op, nc_out, n, x, x_mc, y, y_mc, out, s);
    case 3: return ew_dispatch_nc<T, 3>(op, nc_out, n, x, x_mc, y, y_mc, out, s);
    case 4: return ew_dispatch_nc<T, 4>(op, nc_out, n, x, x_mc, y, y_mc, out, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_elementwise(int dtype, int op, int nc, int nc_out, int64_t n, const void *x, int x_mc,
                              const void *y, int y_mc, void *out, hipStream_t stream) {
  if (dtype == 0) return ew_dispatch<_Float16>(op, nc, nc_out, n, x, x_mc, y, y_mc, out, stream);
  if (dtype == 2) return ew_dispatch<double>(op, nc, nc_out, n, x, x_mc, y, y_mc, out, stream);
  return ew_dispatch<float>(op, nc, nc_out, n, x, x_mc, y, y_mc, out, stream);
}

// ---------------------------------------------------------------------------------
// Exp-MCN, binary16
// ---------------------------------------------------------------------------------

// Correctly rounded binary16 exponential for all 65536 encodings, one table per
// device.  e^x is evaluated in binary64 (error below 2^-50 relative) and rounded once
// to binary16.  Over all finite binary16 x, e^x lies at least 2^-26.4 (relative) away
// from any binary16 rounding boundary, so the binary64 evaluation always rounds to
// the correctly rounded binary16 value.
__device__ _Float16 g_exp16_table[65536];

__global__ __launch_bounds__(256) void exp16_table_kernel(_Float16 *tab) {
  const int h = blockIdx.x * 256 + threadIdx.x;
  const unsigned short bits = (unsigned short)h;
  _Float16 x;
  __builtin_memcpy(&x, &bits, 2);
  tab[h] = (_Float16)exp((double)x);
}

static std::mutex g_exp_mutex;
static _Float16 *g_exp_table_ptr[64];
static std::atomic<bool> g_exp_ready[64];

static hipError_t exp_table(_Float16 **tab, hipStream_t s) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (!g_exp_ready[dev].load(std::memory_order_acquire)) {
    std::lock_guard<std::mutex> lock(g_exp_mutex);
    if (!g_exp_ready[dev].load(std::memory_order_relaxed)) {
      void *p = nullptr;
      err = hipGetSymbolAddress(&p, HIP_SYMBOL(g_exp16_table));
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(exp16_table_kernel, dim3(65536 / 256), dim3(256), 0, s, (_Float16 *)p);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
      // the table must be complete before any stream reads it
      err = hipStreamSynchronize(s);
      if (err != hipSuccess) return err;
      g_exp_table_ptr[dev] = (_Float16 *)p;
      g_exp_ready[dev].store(true, std::memory_order_release);
    }
  }
  *tab = g_exp_table_ptr[dev];
  return hipSuccess;
}

constexpr int EXP_THREADS = 1024;


// The LDS copy of the table covers |x| < 32 (exponent fields 0..19 of both signs, 80
// KiB); outside it e^x is +inf (x >= 32), +0 (x <= -32) or NaN, which is what the
// full table holds there.
constexpr int EXP_LDS_MAG = 20 << 10;  // magnitudes below 0x5000: |x| < 32

__device__ __forceinline__ unsigned exp16_bits(_Float16 v) {
  unsigned short b;
  __builtin_memcpy(&b, &v, 2);
  return b;
}

// |x| <= 2^-12 (binary16 magnitude bits <= 0x0C00): e^x lies in
// [1 - 2^-12 + 2^-26, 1 + 2^-12 + 2^-24], inside the interval (1 - 2^-12, 1 + 2^-11)
// of reals that round to 1, so its binary16 exponential is exactly 1.
constexpr unsigned EXP16_ONE_MAG = 0x0C00u;

// Table slot of an in-range bit pattern: positive half at 0, negative half after it.
__device__ __forceinline__ _Float16 exp16_fast(const _Float16 *tab, unsigned b) {
  return tab[(b & 0x7fffu) + (b >> 15) * (unsigned)EXP_LDS_MAG];
}

// Any bit pattern: +inf for x >= 32, +0 for x <= -32, NaN for NaN.
__device__ __forceinline__ _Float16 exp16_any(const _Float16 *tab, unsigned b) {
  const unsigned mag = b & 0x7fffu;
  if (mag < (unsigned)EXP_LDS_MAG) return exp16_fast(tab, b);
  _Float16 v;
  const unsigned short bs = (unsigned short)b;
  __builtin_memcpy(&v, &bs, 2);
  if (mag > 0x7c00u) return v;
  return (b >> 15) ? _Float16(0) : _Float16(__builtin_inff16());
}

template <int NC, int W>
__global__ __launch_bounds__(EXP_THREADS) void exp16_kernel(const _Float16 *x, _Float16 *out, int64_t n,
                                                            const _Float16 *table) {
  __shared__ uint4 lds_raw[2 * EXP_LDS_MAG * 2 / 16];
  // positive half: table[0 .. EXP_LDS_MAG), negative half: table[0x8000 ..)
  {
    const uint4 *gp = reinterpret_cast<const uint4 *>(table);
    const uint4 *gn = reinterpret_cast<const uint4 *>(table + 0x8000);
    constexpr int H = EXP_LDS_MAG * 2 / 16;  // uint4 per half
    for (int i = threadIdx.x; i < 2 * H; i += EXP_THREADS) lds_raw[i] = i < H ? gp[i] : gn[i - H];
  }
  __syncthreads();
  const _Float16 *tab = reinterpret_cast<const _Float16 *>(lds_raw);
  const int64_t nchunk = n / W;
  const int64_t stride = (int64_t)gridDim.x * EXP_THREADS;
  const int64_t tid = (int64_t)blockIdx.x * EXP_THREADS + threadIdx.x;
  // UU chunks of WW elements at element indices e0[u]: loads, then arithmetic and stores.
  auto loads = [&](const int64_t *e0, auto wtag, auto utag,
                   Pack<_Float16, decltype(wtag)::value> (&xa)[decltype(utag)::value][NC]) {
    constexpr int WW = decltype(wtag)::value;
    constexpr int UU = decltype(utag)::value;
#pragma unroll
    for (int u = 0; u < UU; ++u)
#pragma unroll
      for (int c = 0; c < NC; ++c) xa[u][c] = load_pack<_Float16, WW>(x + c * n + e0[u]);
  };
  auto compute = [&](const int64_t *e0, auto wtag, auto utag,
                     const Pack<_Float16, decltype(wtag)::value> (&xa)[decltype(utag)::value][NC]) {
    constexpr int WW = decltype(wtag)::value;
    constexpr int UU = decltype(utag)::value;
    Pack<_Float16, WW> res[UU][NC];
    if constexpr (NC == 1) {
#pragma unroll
      for (int u = 0; u < UU; ++u)
#pragma unroll
        for (int w = 0; w < WW; ++w) {
          const unsigned b = exp16_bits(xa[u][0].v[w]);
          res[u][0].v[w] = (b & 0x7fffu) < (unsigned)EXP_LDS_MAG ? exp16_fast(tab, b) : exp16_any(tab, b);
        }
    } else {
      // All components but the last: h = (e^x_0), grown by ScalingN(expand) to nc-1
      // components.  `last_one` stays set while every element of the lane has a last
      // component with |x| <= 2^-12 (its exponential is exactly 1 in binary16) and a
      // finite h: ScalingN of a compact h by exactly 1 with expand is h followed by +0.
      _Float16 hh[UU][WW][NC - 1];
      bool last_one = true;
#pragma unroll
      for (int u = 0; u < UU; ++u)
#pragma unroll
        for (int w = 0; w < WW; ++w) {
          _Float16 ex[NC - 1];
          unsigned bits[NC - 1], big = 0;
#pragma unroll
          for (int c = 0; c < NC - 1; ++c) {
            bits[c] = exp16_bits(xa[u][c].v[w]);
            big = big > (bits[c] & 0x7fffu) ? big : (bits[c] & 0x7fffu);
          }
          if (__builtin_expect(big < (unsigned)EXP_LDS_MAG, 1)) {
#pragma unroll
            for (int c = 0; c < NC - 1; ++c) ex[c] = exp16_fast(tab, bits[c]);
          } else {
#pragma unroll
            for (int c = 0; c < NC - 1; ++c) ex[c] = exp16_any(tab, bits[c]);
          }
          const _Float16 h0[1] = {ex[0]};
          exp_chain<_Float16, NC - 1, 1>(h0, ex, hh[u][w]);
          const unsigned lastmag = exp16_bits(xa[u][NC - 1].v[w]) & 0x7fffu;
          last_one = last_one && lastmag <= EXP16_ONE_MAG && __builtin_isfinite((float)hh[u][w][0]);
        }
      if (__all(last_one)) {
#pragma unroll
        for (int u = 0; u < UU; ++u)
#pragma unroll
          for (int w = 0; w < WW; ++w) {
#pragma unroll
            for (int c = 0; c < NC - 1; ++c) res[u][c].v[w] = hh[u][w][c];
            res[u][NC - 1].v[w] = _Float16(0);
          }
      } else {
#pragma unroll
        for (int u = 0; u < UU; ++u)
#pragma unroll
          for (int w = 0; w < WW; ++w) {
            const unsigned b = exp16_bits(xa[u][NC - 1].v[w]);
            const _Float16 e = (b & 0x7fffu) < (unsigned)EXP_LDS_MAG ? exp16_fast(tab, b) : exp16_any(tab, b);
            _Float16 g[NC];
            scaling_n<_Float16, NC - 1, NC>(hh[u][w], e, g);
#pragma unroll
            for (int c = 0; c < NC; ++c) res[u][c].v[w] = g[c];
          }
      }
    }
#pragma unroll
    for (int u = 0; u < UU; ++u)
#pragma unroll
      for (int c = 0; c < NC; ++c) store_pack<_Float16, WW>(out + c * n + e0[u], res[u][c]);
  };
  using IW = std::integral_constant<int, W>;
  using I1 = std::integral_constant<int, 1>;
  // Grid-stride over chunks, software-pipelined one chunk deep: the next chunk's loads
  // are issued before the current chunk's arithmetic, so HBM requests stay in flight
  // while the wave computes (at nc = 3 the registers, 80 per lane, leave room for one
  // workgroup of 16 waves per CU; measured at 2^26 elements, nc = 3: 148 -> 140 us
  // against two chunks per step without the pipeline).
  int64_t ch = tid;
  if (ch < nchunk) {
    Pack<_Float16, W> cur[1][NC];
    int64_t e0[1] = {ch * W};
    loads(e0, IW(), I1(), cur);
    while (true) {
      const int64_t nx = ch + stride;
      const bool more = nx < nchunk;
      Pack<_Float16, W> nxt[1][NC];
      const int64_t e1[1] = {nx * W};
      if (more) loads(e1, IW(), I1(), nxt);
      compute(e0, IW(), I1(), cur);
      if (!more) break;
      ch = nx;
      e0[0] = e1[0];
#pragma unroll
      for (int c = 0; c < NC; ++c) cur[0][c] = nxt[0][c];
    }
  }
  if constexpr (W > 1) {
    const int64_t tail = n - nchunk * W;
    if (tid < tail) {
      const int64_t e0[1] = {nchunk * W + tid};
      Pack<_Float16, 1> xt[1][NC];
      loads(e0, I1(), I1(), xt);
      compute(e0, I1(), I1(), xt);
    }
  }
}

template <int NC>
static hipError_t exp16_launch(int64_t n, const void *x, void *out, const _Float16 *tab, hipStream_t s) {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  bool vec = (n % 8 == 0) && ((uintptr_t)x % 16 == 0) && ((uintptr_t)out % 16 == 0);
  int64_t work = vec ? n / 8 : n;
  int64_t blocks = (work + EXP_THREADS - 1) / EXP_THREADS;
  if (blocks > 2 * cus) blocks = 2 * cus;  // at most two resident per CU (80 KiB of LDS each)
  if (blocks < 1) blocks = 1;
  if (vec)
    hipLaunchKernelGGL((exp16_kernel<NC, 8>), dim3(blocks), dim3(EXP_THREADS), 0, s, (const _Float16 *)x,
                       (_Float16 *)out, n, tab);
  else
    hipLaunchKernelGGL((exp16_kernel<NC, 1>), dim3(blocks), dim3(EXP_THREADS), 0, s, (const _Float16 *)x,
                       (_Float16 *)out, n, tab);
  return hipGetLastError();
}

hipError_t launch_exp_f32(int nc, int64_t n, const void *x, void *out, hipStream_t stream) {
  switch (nc) {
    case 1: return ew_launch<float, 1, EW_EXP, true, false, 1>(n, x, nullptr, out, stream);
    case 2: return ew_launch<float, 2, EW_EXP, true, false, 2>(n, x, nullptr, out, stream);
    case 3: return ew_launch<float, 3, EW_EXP, true, false, 3>(n, x, nullptr, out, stream);
    case 4: return ew_launch<float, 4, EW_EXP, true, false, 4>(n, x, nullptr, out, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_exp_f16(int nc, int64_t n, const void *x, void *out, hipStream_t stream) {
  _Float16 *tab = nullptr;
  hipError_t err = exp_table(&tab, stream);
  if (err != hipSuccess) return err;
  switch (nc) {
    case 1: return exp16_launch<1>(n, x, out, tab, stream);
    case 2: return exp16_launch<2>(n, x, out, tab, stream);
    case 3: return exp16_launch<3>(n, x, out, tab, stream);
    case 4: return exp16_launch<4>(n, x, out, tab, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace mcf
