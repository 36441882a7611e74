// exact.hip -- the exact MC matrix product for binary16 components, on the int8
// matrix cores of gfx950, rounded into nc components.
//
// What is computed.  An MC number is the unevaluated sum of its components (Section
// 2.1), so each output of an MC product has one exact value
//     P_ij = sum_k (sum_c A^(c)_ik)(sum_c B^(c)_kj),
// which MM-MCN (Section 2.2) approximates to about 4 K u^nc sum_k |A_ik||B_kj|
// (Section 2.4).  This product returns P_ij itself, split into nc binary16 components
// by successive round-to-nearest-even: c_0 = RN(P), c_1 = RN(P - c_0), ...  Readings
// fixed here: an overflowing c_0 gives (+-inf, +0, ...); an output whose row of A or
// column of B holds an infinite or NaN component is NaN in every component.
//
// How.  Every binary16 value is an integer multiple of 2^-24, so an MC entry with at
// most four components is an exact integer X = sum_c x_c 2^24 with |X| < 2^42.  X is
// cut into XD = 6 balanced base-256 digits d_s in [-128, 127] (X = sum_s d_s 256^s),
// stored as int8 planes.  Then
//     P_ij 2^48 = sum_{s,t} 256^(s+t) sum_k DA[s]_ik DB[t]_kj,
// and every inner sum is an int8 x int8 contraction with int32 accumulation: exact
// as long as it cannot overflow.  Each product is at most 2^14 in magnitude and at
// most DM digit pairs share a shift class s + t, where DM is the number of digit
// levels a code path handles, so a chunk of 2^31 / (DM 2^14) reduction steps
// cannot overflow: 32768 for DM = 3, 16384 for DM = 4 and 6.  The classes are combined
// exactly in 128-bit integers (|P 2^48| < K 2^84 < 2^127 for K <= 2^40) and rounded in
// integer arithmetic.
//
// Digit layout ("fragment order").  Planes are cut into blocks of 16 rows x 64 k
// (1 KiB); inside a block, byte (r, k) sits at ((k / 16) * 16 + r) * 16 + k % 16, so
// that the 64 lanes of a wavefront read a block as one contiguous KiB with lane l
// holding row l % 16, k = 16 (l / 16) .. 16 (l / 16) + 15 -- the operand layout of
// v_mfma_i32_16x16x64_i8.  Block (s, kb, rb) of an operand with RB row blocks and KB
// k blocks starts at ((s * KB + kb) * RB + rb) KiB.
//
// Kernels: xs_init clears the level statistics and the non-finite flags; xs_slice
// writes the digit planes of both operands (four bytes of every level per lane, so
// that stores are contiguous) and records, per operand, the lowest and highest
// digit level in use; xm_kernel runs the contraction over the levels in use, with one
// code path each for operands whose digits span at most three levels (DM = 3), at most
// four (DM = 4) and up to six (DM = 6), chosen on the device from the statistics so
// that the host never waits; xm_finish adds K-chunk partial sums when K exceeds one
// chunk.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_internal.hpp"

namespace mcf {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __int128 i128;
typedef unsigned __int128 u128;

constexpr int XD = 6;                    // digits per entry
constexpr int XPAD = 128;                // row padding of the digit planes
constexpr int XKSTEP = 64;               // k per matrix-core instruction (one k block)
constexpr int XS_THREADS = 256;

// k per int32 accumulation chunk of a code path handling DM levels
__host__ __device__ constexpr int64_t x_chunk(int dm) { return dm <= 3 ? 32768 : 16384; }

// Statistics, four kinds: [0] A's highest level + 1, [1] B's, [2] XD - A's lowest
// level, [3] XD - B's lowest level, each max-reduced from zero.  Each kind is spread
// over XSLOTS words 256 bytes apart (workgroup b updates slot b % XSLOTS), so that
// concurrent updates do not all meet on one address; readers take the maximum over
// the slots.  Word (kind, slot) is at index (kind * XSLOTS + slot) * 64.
constexpr int XSLOTS = 64;
// After the slots, one word set to 1 when either operand holds a non-finite component.
constexpr int XBADW = 4 * XSLOTS * 64;
constexpr int XSTAT_WORDS = XBADW + 64;

// binary16 bits -> the exact integer value * 2^24 (finite inputs)
__device__ __forceinline__ int64_t f16_units(uint32_t b) {
  const uint32_t e = (b >> 10) & 31u, m = b & 1023u;
  const int64_t mag = e == 0 ? (int64_t)m : ((int64_t)(1024u + m) << (e - 1));
  return (b & 0x8000u) ? -mag : mag;
}

__device__ __forceinline__ bool f16_nonfinite(uint32_t b) { return (b & 0x7C00u) == 0x7C00u; }

struct SliceOp {
  const uint16_t *src;   // planes of binary16
  int planes;            // nc for an MC operand, 1 for a plain one
  int kcontig;           // 1: k is the fast index of src; 0: rows are
  int vec;               // 1: rows of src may be read 8 bytes at a time (kcontig, K % 4 == 0, aligned)
  int64_t plane, rs, ks; // element (row, k) of plane c at c*plane + row*rs + k*ks
  int64_t R, Rp;         // rows, rows padded to XPAD
  int8_t *D;             // XD planes of Rp x Kp digits in fragment order
  uint8_t *bad;          // per-row non-finite flags
  uint32_t *stats;       // the statistics block
  int64_t chunks;        // 16-byte chunks per level: Rp * Kp / 16
};

// Level statistics of a workgroup: wavefront maxima, then the workgroup maximum, then
// one atomic maximum per kind into the workgroup's slot (no value returned, so the
// workgroup does not wait for it; the XSLOTS slots keep same-address atomics few).
// Every lane of the workgroup must call this.
__device__ __forceinline__ void x_stats(uint32_t *stats, int kind_hi, int kind_lo, uint32_t top, uint32_t low) {
  __shared__ uint32_t red[2][XS_THREADS / 64];
  const uint32_t wtop = __ockl_wfred_max_u32(top);
  const uint32_t wlow = __ockl_wfred_max_u32(XD - low);
  const int wave = threadIdx.x / 64;
  if (threadIdx.x % 64 == 0) {
    red[0][wave] = wtop;
    red[1][wave] = wlow;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t bt = 0, bl = 0;
    for (int w = 0; w < XS_THREADS / 64; ++w) {
      bt = max(bt, red[0][w]);
      bl = max(bl, red[1][w]);
    }
    const int slot = (int)(blockIdx.x % XSLOTS) * 64;
    uint32_t *hi = stats + (kind_hi * XSLOTS) * 64 + slot, *lo = stats + (kind_lo * XSLOTS) * 64 + slot;
    if (bt) atomicMax(hi, bt);
    if (bl) atomicMax(lo, bl);
  }
}

__global__ void xs_init(uint32_t *stats, uint8_t *bad_a, int64_t na, uint8_t *bad_b, int64_t nb) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = t; i < 4 * XSLOTS; i += stride) stats[i * 64] = 0;
  if (t == 0) stats[XBADW] = 0;
  for (int64_t i = t; i < na; i += stride) bad_a[i] = 0;
  for (int64_t i = t; i < nb; i += stride) bad_b[i] = 0;
}

// Balanced digits without per-digit arithmetic: with Y = X + 128 (1 + 256 + ... +
// 256^5), which is non-negative for |X| < 2^47, byte s of Y is d_s + 128, so the int8
// digit d_s is byte s of Y with its top bit flipped.
constexpr uint64_t XBIAS = 0x808080808080ull;

// The exact integers (units of 2^-24) of entries (row, k0 .. k0+3) of an operand with
// P planes; p points at entry (row, k0) of plane 0.  All loads are issued first.
template <int P>
__device__ __forceinline__ void slice_entries(const SliceOp &o, const uint16_t *p, int64_t k0, int64_t K,
                                              int64_t (&X)[4], bool &bad) {
  uint32_t bits[P][4];
  if (o.vec && k0 + 4 <= K) {
#pragma unroll
    for (int c = 0; c < P; ++c) {
      const uint2 v = *(const uint2 *)(p + c * o.plane);
#pragma unroll
      for (int j = 0; j < 4; ++j) bits[c][j] = ((j < 2 ? v.x : v.y) >> (16 * (j % 2))) & 0xFFFFu;
    }
  } else {
    // an entry beyond K reads the operand's first entry instead and is discarded
#pragma unroll
    for (int c = 0; c < P; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool ok = k0 + j < K;
        const uint32_t v = ok ? p[c * o.plane + j * o.ks] : o.src[0];
        bits[c][j] = ok ? v : 0u;
      }
  }
#pragma unroll
  for (int c = 0; c < P; ++c)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (f16_nonfinite(bits[c][j])) bad = true;
      else X[j] += f16_units(bits[c][j]);
    }
}

// Lane t writes bytes 4 (t % 4) .. 4 (t % 4) + 3 of 16-byte chunk t / 4 of every level
// plane.  In fragment order chunk u is row block rb = (u / 64) % RB, k block
// kb = u / (64 RB), and inside the block lane l = u % 64 holds row 16 rb + l % 16,
// k = 64 kb + 16 (l / 16) .. + 15.  Entries beyond R or K are zero.
__global__ __launch_bounds__(XS_THREADS) void xs_slice(SliceOp a, SliceOp b, int64_t K, int64_t Kp,
                                                       int64_t a_blocks) {
  const bool is_a = blockIdx.x < a_blocks;
  const SliceOp &o = is_a ? a : b;
  const int64_t t = (int64_t)(is_a ? blockIdx.x : blockIdx.x - a_blocks) * XS_THREADS + threadIdx.x;
  uint32_t top = 0, low = XD;
  if (t < 4 * o.chunks) {
    const int64_t u = t / 4;
    const int part = (int)(t % 4);
    const int64_t RB = o.Rp / 16;
    const int64_t blk = u / 64;
    const int l = (int)(u % 64);
    const int64_t kb = blk / RB, rb = blk - kb * RB;
    const int64_t row = rb * 16 + l % 16;
    const int64_t k0 = kb * 64 + 16 * (l / 16) + 4 * part;
    int64_t X[4] = {0, 0, 0, 0};
    bool bad = false;
    if (row < o.R) {
      // Every load of the lane is issued before any is used, so the lane waits for
      // memory once rather than once per plane (the plane count is uniform per
      // workgroup: one operand per workgroup).
      const uint16_t *p = o.src + row * o.rs + k0 * o.ks;
      switch (o.planes) {
        case 1: slice_entries<1>(o, p, k0, K, X, bad); break;
        case 2: slice_entries<2>(o, p, k0, K, X, bad); break;
        case 3: slice_entries<3>(o, p, k0, K, X, bad); break;
        default: slice_entries<4>(o, p, k0, K, X, bad); break;
      }
      if (bad) {
        o.bad[row] = 1;
        o.stats[XBADW] = 1;
      }
    }
    uint32_t lo[4], hi[4];
    uint64_t any = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t D = ((uint64_t)X[j] + XBIAS) ^ XBIAS;  // the digits as bytes; zero digits are zero bytes
      any |= D;
      lo[j] = (uint32_t)D;
      hi[j] = (uint32_t)(D >> 32);
      const int bl = D ? 64 - __builtin_clzll(D) : 0;
      top = max(top, (uint32_t)((bl + 7) / 8));
    }
    if (any) low = (uint32_t)(__builtin_ctzll(any) / 8);
    const int64_t level = o.chunks * 16;
    int8_t *dst = o.D + t * 4;
#pragma unroll
    for (int s = 0; s < XD; ++s) {
      uint32_t v = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t byte = s < 4 ? (lo[j] >> (8 * s)) & 0xFFu : (hi[j] >> (8 * (s - 4))) & 0xFFu;
        v |= byte << (8 * j);
      }
      *(uint32_t *)(dst + s * level) = v;
    }
  }
  // every lane of the workgroup takes part in the reductions
  x_stats(o.stats, is_a ? 0 : 1, is_a ? 2 : 3, top, low);
}

// ---------------------------------------------------------------------------------
// rounding of an exact value (units of 2^-48) into binary16
// ---------------------------------------------------------------------------------

__device__ __forceinline__ int bitlen(u128 a) {
  const uint64_t hi = (uint64_t)(a >> 64), lo = (uint64_t)a;
  return hi ? 128 - __builtin_clzll(hi) : (lo ? 64 - __builtin_clzll(lo) : 0);
}

// Rounds rem * 2^-48 to the nearest binary16 (ties to even, gradual underflow),
// subtracts the rounded value from rem and returns its bits; on overflow returns the
// infinity of rem's sign and sets ovf.  W is the integer type of rem (int64_t when
// |rem| < 2^62, which cannot overflow binary16, else i128).
template <typename W, typename UW>
__device__ __forceinline__ uint32_t take_f16(W &rem, bool &ovf) {
  if (rem == 0) return 0;
  const bool neg = rem < 0;
  const UW a = neg ? (UW)0 - (UW)rem : (UW)rem;
  int e;
  if constexpr (sizeof(W) == 8) e = 63 - __builtin_clzll((uint64_t)a);
  else e = bitlen(a) - 1;
  const int qe = e - 10 > 24 ? e - 10 : 24;  // quantum 2^(qe-48): 11 significant bits, 2^-24 floor
  UW n = a >> qe;
  const UW r = a - (n << qe);
  const UW half = (UW)1 << (qe - 1);
  if (r > half || (r == half && (n & 1))) n += 1;
  // binary16 bits rise by 1024 per binade and by 1 per quantum, continuously through
  // the subnormals: bits = (qe - 24) * 1024 + n
  const int64_t enc = (int64_t)(qe - 24) * 1024 + (int64_t)n;
  const uint32_t sign = neg ? 0x8000u : 0u;
  if (enc >= 0x7C00) {
    ovf = true;
    return sign | 0x7C00u;
  }
  const W v = (W)(n << qe);
  rem = neg ? rem + v : rem - v;
  return sign | (uint32_t)enc;
}

// Splits V * 2^-48 into nc binary16 components by successive rounding and stores them
// (NaN in every component when nan is set).
__device__ __forceinline__ void store_split(i128 V, int nc, bool nan, uint16_t *C, int64_t plane, int64_t idx) {
  uint32_t bits[4] = {0, 0, 0, 0};
  if (nan) {
    for (int c = 0; c < 4; ++c) bits[c] = 0x7E00;
  } else {
    const u128 a = V < 0 ? (u128)0 - (u128)V : (u128)V;
    bool ovf = false;
    if ((a >> 62) == 0) {  // the common case: 64-bit arithmetic
      int64_t v = (int64_t)V;
      for (int c = 0; c < nc; ++c) bits[c] = take_f16<int64_t, uint64_t>(v, ovf);
    } else {
      for (int c = 0; c < nc; ++c) bits[c] = ovf ? 0u : take_f16<i128, u128>(V, ovf);
    }
  }
  for (int c = 0; c < nc; ++c) C[c * plane + idx] = (uint16_t)bits[c];
}

// ---------------------------------------------------------------------------------
// the contraction
// ---------------------------------------------------------------------------------

struct XmArgs {
  const int8_t *DA, *DB;
  const uint8_t *bad_a, *bad_b;
  const uint32_t *stats;
  int64_t M, N, Kp, Mp, Np;
  int nc;
  uint16_t *C;       // [nc][M][N]
  int cvec;          // rows of C may be written 16 bytes at a time (N % 8 == 0, C aligned)
  const uint16_t *bias;  // [nc][N] MC row added to every output row, or null
  i128 *partial;     // [S][M][N] when the code path that runs needs S > 1 chunks
  int64_t tiles_n;   // workgroup tiles along N
};

struct XLevels {
  int loA, loB, nA, nB;
  bool small;   // both operands within three levels: the DM = 3 code path runs
  bool anybad;  // some input component is infinite or NaN
};

// The first wavefront reads slot l of each kind in lane l and reduces; the result
// reaches the other wavefronts through LDS.  Every lane of the workgroup must call
// this (it holds a barrier).
__device__ __forceinline__ XLevels x_levels(const uint32_t *stats) {
  __shared__ uint32_t sw[5];
  XLevels v;
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
#pragma unroll
    for (int kind = 0; kind < 4; ++kind) {
      const uint32_t m = __ockl_wfred_max_u32(stats[(kind * XSLOTS + l) * 64]);
      if (l == 0) sw[kind] = m;
    }
    if (l == 0) sw[4] = stats[XBADW];
  }
  __syncthreads();
  v.anybad = sw[4] != 0;
  uint32_t w[4];
#pragma unroll
  for (int kind = 0; kind < 4; ++kind) w[kind] = sw[kind];
  const int hiA = (int)w[0], hiB = (int)w[1];
  v.loA = XD - (int)w[2];
  v.loB = XD - (int)w[3];
  v.nA = hiA > v.loA ? hiA - v.loA : 0;
  v.nB = hiB > v.loB ? hiB - v.loB : 0;
  v.small = v.nA <= 3 && v.nB <= 3;
  return v;
}

// The bias of column col as an exact integer in units of 2^-24 (0 without a bias);
// bad is set when one of its components is infinite or NaN.
__device__ __forceinline__ int64_t bias_units(const XmArgs &g, int64_t col, bool &bad) {
  if (g.bias == nullptr) return 0;
  int64_t X = 0;
  for (int c = 0; c < g.nc; ++c) {
    const uint32_t b = g.bias[c * g.N + col];
    if (f16_nonfinite(b)) bad = true;
    else X += f16_units(b);
  }
  return X;
}

// Branch-free rounding for |rem| < 2^62 (which cannot overflow binary16): as
// take_f16 with the sign folded in by two's-complement identities.
__device__ __forceinline__ uint32_t take_f16_fast(int64_t &rem) {
  const uint64_t sgn = (uint64_t)(rem >> 63);      // 0 or all ones
  const uint64_t a = ((uint64_t)rem ^ sgn) - sgn;  // |rem|
  const int e = 63 - __builtin_clzll(a | 1);
  const int qe = e - 10 > 24 ? e - 10 : 24;
  const uint64_t n0 = a >> qe;
  const uint64_t r = a - (n0 << qe);
  const uint64_t half = 1ull << (qe - 1);
  const uint64_t n = n0 + (uint64_t)((r > half) | ((r == half) & (bool)(n0 & 1)));
  const uint64_t v = n << qe;
  rem -= (int64_t)((v ^ sgn) - sgn);  // rem - sign(rem) v
  return ((uint32_t)sgn & 0x8000u) | (uint32_t)((qe - 24) * 1024 + (int)n);
}

// take_f16_fast for a remainder held as a binary64 value (d = rem 2^-48, exact: the
// remainder is an integer below 2^53 in magnitude): d is rounded to binary32 toward
// odd (round to nearest, then, if inexact, the neighbour with an odd last bit), which
// keeps the information a second rounding to binary16 needs (24 >= 11 + 2 bits), and
// then to binary16; d minus the binary16 value is exact in binary64.
__device__ __forceinline__ uint32_t take_f16_binary64(double &d) {
  const float f = (float)d;
  const double fd = (double)f;
  uint32_t fb = __builtin_bit_cast(uint32_t, f);
  if (fd != d && (fb & 1u) == 0u) fb = __builtin_fabs(fd) < __builtin_fabs(d) ? fb + 1u : fb - 1u;
  const _Float16 h = (_Float16)__builtin_bit_cast(float, fb);
  d -= (double)(float)h;
  return __builtin_bit_cast(uint16_t, h);
}

// Epilogue of one wavefront's WTR x WTC tiles of 16 x 16 outputs (accumulator element
// i of lane l is row 4 (l / 16) + i, column l % 16 of its tile, one int32 accumulator
// per tile and shift class).  stage: 16-byte aligned LDS of at least 2560 bytes owned by
// this wavefront.
template <int DM, int WTR, int WTC>
__device__ __forceinline__ void xm_epilogue(const XmArgs &g, const XLevels &lv, v4i (&acc)[2 * DM - 1][WTR][WTC],
                                            int64_t row0, int64_t col0, int64_t chunk, int64_t S, uint16_t *st) {
  constexpr int NCLS = 2 * DM - 1;
  const int lane = threadIdx.x % 64;
  // V = sum_q acc[q] 256^q 2^shift0 (+ bias 2^24) exactly.  First a conservative test
  // that every value of the wavefront stays below 2^62 in magnitude: each term is below
  // 2^(bitlen|acc[q]| + 8 q + shift0) and there are at most 12 terms.  Then, when it
  // holds, V is summed in wrapping 64-bit arithmetic, which is exact because the true
  // sum fits; otherwise in 128-bit integers.
  const int shift0 = 8 * (lv.loA + lv.loB);
  bool fits = true;
  // The test, term by term: a non-zero term with bit length b at shift h needs
  // b + h + 4 <= 62, i.e. its magnitude below 2^(58 - h).  lim(h) is the largest
  // magnitude allowed (uniform across the wavefront).
  auto lim = [&](int h) -> uint64_t {
    const int e = 58 - h;
    return e <= 0 ? 0ull : (e >= 64 ? ~0ull : (1ull << e) - 1);
  };
  // each lane's columns: their bias (units of 2^-24, added 24 bits up) joins the sum
  int64_t bu[WTC];
#pragma unroll
  for (int c = 0; c < WTC; ++c) {
    const int64_t col = col0 + 16 * c + lane % 16;
    bool bb = false;
    bu[c] = col < g.N ? bias_units(g, col, bb) : 0;
    const uint64_t ab = (uint64_t)(bu[c] < 0 ? -bu[c] : bu[c]);
    fits = fits && !bb && ab <= lim(24 + shift0);
  }
  uint32_t lq[NCLS];
#pragma unroll
  for (int q = 0; q < NCLS; ++q) {
    const uint64_t l = lim(8 * q + shift0);
    lq[q] = l > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)l;
  }
#pragma unroll
  for (int r = 0; r < WTR; ++r)
#pragma unroll
    for (int c = 0; c < WTC; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int q = 0; q < NCLS; ++q) {
          const int32_t x = acc[q][r][c][i];
          const uint32_t ux = (uint32_t)x, ax = x < 0 ? 0u - ux : ux;  // |x|, also for -2^31
          fits = fits && ax <= lq[q];
        }
  const bool fast = __all(fits) && !lv.anybad && S == 1;  // uniform across the wavefront
  const int64_t MN = g.M * g.N;
  if (fast) {
    // V in wrapping 64-bit arithmetic (exact: |V| < 2^62), then one component at a
    // time: each lane rounds its outputs and writes them to the wavefront's LDS tile,
    // which goes back to C row by row in 16-byte pieces.
    int64_t v[WTR][WTC][4];
#pragma unroll
    for (int r = 0; r < WTR; ++r)
#pragma unroll
      for (int c = 0; c < WTC; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          uint64_t vu = (uint64_t)bu[c] << 24;
#pragma unroll
          for (int q = 0; q < NCLS; ++q) {
            const int sh = 8 * q + shift0;
            vu += sh < 64 ? (uint64_t)(int64_t)acc[q][r][c][i] << sh : 0;
          }
          v[r][c][i] = (int64_t)vu;
        }
    // When every |V| of the wavefront is below 2^53 (the usual case: V is the output in
    // units of 2^-48), V * 2^-48 is exact in binary64 and the components are taken in
    // binary64 arithmetic, a third of the integer path's instructions.
    bool below53 = true;
    double dv[WTR][WTC][4];
#pragma unroll
    for (int r = 0; r < WTR; ++r)
#pragma unroll
      for (int c = 0; c < WTC; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t x = v[r][c][i];
          below53 = below53 && (uint64_t)(x + (1ll << 53)) < (1ull << 54);
          dv[r][c][i] = __builtin_fma((double)(int32_t)(x >> 32), 0x1p32, (double)(uint32_t)x) * 0x1p-48;
        }
    const bool f64path = __all(below53);
    constexpr int TR = 16 * WTR, TC = 16 * WTC, LD = TC + 8;
    static_assert(TR * LD * 2 <= 2560, "stage tile too small");
    const bool vec = g.cvec && col0 + TC <= g.N;
    for (int k = 0; k < g.nc; ++k) {
      if (f64path) {
#pragma unroll
        for (int r = 0; r < WTR; ++r)
#pragma unroll
          for (int c = 0; c < WTC; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              st[(16 * r + 4 * (lane / 16) + i) * LD + 16 * c + lane % 16] = (uint16_t)take_f16_binary64(dv[r][c][i]);
      } else {
#pragma unroll
        for (int r = 0; r < WTR; ++r)
#pragma unroll
          for (int c = 0; c < WTC; ++c)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              st[(16 * r + 4 * (lane / 16) + i) * LD + 16 * c + lane % 16] = (uint16_t)take_f16_fast(v[r][c][i]);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      uint16_t *Ck = g.C + k * MN;
#pragma unroll
      for (int q0 = 0; q0 < TR * TC / 8; q0 += 64) {
        const int q = q0 + lane;
        const int rr = q / (TC / 8), cc = (q % (TC / 8)) * 8;
        const int64_t row = row0 + rr;
        if (q < TR * TC / 8 && row < g.M) {
          const uint16_t *src = st + rr * LD + cc;
          if (vec) {
            *(uint4 *)(Ck + row * g.N + col0 + cc) = *(const uint4 *)src;
          } else {
            for (int e = 0; e < 8; ++e)
              if (col0 + cc + e < g.N) Ck[row * g.N + col0 + cc + e] = src[e];
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    return;
  }
#pragma unroll
  for (int r = 0; r < WTR; ++r) {
#pragma unroll
    for (int c = 0; c < WTC; ++c) {
      const int64_t col = col0 + 16 * c + lane % 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t row = row0 + 16 * r + 4 * (lane / 16) + i;
        if (row < g.M && col < g.N) {
          const int64_t idx = row * g.N + col;
          // four consecutive classes fit one int64 (|acc| < 2^31, relative shifts up
          // to 24 bits); the groups are combined 32 bits apart in 128 bits
          constexpr int NG = (NCLS + 3) / 4;
          int64_t part[NG];
#pragma unroll
          for (int q = 0; q < NG; ++q) part[q] = 0;
#pragma unroll
          for (int q = 0; q < NCLS; ++q) part[q / 4] += (int64_t)acc[q][r][c][i] * ((int64_t)1 << (8 * (q % 4)));
          u128 Vu = 0;
#pragma unroll
          for (int q = 0; q < NG; ++q) Vu += (u128)(i128)part[q] << (32 * q);
          const i128 V = (i128)(Vu << shift0);
          if (S > 1) {
            g.partial[chunk * MN + idx] = V;  // the bias joins in the finishing kernel
          } else {
            bool bb = false;
            const int64_t b = bias_units(g, col, bb);
            store_split(V + (i128)((u128)(i128)b << 24), g.nc, g.bad_a[row] | g.bad_b[col] | bb, g.C, MN, idx);
          }
        }
      }
    }
  }
}

// One wavefront's WTR x WTC tiles over k blocks [kb0, kb1), operand fragments read
// straight from the digit planes; the fragments of the next k block are loaded while
// the current one is multiplied.
//
// KS = 2: two wavefronts share each tile, one per half of the k blocks (khalf); they
// exchange accumulators through LDS (red: 16 KiB, exact integer sums) so that each
// holds the complete sums of one tile row, and each rounds its row.  Every lane of the
// workgroup must call it then (it holds barriers).
template <int DM, int WTR, int WTC, int KS = 1>
__device__ __forceinline__ void xm_tile(const XmArgs &g, const XLevels &lv, int64_t row0, int64_t col0,
                                        int64_t chunk, int64_t kb0, int64_t kb1, int64_t S, uint16_t *st,
                                        int khalf = 0, int *red = nullptr) {
  constexpr int NCLS = 2 * DM - 1;
  const int lane = threadIdx.x % 64;
  const int64_t KB = g.Kp / 64;
  if constexpr (KS == 2) {
    const int64_t mid = kb0 + (kb1 - kb0 + 1) / 2;
    if (khalf) kb0 = mid;
    else kb1 = mid;
  }
  // the k range is uniform across the wavefront: keep the loop control scalar, so that
  // the loop is not run under an execution mask and the waits for the prefetched
  // fragments are counted
  kb0 = ((int64_t)__builtin_amdgcn_readfirstlane((int)(kb0 >> 32)) << 32) |
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)kb0);
  kb1 = ((int64_t)__builtin_amdgcn_readfirstlane((int)(kb1 >> 32)) << 32) |
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)kb1);

  v4i acc[NCLS][WTR][WTC];
#pragma unroll
  for (int q = 0; q < NCLS; ++q)
#pragma unroll
    for (int r = 0; r < WTR; ++r)
#pragma unroll
      for (int c = 0; c < WTC; ++c) acc[q][r][c] = v4i{0, 0, 0, 0};

  // fragment (level s, k block kb, row block rb) at ((s KB + kb) RB + rb) KiB.  Every
  // level slot up to DM is loaded (a slot beyond the levels in use reads an existing
  // level and is never multiplied), so that the loads of a k block form one straight
  // block of code whose completion the compiler can wait for by count.
  const int64_t RBa = g.Mp / 16, RBb = g.Np / 16;
  const int nA = __builtin_amdgcn_readfirstlane(lv.nA), nB = __builtin_amdgcn_readfirstlane(lv.nB);
  const int loA = __builtin_amdgcn_readfirstlane(lv.loA), loB = __builtin_amdgcn_readfirstlane(lv.loB);
  const int8_t *pa = g.DA + (row0 / 16) * 1024 + lane * 16;
  const int8_t *pb = g.DB + (col0 / 16) * 1024 + lane * 16;
  const int64_t la = KB * RBa * 1024, lb = KB * RBb * 1024;  // level strides
  const int64_t ka = RBa * 1024, kbs = RBb * 1024;          // k-block strides

  auto load = [&](int64_t kb, v4i (&xa)[DM][WTR], v4i (&xb)[DM][WTC]) {
#pragma unroll
    for (int s = 0; s < DM; ++s) {
      const int64_t oa = min(loA + s, XD - 1) * la + kb * ka, ob = min(loB + s, XD - 1) * lb + kb * kbs;
#pragma unroll
      for (int r = 0; r < WTR; ++r) xa[s][r] = *(const v4i *)(pa + oa + r * 1024);
#pragma unroll
      for (int c = 0; c < WTC; ++c) xb[s][c] = *(const v4i *)(pb + ob + c * 1024);
    }
  };
  auto mfmas = [&](const v4i (&xa)[DM][WTR], const v4i (&xb)[DM][WTC]) {
#pragma unroll
    for (int s = 0; s < DM; ++s) {
      if (s < nA) {
#pragma unroll
        for (int t = 0; t < DM; ++t) {
          if (t < nB) {
#pragma unroll
            for (int r = 0; r < WTR; ++r)
#pragma unroll
              for (int c = 0; c < WTC; ++c)
                acc[s + t][r][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xa[s][r], xb[t][c], acc[s + t][r][c], 0, 0, 0);
          }
        }
      }
    }
  };
  // two register sets in alternation (no copies between them): the loads of the next
  // k block are issued before the current block's matrix-core instructions
  v4i fa[DM][WTR], fb[DM][WTC], na[DM][WTR], nb[DM][WTC];
  if (kb0 < kb1) load(kb0, fa, fb);
  for (int64_t kb = kb0; kb < kb1; kb += 2) {
    if (kb + 1 < kb1) load(kb + 1, na, nb);
    mfmas(fa, fb);
    if (kb + 1 >= kb1) break;
    if (kb + 2 < kb1) load(kb + 2, fa, fb);
    mfmas(na, nb);
  }
  if constexpr (KS == 2) {
    // The two wavefronts of a tile split its rows: the one with khalf = h completes tile
    // row h (exact integer sums of both halves' accumulators, exchanged through LDS) and
    // rounds it, so both run the epilogue on half the outputs.
    static_assert(WTR == 2 && WTC * 4 <= 8, "reduction buffer layout");
    const int qw = (threadIdx.x / 64) % 4;
    v4i mine[NCLS][1][WTC];
#pragma unroll
    for (int q = 0; q < NCLS; ++q) {
      // give away the other half's row, keep this half's row
#pragma unroll
      for (int c = 0; c < WTC; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          red[((qw * 2 + khalf) * 8 + c * 4 + i) * 64 + lane] = khalf ? acc[q][0][c][i] : acc[q][1][c][i];
          mine[q][0][c][i] = khalf ? acc[q][1][c][i] : acc[q][0][c][i];
        }
      __syncthreads();
#pragma unroll
      for (int c = 0; c < WTC; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) mine[q][0][c][i] += red[((qw * 2 + (1 - khalf)) * 8 + c * 4 + i) * 64 + lane];
      __syncthreads();
    }
    xm_epilogue<DM, 1, WTC>(g, lv, mine, row0 + 16 * khalf, col0, chunk, S, st);
    return;
  }
  xm_epilogue<DM, WTR, WTC>(g, lv, acc, row0, col0, chunk, S, st);
}

// One workgroup of 4 KS wavefronts per 64 x 64 tile of C; blockIdx.y is the K chunk.
// Operands within three digit levels: each wavefront takes a 32 x 32 quarter (2 x 2
// tiles, five shift classes), with KS = 2 two wavefronts per quarter splitting the k
// blocks (for grids too small to fill the chip).  Within four levels: two passes over
// 64 x 32 halves, each wavefront taking 32 x 16 (2 x 1 tiles, seven classes).
// Otherwise: four passes over the 32 x 32 quarters, each wavefront taking one 16 x 16
// tile (eleven classes).  The second group of wavefronts of a KS = 2 workgroup takes
// part in the three-level path only.
template <int KS>
__global__ __attribute__((amdgpu_flat_work_group_size(1, 256 * KS), amdgpu_waves_per_eu(2))) void xm_kernel(
    XmArgs g) {
  // epilogue staging: 2560 bytes per wavefront; KS = 2 exchange: 16 KiB of the same
  // memory, used before the epilogue
  __shared__ __attribute__((aligned(16))) int8_t smem[KS == 2 ? 8 * 2560 : 4 * 2560];
  const XLevels lv = x_levels(g.stats);
  const int wave = (threadIdx.x / 64) % 4;
  const int khalf = threadIdx.x / 256;
  const int64_t tile = blockIdx.x;
  const int64_t tm = tile / g.tiles_n, tn = tile - tm * g.tiles_n;
  const int64_t KB = g.Kp / 64;
  const int64_t chunk = blockIdx.y;
  const int dm = lv.small ? 3 : (lv.nA <= 4 && lv.nB <= 4 ? 4 : 6);
  const int64_t CKB = x_chunk(dm) / 64;
  const int64_t kb0 = chunk * CKB;
  if (kb0 >= KB && KB > 0) return;  // the grid holds the chunks of the smallest chunk size
  const int64_t kb1 = min(KB, kb0 + CKB);
  const int64_t S = KB == 0 ? 1 : (KB + CKB - 1) / CKB;
  uint16_t *st = (uint16_t *)(smem + (threadIdx.x / 64) * 2560);
  if (dm == 3) {
    xm_tile<3, 2, 2, KS>(g, lv, tm * 64 + (wave / 2) * 32, tn * 64 + (wave % 2) * 32, chunk, kb0, kb1, S, st, khalf,
                         (int *)smem);
    return;
  }
  if (khalf) return;
  if (dm == 4) {
    for (int sub = 0; sub < 2; ++sub)
      xm_tile<4, 2, 1>(g, lv, tm * 64 + (wave / 2) * 32, tn * 64 + sub * 32 + (wave % 2) * 16, chunk, kb0, kb1, S, st);
  } else {
    for (int sub = 0; sub < 4; ++sub)
      xm_tile<6, 1, 1>(g, lv, tm * 64 + (sub / 2) * 32 + (wave / 2) * 16, tn * 64 + (sub % 2) * 32 + (wave % 2) * 16,
                       chunk, kb0, kb1, S, st);
  }
}

__global__ void xm_finish(XmArgs g) {
  const XLevels lv = x_levels(g.stats);  // every lane, before any returns
  const int dm = lv.small ? 3 : (lv.nA <= 4 && lv.nB <= 4 ? 4 : 6);
  const int64_t chunk_kb = x_chunk(dm) / 64;
  const int64_t KB = g.Kp / 64;
  const int64_t S = (KB + chunk_kb - 1) / chunk_kb;
  if (S <= 1) return;  // the product kernel wrote C itself
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = g.M * g.N;
  if (t >= MN) return;
  i128 V = 0;
  for (int64_t s = 0; s < S; ++s) V += g.partial[s * MN + t];
  const int64_t row = t / g.N, col = t - row * g.N;
  bool bb = false;
  const int64_t b = bias_units(g, col, bb);
  store_split(V + (i128)((u128)(i128)b << 24), g.nc, g.bad_a[row] | g.bad_b[col] | bb, g.C, MN, t);
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct XLayout {
  int64_t Mp, Np, Kp, Smax;
  int64_t off_stats, off_bad_a, off_bad_b, off_da, off_db, off_part, total;
};

XLayout x_layout(int64_t M, int64_t N, int64_t K) {
  XLayout L;
  L.Mp = round_up(M, XPAD);
  L.Np = round_up(N, XPAD);
  L.Kp = round_up(K, XKSTEP);
  L.Smax = L.Kp == 0 ? 1 : (L.Kp + x_chunk(6) - 1) / x_chunk(6);
  int64_t o = 0;
  L.off_stats = o;
  o += XSTAT_WORDS * 4;
  L.off_bad_a = o;
  o += round_up(M, 256);
  L.off_bad_b = o;
  o += round_up(N, 256);
  L.off_da = o;
  o += round_up(XD * L.Mp * L.Kp, 256);
  L.off_db = o;
  o += round_up(XD * L.Np * L.Kp, 256);
  L.off_part = o;
  if (L.Smax > 1) o += L.Smax * M * N * (int64_t)sizeof(i128);
  L.total = o;
  return L;
}

}  // namespace

int64_t exact_workspace_bytes(int64_t M, int64_t N, int64_t K) { return x_layout(M, N, K).total; }

hipError_t launch_matmul_exact(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                               int b_mc, int b_trans, const void *bias, void *W, void *C, hipStream_t stream) {
  const XLayout L = x_layout(M, N, K);
  char *w = (char *)W;
  uint32_t *stats = (uint32_t *)(w + L.off_stats);
  uint8_t *bad_a = (uint8_t *)(w + L.off_bad_a), *bad_b = (uint8_t *)(w + L.off_bad_b);
  int8_t *DA = (int8_t *)(w + L.off_da), *DB = (int8_t *)(w + L.off_db);

  {
    const int64_t n = M > N ? M : N;
    const int64_t nb = (n > 4 * XSLOTS ? n : 4 * XSLOTS);
    const int blocks = (int)((nb + 255) / 256 < 1024 ? (nb + 255) / 256 : 1024);
    hipLaunchKernelGGL(xs_init, dim3(blocks), dim3(256), 0, stream, stats, bad_a, M, bad_b, N);
  }
  if (L.Kp > 0) {
    SliceOp a, b;
    a.src = (const uint16_t *)A;
    a.planes = a_mc ? nc : 1;
    a.kcontig = 1;
    a.vec = (K % 4 == 0) && ((uintptr_t)A % 8 == 0);
    a.plane = M * K;
    a.rs = K;
    a.ks = 1;
    a.R = M;
    a.Rp = L.Mp;
    a.D = DA;
    a.bad = bad_a;
    a.stats = stats;
    a.chunks = L.Mp * L.Kp / 16;
    b.src = (const uint16_t *)B;
    b.planes = b_mc ? nc : 1;
    b.kcontig = b_trans ? 1 : 0;
    b.vec = b_trans && (K % 4 == 0) && ((uintptr_t)B % 8 == 0);
    b.plane = K * N;
    b.rs = b_trans ? K : 1;
    b.ks = b_trans ? 1 : N;
    b.R = N;
    b.Rp = L.Np;
    b.D = DB;
    b.bad = bad_b;
    b.stats = stats;
    b.chunks = L.Np * L.Kp / 16;
    const int64_t ab = (4 * a.chunks + XS_THREADS - 1) / XS_THREADS;
    const int64_t bb = (4 * b.chunks + XS_THREADS - 1) / XS_THREADS;
    hipLaunchKernelGGL(xs_slice, dim3((unsigned)(ab + bb)), dim3(XS_THREADS), 0, stream, a, b, K, L.Kp, ab);
  }
  XmArgs g;
  g.DA = DA;
  g.DB = DB;
  g.bad_a = bad_a;
  g.bad_b = bad_b;
  g.stats = stats;
  g.M = M;
  g.N = N;
  g.Kp = L.Kp;
  g.Mp = L.Mp;
  g.Np = L.Np;
  g.nc = nc;
  g.C = (uint16_t *)C;
  g.cvec = (N % 8 == 0) && ((uintptr_t)C % 16 == 0);
  g.bias = (const uint16_t *)bias;
  g.partial = (i128 *)(w + L.off_part);
  {
    g.tiles_n = L.Np / 64;
    const int64_t tiles = (L.Mp / 64) * g.tiles_n;
    // fewer workgroups than two per compute unit: split each tile's k blocks over two
    // wavefronts per quarter
    if (tiles * L.Smax < 512)
      hipLaunchKernelGGL(xm_kernel<2>, dim3((unsigned)tiles, (unsigned)L.Smax), dim3(512), 0, stream, g);
    else
      hipLaunchKernelGGL(xm_kernel<1>, dim3((unsigned)tiles, (unsigned)L.Smax), dim3(256), 0, stream, g);
  }
  if (L.Smax > 1) {
    const int64_t n = M * N;
    hipLaunchKernelGGL(xm_finish, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, g);
  }
  return hipGetLastError();
}

}  // namespace mcf
