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
// cut into XD = 7 balanced base-128 digits d_s in [-64, 63] (X = sum_s d_s 128^s),
// stored as int8 planes D[s][row][k].  Then
//     P_ij 2^48 = sum_{s,t} 128^(s+t) sum_k DA[s]_ik DB[t]_kj,
// and every inner sum is an int8 x int8 contraction with int32 accumulation: exact
// as long as it cannot overflow.  At most 7 digit pairs share a shift class s + t and
// each product is at most 4096 in magnitude, so 65536 reduction steps stay below
// 7 * 4096 * 65536 < 2^31.  The classes are combined exactly in 128-bit integers
// (|P 2^48| < K 2^84 < 2^127 for K <= 2^40) and rounded in integer arithmetic.
//
// Kernels: xs_init clears the level statistics and the non-finite flags; xs_slice
// writes the digit planes of both operands and records, per operand, the lowest and
// highest digit level in use; xm_kernel<DM> runs the contraction over the levels in
// use (two instantiations, DM = 4 for operands whose digits span at most four levels
// and DM = 7 otherwise, both launched: each reads the statistics on the device and
// the one that does not apply returns at once, so the host never waits); xm_finish
// adds K-chunk partial sums when K exceeds one chunk.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_internal.hpp"

namespace mcf {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __int128 i128;
typedef unsigned __int128 u128;

constexpr int XD = 7;                    // digits per entry
constexpr int XPAD = 64;                 // row padding of the digit planes (a workgroup tile)
constexpr int XKSTEP = 64;               // k per matrix-core instruction
constexpr int64_t XKCHUNK = 65536;       // k per int32 accumulation (see the overflow bound above)
constexpr int XS_THREADS = 256;

// statistics words: [0] A's highest level + 1, [1] B's, [2] XD - A's lowest level,
// [3] XD - B's lowest level (all max-reduced from zero)
constexpr int XSTAT_WORDS = 4;

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
  int64_t plane, rs, ks; // element (row, k) of plane c at c*plane + row*rs + k*ks
  int64_t R, Rp;         // rows, rows padded to XPAD
  int8_t *D;             // XD planes of Rp x Kp digits
  uint8_t *bad;          // per-row non-finite flags
  uint32_t *hi, *loinv;  // statistics words of this operand
  int64_t threads;       // Rp * Kp / 16
};

__global__ void xs_init(uint32_t *stats, uint8_t *bad_a, int64_t na, uint8_t *bad_b, int64_t nb) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (t < XSTAT_WORDS) stats[t] = 0;
  for (int64_t i = t; i < na; i += stride) bad_a[i] = 0;
  for (int64_t i = t; i < nb; i += stride) bad_b[i] = 0;
}

// One lane per (row, run of 16 consecutive k): forms the 16 exact integers, cuts them
// into digits and stores 16 bytes per digit plane.  Entries beyond R or K are zero.
__global__ __launch_bounds__(XS_THREADS) void xs_slice(SliceOp a, SliceOp b, int64_t K, int64_t Kp,
                                                       int64_t a_blocks) {
  const bool is_a = blockIdx.x < a_blocks;
  const SliceOp &o = is_a ? a : b;
  const int64_t t = (int64_t)(is_a ? blockIdx.x : blockIdx.x - a_blocks) * XS_THREADS + threadIdx.x;
  const int64_t runs = Kp / 16;
  uint32_t top = 0, low = XD;  // highest level + 1 and lowest non-zero level of this lane
  if (t < o.threads) {
    int64_t row, run;
    if (o.kcontig) {
      row = t / runs;
      run = t - row * runs;
    } else {
      run = t / o.Rp;
      row = t - run * o.Rp;
    }
    const int64_t k0 = run * 16;
    uint32_t dig[XD][4];
#pragma unroll
    for (int s = 0; s < XD; ++s)
#pragma unroll
      for (int w = 0; w < 4; ++w) dig[s][w] = 0;
    bool bad = false;
    if (row < o.R) {
      const uint16_t *p = o.src + row * o.rs;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t k = k0 + j;
        int64_t X = 0;
        if (k < K) {
          for (int c = 0; c < o.planes; ++c) {
            const uint32_t bits = p[c * o.plane + k * o.ks];
            if (f16_nonfinite(bits)) bad = true;
            else X += f16_units(bits);
          }
        }
#pragma unroll
        for (int s = 0; s < XD; ++s) {
          const int64_t d = ((X + 64) & 127) - 64;  // balanced digit in [-64, 63]
          X = (X - d) >> 7;                          // exact: X - d is a multiple of 128
          dig[s][j >> 2] |= ((uint32_t)d & 0xFFu) << (8 * (j & 3));
          if (d != 0) {
            top = max(top, (uint32_t)s + 1);
            low = min(low, (uint32_t)s);
          }
        }
      }
      if (bad) o.bad[row] = 1;
    }
    const int64_t plane = o.Rp * Kp;
    int8_t *dst = o.D + row * Kp + k0;
#pragma unroll
    for (int s = 0; s < XD; ++s)
      *(uint4 *)(dst + s * plane) = make_uint4(dig[s][0], dig[s][1], dig[s][2], dig[s][3]);
  }
  // every lane of the wavefront takes part in the reductions
  const uint32_t wtop = __ockl_wfred_max_u32(top);
  const uint32_t wlow = __ockl_wfred_max_u32(XD - low);
  if (threadIdx.x % warpSize == 0) {
    if (wtop) atomicMax(o.hi, wtop);
    if (wlow) atomicMax(o.loinv, wlow);
  }
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
// infinity of rem's sign and sets *ovf.
__device__ __forceinline__ uint32_t take_f16(i128 &rem, bool &ovf) {
  if (rem == 0) return 0;
  const bool neg = rem < 0;
  const u128 a = neg ? (u128)0 - (u128)rem : (u128)rem;
  const int e = bitlen(a) - 1;
  const int qe = e - 10 > 24 ? e - 10 : 24;  // quantum 2^(qe-48): 11 significant bits, 2^-24 floor
  u128 n = a >> qe;
  const u128 r = a - (n << qe);
  const u128 half = (u128)1 << (qe - 1);
  if (r > half || (r == half && (n & 1))) n += 1;
  // binary16 bits rise by 1024 per binade and by 1 per quantum, continuously through
  // the subnormals: bits = (qe - 24) * 1024 + n
  const int64_t enc = (int64_t)(qe - 24) * 1024 + (int64_t)n;
  const uint32_t sign = neg ? 0x8000u : 0u;
  if (enc >= 0x7C00) {
    ovf = true;
    return sign | 0x7C00u;
  }
  const i128 v = (i128)(n << qe);
  rem = neg ? rem + v : rem - v;
  return sign | (uint32_t)enc;
}

__device__ __forceinline__ void store_split(i128 V, int nc, bool nan, uint16_t *C, int64_t plane, int64_t idx) {
  if (nan) {
    for (int c = 0; c < nc; ++c) C[c * plane + idx] = 0x7E00;
    return;
  }
  bool ovf = false;
  for (int c = 0; c < nc; ++c) {
    const uint32_t bits = ovf ? 0u : take_f16(V, ovf);
    C[c * plane + idx] = (uint16_t)bits;
  }
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
  i128 *partial;     // [S][M][N] when S > 1
  int64_t S;         // K chunks (gridDim.y)
  int64_t tiles_n;   // workgroup tiles along N
};

// Workgroup of 4 wavefronts in a 2 x 2 arrangement; each wavefront computes WT x WT
// tiles of 16 x 16 outputs with v_mfma_i32_16x16x64_i8.  Operand layout of that
// instruction (64 lanes): lane l supplies row (l % 16) of its 16 x 64 operand slice,
// bytes k = 16 (l / 16) .. 16 (l / 16) + 15; the result element i of lane l is row
// 4 (l / 16) + i, column l % 16 of the 16 x 16 tile.
template <int DM, int WT>
__global__ __launch_bounds__(256) void xm_kernel(XmArgs g) {
  constexpr int NCLS = 2 * DM - 1;
  const uint32_t hiA = g.stats[0], hiB = g.stats[1];
  const int loA = XD - (int)g.stats[2], loB = XD - (int)g.stats[3];
  const int nA = (int)hiA > loA ? (int)hiA - loA : 0;
  const int nB = (int)hiB > loB ? (int)hiB - loB : 0;
  const bool small = nA <= 4 && nB <= 4;
  if ((DM == 4) != small) return;  // the other instantiation handles these operands

  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const int64_t tile = blockIdx.x;
  const int64_t tm = tile / g.tiles_n, tn = tile - tm * g.tiles_n;
  const int64_t row0 = tm * (32 * WT) + (wave / 2) * (16 * WT);
  const int64_t col0 = tn * (32 * WT) + (wave % 2) * (16 * WT);
  const int64_t chunk = blockIdx.y;
  const int64_t kbeg = chunk * XKCHUNK;
  const int64_t kend = min(g.Kp, kbeg + XKCHUNK);

  v4i acc[NCLS][WT][WT];
#pragma unroll
  for (int q = 0; q < NCLS; ++q)
#pragma unroll
    for (int r = 0; r < WT; ++r)
#pragma unroll
      for (int c = 0; c < WT; ++c) acc[q][r][c] = v4i{0, 0, 0, 0};

  const int64_t pa = g.Mp * g.Kp, pb = g.Np * g.Kp;
  const int8_t *baseA = g.DA + (int64_t)loA * pa + (row0 + lane % 16) * g.Kp + 16 * (lane / 16);
  const int8_t *baseB = g.DB + (int64_t)loB * pb + (col0 + lane % 16) * g.Kp + 16 * (lane / 16);

  for (int64_t k0 = kbeg; k0 < kend; k0 += XKSTEP) {
    v4i fa[DM][WT], fb[DM][WT];
#pragma unroll
    for (int s = 0; s < DM; ++s) {
      if (s < nA) {
#pragma unroll
        for (int r = 0; r < WT; ++r) fa[s][r] = *(const v4i *)(baseA + s * pa + (int64_t)(16 * r) * g.Kp + k0);
      }
      if (s < nB) {
#pragma unroll
        for (int c = 0; c < WT; ++c) fb[s][c] = *(const v4i *)(baseB + s * pb + (int64_t)(16 * c) * g.Kp + k0);
      }
    }
#pragma unroll
    for (int s = 0; s < DM; ++s) {
      if (s < nA) {
#pragma unroll
        for (int t = 0; t < DM; ++t) {
          if (t < nB) {
#pragma unroll
            for (int r = 0; r < WT; ++r)
#pragma unroll
              for (int c = 0; c < WT; ++c)
                acc[s + t][r][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[s][r], fb[t][c], acc[s + t][r][c], 0, 0, 0);
          }
        }
      }
    }
  }

  // combine the shift classes exactly: V = sum_q acc[q] 128^(q + loA + loB)
  const int shift0 = 7 * (loA + loB);
#pragma unroll
  for (int r = 0; r < WT; ++r) {
#pragma unroll
    for (int c = 0; c < WT; ++c) {
      const int64_t col = col0 + 16 * c + lane % 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t row = row0 + 16 * r + 4 * (lane / 16) + i;
        // five consecutive classes fit one int64 (|acc| < 2^31, relative shifts up to
        // 28 bits); the groups are then combined 35 bits apart in 128 bits
        constexpr int NG = (NCLS + 4) / 5;
        int64_t part[NG];
#pragma unroll
        for (int q = 0; q < NG; ++q) part[q] = 0;
#pragma unroll
        for (int q = 0; q < NCLS; ++q) part[q / 5] += (int64_t)acc[q][r][c][i] * ((int64_t)1 << (7 * (q % 5)));
        u128 Vu = 0;
#pragma unroll
        for (int q = 0; q < NG; ++q) Vu += (u128)(i128)part[q] << (35 * q);
        const i128 V = (i128)(Vu << shift0);
        if (row < g.M && col < g.N) {
          if (g.S == 1) {
            store_split(V, g.nc, g.bad_a[row] | g.bad_b[col], g.C, g.M * g.N, row * g.N + col);
          } else {
            g.partial[(chunk * g.M + row) * g.N + col] = V;
          }
        }
      }
    }
  }
}

__global__ void xm_finish(XmArgs g) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = g.M * g.N;
  if (t >= MN) return;
  i128 V = 0;
  for (int64_t s = 0; s < g.S; ++s) V += g.partial[s * MN + t];
  const int64_t row = t / g.N, col = t - row * g.N;
  store_split(V, g.nc, g.bad_a[row] | g.bad_b[col], g.C, MN, t);
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct XLayout {
  int64_t Mp, Np, Kp, S;
  int64_t off_stats, off_bad_a, off_bad_b, off_da, off_db, off_part, total;
};

XLayout x_layout(int64_t M, int64_t N, int64_t K) {
  XLayout L;
  L.Mp = round_up(M, XPAD);
  L.Np = round_up(N, XPAD);
  L.Kp = round_up(K, XKSTEP);
  L.S = L.Kp == 0 ? 1 : (L.Kp + XKCHUNK - 1) / XKCHUNK;
  int64_t o = 0;
  L.off_stats = o;
  o += 256;
  L.off_bad_a = o;
  o += round_up(M, 256);
  L.off_bad_b = o;
  o += round_up(N, 256);
  L.off_da = o;
  o += round_up(XD * L.Mp * L.Kp, 256);
  L.off_db = o;
  o += round_up(XD * L.Np * L.Kp, 256);
  L.off_part = o;
  if (L.S > 1) o += L.S * M * N * (int64_t)sizeof(i128);
  L.total = o;
  return L;
}

}  // namespace

int64_t exact_workspace_bytes(int64_t M, int64_t N, int64_t K) { return x_layout(M, N, K).total; }

hipError_t launch_matmul_exact(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                               int b_mc, int b_trans, void *W, void *C, hipStream_t stream) {
  const XLayout L = x_layout(M, N, K);
  char *w = (char *)W;
  uint32_t *stats = (uint32_t *)(w + L.off_stats);
  uint8_t *bad_a = (uint8_t *)(w + L.off_bad_a), *bad_b = (uint8_t *)(w + L.off_bad_b);
  int8_t *DA = (int8_t *)(w + L.off_da), *DB = (int8_t *)(w + L.off_db);

  {
    const int64_t n = M > N ? M : N;
    const int blocks = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 + 1 : 1024);
    hipLaunchKernelGGL(xs_init, dim3(blocks), dim3(256), 0, stream, stats, bad_a, M, bad_b, N);
  }
  if (L.Kp > 0) {
    SliceOp a, b;
    a.src = (const uint16_t *)A;
    a.planes = a_mc ? nc : 1;
    a.kcontig = 1;
    a.plane = M * K;
    a.rs = K;
    a.ks = 1;
    a.R = M;
    a.Rp = L.Mp;
    a.D = DA;
    a.bad = bad_a;
    a.hi = stats + 0;
    a.loinv = stats + 2;
    a.threads = L.Mp * L.Kp / 16;
    b.src = (const uint16_t *)B;
    b.planes = b_mc ? nc : 1;
    b.kcontig = b_trans ? 1 : 0;
    b.plane = K * N;
    b.rs = b_trans ? K : 1;
    b.ks = b_trans ? 1 : N;
    b.R = N;
    b.Rp = L.Np;
    b.D = DB;
    b.bad = bad_b;
    b.hi = stats + 1;
    b.loinv = stats + 3;
    b.threads = L.Np * L.Kp / 16;
    const int64_t ab = (a.threads + XS_THREADS - 1) / XS_THREADS;
    const int64_t bb = (b.threads + XS_THREADS - 1) / XS_THREADS;
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
  g.partial = (i128 *)(w + L.off_part);
  g.S = L.S;
  // DM = 4: 2 x 2 tiles per wavefront (64 x 64 per workgroup); DM = 7: 1 x 1 (32 x 32)
  {
    g.tiles_n = L.Np / 64;
    const int64_t tiles = (L.Mp / 64) * g.tiles_n;
    hipLaunchKernelGGL((xm_kernel<4, 2>), dim3((unsigned)tiles, (unsigned)L.S), dim3(256), 0, stream, g);
  }
  {
    g.tiles_n = L.Np / 32;
    const int64_t tiles = (L.Mp / 32) * g.tiles_n;
    hipLaunchKernelGGL((xm_kernel<7, 1>), dim3((unsigned)tiles, (unsigned)L.S), dim3(256), 0, stream, g);
  }
  if (L.S > 1) {
    const int64_t n = M * N;
    hipLaunchKernelGGL(xm_finish, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, g);
  }
  return hipGetLastError();
}

}  // namespace mcf
