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

#include <type_traits>

#include "mcf_arith.hpp"
#include "mcf_internal.hpp"
#include "mm_steps.hpp"

namespace mcf {

constexpr int MM_THREADS = 256;

// The operands of reduction step kk of the LDS tiles for the TM x TN outputs of a
// lane: the A values of its rows, the B values of its columns (all components).
template <typename T, int NA, int NB, int TM, int TN, int KT, int BM, int BN>
struct Operands {
  T a[TM][NA], b[TN][NB];
  __device__ __forceinline__ void load(const T (*As)[KT][BM], const T (*Bs)[KT][BN], int kk, int tx, int ty) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int c = 0; c < NA; ++c) a[i][c] = As[c][kk][ty * TM + i];
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int c = 0; c < NB; ++c) b[j][c] = Bs[c][kk][tx * TN + j];
  }
};

// Per-lane state of the product: the accumulators of every (component p of B, row i,
// column j) the lane owns.  PMASK selects the components p of B that take part
// (MC x MC; bit p clear: B^(p) is zero across the whole tile, so the term is skipped
// -- ScalingN gives zeros and Add-MCN(acc, zeros) returns acc, a Simple-Renorm output,
// unchanged).  GROUP = false: each term's general-compaction branch follows its own
// arithmetic; GROUP = true: the arithmetic of all terms of a step shares one
// straight-line block and one (rarely taken) compaction branch.
template <typename T, int NC, bool AMC, bool BMC, int TM, int TN, int KT, int BM, int BN, int SPOL, int APOL,
          bool GROUP, bool PRUNE>
struct Lane {
  static constexpr int NA = AMC ? NC : 1;
  static constexpr int NB = BMC ? NC : 1;
  static constexpr int NP = (AMC && BMC) ? NC : 1;
  using Ops = Operands<T, NA, NB, TM, TN, KT, BM, BN>;
  T acc[NP][TM][TN][NC];

  // dst = ScalingN terms of step o (FIRST: into acc)
  template <int PMASK>
  __device__ __forceinline__ void scale(const Ops &o, T (&dst)[NP][TM][TN][NC]) {
    T hs[NP][TM][TN][NC + 1];
    bool slow[NP][TM][TN];
    bool any = false;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (!((PMASK >> p) & 1)) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const T v = AMC ? o.b[j][p] : o.a[i][0];
          if constexpr (AMC)
            scaling_terms<T, NC>(o.a[i], v, hs[p][i][j]);
          else
            scaling_terms<T, NC>(o.b[j], v, hs[p][i][j]);
          slow[p][i][j] = sr_try<T, NC, SPOL>(hs[p][i][j], dst[p][i][j], v == T(0));
          if constexpr (GROUP)
            any = any || slow[p][i][j];
          else if (__builtin_expect(slow[p][i][j], 0))
            compact_nz<T, NC + 1, NC>(hs[p][i][j], dst[p][i][j]);
        }
    }
    if constexpr (GROUP) {
      if (__builtin_expect(any, 0)) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          if (!((PMASK >> p) & 1)) continue;
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              if (slow[p][i][j]) compact_nz<T, NC + 1, NC>(hs[p][i][j], dst[p][i][j]);
        }
      }
    }
  }

  // acc = Add-MCN(acc, term) for every term
  template <int PMASK>
  __device__ __forceinline__ void add(const T (&term)[NP][TM][TN][NC]) {
    T ha[NP][TM][TN][NC + 1];
    bool slow[NP][TM][TN];
    bool any = false;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (!((PMASK >> p) & 1)) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          add_terms<T, NC>(acc[p][i][j], term[p][i][j], ha[p][i][j]);
          slow[p][i][j] = sr_try<T, NC, APOL>(ha[p][i][j], acc[p][i][j]);
          if constexpr (GROUP)
            any = any || slow[p][i][j];
          else if (__builtin_expect(slow[p][i][j], 0))
            compact_nz<T, NC + 1, NC>(ha[p][i][j], acc[p][i][j]);
        }
    }
    if constexpr (GROUP) {
      if (__builtin_expect(any, 0)) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          if (!((PMASK >> p) & 1)) continue;
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              if (slow[p][i][j]) compact_nz<T, NC + 1, NC>(ha[p][i][j], acc[p][i][j]);
        }
      }
    }
  }

  // ScalingN of term (x, v) in kept-terms form; lanes failing the test run the
  // general step.  HEAD / TAIL: the products' errors are known to be zero (see mm_kernel).
  // With several outputs per lane (the MC-Linear shape) the tests are wavefront masks
  // and a failing lane sends its wavefront through the general step (3.26 -> 3.20 ms
  // per 4096 x 1024 x 1024 layer); with one output per lane the per-lane branch
  // measured 1% faster.
  static constexpr bool KEPT_MASK = TM * TN > 1;
  template <bool HEAD, bool TAIL>
  __device__ __forceinline__ void scale_kept(const T (&x)[NC], T v, T (&t)[NC]) {
    kept_scale<T, NC, HEAD, TAIL, KEPT_MASK>(x, v, t);
  }

  // a = Add-MCN(a, t) in kept-terms form (TINY: the add_tiny form)
  template <bool TINY>
  __device__ __forceinline__ void add_kept_into(T (&a)[NC], const T (&t)[NC]) {
    kept_add<T, NC, TINY, KEPT_MASK>(a, t);
  }

  // ScalingN of (x, v) when every product x_i v is exact and |x_0| >= |x_1| >= ...
  // (tile flags TPS and ORD): the terms are the products themselves, in magnitude
  // order, so the kept-terms test cannot fail and is not run.
  __device__ __forceinline__ void scale_exact(const T (&x)[NC], T v, T (&t)[NC]) {
    T last;
    scaling_kept<T, NC, true, true>(x, v, t, last);
  }
  template <bool ORD>
  __device__ __forceinline__ void scale_low(const T (&x)[NC], T v, T (&t)[NC]) {
    if constexpr (ORD)
      scale_exact(x, v, t);
    else
      scale_kept<true, true>(x, v, t);
  }

  // Pruned MC x MC product: component P of B multiplies the first NC - P components
  // of A in MM-MCN order with NC - P components; the accumulator of P keeps zeros in
  // its other components, so the epilogue's Add-MCN combination pads it with zeros.
  // FIRST: the step initialises the accumulators (every P, whatever PMASK says).
  template <int P, int PMASK, bool TPS, bool FIRST>
  __device__ __forceinline__ void prune_step(const Ops &o) {
    if constexpr (P < NP) {
      if constexpr (FIRST || ((PMASK >> P) & 1)) {
        constexpr int NCP = NC - P;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const T(&a)[NCP] = *reinterpret_cast<const T(*)[NCP]>(&o.a[i][0]);
            T(&ac)[NCP] = *reinterpret_cast<T(*)[NCP]>(&acc[P][i][j][0]);
            const T v = o.b[j][P];
            T t[NCP];
            if constexpr (SPOL == SR_SUFFIX) {
              kept_scale<T, NCP, TPS && (P > 0), TPS>(a, v, t);
            } else {
              T h[NCP + 1];
              scaling_terms<T, NCP>(a, v, h);
              if (__builtin_expect(sr_try<T, NCP, SPOL>(h, t, v == T(0)), 0)) compact_nz<T, NCP + 1, NCP>(h, t);
            }
            if constexpr (FIRST) {
              nonfinite_tail<T, NCP>(t);
#pragma unroll
              for (int c = 0; c < NCP; ++c) ac[c] = t[c];
#pragma unroll
              for (int c = NCP; c < NC; ++c) acc[P][i][j][c] = T(0);
            } else if constexpr (SPOL == SR_SUFFIX) {
              kept_add<T, NCP, TPS && (P > 0)>(ac, t);
            } else {
              T h[NCP + 1];
              add_terms<T, NCP>(ac, t, h);
              if (__builtin_expect(sr_try<T, NCP, APOL>(h, ac), 0)) compact_nz<T, NCP + 1, NCP>(h, ac);
            }
          }
      }
      prune_step<P + 1, PMASK, TPS, FIRST>(o);
    }
  }

  // term k = 0 initialises the accumulators
  template <bool TPS, bool ORD>
  __device__ __forceinline__ void first(const Ops &o) {
    first_terms<TPS, ORD>(o);
    if constexpr (!PRUNE) {  // (the pruned parts are patched in prune_step)
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) nonfinite_tail<T, NC>(acc[p][i][j]);
    }
  }
  template <bool TPS, bool ORD>
  __device__ __forceinline__ void first_terms(const Ops &o) {
    if constexpr (PRUNE) {
      prune_step<0, (1 << NP) - 1, TPS, true>(o);
    } else if constexpr (SPOL == SR_SUFFIX) {
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            if constexpr (!AMC)
              scale_kept<false, TPS>(o.b[j], o.a[i][0], acc[p][i][j]);
            else if (TPS && p > 0)
              scale_low<ORD>(o.a[i], o.b[j][p], acc[p][i][j]);
            else
              scale_kept<false, TPS>(o.a[i], o.b[j][p], acc[p][i][j]);
          }
    } else {
      scale<(1 << NP) - 1>(o, acc);
    }
  }

  // S consecutive reduction steps kk .. kk+S-1 in kept-terms form, all terms of all
  // S steps behind one test: when a lane's test fails anywhere, the wavefront restores
  // its accumulators and redoes the S steps with the general steps (full terms and the
  // compaction network; a lane whose kept terms were valid gets the same values), so a
  // wavefront takes one rarely-taken uniform branch per S steps.
  template <int PMASK, bool TPS, int S, bool ORD>
  __device__ __forceinline__ void group_kept(const T (*As)[KT][BM], const T (*Bs)[KT][BN], int kk, int tx, int ty) {
    T saved[NP][TM][TN][NC];
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int c = 0; c < NC; ++c) saved[p][i][j][c] = acc[p][i][j][c];
    uint64_t bad = 0;  // lanes failing a test, as a wavefront mask
#pragma unroll
    for (int st = 0; st < S; ++st) {
      Ops o;
      o.load(As, Bs, kk + st, tx, ty);
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        if (!((PMASK >> p) & 1)) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            T t[NC], sum[NC], last;
            if constexpr (!AMC) {
              scaling_kept<T, NC, false, TPS>(o.b[j], o.a[i][0], t, last);
              bad |= kept_invalid_mask<T, NC, TPS, true>(t, last);
            } else if (TPS && p > 0) {
              scaling_kept<T, NC, true, true>(o.a[i], o.b[j][p], t, last);
              if constexpr (!ORD) bad |= kept_invalid_mask<T, NC, true, true>(t, last);
            } else {
              scaling_kept<T, NC, false, TPS>(o.a[i], o.b[j][p], t, last);
              bad |= kept_invalid_mask<T, NC, TPS, true>(t, last);
            }
            if (AMC && BMC && TPS && p > 0) {
              bad |= add_tiny_mask<T, NC>(acc[p][i][j], t, sum);
            } else {
              add_kept<T, NC>(acc[p][i][j], t, sum, last);
              bad |= kept_invalid_mask<T, NC, false>(sum, last);
            }
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[p][i][j][c] = sum[c];
          }
      }
    }
    if (__builtin_expect(bad != 0, 0)) {
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int c = 0; c < NC; ++c) acc[p][i][j][c] = saved[p][i][j][c];
#pragma unroll
      for (int st = 0; st < S; ++st) {
        Ops o;
        o.load(As, Bs, kk + st, tx, ty);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          if (!((PMASK >> p) & 1)) continue;
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              T h[NC + 1], t[NC];
              if constexpr (AMC)
                scaling_terms<T, NC>(o.a[i], BMC ? o.b[j][p] : o.b[j][0], h);
              else
                scaling_terms<T, NC>(o.b[j], o.a[i][0], h);
              compact_nz<T, NC + 1, NC>(h, t);
              add_terms<T, NC>(acc[p][i][j], t, h);
              compact_nz<T, NC + 1, NC>(h, acc[p][i][j]);
            }
        }
      }
    }
  }

  // steps kk0 .. kt-1 of a tile.  GROUP = false: each term's ScalingN and Add-MCN run
  // back to back, so only one term is live at a time.
  template <int PMASK, bool TPS, bool ORD, int DEPTH = 1>
  __device__ __forceinline__ void run(const T (*As)[KT][BM], const T (*Bs)[KT][BN], int kk0, int kt, int tx,
                                      int ty) {
    // two steps per loop iteration, so the accumulators keep their registers across
    // the back edge instead of being copied
    if constexpr (PRUNE) {
#pragma unroll 2
      for (int kk = kk0; kk < kt; ++kk) {
        Ops o;
        o.load(As, Bs, kk, tx, ty);
        prune_step<0, PMASK, TPS, false>(o);
      }
      return;
    }
    if constexpr (SPOL == SR_SUFFIX && NC == 2) {
      // nc = 2: the tests of two steps share one branch.  (For nc >= 3 grouping keeps
      // more temporaries live, lowers the wavefronts per SIMD and was measured
      // slower; there each step tests and branches on its own, below.)
      // Two groups per iteration: each group keeps its input accumulators live for the
      // redo, so with one group per iteration the new accumulators were copied back
      // into the old registers at the back edge (4 of 54 VALU instructions per two
      // steps); with two the registers alternate.  Together with the mask tests:
      // 1024^3 nc = 2 0.733 -> 0.699 ms.
      int kk = kk0;
      for (; kk + 3 < kt; kk += 4) {
        group_kept<PMASK, TPS, 2, ORD>(As, Bs, kk, tx, ty);
        group_kept<PMASK, TPS, 2, ORD>(As, Bs, kk + 2, tx, ty);
      }
      if (kk + 1 < kt) {
        group_kept<PMASK, TPS, 2, ORD>(As, Bs, kk, tx, ty);
        kk += 2;
      }
      if (kk < kt) group_kept<PMASK, TPS, 1, ORD>(As, Bs, kk, tx, ty);
      return;
    }
    if constexpr (DEPTH > 1 && !GROUP) {
      // The operands of DEPTH steps are read from LDS first, then the steps run on them
      // in k order: for binary32 grids of few wavefronts, where nothing hides a step's
      // LDS latency, and for the binary16 MC-Linear kernel.
      int kk = kk0;
      for (; kk + DEPTH <= kt; kk += DEPTH) {
        Ops os[DEPTH];
#pragma unroll
        for (int u = 0; u < DEPTH; ++u) os[u].load(As, Bs, kk + u, tx, ty);
#pragma unroll
        for (int u = 0; u < DEPTH; ++u) {
          if constexpr (SPOL == SR_SUFFIX)
            kept_step<PMASK, TPS, ORD>(os[u]);
          else
            full_step<PMASK>(os[u]);
        }
      }
      for (; kk < kt; ++kk) {
        Ops o;
        o.load(As, Bs, kk, tx, ty);
        if constexpr (SPOL == SR_SUFFIX)
          kept_step<PMASK, TPS, ORD>(o);
        else
          full_step<PMASK>(o);
      }
      return;
    }
#pragma unroll 2
    for (int kk = kk0; kk < kt; ++kk) {
      Ops o;
      o.load(As, Bs, kk, tx, ty);
      if constexpr (SPOL == SR_SUFFIX) {
        kept_step<PMASK, TPS, ORD>(o);
      } else if constexpr (GROUP) {
        T term[NP][TM][TN][NC];
        scale<PMASK>(o, term);
        add<PMASK>(term);
      } else {
        full_step<PMASK>(o);
      }
    }
  }

  // One reduction step in kept-terms form, term by term.
  template <int PMASK, bool TPS, bool ORD>
  __device__ __forceinline__ void kept_step(const Ops &o) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (!((PMASK >> p) & 1)) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          T term[NC];
          if constexpr (!AMC) {
            scale_kept<false, TPS>(o.b[j], o.a[i][0], term);
            add_kept_into<false>(acc[p][i][j], term);
          } else if (BMC && TPS && p > 0) {
            scale_low<ORD>(o.a[i], o.b[j][p], term);
            add_kept_into<true>(acc[p][i][j], term);
          } else {
            scale_kept<false, TPS>(o.a[i], o.b[j][p], term);
            add_kept_into<false>(acc[p][i][j], term);
          }
        }
    }
  }

  // One reduction step in the general form: each term's ScalingN and Add-MCN back to
  // back, with Simple-Renorm's fast path (SPOL / APOL) and the compaction network for
  // lanes that fail its test.
  template <int PMASK>
  __device__ __forceinline__ void full_step(const Ops &o) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if (!((PMASK >> p) & 1)) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const T v = AMC ? o.b[j][p] : o.a[i][0];
          T h[NC + 1], term[NC];
          if constexpr (AMC)
            scaling_terms<T, NC>(o.a[i], v, h);
          else
            scaling_terms<T, NC>(o.b[j], v, h);
          if (__builtin_expect(sr_try<T, NC, SPOL>(h, term, v == T(0)), 0)) compact_nz<T, NC + 1, NC>(h, term);
          add_terms<T, NC>(acc[p][i][j], term, h);
          if (__builtin_expect(sr_try<T, NC, APOL>(h, acc[p][i][j]), 0)) compact_nz<T, NC + 1, NC>(h, acc[p][i][j]);
        }
    }
  }
};

// Tile of C for workgroup `id` of a 1-D grid of gx * gy tiles (gx along N, gy along
// M).  The dispatcher hands workgroup id to XCD id % 8, and each XCD has its own L2,
// so the ids are first regrouped to give every XCD a contiguous run of the tile
// order; the tile order then walks bands of TILE_GROUP tile-rows column by column, so
// the workgroups an XCD runs together share their A rows and B columns in its L2.
// (The remainder of an id count not divisible by 8 keeps its own order.)  Results do
// not depend on this mapping: every output is reduced in k order by one lane.
constexpr uint32_t TILE_GROUP = 16;
constexpr uint32_t N_XCD = 8;

__device__ __forceinline__ void tile_of(uint32_t id, uint32_t total, uint32_t gx, uint32_t gy, int64_t &tm,
                                        int64_t &tn) {
  const uint32_t t8 = total - total % N_XCD;
  const uint32_t v = id < t8 ? (id % N_XCD) * (t8 / N_XCD) + id / N_XCD : id;
  const uint32_t band = v / (TILE_GROUP * gx);
  const uint32_t row0 = band * TILE_GROUP;
  const uint32_t rows = (gy - row0) < TILE_GROUP ? (gy - row0) : TILE_GROUP;
  const uint32_t local = v - band * TILE_GROUP * gx;
  tm = row0 + local % rows;
  tn = local / rows;
}

// Shapes, strides and epilogue of one product launch.  Each batch index bb (grid y
// plus bb0) is split into (bb / B2, bb % B2); operand planes start a_plane / b_plane
// components apart and a batch at i1 * s1 + i2 * s2 components (a stride of 0
// broadcasts the operand); C is dense: [nc][batches][M][N].
template <typename T>
struct MmArgs {
  int64_t M, N, K;
  int64_t a_plane, b_plane, c_plane;
  int64_t B2, bb0;
  int64_t a_s1, a_s2, b_s1, b_s2;
  // epilogue: 0 none; 1 Add-MCN(acc, y) (MC-Linear bias); 2 AddMM:
  // Add-MCN(ScalingN(acc, alpha), ScalingN(y, beta)).  y planes y_plane apart, rows
  // y_ld apart (0: one row for every output row).
  int mode;
  const T *y;
  int64_t y_plane, y_ld;
  T alpha, beta;
};

// A: [NA][M][K] row-major planes.  B: [NB][K][N] (BT = false) or [NB][N][K] (BT =
// true).  NA = NC when A is MC else 1, likewise NB.
// Occupancy: with nc <= 3, binary32 kernels run at least 5 wavefronts per SIMD (at most
// 96 VGPRs); they sit just under that bound (the 8192^3 one spills one 8-byte value
// outside its loop) and one register more would drop them to 4.  The binary16 kernels
// (but the pruned ones) run 7 or 8.  MC-Linear (BT) and nc = 1 run 8, the most a SIMD
// holds: at 64 VGPRs the few values that no longer fit are per-tile addresses,
// reloaded once per tile.  The other nc = 2 and 3 products run 7 (72 VGPRs: fewer
// spills around the tile loop): 1024^3 nc = 2 0.70 -> 0.67 ms, nc = 3 1.30 -> 1.26 ms
// (6 wavefronts: 0.67 / 1.29, 5: 0.72 ms); MC-Linear is 1% slower at 7.  nc = 4 needs
// more registers.
template <int NC, bool BT>
constexpr int f16_waves() {
  return NC >= 2 && !BT ? 7 : 8;
}
template <typename T, int NC, bool AMC, bool BMC, bool BT, int TM, int TN, int KT, int SPOL, int APOL,
          bool GROUP, bool ADDMM, bool PRUNE, int DEPTH = 1>
__global__ __attribute__((amdgpu_flat_work_group_size(1, MM_THREADS),
                          amdgpu_waves_per_eu(sizeof(T) == 2 && NC <= 3 && !PRUNE ? f16_waves<NC, BT>()
                                              : (NC <= 3 && sizeof(T) <= 4 ? 5 : 1)))) void
mm_kernel(const T *__restrict__ A, const T *__restrict__ B,
                                                        T *__restrict__ C, const MmArgs<T> g) {
  const int64_t M = g.M, N = g.N, K = g.K;
  {
    const int64_t bb = g.bb0 + blockIdx.y;
    const int64_t i1 = bb / g.B2, i2 = bb - (bb / g.B2) * g.B2;
    A += i1 * g.a_s1 + i2 * g.a_s2;
    B += i1 * g.b_s1 + i2 * g.b_s2;
    C += bb * M * N;
  }
  constexpr int NA = AMC ? NC : 1;
  constexpr int NB = BMC ? NC : 1;
  constexpr int TX = 16, TY = 16;  // lanes along N and along M
  constexpr int BM = TY * TM, BN = TX * TN;
  constexpr int NP = (AMC && BMC) ? NC : 1;  // components of B swept (MC x MC)
  constexpr int ALL = (1 << NP) - 1;
  constexpr int EPOL = APOL == SR_SUFFIX ? SR_NET : APOL;  // the epilogue's Add-MCN
  __shared__ T As[NA][KT][BM];
  __shared__ T Bs[NB][KT][BN];

  const int tx = threadIdx.x % TX, ty = threadIdx.x / TX;
  int64_t m0, n0;
  tile_of(blockIdx.x, gridDim.x, (uint32_t)((N + BN - 1) / BN), (uint32_t)((M + BM - 1) / BM), m0, n0);
  m0 *= BM;
  n0 *= BN;

  Lane<T, NC, AMC, BMC, TM, TN, KT, BM, BN, SPOL, APOL, GROUP, PRUNE> lane;
  auto &acc = lane.acc;

  // Each thread stages A_PER elements of the A tile and B_PER of the B tile per
  // component plane.  The next tile's global loads are issued into registers before
  // the current tile's arithmetic, so their latency hides behind it; the registers
  // go to LDS at the top of the next iteration.
  constexpr int A_PER = (BM * KT + MM_THREADS - 1) / MM_THREADS;
  constexpr int B_PER = (BN * KT + MM_THREADS - 1) / MM_THREADS;
  T ra[A_PER][NA], rb[B_PER][NB];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int t = 0; t < A_PER; ++t) {
      const int idx = threadIdx.x + t * MM_THREADS;
      const int r = idx / KT, kk = idx % KT;
      const int64_t gm = m0 + r, gk = k0 + kk;
      const bool ok = idx < BM * KT && gm < M && gk < K;
#pragma unroll
      for (int c = 0; c < NA; ++c) ra[t][c] = ok ? A[c * g.a_plane + gm * K + gk] : T(0);
    }
#pragma unroll
    for (int t = 0; t < B_PER; ++t) {
      const int idx = threadIdx.x + t * MM_THREADS;
      int col, kk;
      if constexpr (BT) {
        col = idx / KT;
        kk = idx % KT;
      } else {
        kk = idx / BN;
        col = idx % BN;
      }
      const int64_t gn = n0 + col, gk = k0 + kk;
      const bool ok = idx < BN * KT && gn < N && gk < K;
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const int64_t off = c * g.b_plane + (BT ? (gn * K + gk) : (gk * N + gn));
        rb[t][c] = ok ? B[off] : T(0);
      }
    }
  };

  // Kept-terms policy: the largest magnitude of each component plane of the A and B
  // tiles (binary32 bit patterns of |value|, which order like the values; a NaN or an
  // infinity is above every finite value), in LDS slots alternating between tiles.
  // It decides per tile whether every product of a low component, x_c * v_p with
  // c + p >= 1 (x the MC operand, v_p the other operand's components), is below
  // exact_limit, so that its Two-Prod error is zero (a product's error is at most half
  // the spacing of the format at the product, which below exact_limit is half the
  // smallest subnormal, and that rounds to zero).  For MC x MC one more slot notes
  // whether some value of A in the tile has components out of magnitude order
  // (|a_c| < |a_{c+1}|, or a NaN); when none has and the products are exact, the
  // ScalingN terms of B's low components are exact products in magnitude order and
  // need no kept-terms test (ORD).
  constexpr bool TRACK = SPOL == SR_SUFFIX && NC > 1;
  constexpr bool ORD_OK = TRACK && AMC && BMC && !PRUNE;
  constexpr int NSLOT = NA + NB + (ORD_OK ? 1 : 0);
  __shared__ uint32_t mx[2][NSLOT];
  if constexpr (TRACK) {
    if (threadIdx.x < 2 * NSLOT) (&mx[0][0])[threadIdx.x] = 0;
    __syncthreads();
  }

  if (K > 0) fetch(0);
  int tile = 0;
  for (int64_t k0 = 0; k0 < K; k0 += KT, ++tile) {
    const int kt = (int)((K - k0) < KT ? (K - k0) : KT);
    // registers -> LDS: A transposed to [k][m]; note which planes of B hold a non-zero
    int nonzero_planes = 0;
    uint32_t lmax[NSLOT];
#pragma unroll
    for (int c = 0; c < NSLOT; ++c) lmax[c] = 0;
#pragma unroll
    for (int t = 0; t < A_PER; ++t) {
      const int idx = threadIdx.x + t * MM_THREADS;
      if (idx < BM * KT) {
#pragma unroll
        for (int c = 0; c < NA; ++c) {
          As[c][idx % KT][idx / KT] = ra[t][c];
          if constexpr (TRACK) lmax[c] = max(lmax[c], __float_as_uint(__builtin_fabsf((float)ra[t][c])));
          if constexpr (ORD_OK)
            if (c + 1 < NA && out_of_order(ra[t][c], ra[t][c + 1 < NA ? c + 1 : c])) lmax[NA + NB] = 1;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < B_PER; ++t) {
      const int idx = threadIdx.x + t * MM_THREADS;
      if (idx < BN * KT) {
        const int col = BT ? idx / KT : idx % BN, kk = BT ? idx % KT : idx / BN;
#pragma unroll
        for (int c = 0; c < NB; ++c) {
          Bs[c][kk][col] = rb[t][c];
          if (rb[t][c] != T(0)) nonzero_planes |= 1 << c;
          if constexpr (TRACK) lmax[NA + c] = max(lmax[NA + c], __float_as_uint(__builtin_fabsf((float)rb[t][c])));
        }
      }
    }
    if constexpr (TRACK) {
      // wavefront maximum (DPP), then one LDS atomic per wavefront and plane
#pragma unroll
      for (int c = 0; c < NSLOT; ++c) {
        const uint32_t w = __ockl_wfred_max_u32(lmax[c]);
        if (threadIdx.x % warpSize == 0) atomicMax(&mx[tile & 1][c], w);
      }
    }
    int pmask = ALL;
    if constexpr (AMC && BMC) {
      // the last component plane of B is often zero throughout a tile (binary16)
      pmask = __syncthreads_or(nonzero_planes & (1 << (NP - 1))) ? ALL : (ALL >> 1);
    } else {
      __syncthreads();
    }
    bool tps = false, ord = false;
    if constexpr (TRACK) {
      // X: the MC operand's planes, V: the other operand's planes
      constexpr int X0 = AMC ? 0 : NA, NX = AMC ? NA : NB;
      constexpr int V0 = AMC ? NA : 0, NV = AMC ? NB : NA;
      tps = true;
#pragma unroll
      for (int c = 0; c < NX; ++c)
#pragma unroll
        for (int p = 0; p < NV; ++p)
          if (c + p >= 1)
            tps = tps && __uint_as_float(mx[tile & 1][X0 + c]) * __uint_as_float(mx[tile & 1][V0 + p]) <
                             exact_limit<T>();
      if constexpr (ORD_OK) ord = mx[tile & 1][NA + NB] == 0;
      // the other slot set was last read during the previous tile, before its final
      // barrier, and is next written by the next tile, after this tile's final barrier
      if (threadIdx.x < NSLOT) mx[(tile & 1) ^ 1][threadIdx.x] = 0;
    }
    if (k0 + KT < K) fetch(k0 + KT);  // next tile, in flight during this one
    auto steps = [&](auto tps_c, auto ord_c) {
      constexpr bool TPS = decltype(tps_c)::value;
      constexpr bool ORD = decltype(ord_c)::value;
      int kk0 = 0;
      if (k0 == 0) {  // term k = 0 initialises the accumulators
        typename decltype(lane)::Ops o;
        o.load(As, Bs, 0, tx, ty);
        lane.template first<TPS, ORD>(o);
        kk0 = 1;
      }
      if (NP > 1 && pmask != ALL)
        lane.template run<(ALL >> 1), TPS, ORD, DEPTH>(As, Bs, kk0, kt, tx, ty);
      else
        lane.template run<ALL, TPS, ORD, DEPTH>(As, Bs, kk0, kt, tx, ty);
    };
    using no = std::integral_constant<bool, false>;
    if (TRACK && tps && ord)
      steps(std::integral_constant<bool, TRACK>{}, std::integral_constant<bool, ORD_OK>{});
    else if (TRACK && tps)
      steps(std::integral_constant<bool, TRACK>{}, no{});
    else
      steps(no{}, no{});
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
        for (int p = 1; p < NP; ++p) mm_add<T, NC, EPOL>(r, acc[p][i][j], r);
      }
      if (gm < M && gn < N) {
        if (g.mode != 0) {
          T yv[NC];
#pragma unroll
          for (int c = 0; c < NC; ++c) yv[c] = g.y[c * g.y_plane + gm * g.y_ld + gn];
          if constexpr (ADDMM) {  // AddMM-MCN: both operands scaled first (ScalingN, expand off)
            scaling_n<T, NC, NC>(r, g.alpha, r);
            scaling_n<T, NC, NC>(yv, g.beta, yv);
          }
          mm_add<T, NC, EPOL>(r, yv, r);
        }
        // Zero components leave as +0, the padding Simple-Renorm writes (a zero term
        // that was skipped or selected above may carry the sign of -0).
#pragma unroll
        for (int c = 0; c < NC; ++c) C[c * g.c_plane + gm * N + gn] = (r[c] != T(0)) ? r[c] : T(0);
      }
    }
}

// Batches go to grid y, at most MM_MAX_GRID_Y per launch.
constexpr int64_t MM_MAX_GRID_Y = 65535;

template <typename T, int NC, bool AMC, bool BMC, bool BT, int TM, int TN, int SPOL, int APOL, int KT = 16,
          bool PRUNE = false, int DEPTH = 1>
static hipError_t mm_launch_tile(MmArgs<T> g, int64_t batches, const void *A, const void *B, void *C,
                                 hipStream_t s) {
  constexpr int BM = 16 * TM, BN = 16 * TN;
  const unsigned gx = (unsigned)(((g.N + BN - 1) / BN) * ((g.M + BM - 1) / BM));
  for (int64_t b0 = 0; b0 < batches; b0 += MM_MAX_GRID_Y) {
    g.bb0 = b0;
    const int64_t nb = (batches - b0) < MM_MAX_GRID_Y ? (batches - b0) : MM_MAX_GRID_Y;
    if (g.mode == 2)  // the AddMM epilogue is a separate instantiation: it needs more registers
      hipLaunchKernelGGL((mm_kernel<T, NC, AMC, BMC, BT, TM, TN, KT, SPOL, APOL, false, true, PRUNE, DEPTH>),
                         dim3(gx, (unsigned)nb), dim3(MM_THREADS), 0, s, (const T *)A, (const T *)B, (T *)C, g);
    else
      hipLaunchKernelGGL((mm_kernel<T, NC, AMC, BMC, BT, TM, TN, KT, SPOL, APOL, false, false, PRUNE, DEPTH>),
                         dim3(gx, (unsigned)nb), dim3(MM_THREADS), 0, s, (const T *)A, (const T *)B, (T *)C, g);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Launch shape and Simple-Renorm policies (measured on the product workloads):
//   binary32: every kept term is non-zero almost always -> SR_FULL for both steps;
//             two outputs per lane once the output has 2^25 entries or more, else one;
//   binary16: one output per lane (two rows per lane for MC-Linear, 6% faster than one
//             on its 4096 x 1024 x 1024 layer); the low terms of a step are often zero (they fall
//             below the subnormal grid), almost always as a trailing run, so both steps
//             use the kept-terms form (SR_SUFFIX), which skips the final carry.
template <typename T, int NC, bool AMC, bool BMC, bool BT, bool PRUNE = false>
static hipError_t mm_launch(const MmArgs<T> &g, int64_t batches, const void *A, const void *B, void *C,
                            hipStream_t s) {
  if constexpr (sizeof(T) == 8) {  // binary64: as binary32, one output per lane (twice the registers)
    return mm_launch_tile<T, NC, AMC, BMC, BT, 1, 1, SR_FULL, SR_FULL, 16, PRUNE>(g, batches, A, B, C, s);
  } else if constexpr (sizeof(T) == 4) {
    if (g.M * g.N >= ((int64_t)1 << 25))
      return mm_launch_tile<T, NC, AMC, BMC, BT, 1, 2, SR_FULL, SR_FULL, 16, PRUNE>(g, batches, A, B, C, s);
    // up to 2^20 outputs in all (at most 4 wavefronts per SIMD): the operands of 8 steps
    // are read from LDS before the steps run
    if constexpr (!PRUNE)
      if (g.M * g.N <= ((int64_t)1 << 20) / (batches > 0 ? batches : 1))
        return mm_launch_tile<T, NC, AMC, BMC, BT, 1, 1, SR_FULL, SR_FULL, 16, PRUNE, 8>(g, batches, A, B, C, s);
    return mm_launch_tile<T, NC, AMC, BMC, BT, 1, 1, SR_FULL, SR_FULL, 16, PRUNE>(g, batches, A, B, C, s);
  } else {
    // MC-Linear: two rows of x per lane share each weight value; 32-step tiles (2.5%
    // faster); at nc = 3 the operands of two steps are read before they run (3.18 ->
    // 3.05 ms per 4096 x 1024 x 1024 layer; the same for the 1024^3 MC x MC product was
    // slower: 1.26 -> 1.31 ms)
    if constexpr (BT && NC == 3)
      return mm_launch_tile<T, NC, AMC, BMC, BT, 2, 1, SR_SUFFIX, SR_SUFFIX, 32, false, 2>(g, batches, A, B, C, s);
    if constexpr (BT)
      return mm_launch_tile<T, NC, AMC, BMC, BT, 2, 1, SR_SUFFIX, SR_SUFFIX, NC <= 3 ? 32 : 16>(g, batches, A, B, C, s);
    // 32-step LDS tiles halve the per-tile staging and barriers (1024^3: nc = 2 8%
    // faster than 16 steps, nc = 3 4% at eight wavefronts per SIMD; 64 steps slower)
    constexpr int KT = NC <= 3 ? 32 : 16;
    return mm_launch_tile<T, NC, AMC, BMC, BT, 1, 1, SR_SUFFIX, SR_SUFFIX, KT, PRUNE>(g, batches, A, B, C, s);
  }
}

template <typename T, int NC>
static hipError_t mm_kinds(const MmArgs<T> &g, int64_t batches, const void *A, int a_mc, const void *B, int b_mc,
                           int b_trans, int prune, void *C, hipStream_t s) {
  if (prune) {  // pruned MC x MC product
    if (a_mc && b_mc && !b_trans) return mm_launch<T, NC, true, true, false, true>(g, batches, A, B, C, s);
    return hipErrorInvalidValue;
  }
  if (b_trans) {
    // linear layer: plain input times MC weight stored [out][in]
    if (!a_mc && b_mc) return mm_launch<T, NC, false, true, true>(g, batches, A, B, C, s);
    return hipErrorInvalidValue;
  }
  if (a_mc && b_mc) return mm_launch<T, NC, true, true, false>(g, batches, A, B, C, s);
  if (a_mc) return mm_launch<T, NC, true, false, false>(g, batches, A, B, C, s);
  return mm_launch<T, NC, false, true, false>(g, batches, A, B, C, s);
}

template <typename T>
static hipError_t mm_dispatch(int nc, const MmArgs<T> &g, int64_t batches, const void *A, int a_mc, const void *B,
                              int b_mc, int b_trans, int prune, void *C, hipStream_t s) {
  switch (nc) {
    case 1: return mm_kinds<T, 1>(g, batches, A, a_mc, B, b_mc, b_trans, prune, C, s);
    case 2: return mm_kinds<T, 2>(g, batches, A, a_mc, B, b_mc, b_trans, prune, C, s);
    case 3: return mm_kinds<T, 3>(g, batches, A, a_mc, B, b_mc, b_trans, prune, C, s);
    case 4: return mm_kinds<T, 4>(g, batches, A, a_mc, B, b_mc, b_trans, prune, C, s);
  }
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t mm_typed(const MmLaunch &L, hipStream_t s) {
  MmArgs<T> g;
  g.M = L.M;
  g.N = L.N;
  g.K = L.K;
  g.a_plane = L.a_plane;
  g.b_plane = L.b_plane;
  g.c_plane = L.B1 * L.B2 * L.M * L.N;
  g.B2 = L.B2;
  g.bb0 = 0;
  g.a_s1 = L.a_s1;
  g.a_s2 = L.a_s2;
  g.b_s1 = L.b_s1;
  g.b_s2 = L.b_s2;
  g.mode = L.mode;
  g.y = (const T *)L.y;
  g.y_plane = L.y_plane;
  g.y_ld = L.y_ld;
  g.alpha = (T)L.alpha;
  g.beta = (T)L.beta;
  return mm_dispatch<T>(L.nc, g, L.B1 * L.B2, L.A, L.a_mc, L.B, L.b_mc, L.b_trans, L.prune, L.C, s);
}

hipError_t launch_matmul_general(const MmLaunch &L, hipStream_t stream) {
  if (L.dtype == 0) return mm_typed<_Float16>(L, stream);
  if (L.dtype == 2) return mm_typed<double>(L, stream);
  return mm_typed<float>(L, stream);
}

hipError_t launch_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                         const void *B, int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream) {
  MmLaunch L;
  L.dtype = dtype;
  L.nc = nc;
  L.M = M;
  L.N = N;
  L.K = K;
  L.A = A;
  L.a_mc = a_mc;
  L.a_plane = M * K;
  L.B = B;
  L.b_mc = b_mc;
  L.b_trans = b_trans;
  L.b_plane = K * N;
  L.C = C;
  if (bias != nullptr) {
    L.mode = 1;
    L.y = bias;
    L.y_plane = N;
    L.y_ld = 0;
  }
  return launch_matmul_general(L, stream);
}

}  // namespace mcf
