/*
 * mcf_oracle.c -- plain, slow CPU oracle for multi-component floating point (MCF)
 * arithmetic as defined in "MCTensor: A High-Precision Deep Learning Library with
 * Multi-Component Floating-Point" (Yu, Guo, Li, Yuan, De Sa; arXiv 2207.08867).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * includes this file; only the test-suite, the smoke check and the CPU-baseline leg
 * of the benchmark load it.  It shares no code, header, table or constant with the
 * HIP implementation.
 *
 * Number model (Section 2.1 and Appendix A.2.1 write every step as fl(.), one
 * rounding in the component format):
 *   - A component value is held in a C double.  Every double handled here is
 *     exactly representable in the component format (binary16, binary32 or
 *     binary64).
 *   - fl(.) is IEEE-754 round-to-nearest-even into the component format, with
 *     gradual underflow and overflow to infinity.  It is implemented from the IEEE
 *     definition in round_to() below, on top of an exact or correctly-rounded double.
 *   - + - : the double sum of two binary16 values is exact; for binary32 the double
 *     sum is one extra rounding that is innocuous because 53 >= 2*24+2 (Figueroa,
 *     "When is double rounding innocuous?", SIGNUM 1995).
 *   - *   : the double product of two binary16/binary32 values is exact.
 *   - /   : correctly-rounded double quotient, then fl(.); innocuous by the same
 *     theorem (53 >= 2p+2 for p = 11 and p = 24).
 *   - fma : exact product, double sum with its exact remainder, then fl(.) with the
 *     remainder's sign used to break a tie (see fl_fma); binary64: the C library's
 *     fma, which rounds once.
 *   - binary64 components: every double operation above is already the correctly
 *     rounded binary64 result, and fl(.) is the identity on doubles.  The binary64
 *     component exponential is e^x in binary128 (libquadmath's expq), accepted when a
 *     2^-100 relative margin around it rounds to one binary64 value; the few other
 *     arguments are decided in oracle/__init__.py with 80-digit decimal arithmetic, and
 *     Exp-MCN then takes the component exponentials as inputs.
 *   - exp : the component exponential is taken to be correctly rounded (the paper
 *     calls torch.exp and fixes no accuracy); computed as fl(.) of a double
 *     (binary16) or long double (binary32) exponential.  Exhaustive pinning for
 *     binary16 lives in the tests.
 * Build with -ffp-contract=off and without fast-math; mcf_oracle_check_env()
 * verifies that the SSE flush-to-zero / denormals-are-zero bits are clear.
 *
 * Layout of array arguments: component-major ("planar") -- component c of element i
 * is at index c*n + i.  binary16 data are passed as raw uint16 bit patterns,
 * binary32 data as float.
 */
#include <math.h>
#include <quadmath.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <xmmintrin.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define FMT_F16 0
#define FMT_F32 1
#define FMT_F64 2
#define MAXC 8 /* largest component count handled by the fixed-size scratch arrays */

/* ------------------------------------------------------------------------------ */
/* Component formats and rounding                                                   */
/* ------------------------------------------------------------------------------ */

typedef struct {
  int p;    /* significand bits, hidden bit included */
  int emin; /* exponent of the smallest normal number */
  int emax; /* exponent of the largest finite number */
} fmt_desc;

static const fmt_desc FMTS[3] = {{11, -14, 15}, {24, -126, 127}, {53, -1022, 1023}};

/* Round the real number x + r to the format, where x is a double and r is an
 * infinitesimal remainder whose sign is dir (-1, 0 or +1).  IEEE round to nearest,
 * ties to even, gradual underflow, overflow to infinity. */
static double round_to(int f, double x, int dir) {
  const fmt_desc *d = &FMTS[f];
  if (isnan(x) || isinf(x)) return x;
  if (x == 0.0) {
    if (dir == 0) return x;
    return dir > 0 ? 0.0 : -0.0; /* |x + r| is far below half the smallest subnormal */
  }
  int neg = signbit(x) ? 1 : 0;
  double ax = fabs(x);
  int mdir = neg ? -dir : dir; /* direction of the remainder for the magnitude */
  int e2;
  frexp(ax, &e2);          /* ax = m * 2^e2 with m in [0.5, 1): leading bit at 2^(e2-1) */
  int lead = e2 - 1;
  int q = lead - (d->p - 1); /* exponent of the last significand bit */
  int qmin = d->emin - (d->p - 1);
  if (q < qmin) q = qmin;    /* subnormal range: fixed quantum 2^qmin */
  double scaled = ldexp(ax, -q); /* exact: power-of-two scaling, scaled < 2^p */
  double n = floor(scaled);
  double frac = scaled - n;      /* exact: scaled < 2^53 */
  if (frac > 0.5) {
    n += 1.0;
  } else if (frac == 0.5) {
    if (mdir > 0)
      n += 1.0;
    else if (mdir == 0 && fmod(n, 2.0) != 0.0)
      n += 1.0;
  }
  double r = ldexp(n, q);
  if (r >= ldexp(1.0, d->emax + 1)) r = INFINITY;
  return neg ? -r : r;
}

static double fl(int f, double x) { return round_to(f, x, 0); }

static double fl_add(int f, double a, double b) { return fl(f, a + b); }
static double fl_sub(int f, double a, double b) { return fl(f, a - b); }
static double fl_mul(int f, double a, double b) { return fl(f, a * b); }
static double fl_div(int f, double a, double b) { return fl(f, a / b); }

/* fma(a, b, c) rounded once.  a*b is exact in double; s = a*b + c is rounded in
 * double and t is its exact remainder (Knuth's six-operation sum in double, used here
 * only as exact double-precision bookkeeping).  fl(s) is the correctly rounded result
 * unless s sits exactly on a tie of the component format, where t decides. */
static double fl_fma(int f, double a, double b, double c) {
  if (f == FMT_F64) return fma(a, b, c); /* the C library's fma rounds once */
  double pr = a * b;
  double s = pr + c;
  double bv = s - pr;
  double av = s - bv;
  double t = (pr - av) + (c - bv);
  if (isnan(t) || isinf(s)) return fl(f, s);
  return round_to(f, s, t > 0 ? 1 : (t < 0 ? -1 : 0));
}

/* Correctly rounded component exponential (a reading: the paper calls torch.exp). */
static double fl_exp(int f, double a) {
  if (f == FMT_F16) return fl(f, exp(a));
  long double e = expl((long double)a);
  double hi = (double)e;
  long double lo = e - (long double)hi;
  return round_to(f, hi, lo > 0 ? 1 : (lo < 0 ? -1 : 0));
}

/* binary16 bit pattern <-> double, from the IEEE-754 definition. */
static double f16_decode(uint16_t h) {
  int s = h >> 15, e = (h >> 10) & 0x1f, m = h & 0x3ff;
  double v;
  if (e == 0x1f)
    v = m ? NAN : INFINITY;
  else if (e == 0)
    v = ldexp((double)m, -24);
  else
    v = ldexp((double)(m + 1024), e - 25);
  return s ? -v : v;
}

static uint16_t f16_encode(double v) { /* v must be exactly representable */
  uint16_t s = signbit(v) ? 0x8000 : 0;
  double a = fabs(v);
  if (isnan(v)) return 0x7e00;
  if (isinf(v)) return s | 0x7c00;
  if (a == 0.0) return s;
  if (a < ldexp(1.0, -14)) return s | (uint16_t)(a * ldexp(1.0, 24));
  int e2;
  double m = frexp(a, &e2); /* a = m 2^e2, m in [0.5,1) */
  int e = e2 - 1;           /* a = (1.f) 2^e */
  uint16_t mant = (uint16_t)((m * 2.0 - 1.0) * 1024.0);
  return s | (uint16_t)((e + 15) << 10) | mant;
}

static double load_c(int f, const void *base, int64_t idx) {
  if (f == FMT_F16) return f16_decode(((const uint16_t *)base)[idx]);
  if (f == FMT_F64) return ((const double *)base)[idx];
  return (double)((const float *)base)[idx];
}

static void store_c(int f, void *base, int64_t idx, double v) {
  if (f == FMT_F16)
    ((uint16_t *)base)[idx] = f16_encode(v);
  else if (f == FMT_F64)
    ((double *)base)[idx] = v;
  else
    ((float *)base)[idx] = (float)v;
}

/* ------------------------------------------------------------------------------ */
/* Error-free transformations (Appendix A.2.1)                                      */
/* ------------------------------------------------------------------------------ */

/* Two-Sum (Knuth's error-free sum): s = fl(a+b) and the exact rounding error
 * a + b - s, recovered from each operand's share of s (s - a, then s minus that
 * share) and what rounding removed from each operand; the error is the sum of the
 * two removed parts.  Six operations, in the order that fixes the sign of a zero
 * error. */
static void two_sum(int f, double a, double b, double *s, double *e) {
  double sum = fl_add(f, a, b);
  double share_b = fl_sub(f, sum, a);
  double share_a = fl_sub(f, sum, share_b);
  double lost_b = fl_sub(f, b, share_b);
  double lost_a = fl_sub(f, a, share_a);
  *s = sum;
  *e = fl_add(f, lost_a, lost_b);
}

/* Two-Prod, FMA variant: p = fl(a*b), e = fl(a*b - p) in one rounding. */
static void two_prod(int f, double a, double b, double *p, double *e) {
  *p = fl_mul(f, a, b);
  *e = fl_fma(f, a, b, -*p);
}

/* Simple-Renorm: move the zero components back.  Reading used throughout: every one
 * of the m inputs is scanned (the prose says all non-zero values are extracted) and
 * the first r non-zero ones are kept in order; empty slots are +0. */
static void simple_renorm(const double *h, int m, int r, double *b) {
  int k = 0;
  for (int i = 0; i < r; ++i) b[i] = 0.0;
  for (int i = 0; i < m; ++i) {
    if (h[i] != 0.0 && k < r) {
      b[k] = h[i];
      k += 1;
    }
  }
}

/* Renormalize (Priest variant, Appendix A.2.1).  Readings: the first sweep runs over
 * the components that exist (i = 1..n-1); t_0 = 0 is kept; the value left in s after
 * the second sweep is emitted if a slot is free, so no part of the sum is dropped. */
static void renormalize(int f, const double *x, int n, int r, double *b) {
  double t[MAXC + 1];
  double s = x[0];
  t[0] = 0.0;
  for (int i = 1; i < n; ++i) two_sum(f, x[i], s, &s, &t[i]);
  int k = 0;
  for (int i = 0; i < r; ++i) b[i] = 0.0;
  for (int i = 0; i < n; ++i) {
    double e;
    two_sum(f, s, t[i], &s, &e);
    if (e != 0.0) {
      if (k < r) b[k] = s;
      s = e;
      k += 1;
    }
  }
  if (k < r) b[k] = s;
}

/* Grow-ExpN (Section 2.1): an n-component value plus a plain value v. */
static void grow_expn(int f, const double *x, int n, double v, double *out) {
  double h[MAXC + 1];
  double Q = v;
  for (int i = 1; i <= n; ++i) {
    int k = n + 1 - i;
    two_sum(f, x[k - 1], Q, &Q, &h[k]);
  }
  h[0] = Q;
  simple_renorm(h, n + 1, n, out);
}

/* ScalingN (Appendix A.2.1): an m-component value times a plain value v.  With
 * expand the m+1 terms are all kept, otherwise m. */
static void scaling_n(int f, const double *x, int m, double v, int expand, double *out) {
  double h[MAXC + 1];
  double e = 0.0;
  for (int i = 0; i < m; ++i) {
    double hp, e1, e2;
    two_prod(f, x[i], v, &hp, &e1);
    two_sum(f, hp, e, &h[i], &e2);
    e = fl_add(f, e1, e2);
  }
  h[m] = e;
  simple_renorm(h, m + 1, expand ? m + 1 : m, out);
}

/* Add-MCN (Appendix A.2.1): sum of two n-component values. */
static void add_mcn(int f, const double *x, const double *y, int n, double *out) {
  double h[MAXC + 1];
  double e = 0.0;
  for (int i = 0; i < n; ++i) {
    double hp, e1, e2;
    two_sum(f, x[i], y[i], &hp, &e1);
    two_sum(f, hp, e, &h[i], &e2);
    e = fl_add(f, e1, e2);
  }
  h[n] = e;
  simple_renorm(h, n + 1, n, out);
}

/* Div-MCN (Appendix A.2.1): long division, n+1 quotient digits, n corrections. */
static void div_mcn(int f, const double *x_in, const double *y, int n, double *out) {
  double h[MAXC + 1], x[MAXC] = {0.0}, s[MAXC], neg[MAXC];
  for (int i = 0; i < n; ++i) x[i] = x_in[i];
  double q = fl_div(f, x[0], y[0]);
  h[0] = q;
  for (int i = 1; i <= n; ++i) {
    scaling_n(f, y, n, q, 0, s);
    for (int c = 0; c < n; ++c) neg[c] = -s[c]; /* negation is exact */
    double r[MAXC];
    add_mcn(f, x, neg, n, r);
    for (int c = 0; c < n; ++c) x[c] = r[c];
    q = fl_div(f, x[0], y[0]);
    h[i] = q;
  }
  simple_renorm(h, n + 1, n, out);
}

/* DivN (Appendix A.2.1): plain value over an n-component value, by padding the
 * plain value with zero components. */
static void div_n(int f, double v, const double *y, int n, double *out) {
  double x[MAXC];
  x[0] = v;
  for (int i = 1; i < n; ++i) x[i] = 0.0;
  div_mcn(f, x, y, n, out);
}

/* Mult-MCN, fast version (Appendix A.2.1): x / (1/y), each quotient renormalized. */
static void mult_mcn(int f, const double *x, const double *y, int n, double *out) {
  double one[MAXC], q[MAXC], yinv[MAXC];
  one[0] = 1.0;
  for (int i = 1; i < n; ++i) one[i] = 0.0;
  div_mcn(f, one, y, n, q);
  renormalize(f, q, n, n, yinv);
  div_mcn(f, x, yinv, n, q);
  renormalize(f, q, n, n, out);
}

/* Mult-MCN-Slow (Appendix A.2.1): product digits by repeated division.  p = fl(x_0
 * y_0) is the first digit; then n times the remainder x = Add-MCN(x, -DivN(p, y)) is
 * formed and its next digit p = fl(x_0 y_0) taken; the n+1 digits pass through
 * Simple-Renorm. */
static void mult_mcn_slow(int f, const double *x_in, const double *y, int n, double *out) {
  double h[MAXC + 1], x[MAXC] = {0.0}, d[MAXC], neg[MAXC], r[MAXC];
  for (int i = 0; i < n; ++i) x[i] = x_in[i];
  double p = fl_mul(f, x[0], y[0]);
  h[0] = p;
  for (int i = 1; i <= n; ++i) {
    div_n(f, p, y, n, d);
    for (int c = 0; c < n; ++c) neg[c] = -d[c]; /* negation is exact */
    add_mcn(f, x, neg, n, r);
    for (int c = 0; c < n; ++c) x[c] = r[c];
    p = fl_mul(f, x[0], y[0]);
    h[i] = p;
  }
  simple_renorm(h, n + 1, n, out);
}

/* Square-MCN (Appendix A.2.1).  Reading: the printed first step fl(2^{x_0}) is taken
 * as fl(x_0 x_0) (the algorithm squares x).  h = (fl(x_0 x_0), 0, ..., 0), then
 * h = Grow-ExpN(h, fl(2 x_0 x_1)) (2 x_0 is exact, so this is one rounding of the
 * product); with n = 1 there is no x_1 and the addend is zero. */
static void square_mcn(int f, const double *x, int n, double *out) {
  double h[MAXC];
  h[0] = fl_mul(f, x[0], x[0]);
  for (int i = 1; i < n; ++i) h[i] = 0.0;
  double v = n > 1 ? fl_mul(f, fl_mul(f, 2.0, x[0]), x[1]) : 0.0;
  grow_expn(f, h, n, v, out);
}

/* Exp-MCN (Appendix A.2.1).  Reading: the factor of step i is exp(x_i) (the printed
 * exp(h_i) is taken as a typo); h starts with one component and ScalingN with expand
 * grows it by one per step, to n components. */
static void exp_mcn(int f, const double *x, int n, double *out) {
  double h[MAXC + 1], t[MAXC + 1];
  int m = 1;
  h[0] = fl_exp(f, x[0]);
  for (int i = 1; i < n; ++i) {
    scaling_n(f, h, m, fl_exp(f, x[i]), 1, t);
    m += 1;
    for (int c = 0; c < m; ++c) h[c] = t[c];
  }
  for (int c = 0; c < n; ++c) out[c] = h[c];
}

/* ------------------------------------------------------------------------------ */
/* Environment check                                                                */
/* ------------------------------------------------------------------------------ */

/* Returns 0 when the SSE control word has flush-to-zero and denormals-are-zero clear
 * (gradual underflow is part of the number model). */
int mcf_oracle_check_env(void) {
  unsigned int csr = _mm_getcsr();
  return (csr & 0x8040u) ? -1 : 0;
}

int mcf_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------------ */
/* Scalar primitives exported for pinning tests (values as doubles)                  */
/* ------------------------------------------------------------------------------ */

double mcf_oracle_round(int f, double x) { return fl(f, x); }
double mcf_oracle_fl_add(int f, double a, double b) { return fl_add(f, a, b); }
double mcf_oracle_fl_sub(int f, double a, double b) { return fl_sub(f, a, b); }
double mcf_oracle_fl_mul(int f, double a, double b) { return fl_mul(f, a, b); }
double mcf_oracle_fl_div(int f, double a, double b) { return fl_div(f, a, b); }
double mcf_oracle_fl_fma(int f, double a, double b, double c) { return fl_fma(f, a, b, c); }
double mcf_oracle_fl_exp(int f, double a) { return fl_exp(f, a); }
double mcf_oracle_f16_decode(uint16_t h) { return f16_decode(h); }
uint16_t mcf_oracle_f16_encode(double v) { return f16_encode(v); }

/* Vectorised versions over arrays of doubles (for exhaustive pins). op: 0 add, 1 sub,
 * 2 mul, 3 div, 4 fma(a,b,-fl(a*b)) i.e. the Two-Prod error, 5 exp(a), 6 round(a). */
void mcf_oracle_binop_array(int f, int op, int64_t n, const double *a, const double *b, double *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double r;
    switch (op) {
      case 0: r = fl_add(f, a[i], b[i]); break;
      case 1: r = fl_sub(f, a[i], b[i]); break;
      case 2: r = fl_mul(f, a[i], b[i]); break;
      case 3: r = fl_div(f, a[i], b[i]); break;
      case 4: r = fl_fma(f, a[i], b[i], -fl_mul(f, a[i], b[i])); break;
      case 5: r = fl_exp(f, a[i]); break;
      default: r = fl(f, a[i]); break;
    }
    out[i] = r;
  }
}

/* Pinning aid for the binary32 exponential.  fl_exp rounds the long double e^x of
 * expl to binary32; that is the correctly rounded result unless e^x lies closer to a
 * binary32 rounding boundary than expl's error.  This scans every binary32 x with
 * 2^-30 <= |x| <= 105 (outside that range e^x rounds to 1, or to 0 or infinity, far
 * from any boundary) and reports the x whose expl value, moved by the relative amount
 * rel_margin either way, rounds to two different binary32 values.  Up to max_out bit
 * patterns go to out; the return value is how many there are. */
static double round_ld_f32(long double v) {
  double hi = (double)v;
  long double lo = v - (long double)hi;
  return round_to(FMT_F32, hi, lo > 0 ? 1 : (lo < 0 ? -1 : 0));
}

int64_t mcf_oracle_exp32_near_ties(double rel_margin, uint32_t *out, int64_t max_out) {
  int64_t count = 0;
#pragma omp parallel for schedule(dynamic, 1 << 16) reduction(+ : count)
  for (int64_t b = 0; b < ((int64_t)1 << 32); ++b) {
    uint32_t bits = (uint32_t)b;
    float xf;
    memcpy(&xf, &bits, 4);
    double ax = fabs((double)xf);
    if (!(ax >= 0x1p-30 && ax <= 105.0)) continue;
    long double e = expl((long double)xf);
    long double m = (long double)rel_margin;
    if (round_ld_f32(e * (1.0L - m)) != round_ld_f32(e * (1.0L + m))) {
      int64_t slot;
#pragma omp atomic capture
      slot = count++;
      if (slot < max_out) out[slot] = bits;
    }
  }
  return count;
}

/* Two-Sum / Two-Prod on arrays of doubles: outputs s (or p) and e. */
void mcf_oracle_eft_array(int f, int prod, int64_t n, const double *a, const double *b, double *s, double *e) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    if (prod)
      two_prod(f, a[i], b[i], &s[i], &e[i]);
    else
      two_sum(f, a[i], b[i], &s[i], &e[i]);
  }
}

/* ------------------------------------------------------------------------------ */
/* Elementwise MC operations over planar arrays                                     */
/* ------------------------------------------------------------------------------ */

/* Gather element i of a planar operand with xn planes. */
static void gather(int f, const void *base, int xn, int64_t n, int64_t i, double *v) {
  for (int c = 0; c < xn; ++c) v[c] = load_c(f, base, (int64_t)c * n + i);
}

static void scatter(int f, void *base, int nc, int64_t n, int64_t i, const double *v) {
  for (int c = 0; c < nc; ++c) store_c(f, base, (int64_t)c * n + i, v[c]);
}

/* Operation codes for mcf_oracle_elementwise. */
enum { OP_ADD = 0, OP_MUL = 1, OP_DIV = 2, OP_EXP = 3, OP_RENORM = 4, OP_SIMPLE_RENORM = 5,
       OP_SCALING_EXPAND = 6, OP_MUL_SLOW = 7, OP_SQUARE = 8 };

/* out = op(x, y) elementwise over n elements.  x_mc / y_mc say whether an operand is
 * an MC value (nc planes) or a plain tensor (one plane).
 *   ADD : (MC,MC) Add-MCN; (MC,T) and (T,MC) Grow-ExpN.
 *   MUL : (MC,MC) Mult-MCN (fast); (MC,T) and (T,MC) ScalingN without expand.
 *   DIV : (MC,MC) Div-MCN; (T,MC) DivN; (MC,T) Div-MCN with the divisor padded by zeros.
 *   EXP : Exp-MCN of x (MC).
 *   RENORM / SIMPLE_RENORM : x (MC) has nc components, out has nc_out.
 *   SCALING_EXPAND : (MC,T) ScalingN with expand, out has nc+1 components.
 *   MUL_SLOW : (MC,MC) Mult-MCN-Slow.
 *   SQUARE : Square-MCN of x (MC).
 * Returns 0, or -1 on bad arguments. */
int mcf_oracle_elementwise(int f, int op, int nc, int nc_out, int64_t n, const void *x, int x_mc,
                           const void *y, int y_mc, void *out) {
  if (nc < 1 || nc > MAXC || f < FMT_F16 || f > FMT_F64) return -1;
  if (op == OP_EXP && f == FMT_F64) return -1; /* no correctly rounded binary64 exp here */
  int binary = (op == OP_ADD || op == OP_MUL || op == OP_DIV || op == OP_SCALING_EXPAND || op == OP_MUL_SLOW);
  if (binary && !x_mc && !y_mc) return -1;
  if (op == OP_MUL_SLOW && !(x_mc && y_mc)) return -1;
  if (op < OP_ADD || op > OP_SQUARE) return -1;
  if ((op == OP_RENORM || op == OP_SIMPLE_RENORM) && (nc_out < 1 || nc_out > nc)) return -1;
  int xn = x_mc ? nc : 1, yn = y_mc ? nc : 1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double a[MAXC + 1], b[MAXC + 1], r[MAXC + 1];
    for (int c = 0; c < MAXC + 1; ++c) a[c] = b[c] = r[c] = 0.0;
    gather(f, x, xn, n, i, a);
    if (binary) gather(f, y, yn, n, i, b);
    int rn = nc;
    switch (op) {
      case OP_ADD:
        if (x_mc && y_mc)
          add_mcn(f, a, b, nc, r);
        else if (x_mc)
          grow_expn(f, a, nc, b[0], r);
        else
          grow_expn(f, b, nc, a[0], r);
        break;
      case OP_MUL:
        if (x_mc && y_mc)
          mult_mcn(f, a, b, nc, r);
        else if (x_mc)
          scaling_n(f, a, nc, b[0], 0, r);
        else
          scaling_n(f, b, nc, a[0], 0, r);
        break;
      case OP_DIV:
        if (x_mc && y_mc)
          div_mcn(f, a, b, nc, r);
        else if (y_mc)
          div_n(f, a[0], b, nc, r);
        else
          div_mcn(f, a, b, nc, r); /* (MC,T): the divisor is (v, 0, ..., 0) */
        break;
      case OP_EXP:
        exp_mcn(f, a, nc, r);
        break;
      case OP_RENORM:
        renormalize(f, a, nc, nc_out, r);
        rn = nc_out;
        break;
      case OP_SIMPLE_RENORM:
        simple_renorm(a, nc, nc_out, r);
        rn = nc_out;
        break;
      case OP_SCALING_EXPAND:
        scaling_n(f, a, nc, b[0], 1, r);
        rn = nc + 1;
        break;
      case OP_MUL_SLOW:
        mult_mcn_slow(f, a, b, nc, r);
        break;
      case OP_SQUARE:
        square_mcn(f, a, nc, r);
        break;
    }
    scatter(f, out, rn, n, i, r);
  }
  return 0;
}

/* ------------------------------------------------------------------------------ */
/* Matrix products (Appendix A.2.2)                                                  */
/* ------------------------------------------------------------------------------ */

typedef struct {
  int f;
  const void *A; /* MC (nc planes) when a_mc, else one plane */
  int a_mc;
  const void *B;
  int b_mc;
  int64_t K;
  int64_t lda_m, lda_k; /* element strides of A along its row index and along k */
  int64_t ldb_k, ldb_n; /* element strides of B along k and along its column index */
  int64_t a_plane, b_plane;
} mm_args;

/* Term k of output (i, j): the MC factor (nc components) and the plain factor.  When
 * both operands are MC, the plain factor is component `bcomp` of B[k][j]. */
static void mm_term(const mm_args *g, int nc, int64_t i, int64_t j, int64_t k, int bcomp, double *mc,
                    double *plain) {
  if (g->a_mc) {
    for (int c = 0; c < nc; ++c) mc[c] = load_c(g->f, g->A, c * g->a_plane + i * g->lda_m + k * g->lda_k);
    *plain = load_c(g->f, g->B, bcomp * g->b_plane + k * g->ldb_k + j * g->ldb_n);
  } else {
    for (int c = 0; c < nc; ++c) mc[c] = load_c(g->f, g->B, c * g->b_plane + k * g->ldb_k + j * g->ldb_n);
    *plain = load_c(g->f, g->A, i * g->lda_m + k * g->lda_k);
  }
}

/* MM-MCN for one output of an MC matrix times a plain matrix, over the reduction
 * indices k = k0, k0 + kstep, k0 + 2 kstep, ... below K:
 * acc = ScalingN(first term); acc = Add-MCN(acc, ScalingN(next term)) for each
 * further k, the sequential order in which the paper propagates the addition error
 * (Section 2.2; Appendix A.2.2, MV-MCN and MM-MCN).  The full product is k0 = 0,
 * kstep = 1.  No term gives +0 in every component. */
static void mm_entry_plain(const mm_args *g, int nc, int64_t i, int64_t j, int bcomp, int64_t k0, int64_t kstep,
                           double *acc) {
  double mc[MAXC], term[MAXC], t[MAXC], v;
  for (int c = 0; c < nc; ++c) acc[c] = 0.0;
  for (int64_t k = k0; k < g->K; k += kstep) {
    mm_term(g, nc, i, j, k, bcomp, mc, &v);
    scaling_n(g->f, mc, nc, v, 0, term);
    if (k == k0) {
      for (int c = 0; c < nc; ++c) acc[c] = term[c];
    } else {
      add_mcn(g->f, acc, term, nc, t);
      for (int c = 0; c < nc; ++c) acc[c] = t[c];
    }
  }
}

/* One output C[i][j].  MC x plain and plain x MC follow MM-MCN directly.  MC x MC is
 * not defined in the paper (its matrix operators take one MC and one plain operand);
 * reading: linearity over the components of B,
 *   C = MM(A, B^(0)) (+) MM(A, B^(1)) (+) ... (+) MM(A, B^(nc-1)),
 * with (+) = Add-MCN applied left to right. */
static void mm_entry(const mm_args *g, int nc, int64_t i, int64_t j, double *out) {
  if (g->a_mc && g->b_mc) {
    double part[MAXC], t[MAXC];
    mm_entry_plain(g, nc, i, j, 0, 0, 1, out);
    for (int b = 1; b < nc; ++b) {
      mm_entry_plain(g, nc, i, j, b, 0, 1, part);
      add_mcn(g->f, out, part, nc, t);
      for (int c = 0; c < nc; ++c) out[c] = t[c];
    }
  } else {
    mm_entry_plain(g, nc, i, j, 0, 0, 1, out);
  }
}

/* Pruned MC x MC product, one output (a reading of the faster contraction the paper
 * leaves open, Section 2.2: the component products A^(a) B^(b) with a + b >= nc are
 * of the order of u^nc relative, the size of MM-MCN's own error, and are left out).
 * Component b of B multiplies the first nc - b components of A in MM-MCN order with
 * nc - b components; the parts, padded with zeros to nc components, are combined
 * left to right with Add-MCN:
 *   C = MM_nc(A, B^(0)) (+) MM_{nc-1}(A[:nc-1], B^(1)) (+) ... (+) MM_1(A[:1], B^(nc-1)). */
static void mm_entry_pruned(const mm_args *g, int nc, int64_t i, int64_t j, double *out) {
  double part[MAXC], t[MAXC];
  mm_entry_plain(g, nc, i, j, 0, 0, 1, out);
  for (int b = 1; b < nc; ++b) {
    for (int c = 0; c < MAXC; ++c) part[c] = 0.0;
    mm_entry_plain(g, nc - b, i, j, b, 0, 1, part);
    add_mcn(g->f, out, part, nc, t);
    for (int c = 0; c < nc; ++c) out[c] = t[c];
  }
}

/* The pruned product of two MC matrices at the `count` positions (as
 * mcf_oracle_matmul with both operands MC). */
int mcf_oracle_matmul_pruned(int f, int nc, int64_t M, int64_t N, int64_t K, const void *A, const void *B,
                             const int64_t *rows, const int64_t *cols, int64_t count, void *out) {
  if (nc < 1 || nc > MAXC) return -1;
  mm_args g = {f, A, 1, B, 1, K, K, 1, N, 1, M * K, K * N};
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / N;
    int64_t j = rows ? cols[t] : t % N;
    double r[MAXC];
    mm_entry_pruned(&g, nc, i, j, r);
    scatter(f, out, nc, count, t, r);
  }
  return 0;
}

/* C = A x B with A [M][K] and B [K][N] row-major planes (nc planes when MC, one when
 * plain; at least one MC), evaluated only at the `count` positions (rows[t], cols[t]);
 * out is [nc][count].  rows == NULL means every position in row-major order (count
 * must then be M*N).  Returns 0, or -1 on bad arguments. */
int mcf_oracle_matmul(int f, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                      const void *B, int b_mc, const int64_t *rows, const int64_t *cols, int64_t count,
                      void *out) {
  if (nc < 1 || nc > MAXC || (!a_mc && !b_mc)) return -1;
  mm_args g = {f, A, a_mc, B, b_mc, K, K, 1, N, 1, M * K, K * N};
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / N;
    int64_t j = rows ? cols[t] : t % N;
    double r[MAXC];
    mm_entry(&g, nc, i, j, r);
    scatter(f, out, nc, count, t, r);
  }
  return 0;
}

/* K-split product, one output and one component of B (the whole B when it is
 * plain).  Reading of the paper's remark that an accurate sum of N MC values can be
 * had in O(nc log N) depth (Section 2.2): the K reduction steps are dealt out
 * round-robin to S = min(S, K) slices, slice s taking k = s, s + S, s + 2S, ...;
 * each slice accumulates its terms in MM-MCN order; the S slice sums are then
 * combined by a pairwise tree of Add-MCN: at each level, entry q of the next level
 * is Add-MCN(entry 2q, entry 2q+1), and an odd last entry moves up unchanged, until
 * one value is left.  S = 1 is MM-MCN itself. */
static void mm_entry_split_plain(const mm_args *g, int nc, int64_t i, int64_t j, int bcomp, int64_t S,
                                 double *work, double *out) {
  if (g->K == 0) {
    for (int c = 0; c < nc; ++c) out[c] = 0.0;
    return;
  }
  if (S > g->K) S = g->K;
  for (int64_t s = 0; s < S; ++s) mm_entry_plain(g, nc, i, j, bcomp, s, S, work + s * nc);
  for (int64_t count = S; count > 1; count = (count + 1) / 2) {
    for (int64_t q = 0; 2 * q < count; ++q) {
      double t[MAXC];
      if (2 * q + 1 < count)
        add_mcn(g->f, work + 2 * q * nc, work + (2 * q + 1) * nc, nc, t);
      else
        for (int c = 0; c < nc; ++c) t[c] = work[2 * q * nc + c];
      for (int c = 0; c < nc; ++c) work[q * nc + c] = t[c];
    }
  }
  for (int c = 0; c < nc; ++c) out[c] = work[c];
}

/* C = A x B by the K-split above (MC x MC: one K-split product per component of B,
 * combined left to right with Add-MCN, as in mm_entry).  Arguments as for
 * mcf_oracle_matmul, plus the slice count S >= 1.  Returns 0, or -1 on bad
 * arguments or when scratch memory cannot be had. */
int mcf_oracle_matmul_splitk(int f, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                             const void *B, int b_mc, int64_t S, const int64_t *rows, const int64_t *cols,
                             int64_t count, void *out) {
  if (nc < 1 || nc > MAXC || (!a_mc && !b_mc) || S < 1) return -1;
  mm_args g = {f, A, a_mc, B, b_mc, K, K, 1, N, 1, M * K, K * N};
  int64_t slots = S < K ? S : (K > 0 ? K : 1);
  int failed = 0;
#pragma omp parallel
  {
    double *work = (double *)malloc((size_t)slots * nc * sizeof(double));
    if (!work) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < count; ++t) {
      if (!work) continue;
      int64_t i = rows ? rows[t] : t / N;
      int64_t j = rows ? cols[t] : t % N;
      double r[MAXC];
      mm_entry_split_plain(&g, nc, i, j, 0, S, work, r);
      if (a_mc && b_mc) {
        for (int b = 1; b < nc; ++b) {
          double part[MAXC], sum[MAXC];
          mm_entry_split_plain(&g, nc, i, j, b, S, work, part);
          add_mcn(f, r, part, nc, sum);
          for (int c = 0; c < nc; ++c) r[c] = sum[c];
        }
      }
      scatter(f, out, nc, count, t, r);
    }
    free(work);
  }
  return failed ? -1 : 0;
}

/* MC-Linear forward (Section 2.3): the product of the MC weight and the plain input,
 * Y[t][o] = sum over i of W[o][i] * X[t][i] in MM-MCN order, then Add-MCN with the
 * MC bias[o] when bias is given.  X is plain [T][I], W is [nc][O][I], bias [nc][O].
 * Evaluated at the positions (rows[t], cols[t]) = (token, output feature); out is
 * [nc][count]. */
int mcf_oracle_linear(int f, int nc, int64_t T, int64_t I, int64_t O, const void *X, const void *W,
                      const void *bias, const int64_t *rows, const int64_t *cols, int64_t count, void *out) {
  if (nc < 1 || nc > MAXC) return -1;
  /* As a product A x B: A = X (plain), B[k=i][j=o] = W[o][i] (MC). */
  mm_args g = {f, X, 0, W, 1, I, I, 1, 1, I, T * I, O * I};
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / O;
    int64_t j = rows ? cols[t] : t % O;
    double r[MAXC];
    mm_entry_plain(&g, nc, i, j, 0, 0, 1, r);
    if (bias) {
      double b[MAXC], s[MAXC];
      for (int c = 0; c < nc; ++c) b[c] = load_c(f, bias, (int64_t)c * O + j);
      add_mcn(f, r, b, nc, s);
      for (int c = 0; c < nc; ++c) r[c] = s[c];
    }
    scatter(f, out, nc, count, t, r);
  }
  return 0;
}

/* ------------------------------------------------------------------------------ */
/* Correctly rounded binary64 exponential (first step) and Exp-MCN from given         */
/* component exponentials                                                             */
/* ------------------------------------------------------------------------------ */

/* e^a in binary128, rounded to binary64 when every value within 2^-100 (relative) of it
 * rounds to the same binary64 number; *unsure = 1 otherwise. */
static double exp64_first(double a, int *unsure) {
  *unsure = 0;
  if (isnan(a)) return a;
  if (a > 710.0) return INFINITY; /* e^710 exceeds the largest binary64 number */
  if (a < -746.0) return 0.0;     /* e^-746 is below half the smallest subnormal */
  __float128 q = expq((__float128)a);
  __float128 d = q * (__float128)ldexp(1.0, -100);
  double lo = (double)(q - d), hi = (double)(q + d);
  if (lo != hi) *unsure = 1;
  return (double)q;
}

void mcf_oracle_exp64_first(int64_t n, const double *x, double *out, int32_t *unsure) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    int u;
    out[i] = exp64_first(x[i], &u);
    unsure[i] = u;
  }
}

/* Exp-MCN (Appendix A.2.1, reading E1) from the component exponentials E[c][i] (values
 * of the format f): h = (E_0), then h = ScalingN(h, E_c) with expand. */
int mcf_oracle_exp_mcn_given(int f, int nc, int64_t n, const void *E, void *out) {
  if (nc < 1 || nc > MAXC) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double h[MAXC + 1], t[MAXC + 1];
    int m = 1;
    h[0] = load_c(f, E, i);
    for (int c = 1; c < nc; ++c) {
      scaling_n(f, h, m, load_c(f, E, (int64_t)c * n + i), 1, t);
      m += 1;
      for (int k = 0; k < m; ++k) h[k] = t[k];
    }
    for (int c = 0; c < nc; ++c) store_c(f, out, (int64_t)c * n + i, h[c]);
  }
  return 0;
}

/* Test-input search: random binary64 x uniform in [lo, hi] (a SplitMix64 sequence from
 * seed) whose e^x lies within rel (relative, rel >> 2^-100) of a binary64 rounding
 * boundary.  Writes up to max_out of them to out and returns how many were found. */
int64_t mcf_oracle_exp64_near_midpoints(double lo, double hi, uint64_t seed, int64_t tries, double rel,
                                        double *out, int64_t max_out) {
  int64_t found = 0;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < tries; ++t) {
    uint64_t z = seed + (uint64_t)t * 0x9e3779b97f4a7c15ull;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z = z ^ (z >> 31);
    double x = lo + (hi - lo) * ((double)(z >> 11) * ldexp(1.0, -53));
    __float128 q = expq((__float128)x);
    double r = (double)q;
    if (r == 0.0 || isinf(r)) continue;
    __float128 up = ((__float128)r + (__float128)nextafter(r, INFINITY)) / 2;
    __float128 dn = ((__float128)r + (__float128)nextafter(r, -INFINITY)) / 2;
    __float128 d1 = fabsq(q - up), d2 = fabsq(q - dn);
    __float128 d = d1 < d2 ? d1 : d2;
    if (d < q * (__float128)rel) {
      int64_t k;
#pragma omp atomic capture
      k = found++;
      if (k < max_out) out[k] = x;
    }
  }
  return found;
}

/* ------------------------------------------------------------------------------ */
/* binary16 components with scaled low components (reading SC1)                      */
/* ------------------------------------------------------------------------------ */

/* The paper observes that binary16 components cannot hold errors below the smallest
 * subnormal, 2^-24, and that scaling the smaller components by a factor 2^-k would
 * capture smaller errors (Section 2.4).  Reading SC1: component c of a stored value is
 * a binary16 number y_c that stands for x_c = 2^(-11 c) y_c, so level c of a value lives
 * on the binary16 grid scaled by 2^(-11 c) -- one binary16 precision below level c-1.
 * The algorithms are the paper's, with every quantity given a level and every fl()
 * taken in the binary16 format of the level of its result,
 *     fl_l(v) = 2^(-11 l) RN16(2^(11 l) v):
 *   - the terms an operation combines share one level l (component i of an operand
 *     at slot level L is at level L + i; a product x_i v is at the sum of the levels);
 *   - the rounding error of an operation at level l -- the second output of Two-Sum
 *     or Two-Prod -- and the carry summed from such errors belong to level l + 1;
 *   - Simple-Renorm moving a value to an earlier slot j rounds it into level j.
 * Only operations whose operands pair equal levels are defined this way: Add-MCN,
 * ScalingN, and the products and MC-Linear built from them. */
#define SC_SHIFT 11

static double fl_lv(int lv, double v) {
  return ldexp(round_to(FMT_F16, ldexp(v, SC_SHIFT * lv), 0), -SC_SHIFT * lv);
}

/* Two-Sum at level lv: the six operations of Knuth's error-free sum, each rounded at
 * level lv; the error they return is exact and is used at level lv + 1. */
static void sc_two_sum(int lv, double a, double b, double *s, double *e) {
  double sum = fl_lv(lv, a + b);
  double share_b = fl_lv(lv, sum - a);
  double share_a = fl_lv(lv, sum - share_b);
  double lost_b = fl_lv(lv, b - share_b);
  double lost_a = fl_lv(lv, a - share_a);
  *s = sum;
  *e = fl_lv(lv, lost_a + lost_b);
}

/* Two-Prod (FMA variant) at level lv: p = fl_lv(a b); the fused remainder a b - p,
 * exact in double, is rounded once at level lv + 1. */
static void sc_two_prod(int lv, double a, double b, double *p, double *e) {
  *p = fl_lv(lv, a * b);
  *e = fl_lv(lv + 1, a * b - *p);
}

/* Simple-Renorm of h[0..m-1] (h[i] at level L + i) into r slots: the first r non-zero
 * values in order, the one landing in slot j rounded into level L + j; +0 padding. */
static void sc_simple_renorm(const double *h, int m, int r, int L, double *b) {
  int k = 0;
  for (int i = 0; i < r; ++i) b[i] = 0.0;
  for (int i = 0; i < m; ++i) {
    if (h[i] != 0.0 && k < r) {
      b[k] = fl_lv(L + k, h[i]);
      k += 1;
    }
  }
}

/* ScalingN without expand: x[0..m-1] at levels L.. times a plain value v at level mu. */
static void sc_scaling_n(const double *x, int m, int L, double v, int mu, double *out) {
  double h[MAXC + 1];
  double e = 0.0;
  for (int i = 0; i < m; ++i) {
    const int lv = L + i + mu;
    double hp, e1, e2;
    sc_two_prod(lv, x[i], v, &hp, &e1);
    sc_two_sum(lv, hp, e, &h[i], &e2);
    e = fl_lv(lv + 1, e1 + e2);
  }
  h[m] = e;
  sc_simple_renorm(h, m + 1, m, L + mu, out);
}

/* Add-MCN of x and y, both n components at levels L.. */
static void sc_add_mcn(const double *x, const double *y, int n, int L, double *out) {
  double h[MAXC + 1];
  double e = 0.0;
  for (int i = 0; i < n; ++i) {
    const int lv = L + i;
    double hp, e1, e2;
    sc_two_sum(lv, x[i], y[i], &hp, &e1);
    sc_two_sum(lv, hp, e, &h[i], &e2);
    e = fl_lv(lv + 1, e1 + e2);
  }
  h[n] = e;
  sc_simple_renorm(h, n + 1, n, L, out);
}

static double sc_load(const void *base, int c, int64_t idx) {
  return ldexp(f16_decode(((const uint16_t *)base)[idx]), -SC_SHIFT * c);
}

static void sc_store(void *base, int c, int64_t idx, double v) {
  ((uint16_t *)base)[idx] = f16_encode(ldexp(v, SC_SHIFT * c));
}

/* Elementwise: op 0 = Add-MCN of two MC values, op 1 = ScalingN of an MC value by a
 * plain one (either order).  Arrays are scaled binary16 planes [nc or 1][n]. */
int mcf_oracle_scaled_elementwise(int op, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc,
                                  void *out) {
  if (nc < 1 || nc > MAXC) return -1;
  if (op == 0 && !(x_mc && y_mc)) return -1;
  if (op == 1 && x_mc == y_mc) return -1;
  if (op != 0 && op != 1) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double a[MAXC], b[MAXC], r[MAXC];
    for (int c = 0; c < (x_mc ? nc : 1); ++c) a[c] = sc_load(x, c, (int64_t)c * n + i);
    for (int c = 0; c < (y_mc ? nc : 1); ++c) b[c] = sc_load(y, c, (int64_t)c * n + i);
    if (op == 0)
      sc_add_mcn(a, b, nc, 0, r);
    else if (x_mc)
      sc_scaling_n(a, nc, 0, b[0], 0, r);
    else
      sc_scaling_n(b, nc, 0, a[0], 0, r);
    for (int c = 0; c < nc; ++c) sc_store(out, c, (int64_t)c * n + i, r[c]);
  }
  return 0;
}

/* MM-MCN for one output over the first m components of the MC factor (A when a_mc,
 * else B), the plain factor being component `bcomp` of B (at level bcomp) or the
 * plain operand (level 0): acc = ScalingN(first term), then Add-MCN of each further
 * ScalingN term in k order.  The accumulator's slot c is at level mu + c. */
static void sc_mm_entry_plain(const mm_args *g, int m, int64_t i, int64_t j, int bcomp, double *acc) {
  const int mu = (g->a_mc && g->b_mc) ? bcomp : 0;
  for (int c = 0; c < m; ++c) acc[c] = 0.0;
  for (int64_t k = 0; k < g->K; ++k) {
    double mc[MAXC], term[MAXC], t[MAXC], v;
    if (g->a_mc) {
      for (int c = 0; c < m; ++c) mc[c] = sc_load(g->A, c, c * g->a_plane + i * g->lda_m + k * g->lda_k);
      v = sc_load(g->B, bcomp, bcomp * g->b_plane + k * g->ldb_k + j * g->ldb_n);
    } else {
      for (int c = 0; c < m; ++c) mc[c] = sc_load(g->B, c, c * g->b_plane + k * g->ldb_k + j * g->ldb_n);
      v = sc_load(g->A, 0, i * g->lda_m + k * g->lda_k);
    }
    sc_scaling_n(mc, m, 0, v, mu, term);
    if (k == 0) {
      for (int c = 0; c < m; ++c) acc[c] = term[c];
    } else {
      sc_add_mcn(acc, term, m, mu, t);
      for (int c = 0; c < m; ++c) acc[c] = t[c];
    }
  }
}

/* One output.  MC x plain and plain x MC: MM-MCN.  MC x MC (reading SC1 with the
 * linearity over B's components of the unscaled product): component b of B sits at
 * level b, so its part A B^(b) has levels b, b+1, ...; the levels below the format's
 * last one (nc - 1) are kept, i.e. the part is MM-MCN over the first nc - b
 * components of A with nc - b components at levels b .. nc-1.  Each part, placed at
 * its levels (b leading zero slots), is added left to right with Add-MCN:
 *   C = P_0 (+) (0, P_1) (+) (0, 0, P_2) (+) ... */
static void sc_mm_entry(const mm_args *g, int nc, int64_t i, int64_t j, double *out) {
  sc_mm_entry_plain(g, nc, i, j, 0, out);
  if (!(g->a_mc && g->b_mc)) return;
  for (int b = 1; b < nc; ++b) {
    double part[MAXC], y[MAXC], t[MAXC];
    sc_mm_entry_plain(g, nc - b, i, j, b, part);
    for (int c = 0; c < nc; ++c) y[c] = c < b ? 0.0 : part[c - b];
    sc_add_mcn(out, y, nc, 0, t);
    for (int c = 0; c < nc; ++c) out[c] = t[c];
  }
}

/* C = A x B on scaled binary16 planes, at the `count` positions (as mcf_oracle_matmul). */
int mcf_oracle_scaled_matmul(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                             int b_mc, const int64_t *rows, const int64_t *cols, int64_t count, void *out) {
  if (nc < 1 || nc > MAXC || (!a_mc && !b_mc)) return -1;
  mm_args g = {FMT_F16, A, a_mc, B, b_mc, K, K, 1, N, 1, M * K, K * N};
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / N;
    int64_t j = rows ? cols[t] : t % N;
    double r[MAXC];
    sc_mm_entry(&g, nc, i, j, r);
    for (int c = 0; c < nc; ++c) sc_store(out, c, (int64_t)c * count + t, r[c]);
  }
  return 0;
}

/* MC-Linear forward on scaled binary16 planes: Y[t][o] = MM-MCN over i of
 * ScalingN(W[o][i], X[t][i]) (X plain, level 0), then Add-MCN with bias[o]. */
int mcf_oracle_scaled_linear(int nc, int64_t T, int64_t I, int64_t O, const void *X, const void *W,
                             const void *bias, const int64_t *rows, const int64_t *cols, int64_t count,
                             void *out) {
  if (nc < 1 || nc > MAXC) return -1;
  mm_args g = {FMT_F16, X, 0, W, 1, I, I, 1, 1, I, T * I, O * I};
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / O;
    int64_t j = rows ? cols[t] : t % O;
    double r[MAXC];
    sc_mm_entry_plain(&g, nc, i, j, 0, r);
    if (bias) {
      double b[MAXC], s2[MAXC];
      for (int c = 0; c < nc; ++c) b[c] = sc_load(bias, c, (int64_t)c * O + j);
      sc_add_mcn(r, b, nc, 0, s2);
      for (int c = 0; c < nc; ++c) r[c] = s2[c];
    }
    for (int c = 0; c < nc; ++c) sc_store(out, c, (int64_t)c * count + t, r[c]);
  }
  return 0;
}

/* ------------------------------------------------------------------------------ */
/* Exact arithmetic checker                                                          */
/* ------------------------------------------------------------------------------ */

/* A long fixed-point accumulator: value = sum_d dig[d] * 2^(32*d - ACC_BIAS), digits
 * held in int64 so that up to 2^31 signed additions need no intermediate carry.
 * Every double is a multiple of 2^-1074 below 2^1024, so the window
 * 2^-1184 .. 2^1120 holds any sum of doubles exactly. */
#define ACC_DIG 72
#define ACC_BIAS 1184

typedef struct {
  int64_t dig[ACC_DIG];
} exact_acc;

static void acc_clear(exact_acc *a) { memset(a->dig, 0, sizeof(a->dig)); }

/* a += sign * v for a finite double v */
static void acc_add(exact_acc *a, double v, int sign) {
  if (v == 0.0) return;
  if (v < 0) {
    v = -v;
    sign = -sign;
  }
  int e2;
  double m = frexp(v, &e2);             /* v = m 2^e2, m in [0.5, 1) */
  uint64_t mi = (uint64_t)ldexp(m, 53); /* v = mi 2^(e2-53) exactly */
  int pos = e2 - 53 + ACC_BIAS;         /* bit position of mi's last bit, >= 58 */
  int d = pos / 32, sh = pos % 32;
  unsigned __int128 w = ((unsigned __int128)mi) << sh; /* at most 85 bits */
  for (int q = 0; q < 3; ++q) {
    int64_t part = (int64_t)(uint32_t)(w >> (32 * q));
    a->dig[d + q] += sign > 0 ? part : -part;
  }
}

/* The accumulated value rounded to double (relative error below 2^-52). */
static double acc_value(const exact_acc *in) {
  int64_t dig[ACC_DIG];
  int64_t carry = 0;
  for (int d = 0; d < ACC_DIG; ++d) { /* normalise to digits in [0, 2^32) plus a sign carry */
    int64_t v = in->dig[d] + carry;
    int64_t lo = v & 0xffffffffLL;
    carry = (v - lo) / 4294967296LL;
    dig[d] = lo;
  }
  int neg = carry < 0; /* carry is 0 or -1: the value is carry * 2^(32*ACC_DIG) + digits */
  if (neg) {           /* magnitude = two's complement of the digit string */
    int64_t c2 = 1;
    for (int d = 0; d < ACC_DIG; ++d) {
      int64_t v = (0xffffffffLL - dig[d]) + c2;
      c2 = v >> 32;
      dig[d] = v & 0xffffffffLL;
    }
  }
  /* sum from the top: the first three non-zero digits carry 64+ significant bits */
  double r = 0.0;
  for (int d = ACC_DIG - 1; d >= 0; --d) r += ldexp((double)dig[d], 32 * d - ACC_BIAS);
  return neg ? -r : r;
}

/* Exact error of a computed MC matrix product (plus an optional MC bias per column).
 * For each requested output t = (rows[t], cols[t]):
 *   err[t]   = (exact sum of the nc components of C_t) - (exact value of
 *              sum_k A^_ik B^_kj + bias^_j), computed exactly and rounded to double,
 *   absab[t] = sum_k |A^_ik| |B^_kj| + |bias^_j| (the bound's denominator; A^, B^ are
 *              the exact values of the MC entries), rounded to double,
 *   exact[t] = the exact product (plus bias) rounded to double.
 * A is [a_planes][M][K], B is [b_planes][K][N] row-major, bias [bias_planes][N] or
 * NULL, C is [nc][count]. */
int mcf_oracle_matmul_exact_err(int f, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_planes,
                                const void *B, int b_planes, const void *bias, int bias_planes,
                                const int64_t *rows, const int64_t *cols, int64_t count, const void *C,
                                double *err, double *absab, double *exact) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < count; ++t) {
    int64_t i = rows ? rows[t] : t / N;
    int64_t j = rows ? cols[t] : t % N;
    exact_acc diff, ex;
    acc_clear(&diff);
    acc_clear(&ex);
    double sab = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      exact_acc ea, eb;
      acc_clear(&ea);
      acc_clear(&eb);
      for (int ca = 0; ca < a_planes; ++ca) {
        double a = load_c(f, A, ca * M * K + i * K + k);
        acc_add(&ea, a, 1);
        for (int cb = 0; cb < b_planes; ++cb) {
          double b = load_c(f, B, cb * K * N + k * N + j);
          /* a*b is exact in double for binary16/32 components; for binary64 ones
           * it is split exactly as p + e, e = fma(a, b, -p) (no underflow assumed) */
          double p = a * b, e = f == FMT_F64 ? fma(a, b, -p) : 0.0;
          acc_add(&diff, p, -1);
          acc_add(&ex, p, 1);
          acc_add(&diff, e, -1);
          acc_add(&ex, e, 1);
        }
      }
      for (int cb = 0; cb < b_planes; ++cb) acc_add(&eb, load_c(f, B, cb * K * N + k * N + j), 1);
      sab += fabs(acc_value(&ea)) * fabs(acc_value(&eb));
    }
    if (bias) {
      exact_acc eb;
      acc_clear(&eb);
      for (int cb = 0; cb < bias_planes; ++cb) {
        double b = load_c(f, bias, cb * N + j);
        acc_add(&eb, b, 1);
        acc_add(&diff, b, -1);
        acc_add(&ex, b, 1);
      }
      sab += fabs(acc_value(&eb));
    }
    for (int c = 0; c < nc; ++c) acc_add(&diff, load_c(f, C, (int64_t)c * count + t), 1);
    err[t] = acc_value(&diff);
    absab[t] = sab;
    exact[t] = acc_value(&ex);
  }
  return 0;
}

/* diff[i] = (exact value of element i of x) - (exact value of element i of y),
 * rounded to double; x has x_planes planes, y has y_planes (y may be NULL). */
void mcf_oracle_exact_diff(int f, int64_t n, const void *x, int x_planes, const void *y, int y_planes,
                           double *diff) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    exact_acc a;
    acc_clear(&a);
    for (int c = 0; c < x_planes; ++c) acc_add(&a, load_c(f, x, (int64_t)c * n + i), 1);
    if (y)
      for (int c = 0; c < y_planes; ++c) acc_add(&a, load_c(f, y, (int64_t)c * n + i), -1);
    diff[i] = acc_value(&a);
  }
}
