/*
 * mcf.h -- C ABI of the MI355X (gfx950) multi-component floating-point library.
 *
 * Arithmetic follows "MCTensor: A High-Precision Deep Learning Library with
 * Multi-Component Floating-Point" (arXiv 2207.08867).  A multi-component (MC) value
 * is an unevaluated sum x = x_0 + x_1 + ... + x_{nc-1} of nc floating-point
 * components of one format, largest first (Section 2, the MCF expansion equation).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  All tensor pointers are DEVICE pointers owned by the caller; the library
 *   allocates nothing per call and keeps no state besides two static per-device
 *   arrays: a binary16 exponential table (128 KiB, built on the first mc_exp call on
 *   a device) and the 8 MiB scratch of mc_matmul_splitk_noalloc.  Calls that need
 *   scratch memory (mc_matmul_splitk, mc_matmul_exact, mc_linreg_gd_step) take a
 *   caller-owned workspace.
 * Layout.  Dense, component-major ("planar"): component c of element i of an MC
 *   array of n elements is at element offset c*n + i.  A plain tensor is one plane.
 *   Matrices are row-major inside each plane.  The paper's interleaved layout
 *   (components in the last dimension) converts with a transpose on the caller side.
 * Formats.  MCF_F16 = IEEE binary16 components, MCF_F32 = IEEE binary32, MCF_F64 =
 *   IEEE binary64 (the paper's MC float64).  Every step of every algorithm is one IEEE
 *   round-to-nearest-even operation in the component format with gradual underflow;
 *   FMA appears only where the algorithm names it (Two-Prod); component division is
 *   correctly rounded; the component exponentials are correctly rounded in every
 *   format.  mc_matmul_exact takes MCF_F16 only.
 *   MCF_F16S = binary16 components with scaled low components (Section 2.4 names
 *   scaling the smaller components as the way past binary16's smallest subnormal):
 *   component c is stored as the binary16 number y_c and stands for 2^(-11 c) y_c.
 *   The algorithms are the same, with every quantity at a level and every rounding
 *   taken in the binary16 format of its level, fl_l(v) = 2^(-11 l) RN16(2^(11 l) v):
 *   the operands of an operation share a level (component i of an operand is at
 *   level i; a product is at the sum of its factors' levels), the errors of Two-Sum
 *   and Two-Prod and the carry built from them are at the next level, and a value
 *   Simple-Renorm moves to an earlier slot j is rounded into level j.  Only
 *   operations whose operands pair equal levels take MCF_F16S: mc_add (MC, MC
 *   only), mc_mul (MC, T and T, MC only), mc_matmul (MC x MC by the level-aligned
 *   parts described there) and mc_linear_fwd; every other call returns MCF_E_DTYPE.
 *   Non-finite components are outside this format's contract.
 * Operand kinds.  Binary operations take an MC value and a plain tensor in either
 *   order, or two MC values (Section 2.1).  The flags x_mc / y_mc / a_mc / b_mc are 1
 *   for an MC operand of nc planes and 0 for a plain tensor of one plane; at least
 *   one operand must be MC.  Results always have nc components.
 * nc.  1 <= nc <= 4.
 * Streams.  Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *   runs asynchronously; nothing synchronises.  Calls on different streams are
 *   independent.  The library is reentrant.
 * Graph capture.  A call launches kernels only (no allocation, memset or
 *   synchronisation), so it may be captured into a HIP graph on `stream` -- except
 *   the first binary16 mc_exp call on a device, which builds the exponential table and
 *   waits for it; make that call once before capturing.
 * Aliasing.  Elementwise calls allow `out` to be exactly `x` or `y` (in place);
 *   any other overlap of out with an input is rejected (MCF_E_ALIAS).  Matrix calls
 *   reject any overlap of the output with an input.
 * Degenerate sizes.  n = 0 (or M*N = 0) returns MCF_OK without launching; a
 *   reduction length of 0 gives +0 in every output component.
 * Size limits.  Each entry point states its own; in addition every matrix of a
 *   product (M*K, K*N, M*N elements per plane) must stay below 2^50 elements, else
 *   MCF_E_SHAPE.
 * Errors.  Every call returns MCF_OK (0) or a negative mcf_status; on error nothing
 *   is launched.  Launch failures are reported as MCF_E_HIP.  Input values are not
 *   inspected: non-finite components propagate by IEEE rules.
 */
#ifndef MCF_H
#define MCF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MCF_F16 = 0, MCF_F32 = 1, MCF_F64 = 2, MCF_F16S = 3 } mcf_dtype;

typedef enum {
  MCF_OK = 0,
  MCF_E_NULL = -1,  /* a required pointer is NULL */
  MCF_E_NC = -2,    /* nc (or nc_out) out of range */
  MCF_E_SHAPE = -3, /* negative size, or a size the kernels cannot index */
  MCF_E_DTYPE = -4, /* unknown format, or an operation not provided for it */
  MCF_E_ALIAS = -5, /* output overlaps an input in a way that is not allowed */
  MCF_E_HIP = -6,   /* the HIP runtime reported an error */
  MCF_E_ARG = -7,   /* any other invalid argument (operand kinds, mode) */
  MCF_E_SCRATCH = -8 /* the call needs more than the library's static scratch */
} mcf_status;

/* Addition (Section 2.1; Appendix A.2.1).
 *   (MC, MC): Add-MCN -- per component, Two-Sum of the operands, Two-Sum with the
 *             carry, carry = fl(e1 + e2); the nc+1 terms pass through Simple-Renorm.
 *   (MC, T), (T, MC): Grow-ExpN -- a chain of Two-Sums from the last component up,
 *             then Simple-Renorm to nc components.
 * x, y: [nc or 1][n]; out: [nc][n]. */
int mc_add(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream);

/* Multiplication (Section 2.1; Appendix A.2.1).
 *   (MC, T), (T, MC): ScalingN without expand -- per component Two-Prod (FMA
 *             variant), Two-Sum with the carry, carry = fl(e1 + e2); Simple-Renorm.
 *   (MC, MC): Mult-MCN, fast version -- Renormalize(Div-MCN(x, Renormalize(
 *             Div-MCN((1, 0, ..., 0), y)))).
 * x, y: [nc or 1][n]; out: [nc][n]. */
int mc_mul(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream);

/* Division (Appendix A.2.1).
 *   (MC, MC): Div-MCN -- long division: q = fl(x_0 / y_0), then nc times
 *             x = Add-MCN(x, -ScalingN(y, q)), q = fl(x_0 / y_0); the nc+1 quotient
 *             digits pass through Simple-Renorm.
 *   (T, MC):  DivN -- the dividend is padded with zero components.
 *   (MC, T):  Div-MCN with the divisor padded with zero components.
 * x, y: [nc or 1][n]; out: [nc][n]. */
int mc_div(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream);

/* Multiplication, Mult-MCN-Slow (Appendix A.2.1), for two MC operands: p = fl(x_0 y_0)
 * is the first product digit; nc times the remainder x = Add-MCN(x, -DivN(p, y)) is
 * formed and its next digit p = fl(x_0 y_0) taken; the nc+1 digits pass through
 * Simple-Renorm.  x, y, out: [nc][n]; out may be x or y exactly. */
int mc_mul_slow(int dtype, int nc, int64_t n, const void *x, const void *y, void *out, void *stream);

/* Square, Square-MCN (Appendix A.2.1).  The printed first step fl(2^{x_0}) is read as
 * fl(x_0 x_0), the square's leading term: h = (fl(x_0 x_0), 0, ..., 0), then
 * h = Grow-ExpN(h, fl(2 x_0 x_1)) (the addend is zero when nc = 1).  As printed, the
 * result is accurate to about one unit of x_0^2 (the rounding of x_0^2 and the terms
 * x_1^2, x_0 x_2, ... are not carried).  x, out: [nc][n]; out == x allowed. */
int mc_square(int dtype, int nc, int64_t n, const void *x, void *out, void *stream);

/* Exponential, Exp-MCN (Appendix A.2.1): h = exp(x_0) (one component), then for
 * i = 1 .. nc-1, h = ScalingN(h, exp(x_i), expand) growing h by one component per
 * step.  The component exponential is correctly rounded in every format (binary16
 * by table lookup; binary32 from a binary64 evaluation, with a double-double one
 * where that lies too close to a rounding boundary; binary64 by a double-double
 * table-driven evaluation, with a 192-bit fixed-point one where that lies too close
 * to a rounding boundary).  x, out: [nc][n]; out == x allowed. */
int mc_exp(int dtype, int nc, int64_t n, const void *x, void *out, void *stream);

/* Renormalization (Appendix A.2.1).
 *   mode 0: Renormalize (Priest variant): a top-down Two-Sum sweep s = x_0 (+) x_1 ...
 *           collecting the errors t_i, then a second sweep s, e = Two-Sum(s, t_i)
 *           that emits s whenever e != 0; the final s is emitted too; the first
 *           nc_out emitted values are returned, +0 padded.
 *   mode 1: Simple-Renorm: the first nc_out non-zero components in order, +0 padded.
 * 1 <= nc_out <= nc_in <= 4.  x: [nc_in][n]; out: [nc_out][n] (out == x allowed
 * only when nc_out == nc_in). */
int mc_renorm(int dtype, int nc_in, int nc_out, int64_t n, const void *x, void *out, int mode, void *stream);

/* Matrix product C = A B (Appendix A.2.2, MM-MCN; MV-MCN is N = 1 and Dot-MCN is
 * M = N = 1).  Each output is accumulated in MM-MCN order: acc = ScalingN(A_i0,
 * B_0j), then acc = Add-MCN(acc, ScalingN(A_ik, B_kj)) for k = 1 .. K-1, so the
 * result is reproducible and independent of the launch geometry.  With both
 * operands MC (not defined by the paper, whose matrix operators multiply an MC
 * matrix by a plain one) the product is taken by linearity over the components of
 * B: C = MM(A, B^(0)) (+) MM(A, B^(1)) (+) ... with (+) = Add-MCN.
 * MCF_F16S, both operands MC: B^(b) is at level b, so the part A B^(b) has levels
 * b, b+1, ..., of which the format keeps those below nc: the part is MM-MCN over the
 * first nc - b components of A with nc - b components at levels b .. nc-1, and the
 * parts, each placed at its levels (b leading zero components), are added left to
 * right: C = P_0 (+) (0, P_1) (+) (0, 0, P_2) ...
 * A: [nc or 1][M][K], B: [nc or 1][K][N], C: [nc][M][N]. */
int mc_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
              int b_mc, void *C, void *stream);

/* Pruned product of two MC matrices, a faster contraction with the accuracy class of
 * mc_matmul (Section 2.2 leaves faster MC products open).  The component products
 * A^(a) B^(b) with a + b >= nc are of the order of u^nc relative to A B -- the size of
 * MM-MCN's own error -- and are left out: component b of B multiplies the first
 * nc - b components of A, in MM-MCN order with nc - b components,
 *   C = MM_nc(A, B^(0)) (+) MM_{nc-1}(A[:nc-1], B^(1)) (+) ... (+) MM_1(A[:1], B^(nc-1)),
 * each part zero-padded to nc components, (+) = Add-MCN left to right.  A fixed
 * function of the inputs (reproducible on any launch geometry) but not mc_matmul's
 * bits: the error bound |C - C*| <= 4 K u^nc (|A||B|) is what it shares.  At nc = 3 it
 * needs 48 essential operations per multiply-add against mc_matmul's 102.
 * A: [nc][M][K], B: [nc][K][N], C: [nc][M][N], C not overlapping A or B. */
int mc_matmul_pruned(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, const void *B, void *C,
                     void *stream);

/* Batched and broadcast matrix products, BMM-MCN and 4DMM-MCN (Appendix A.2.2): for
 * every batch index (i1, i2) in [0, B1) x [0, B2), the matrices of A and B at that
 * index are multiplied exactly as mc_matmul multiplies its operands (MM-MCN order;
 * both MC: by linearity over the components of B).  A batch dimension of size 1
 * broadcast against a larger one (torch.matmul semantics) is a batch stride of 0.
 * A: component plane c starts at A + c*a_plane (elements); the matrix of batch
 *   (i1, i2) starts a_s1*i1 + a_s2*i2 elements into each plane and is [M][K]
 *   row-major.  B likewise, [K][N], with b_plane, b_s1, b_s2.  Every stride is >= 0
 *   and each plane must hold every batch's matrix: (B1-1)*s1 + (B2-1)*s2 + rows*cols
 *   <= plane (else MCF_E_SHAPE); the caller provides planes * plane elements.
 * C: dense [nc][B1][B2][M][N]; it must not overlap A or B.
 * Sizes as mc_matmul; B1, B2 >= 0; B1 * B2 * M * N below 2^40. */
int mc_matmul_batched(int dtype, int nc, int64_t B1, int64_t B2, int64_t M, int64_t N, int64_t K, const void *A,
                      int a_mc, int64_t a_plane, int64_t a_s1, int64_t a_s2, const void *B, int b_mc,
                      int64_t b_plane, int64_t b_s1, int64_t b_s2, void *C, void *stream);

/* AddMM-MCN (Appendix A.2.2): C = Add-MCN(ScalingN(A B, alpha), ScalingN(Y, beta)),
 * the product taken exactly as mc_matmul (any operand kinds), both ScalingN without
 * expand (so the result has nc components).
 * Y: MC, [nc][M][N] (y_rows = M) or [nc][N] added to every row (y_rows = 1).
 * alpha, beta: plain scalars that must be exactly representable in the component
 *   format (else MCF_E_ARG).
 * A: [nc or 1][M][K], B: [nc or 1][K][N], C: [nc][M][N], not overlapping A, B or Y. */
int mc_addmm(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B, int b_mc,
             const void *Y, int64_t y_rows, double alpha, double beta, void *C, void *stream);

/* K-split matrix product, for reductions that are long compared with the number of
 * outputs (Dot-MCN, MV-MCN, small products).  Section 2.2 of the paper notes that an
 * accurate sum of N MC values can be had in O(nc log N) depth; this entry point
 * computes the following log-depth variant of MM-MCN, fixed by the slice count S
 * alone (never by the device or the launch):
 *   the reduction steps are dealt round-robin to S slices, slice s taking
 *   k = s, s + S, s + 2S, ...; each slice is summed in MM-MCN order; the S slice
 *   sums are combined by a pairwise Add-MCN tree -- at each level entry q of the
 *   next level is Add-MCN(entry 2q, entry 2q+1), an odd last entry moves up
 *   unchanged.  With both operands MC, one such product per component of B,
 *   combined left to right with Add-MCN (as mc_matmul).
 * S = 1 gives exactly mc_matmul's result.  Other S give a result of the same
 * accuracy class (the error bound of MM-MCN holds) but not the same bits.
 * slices: S, at most 2^20 (else MCF_E_ARG); values above K are taken as K;
 *   slices <= 0 selects mc_matmul_splitk_slices(M, N, K).
 * workspace: device memory of at least mc_matmul_splitk_workspace(...) bytes (the
 *   partial tree roots: G = ceil(S / 256) entries of planes x nc x M x N components
 *   when S > 256; planes = nc for MC x MC, else 1), owned
 *   by the caller, not overlapping A, B or C; may be NULL when that size is 0.  Its
 *   contents on entry do not matter; calls sharing a workspace must not overlap
 *   in time.  Too small: MCF_E_ARG; NULL when needed: MCF_E_NULL.
 * A: [nc or 1][M][K], B: [nc or 1][K][N], C: [nc][M][N] (C must not overlap A or B);
 * M * N below 2^31. */
int mc_matmul_splitk(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                     int b_mc, int64_t slices, void *workspace, int64_t workspace_bytes, void *C, void *stream);

/* Allocation-free form of mc_matmul_splitk, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, result and rules as mc_matmul_splitk, but the partial
 * tree roots go to a static per-device scratch array inside the library (8 MiB,
 * held by every device the library runs on until the process ends) instead of a
 * caller workspace; the call allocates nothing.
 * Limit: calls whose mc_matmul_splitk_workspace(...) exceeds 8 MiB (8388608 bytes)
 *   return MCF_E_SCRATCH and launch nothing.  With the default slice count the roots
 *   take at most 1 MiB (binary64, nc = 4, MC x MC), so the limit binds only for
 *   large explicit slice counts on many outputs.
 * Sharing: every call on a device uses that device's one scratch array, so calls on
 *   one device that overlap in time (different streams, or different host threads)
 *   race and give undefined results; serialise them.  The contents left by earlier
 *   calls do not matter (nothing is read before it is written).
 * The device is the one that runs `stream` (the current device for NULL).  The first
 * call on a device looks up the array's device address (no allocation). */
int mc_matmul_splitk_noalloc(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                             const void *B, int b_mc, int64_t slices, void *C, void *stream);

/* Default slice count of mc_matmul_splitk, a function of the shape only: enough
 * slices for about 2^20 lanes in total (ceil(2^20 / (M N))), at most K / 64 (so a
 * slice holds at least 64 terms when K allows), at most 2^20, at least 1.
 * Negative sizes: MCF_E_SHAPE. */
int64_t mc_matmul_splitk_slices(int64_t M, int64_t N, int64_t K);

/* Workspace bytes mc_matmul_splitk needs for these arguments (0 when none), or a
 * negative mcf_status for arguments mc_matmul_splitk would reject. */
int64_t mc_matmul_splitk_workspace(int dtype, int nc, int64_t M, int64_t N, int64_t K, int a_mc, int b_mc,
                                   int64_t slices);

/* Exact MC product for binary16 components, rounded into nc components.  An MC
 * number is the unevaluated sum of its components (Section 2.1), so every output has
 * one exact value P_ij = sum_k (sum_c A^(c)_ik)(sum_c B^(c)_kj), the quantity that
 * MM-MCN (Section 2.2) approximates within about 4 K u^nc sum_k |A_ik||B_kj|
 * (Section 2.4).  This call returns P_ij split by successive round-to-nearest-even
 * into binary16: c_0 = RN(P), c_1 = RN(P - c_0), ..., so the components never
 * overlap and their sum is within half an ulp of c_{nc-1} (at most 2^-25 absolute
 * in the subnormal range) of P.  Not mc_matmul's bits: a different, more accurate
 * result.  The contraction runs on the int8 matrix cores: each entry is an exact
 * integer multiple of 2^-24, cut into 8-bit digits whose products are summed
 * exactly.
 * dtype: MCF_F16 only (else MCF_E_DTYPE).
 * Special values (input values ARE inspected here): an output whose row of A or
 *   column of B holds an infinite or NaN component is NaN in every component; if
 *   |P| rounds above 65504 the result is (+-inf, +0, ..., +0); an exact zero gives +0
 *   in every component, a non-zero P that rounds to zero keeps its sign.
 * A: [nc or 1][M][K]; B: [nc or 1][K][N], or [nc or 1][N][K] when b_trans = 1 (a
 *   linear layer's weight); C: [nc][M][N], not overlapping A or B.
 * workspace: device memory of at least mc_matmul_exact_workspace(...) bytes, owned by
 *   the caller, not overlapping A, B or C (else MCF_E_ALIAS); contents on entry do
 *   not matter; calls sharing a workspace must not overlap in time.  Too small:
 *   MCF_E_ARG; NULL: MCF_E_NULL.
 * Sizes: M, N <= 2^31, K <= 2^29, (M + N) K <= 2^40 and M N <= 2^38 (else
 *   MCF_E_SHAPE). */
int mc_matmul_exact(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                    int b_mc, int b_trans, void *workspace, int64_t workspace_bytes, void *C, void *stream);

/* Exact MC-Linear forward for binary16 components: y = x W^T + b with the exact value
 * of every output (x plain, W and b MC; Section 2.3's layer) split into nc components
 * by successive rounding, as mc_matmul_exact -- the bias is added to the exact sum
 * before the split.  An output whose column of W or bias holds an infinite or NaN
 * component, or whose row of x does, is NaN in every component.
 * x: [batch][in] (plain), W: [nc][out][in], b: [nc][out] or NULL, y: [nc][batch][out]
 * (not overlapping x, W, b or the workspace).
 * workspace: as mc_matmul_exact, at least mc_matmul_exact_workspace(dtype, nc, batch,
 *   out, in) bytes.  dtype: MCF_F16 only.  Sizes as mc_matmul_exact with M = batch,
 *   N = out, K = in. */
int mc_linear_fwd_exact(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                        const void *b, void *workspace, int64_t workspace_bytes, void *y, void *stream);

/* Workspace bytes mc_matmul_exact needs (about 6 (M + N) K bytes of digit planes,
 * plus 16 M N ceil(K / 16384) bytes of partial sums when K > 16384), or a negative
 * mcf_status for
 * sizes it would reject. */
int64_t mc_matmul_exact_workspace(int dtype, int nc, int64_t M, int64_t N, int64_t K);

/* MC-Linear forward (Section 2.3): y = x W^T (+ b).  The weight and bias are MC,
 * the input is a plain tensor; each output accumulates ScalingN(W[o][i], x[t][i])
 * over i in MM-MCN order, then adds the bias with Add-MCN.
 * x: [batch][in] (plain), W: [nc][out][in], b: [nc][out] or NULL,
 * y: [nc][batch][out]. */
int mc_linear_fwd(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                  const void *b, void *y, void *stream);

/* MC-Linear backward (the layer of Section 2.3, y = x W^T + b): given the gradient dY
 * of the loss with respect to y, computes
 *   dX = dY W          [batch][in]  (MM-MCN; dY MC: by linearity over W's components)
 *   dW = dY^T x        [out][in]    (MM-MCN over the batch index, in batch order)
 *   db = sum_t dY[t]   [out]        (Add-MCN of the rows of dY in batch order: MM-MCN
 *                                    against a column of ones, ScalingN by 1 being exact)
 * The paper keeps the gradient of an MC value as a plain tensor -- the gradient of
 * its leading component (Section 2.1) -- and takes it from automatic differentiation;
 * here the gradients are MC values whose leading components are those plain
 * gradients, accumulated with MM-MCN's error propagation.  A plain dY (dy_mc = 0)
 * enters dW and db as an MC value with +0 low components.
 * x: [batch][in] plain; W: [nc][out][in]; dY: [nc or 1][batch][out] (dy_mc 1 or 0);
 * dX: [nc][batch][in], dW: [nc][out][in], db: [nc][out] -- each may be NULL (not
 * computed); outputs must not overlap the inputs, each other or the workspace.
 * workspace: device memory of at least mc_linear_bwd_workspace(...) bytes when dW or
 *   db is requested (dY^T staged in nc planes; then a column of ones, or, when both dW
 *   and db are requested, x with a column of ones appended and the [dW | db] product,
 *   which gives both in one pass), owned by the
 *   caller, not overlapping the inputs; contents on entry do not matter; calls sharing
 *   it must not overlap in time.  Too small: MCF_E_ARG; NULL when needed: MCF_E_NULL.
 * dtype: MCF_F16, MCF_F32, MCF_F64.  Sizes: batch, out <= 2^20, in <= 2^30 (and the
 * product limits of mc_matmul). */
int mc_linear_bwd(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                  const void *dY, int dy_mc, void *dX, void *dW, void *db, void *workspace, int64_t workspace_bytes,
                  void *stream);

/* Workspace bytes mc_linear_bwd needs when dW or db is requested, or a negative
 * mcf_status for sizes it would reject. */
int64_t mc_linear_bwd_workspace(int dtype, int nc, int64_t batch, int64_t in, int64_t out);

/* One gradient-descent step of the paper's linear-regression precision experiment
 * (Section 2.4): an MC-Linear layer without bias, W (out = 1 row of d weights), fitted
 * to targets y with the mean-squared error L(W) = (1/n) sum_i (x_i . W - y_i)^2.
 * The paper leaves the optimizer step unprinted and defines the gradient of an MC value
 * as the plain gradient of its leading component (Section 2.1).  This call computes, in
 * stream order:
 *   yhat = MC-Linear(X, W) (MM-MCN order, as mc_linear_fwd);
 *   r = Grow-ExpN(yhat, y_neg), the MC residual;
 *   G = r^T X and RR = r . r, each by the K-split product with its default slice count
 *     (mc_matmul_splitk_slices);
 *   per weight j: g = ScalingN(G_j, fl(2/n)); grad_j = the leading component of g;
 *     W_j = Grow-ExpN(W_j, fl(-lr * grad_j)) (one rounding of the product);
 *   loss = ScalingN(RR, fl(1/n)), the loss at W before the update.
 * fl(2/n), fl(1/n): the binary64 quotients rounded once to the component format;
 * fl(-lr): the binary64 value -lr rounded to the component format.
 * X: [n][d] plain; y_neg: [n] plain, the NEGATED targets (-y); W: [nc][d] MC, updated
 *   in place; loss: [nc] MC, or NULL.  W and loss must not overlap each other, X, y_neg
 *   or the workspace.
 * workspace: device memory of at least mc_linreg_workspace(...) bytes, owned by the
 *   caller (contents on entry do not matter; steps sharing it must not overlap in
 *   time).  Too small: MCF_E_ARG.
 * Sizes: n >= 1, d >= 1, n <= 2^30, d <= 2^20, n d <= 2^40. */
int mc_linreg_gd_step(int dtype, int nc, int64_t n, int64_t d, const void *X, const void *y_neg, void *W, double lr,
                      void *workspace, int64_t workspace_bytes, void *loss, void *stream);

/* Workspace bytes mc_linreg_gd_step needs, or a negative mcf_status for arguments it
 * would reject. */
int64_t mc_linreg_workspace(int dtype, int nc, int64_t n, int64_t d);

/* Human-readable name of a status code (static storage). */
const char *mc_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* MCF_H */
