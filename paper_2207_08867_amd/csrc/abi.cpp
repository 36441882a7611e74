// abi.cpp -- the extern "C" entry points declared in include/mcf.h: argument
// validation, aliasing rules and dispatch to the kernel launchers.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mcf.h"
#include "mcf_internal.hpp"

namespace {

constexpr int MAX_NC = 4;

int64_t elem_size(int dtype) { return (dtype == MCF_F16 || dtype == MCF_F16S) ? 2 : (dtype == MCF_F64 ? 8 : 4); }

bool overlap(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
  if (abytes <= 0 || bbytes <= 0) return false;
  uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bbytes && b0 < a0 + (uintptr_t)abytes;
}

// out may coincide with an input exactly; any other overlap is an error.
bool bad_alias(const void *out, int64_t obytes, const void *in, int64_t ibytes) {
  if (in == nullptr) return false;
  if (out == in && obytes == ibytes) return false;
  return overlap(out, obytes, in, ibytes);
}

// The sequential product launches one workgroup per 16 x 16 (or larger) tile of C in
// a 1-D grid, which must stay below 2^31 workgroups.
bool grid_fits(int64_t M, int64_t N) { return ((M + 15) / 16) * ((N + 15) / 16) < ((int64_t)1 << 31); }

// a * b elements stay below 2^50, so byte counts (times nc and the element size) and
// offsets never overflow int64; a, b >= 0.
bool elems_fit(int64_t a, int64_t b) { return b == 0 || a <= ((int64_t)1 << 50) / b; }

// Operand sizes of an M x K by K x N product.
bool product_fits(int64_t M, int64_t N, int64_t K) {
  return elems_fit(M, K) && elems_fit(K, N) && elems_fit(M, N);
}

int hip_status(hipError_t e) { return e == hipSuccess ? MCF_OK : MCF_E_HIP; }

int check_common(int dtype, int nc, int64_t n) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (n < 0) return MCF_E_SHAPE;
  // plane offsets c * n stay far below 2^62 elements
  if (n > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  return MCF_OK;
}

int binary_op(int op, int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
              void *stream) {
  int st = check_common(dtype, nc, n);
  if (st != MCF_OK) return st;
  if ((x_mc != 0 && x_mc != 1) || (y_mc != 0 && y_mc != 1) || (!x_mc && !y_mc)) return MCF_E_ARG;
  if (n == 0) return MCF_OK;
  if (!x || !y || !out) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t ob = nc * n * es, xb = (x_mc ? nc : 1) * n * es, yb = (y_mc ? nc : 1) * n * es;
  if (bad_alias(out, ob, x, xb) || bad_alias(out, ob, y, yb)) return MCF_E_ALIAS;
  return hip_status(mcf::launch_elementwise(dtype, op, nc, nc, n, x, x_mc, y, y_mc, out, (hipStream_t)stream));
}

// binary16 with scaled low components: Add-MCN of two MC operands (op EW_ADD) and
// ScalingN of an MC operand by a plain one, in either order (op EW_MUL).  The other
// operand kinds pair values of different levels and are not provided (MCF_E_DTYPE).
int scaled_binary_op(int op, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
                     void *stream) {
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (n < 0 || n > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if ((x_mc != 0 && x_mc != 1) || (y_mc != 0 && y_mc != 1) || (!x_mc && !y_mc)) return MCF_E_ARG;
  if (op == mcf::EW_ADD ? !(x_mc && y_mc) : (x_mc && y_mc)) return MCF_E_DTYPE;
  if (n == 0) return MCF_OK;
  if (!x || !y || !out) return MCF_E_NULL;
  const int64_t ob = nc * n * 2, xb = (x_mc ? nc : 1) * n * 2, yb = (y_mc ? nc : 1) * n * 2;
  if (bad_alias(out, ob, x, xb) || bad_alias(out, ob, y, yb)) return MCF_E_ALIAS;
  if (op == mcf::EW_MUL && !x_mc)  // the MC operand goes first
    return hip_status(mcf::launch_scaled_elementwise(op, nc, n, y, x, out, (hipStream_t)stream));
  return hip_status(mcf::launch_scaled_elementwise(op, nc, n, x, y, out, (hipStream_t)stream));
}

// Shared validation of the K-split product; *S receives the slice count used
// (the default for slices <= 0, capped at K).
int splitk_check(int dtype, int nc, int64_t M, int64_t N, int64_t K, int a_mc, int b_mc, int64_t slices,
                 int64_t *S) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if ((a_mc != 0 && a_mc != 1) || (b_mc != 0 && b_mc != 1) || (!a_mc && !b_mc)) return MCF_E_ARG;
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  if (M > ((int64_t)1 << 40) || N > ((int64_t)1 << 40) || K > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (M > 0 && N > (((int64_t)1 << 31) - 1) / M) return MCF_E_SHAPE;  // grid of up to M*N workgroups
  if (!product_fits(M, N, K)) return MCF_E_SHAPE;
  if (slices > mcf::SPLITK_MAX_SLICES) return MCF_E_ARG;
  int64_t s = slices <= 0 ? mcf::splitk_default_slices(M, N, K) : slices;
  if (K > 0 && s > K) s = K;
  *S = s < 1 ? 1 : s;
  return MCF_OK;
}

int64_t splitk_workspace_bytes(int dtype, int nc, int64_t M, int64_t N, int64_t K, int a_mc, int b_mc, int64_t S) {
  if (M == 0 || N == 0 || K == 0) return 0;
  const int64_t np = (a_mc && b_mc) ? nc : 1;
  return mcf::splitk_roots(S) * np * nc * M * N * elem_size(dtype);
}

int exact_check(int dtype, int nc, int64_t M, int64_t N, int64_t K, int a_mc, int b_mc, int b_trans) {
  if (dtype != MCF_F16) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if ((a_mc != 0 && a_mc != 1) || (b_mc != 0 && b_mc != 1) || (b_trans != 0 && b_trans != 1)) return MCF_E_ARG;
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  // digit planes of 6 (M + N) K bytes, grids of (M / 32) (N / 32) workgroups (rows
  // padded to 128) and up to K / 16384 chunks in the second grid dimension
  if (M > ((int64_t)1 << 31) || N > ((int64_t)1 << 31) || K > ((int64_t)1 << 29)) return MCF_E_SHAPE;
  if ((M + N) > 0 && K > ((int64_t)1 << 40) / (M + N + 256)) return MCF_E_SHAPE;
  if (((M + 127) / 32) * ((N + 127) / 32) >= ((int64_t)1 << 31)) return MCF_E_SHAPE;
  if (M > 0 && N > ((int64_t)1 << 38) / M) return MCF_E_SHAPE;
  return MCF_OK;
}

int linreg_check(int dtype, int nc, int64_t n, int64_t d) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (n < 1 || d < 1) return MCF_E_SHAPE;
  // X has n d elements; the sequential product's grid covers n rows, the K-split
  // products' grids d outputs
  if (n > ((int64_t)1 << 30) || d > ((int64_t)1 << 20) || n > (((int64_t)1 << 40) / d)) return MCF_E_SHAPE;
  return MCF_OK;
}

int linear_bwd_check(int dtype, int nc, int64_t batch, int64_t in, int64_t out) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (batch < 0 || in < 0 || out < 0) return MCF_E_SHAPE;
  // the products dX (batch x in, reduction out), dW (out x in, reduction batch) and db
  // (out x 1, reduction batch) and the staging grid (batch / 32 tiles in a y dimension)
  if (batch > ((int64_t)1 << 20) || out > ((int64_t)1 << 20) || in > ((int64_t)1 << 30)) return MCF_E_SHAPE;
  if (!grid_fits(batch, in) || !grid_fits(out, in) || !product_fits(batch, in, out) || !product_fits(out, in, batch))
    return MCF_E_SHAPE;
  return MCF_OK;
}

// The component-format rounding of a binary64 value.
double round_to_format(int dtype, double v) {
  if (dtype == MCF_F16) return (double)(_Float16)v;
  if (dtype == MCF_F64) return v;
  return (double)(float)v;
}

}  // namespace

extern "C" {

int mc_add(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream) {
  if (dtype == MCF_F16S) return scaled_binary_op(mcf::EW_ADD, nc, n, x, x_mc, y, y_mc, out, stream);
  return binary_op(mcf::EW_ADD, dtype, nc, n, x, x_mc, y, y_mc, out, stream);
}

int mc_mul(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream) {
  if (dtype == MCF_F16S) return scaled_binary_op(mcf::EW_MUL, nc, n, x, x_mc, y, y_mc, out, stream);
  return binary_op(mcf::EW_MUL, dtype, nc, n, x, x_mc, y, y_mc, out, stream);
}

int mc_div(int dtype, int nc, int64_t n, const void *x, int x_mc, const void *y, int y_mc, void *out,
           void *stream) {
  return binary_op(mcf::EW_DIV, dtype, nc, n, x, x_mc, y, y_mc, out, stream);
}

int mc_mul_slow(int dtype, int nc, int64_t n, const void *x, const void *y, void *out, void *stream) {
  return binary_op(mcf::EW_MUL_SLOW, dtype, nc, n, x, 1, y, 1, out, stream);
}

int mc_square(int dtype, int nc, int64_t n, const void *x, void *out, void *stream) {
  int st = check_common(dtype, nc, n);
  if (st != MCF_OK) return st;
  if (n == 0) return MCF_OK;
  if (!x || !out) return MCF_E_NULL;
  const int64_t b = nc * n * elem_size(dtype);
  if (bad_alias(out, b, x, b)) return MCF_E_ALIAS;
  return hip_status(mcf::launch_elementwise(dtype, mcf::EW_SQUARE, nc, nc, n, x, 1, nullptr, 0, out,
                                            (hipStream_t)stream));
}

int mc_exp(int dtype, int nc, int64_t n, const void *x, void *out, void *stream) {
  int st = check_common(dtype, nc, n);
  if (st != MCF_OK) return st;
  if (n == 0) return MCF_OK;
  if (!x || !out) return MCF_E_NULL;
  const int64_t b = nc * n * elem_size(dtype);
  if (bad_alias(out, b, x, b)) return MCF_E_ALIAS;
  if (dtype == MCF_F16) return hip_status(mcf::launch_exp_f16(nc, n, x, out, (hipStream_t)stream));
  if (dtype == MCF_F64) return hip_status(mcf::launch_exp_f64(nc, n, x, out, (hipStream_t)stream));
  return hip_status(mcf::launch_exp_f32(nc, n, x, out, (hipStream_t)stream));
}

int mc_renorm(int dtype, int nc_in, int nc_out, int64_t n, const void *x, void *out, int mode, void *stream) {
  int st = check_common(dtype, nc_in, n);
  if (st != MCF_OK) return st;
  if (nc_out < 1 || nc_out > nc_in) return MCF_E_NC;
  if (mode != 0 && mode != 1) return MCF_E_ARG;
  if (n == 0) return MCF_OK;
  if (!x || !out) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  if (bad_alias(out, nc_out * n * es, x, nc_in * n * es)) return MCF_E_ALIAS;
  return hip_status(mcf::launch_elementwise(dtype, mode == 0 ? mcf::EW_RENORM : mcf::EW_SIMPLE_RENORM, nc_in,
                                            nc_out, n, x, 1, nullptr, 0, out, (hipStream_t)stream));
}

int mc_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
              int b_mc, void *C, void *stream) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64 && dtype != MCF_F16S) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if ((a_mc != 0 && a_mc != 1) || (b_mc != 0 && b_mc != 1) || (!a_mc && !b_mc)) return MCF_E_ARG;
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  if (M > ((int64_t)1 << 20) || N > ((int64_t)1 << 30) || K > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (!grid_fits(M, N) || !product_fits(M, N, K)) return MCF_E_SHAPE;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * M * N * es;
  if (overlap(C, cb, A, (a_mc ? nc : 1) * M * K * es) || overlap(C, cb, B, (b_mc ? nc : 1) * K * N * es))
    return MCF_E_ALIAS;
  if (dtype == MCF_F16S)
    return hip_status(
        mcf::launch_scaled_matmul(nc, M, N, K, A, a_mc, B, b_mc, 0, nullptr, C, (hipStream_t)stream));
  return hip_status(mcf::launch_matmul(dtype, nc, M, N, K, A, a_mc, B, b_mc, 0, nullptr, C, (hipStream_t)stream));
}

int mc_matmul_pruned(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, const void *B, void *C,
                     void *stream) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  if (M > ((int64_t)1 << 20) || N > ((int64_t)1 << 30) || K > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (!grid_fits(M, N) || !product_fits(M, N, K)) return MCF_E_SHAPE;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * M * N * es;
  if (overlap(C, cb, A, nc * M * K * es) || overlap(C, cb, B, nc * K * N * es)) return MCF_E_ALIAS;
  mcf::MmLaunch L;
  L.dtype = dtype;
  L.nc = nc;
  L.M = M;
  L.N = N;
  L.K = K;
  L.A = A;
  L.a_plane = M * K;
  L.B = B;
  L.b_plane = K * N;
  L.C = C;
  L.prune = 1;
  return hip_status(mcf::launch_matmul_general(L, (hipStream_t)stream));
}

int mc_matmul_batched(int dtype, int nc, int64_t B1, int64_t B2, int64_t M, int64_t N, int64_t K, const void *A,
                      int a_mc, int64_t a_plane, int64_t a_s1, int64_t a_s2, const void *B, int b_mc,
                      int64_t b_plane, int64_t b_s1, int64_t b_s2, void *C, void *stream) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if ((a_mc != 0 && a_mc != 1) || (b_mc != 0 && b_mc != 1) || (!a_mc && !b_mc)) return MCF_E_ARG;
  if (M < 0 || N < 0 || K < 0 || B1 < 0 || B2 < 0) return MCF_E_SHAPE;
  if (M > ((int64_t)1 << 20) || N > ((int64_t)1 << 30) || K > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (B1 > ((int64_t)1 << 40) || B2 > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (!grid_fits(M, N) || !product_fits(M, N, K)) return MCF_E_SHAPE;
  if (B1 == 0 || B2 == 0 || M == 0 || N == 0) return MCF_OK;
  if (B1 > (((int64_t)1 << 40) / B2) / (M * N)) return MCF_E_SHAPE;
  if (a_s1 < 0 || a_s2 < 0 || b_s1 < 0 || b_s2 < 0 || a_plane < 0 || b_plane < 0) return MCF_E_SHAPE;
  const int64_t lim = (int64_t)1 << 50;
  if (a_s1 > lim / B1 || a_s2 > lim / B2 || b_s1 > lim / B1 || b_s2 > lim / B2 || a_plane > lim || b_plane > lim)
    return MCF_E_SHAPE;
  // every batch's matrix lies inside its plane
  if ((B1 - 1) * a_s1 + (B2 - 1) * a_s2 + M * K > a_plane) return MCF_E_SHAPE;
  if ((B1 - 1) * b_s1 + (B2 - 1) * b_s2 + K * N > b_plane) return MCF_E_SHAPE;
  if (!C || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * B1 * B2 * M * N * es;
  if (overlap(C, cb, A, (a_mc ? nc : 1) * a_plane * es) || overlap(C, cb, B, (b_mc ? nc : 1) * b_plane * es))
    return MCF_E_ALIAS;
  mcf::MmLaunch L;
  L.dtype = dtype;
  L.nc = nc;
  L.M = M;
  L.N = N;
  L.K = K;
  L.B1 = B1;
  L.B2 = B2;
  L.A = A;
  L.a_mc = a_mc;
  L.a_plane = a_plane;
  L.a_s1 = a_s1;
  L.a_s2 = a_s2;
  L.B = B;
  L.b_mc = b_mc;
  L.b_plane = b_plane;
  L.b_s1 = b_s1;
  L.b_s2 = b_s2;
  L.C = C;
  return hip_status(mcf::launch_matmul_general(L, (hipStream_t)stream));
}

int mc_addmm(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B, int b_mc,
             const void *Y, int64_t y_rows, double alpha, double beta, void *C, void *stream) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if ((a_mc != 0 && a_mc != 1) || (b_mc != 0 && b_mc != 1) || (!a_mc && !b_mc)) return MCF_E_ARG;
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  if (M > ((int64_t)1 << 20) || N > ((int64_t)1 << 30) || K > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (!grid_fits(M, N) || !product_fits(M, N, K)) return MCF_E_SHAPE;
  if (y_rows != M && y_rows != 1) return MCF_E_SHAPE;
  // the scalars must be values of the component format
  const bool exact = dtype == MCF_F64   ? true
                     : dtype == MCF_F32 ? (double)(float)alpha == alpha && (double)(float)beta == beta
                                        : (double)(_Float16)alpha == alpha && (double)(_Float16)beta == beta;
  if (!exact) return MCF_E_ARG;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || !Y || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * M * N * es;
  if (overlap(C, cb, A, (a_mc ? nc : 1) * M * K * es) || overlap(C, cb, B, (b_mc ? nc : 1) * K * N * es) ||
      overlap(C, cb, Y, nc * y_rows * N * es))
    return MCF_E_ALIAS;
  mcf::MmLaunch L;
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
  L.b_plane = K * N;
  L.C = C;
  L.mode = 2;
  L.y = Y;
  L.y_plane = y_rows * N;
  L.y_ld = y_rows == 1 ? 0 : N;
  L.alpha = alpha;
  L.beta = beta;
  return hip_status(mcf::launch_matmul_general(L, (hipStream_t)stream));
}

int64_t mc_matmul_splitk_slices(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 0) return MCF_E_SHAPE;
  return mcf::splitk_default_slices(M, N, K);
}

int64_t mc_matmul_splitk_workspace(int dtype, int nc, int64_t M, int64_t N, int64_t K, int a_mc, int b_mc,
                                   int64_t slices) {
  int64_t S = 0;
  int st = splitk_check(dtype, nc, M, N, K, a_mc, b_mc, slices, &S);
  if (st != MCF_OK) return st;
  return splitk_workspace_bytes(dtype, nc, M, N, K, a_mc, b_mc, S);
}

int mc_matmul_splitk(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                     int b_mc, int64_t slices, void *workspace, int64_t workspace_bytes, void *C, void *stream) {
  int64_t S = 0;
  int st = splitk_check(dtype, nc, M, N, K, a_mc, b_mc, slices, &S);
  if (st != MCF_OK) return st;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * M * N * es, ab = (a_mc ? nc : 1) * M * K * es, bb = (b_mc ? nc : 1) * K * N * es;
  if (overlap(C, cb, A, ab) || overlap(C, cb, B, bb)) return MCF_E_ALIAS;
  if (K == 0)  // every output is +0
    return hip_status(mcf::launch_matmul(dtype, nc, M, N, 0, A, a_mc, B, b_mc, 0, nullptr, C, (hipStream_t)stream));
  const int64_t wb = splitk_workspace_bytes(dtype, nc, M, N, K, a_mc, b_mc, S);
  if (wb > 0) {
    if (!workspace) return MCF_E_NULL;
    if (workspace_bytes < wb) return MCF_E_ARG;
    if (overlap(workspace, wb, A, ab) || overlap(workspace, wb, B, bb) || overlap(workspace, wb, C, cb))
      return MCF_E_ALIAS;
  }
  return hip_status(
      mcf::launch_matmul_splitk(dtype, nc, M, N, K, A, a_mc, B, b_mc, S, workspace, C, (hipStream_t)stream));
}

int mc_matmul_splitk_noalloc(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                             const void *B, int b_mc, int64_t slices, void *C, void *stream) {
  int64_t S = 0;
  int st = splitk_check(dtype, nc, M, N, K, a_mc, b_mc, slices, &S);
  if (st != MCF_OK) return st;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t cb = nc * M * N * es, ab = (a_mc ? nc : 1) * M * K * es, bb = (b_mc ? nc : 1) * K * N * es;
  if (overlap(C, cb, A, ab) || overlap(C, cb, B, bb)) return MCF_E_ALIAS;
  if (K == 0)  // every output is +0
    return hip_status(mcf::launch_matmul(dtype, nc, M, N, 0, A, a_mc, B, b_mc, 0, nullptr, C, (hipStream_t)stream));
  const int64_t wb = splitk_workspace_bytes(dtype, nc, M, N, K, a_mc, b_mc, S);
  if (wb > mcf::SPLITK_SCRATCH_BYTES) return MCF_E_SCRATCH;
  void *scratch = nullptr;
  if (wb > 0) {
    const hipError_t e = mcf::splitk_scratch((hipStream_t)stream, &scratch);
    if (e != hipSuccess) return MCF_E_HIP;
    // the static scratch is library memory, so it cannot overlap A, B or C
  }
  return hip_status(
      mcf::launch_matmul_splitk(dtype, nc, M, N, K, A, a_mc, B, b_mc, S, scratch, C, (hipStream_t)stream));
}

int64_t mc_matmul_exact_workspace(int dtype, int nc, int64_t M, int64_t N, int64_t K) {
  int st = exact_check(dtype, nc, M, N, K, 1, 1, 0);
  if (st != MCF_OK) return st;
  if (M == 0 || N == 0) return 0;
  return mcf::exact_workspace_bytes(M, N, K);
}

int mc_matmul_exact(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                    int b_mc, int b_trans, void *workspace, int64_t workspace_bytes, void *C, void *stream) {
  int st = exact_check(dtype, nc, M, N, K, a_mc, b_mc, b_trans);
  if (st != MCF_OK) return st;
  if (M == 0 || N == 0) return MCF_OK;
  if (!C || !workspace || (K > 0 && (!A || !B))) return MCF_E_NULL;
  const int64_t wb = mcf::exact_workspace_bytes(M, N, K);
  if (workspace_bytes < wb) return MCF_E_ARG;
  const int64_t cb = nc * M * N * 2, ab = (a_mc ? nc : 1) * M * K * 2, bb = (b_mc ? nc : 1) * K * N * 2;
  if (overlap(C, cb, A, ab) || overlap(C, cb, B, bb)) return MCF_E_ALIAS;
  if (overlap(workspace, wb, A, ab) || overlap(workspace, wb, B, bb) || overlap(workspace, wb, C, cb))
    return MCF_E_ALIAS;
  return hip_status(
      mcf::launch_matmul_exact(nc, M, N, K, A, a_mc, B, b_mc, b_trans, nullptr, workspace, C, (hipStream_t)stream));
}

int mc_linear_fwd_exact(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                        const void *b, void *workspace, int64_t workspace_bytes, void *y, void *stream) {
  int st = exact_check(dtype, nc, batch, out, in, 0, 1, 1);
  if (st != MCF_OK) return st;
  if (batch == 0 || out == 0) return MCF_OK;
  if (!y || !workspace || (in > 0 && (!x || !W))) return MCF_E_NULL;
  const int64_t wb = mcf::exact_workspace_bytes(batch, out, in);
  if (workspace_bytes < wb) return MCF_E_ARG;
  const int64_t yb = nc * batch * out * 2, xb = batch * in * 2, Wb = nc * out * in * 2, bb = nc * out * 2;
  if (overlap(y, yb, x, xb) || overlap(y, yb, W, Wb) || (b && overlap(y, yb, b, bb))) return MCF_E_ALIAS;
  if (overlap(workspace, wb, x, xb) || overlap(workspace, wb, W, Wb) || overlap(workspace, wb, y, yb) ||
      (b && overlap(workspace, wb, b, bb)))
    return MCF_E_ALIAS;
  return hip_status(
      mcf::launch_matmul_exact(nc, batch, out, in, x, 0, W, 1, 1, b, workspace, y, (hipStream_t)stream));
}

int64_t mc_linear_bwd_workspace(int dtype, int nc, int64_t batch, int64_t in, int64_t out) {
  const int st = linear_bwd_check(dtype, nc, batch, in, out);
  if (st != MCF_OK) return st;
  return mcf::linear_bwd_workspace_bytes(dtype, nc, batch, in, out);
}

int mc_linear_bwd(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                  const void *dY, int dy_mc, void *dX, void *dW, void *db, void *workspace, int64_t workspace_bytes,
                  void *stream) {
  const int st = linear_bwd_check(dtype, nc, batch, in, out);
  if (st != MCF_OK) return st;
  if (dy_mc != 0 && dy_mc != 1) return MCF_E_ARG;
  const int64_t es = elem_size(dtype);
  // outputs with no elements are not computed
  const int64_t dxb = nc * batch * in * es, dwb = nc * out * in * es, dbb = nc * out * es;
  if (dxb == 0) dX = nullptr;
  if (dwb == 0) dW = nullptr;
  if (dbb == 0) db = nullptr;
  if (!dX && !dW && !db) return MCF_OK;
  const int64_t xb = batch * in * es, Wb = nc * out * in * es, yb = (dy_mc ? nc : 1) * batch * out * es;
  if ((dX || dW) && in > 0 && batch > 0 && (!x || !W)) return MCF_E_NULL;
  if (batch > 0 && out > 0 && !dY) return MCF_E_NULL;
  const bool staged = dW || db;
  const int64_t wb = staged ? mcf::linear_bwd_workspace_bytes(dtype, nc, batch, in, out) : 0;
  if (staged) {
    if (!workspace) return MCF_E_NULL;
    if (workspace_bytes < wb) return MCF_E_ARG;
  }
  const void *ins[3] = {x, W, dY};
  const int64_t inb[3] = {xb, Wb, yb};
  void *outs[4] = {dX, dW, db, staged ? workspace : nullptr};
  const int64_t outb[4] = {dxb, dwb, dbb, wb};
  for (int o = 0; o < 4; ++o) {
    if (!outs[o]) continue;
    for (int i = 0; i < 3; ++i)
      if (ins[i] && overlap(outs[o], outb[o], ins[i], inb[i])) return MCF_E_ALIAS;
    for (int p = o + 1; p < 4; ++p)
      if (outs[p] && overlap(outs[o], outb[o], outs[p], outb[p])) return MCF_E_ALIAS;
  }
  return hip_status(mcf::launch_linear_bwd(dtype, nc, batch, in, out, x, W, dY, dy_mc, dX, dW, db, workspace,
                                           (hipStream_t)stream));
}

int64_t mc_linreg_workspace(int dtype, int nc, int64_t n, int64_t d) {
  const int st = linreg_check(dtype, nc, n, d);
  if (st != MCF_OK) return st;
  return mcf::linreg_workspace_bytes(dtype, nc, n, d);
}

int mc_linreg_gd_step(int dtype, int nc, int64_t n, int64_t d, const void *X, const void *y_neg, void *W, double lr,
                      void *workspace, int64_t workspace_bytes, void *loss, void *stream) {
  const int st = linreg_check(dtype, nc, n, d);
  if (st != MCF_OK) return st;
  if (!X || !y_neg || !W || !workspace) return MCF_E_NULL;
  const int64_t wb = mcf::linreg_workspace_bytes(dtype, nc, n, d);
  if (workspace_bytes < wb) return MCF_E_ARG;
  const int64_t es = elem_size(dtype);
  const int64_t xb = n * d * es, yb = n * es, Wb = nc * d * es, lb = nc * es;
  if (overlap(W, Wb, X, xb) || overlap(W, Wb, y_neg, yb) || overlap(W, Wb, workspace, wb)) return MCF_E_ALIAS;
  if (overlap(workspace, wb, X, xb) || overlap(workspace, wb, y_neg, yb)) return MCF_E_ALIAS;
  if (loss && (overlap(loss, lb, W, Wb) || overlap(loss, lb, workspace, wb) || overlap(loss, lb, X, xb) ||
               overlap(loss, lb, y_neg, yb)))
    return MCF_E_ALIAS;
  const double s2n = round_to_format(dtype, 2.0 / (double)n), s1n = round_to_format(dtype, 1.0 / (double)n);
  const double neg_lr = round_to_format(dtype, -lr);
  return hip_status(mcf::launch_linreg_step(dtype, nc, n, d, X, y_neg, W, s2n, s1n, neg_lr, workspace, loss,
                                            (hipStream_t)stream));
}

int mc_linear_fwd(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                  const void *b, void *y, void *stream) {
  if (dtype != MCF_F16 && dtype != MCF_F32 && dtype != MCF_F64 && dtype != MCF_F16S) return MCF_E_DTYPE;
  if (nc < 1 || nc > MAX_NC) return MCF_E_NC;
  if (batch < 0 || in < 0 || out < 0) return MCF_E_SHAPE;
  if (batch > ((int64_t)1 << 20) || out > ((int64_t)1 << 30) || in > ((int64_t)1 << 40)) return MCF_E_SHAPE;
  if (!grid_fits(batch, out) || !product_fits(batch, out, in)) return MCF_E_SHAPE;
  if (batch == 0 || out == 0) return MCF_OK;
  if (!y || (in > 0 && (!x || !W))) return MCF_E_NULL;
  const int64_t es = elem_size(dtype);
  const int64_t yb = nc * batch * out * es;
  if (overlap(y, yb, x, batch * in * es) || overlap(y, yb, W, nc * out * in * es) ||
      (b && overlap(y, yb, b, nc * out * es)))
    return MCF_E_ALIAS;
  if (dtype == MCF_F16S)
    return hip_status(mcf::launch_scaled_matmul(nc, batch, out, in, x, 0, W, 1, 1, b, y, (hipStream_t)stream));
  return hip_status(mcf::launch_matmul(dtype, nc, batch, out, in, x, 0, W, 1, 1, b, y, (hipStream_t)stream));
}

const char *mc_status_str(int status) {
  switch (status) {
    case MCF_OK: return "MCF_OK";
    case MCF_E_NULL: return "MCF_E_NULL: required pointer is NULL";
    case MCF_E_NC: return "MCF_E_NC: component count out of range";
    case MCF_E_SHAPE: return "MCF_E_SHAPE: invalid size";
    case MCF_E_DTYPE: return "MCF_E_DTYPE: unsupported component format";
    case MCF_E_ALIAS: return "MCF_E_ALIAS: output overlaps an input";
    case MCF_E_HIP: return "MCF_E_HIP: HIP runtime error";
    case MCF_E_ARG: return "MCF_E_ARG: invalid argument";
    case MCF_E_SCRATCH: return "MCF_E_SCRATCH: the call needs more scratch than the library's static 8 MiB";
  }
  return "unknown status";
}

}  // extern "C"
