// linear_bwd.hip -- MC-Linear backward on gfx950: the gradients of y = x W^T + b with
// respect to the input, the weight and the bias, given the gradient dY of the output.
//
//   dX = dY W              [batch][in]   (MM-MCN; dY MC: by linearity over W's
//                                         components, as every MC x MC product)
//   dW = dY^T x            [out][in]     (MM-MCN over the batch index)
//   db = sum_t dY[t]       [out]         (MM-MCN against a column of ones: Add-MCN of the
//                                         rows in batch order; ScalingN by 1 is exact)
// A plain dY (the gradient of an MC value is a plain tensor, Section 2.1) enters dW and
// db as an MC value with +0 low components, so the products keep their exact rounding
// errors; the leading component of each result is the plain gradient.  All three are
// the library's sequential product kernels; this file adds the staging of dY^T (and
// the promotion of a plain dY) in the caller's workspace.  When both dW and db are
// wanted they come from one product, dY^T [x | 1], whose last column is db: every
// output of a product depends only on its own row and column, so the columns are the
// values of the two separate products, and the 1024-output column sum (a long
// dependent chain per lane, latency-bound when run alone) runs beside dW's tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_internal.hpp"

namespace mcf {
namespace {

constexpr int TP = 32;  // transpose tile

// dYt[c][o][t] = dY[c][t][o] for c < planes, +0 for planes <= c < nc.  Grid: (tiles of
// O, tiles of T, nc); 32 x 8 lanes move a 32 x 32 tile through LDS.
template <typename T>
__global__ __launch_bounds__(TP * 8) void transpose_promote_kernel(const T *__restrict__ dY, int planes,
                                                                   T *__restrict__ dYt, int64_t Tn, int64_t O) {
  __shared__ T tile[TP][TP + 1];
  const int c = blockIdx.z;
  const int64_t o0 = (int64_t)blockIdx.x * TP, t0 = (int64_t)blockIdx.y * TP;
  const int tx = threadIdx.x % TP, ty = threadIdx.x / TP;
  for (int r = ty; r < TP; r += 8) {
    const int64_t t = t0 + r, o = o0 + tx;
    tile[r][tx] = (c < planes && t < Tn && o < O) ? dY[(int64_t)c * Tn * O + t * O + o] : T(0);
  }
  __syncthreads();
  for (int r = ty; r < TP; r += 8) {
    const int64_t o = o0 + r, t = t0 + tx;
    if (o < O && t < Tn) dYt[(int64_t)c * O * Tn + o * Tn + t] = tile[tx][r];
  }
}

template <typename T>
__global__ void fill_one_kernel(T *__restrict__ v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = T(1);
}

// xo[t][i] = x[t][i] for i < I, xo[t][I] = 1: [Tn][I + 1].
template <typename T>
__global__ void append_ones_kernel(const T *__restrict__ x, T *__restrict__ xo, int64_t Tn, int64_t I) {
  const int64_t n = Tn * (I + 1);
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = k / (I + 1), i = k - t * (I + 1);
    xo[k] = i < I ? x[t * I + i] : T(1);
  }
}

// C [nc][O][I + 1] -> dW [nc][O][I] (columns < I) and db [nc][O] (column I).
template <typename T>
__global__ void split_last_column_kernel(const T *__restrict__ C, T *__restrict__ dW, T *__restrict__ db,
                                         int64_t rows, int64_t I) {
  const int64_t n = rows * (I + 1);
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = k / (I + 1), i = k - r * (I + 1);
    if (i < I)
      dW[r * I + i] = C[k];
    else
      db[r] = C[k];
  }
}

// The [dW | db] product (out x (in + 1), reduction batch) within the product kernel's
// grid (below 2^31 tiles of 16 x 16) and operand-size limits (below 2^50 elements).
bool fused_fits(int64_t O, int64_t I, int64_t Tn) {
  const int64_t N = I + 1;
  return ((O + 15) / 16) * ((N + 15) / 16) < ((int64_t)1 << 31) && Tn <= ((int64_t)1 << 50) / N &&
         O <= ((int64_t)1 << 50) / N;
}

unsigned stride_grid(int64_t n) {
  const int64_t b = (n + 255) / 256;
  return (unsigned)(b < 8192 ? (b < 1 ? 1 : b) : 8192);
}

int64_t es_of(int dtype) { return dtype == 0 ? 2 : (dtype == 2 ? 8 : 4); }
int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

template <typename T>
hipError_t stage(int nc, int planes, int64_t Tn, int64_t O, const void *dY, void *dYt, void *ones, hipStream_t s) {
  const dim3 grid((unsigned)((O + TP - 1) / TP), (unsigned)((Tn + TP - 1) / TP), (unsigned)nc);
  hipLaunchKernelGGL((transpose_promote_kernel<T>), grid, dim3(TP * 8), 0, s, (const T *)dY, planes, (T *)dYt, Tn,
                     O);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ones == nullptr) return e;
  hipLaunchKernelGGL((fill_one_kernel<T>), dim3((unsigned)((Tn + 255) / 256)), dim3(256), 0, s, (T *)ones, Tn);
  return hipGetLastError();
}

}  // namespace

// dY^T, then either the column of ones (db alone) or [x | 1] and the [dW | db] product
// (both): the larger of the two.
int64_t linear_bwd_workspace_bytes(int dtype, int nc, int64_t Tn, int64_t I, int64_t O) {
  const int64_t es = es_of(dtype);
  const int64_t both = align256(Tn * (I + 1) * es) + align256(nc * O * (I + 1) * es);
  const int64_t ones = align256(Tn * es);
  return align256(nc * O * Tn * es) + (both > ones ? both : ones);
}

hipError_t launch_linear_bwd(int dtype, int nc, int64_t Tn, int64_t I, int64_t O, const void *x, const void *W,
                             const void *dY, int dy_mc, void *dX, void *dW, void *db, void *ws, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (dX != nullptr) {
    e = launch_matmul(dtype, nc, Tn, I, O, dY, dy_mc, W, 1, 0, nullptr, dX, s);
    if (e != hipSuccess) return e;
  }
  if (dW == nullptr && db == nullptr) return e;
  char *w = (char *)ws;
  void *dYt = w, *ones = w + align256(nc * O * Tn * es_of(dtype));
  const int planes = dy_mc ? nc : 1;
  const bool fused = dW != nullptr && db != nullptr && Tn > 0 && I > 0 && fused_fits(O, I, Tn);
  const bool ones_needed = db != nullptr && !fused;
  if (Tn > 0) {
    if (dtype == 0)
      e = stage<_Float16>(nc, planes, Tn, O, dY, dYt, ones_needed ? ones : nullptr, s);
    else if (dtype == 2)
      e = stage<double>(nc, planes, Tn, O, dY, dYt, ones_needed ? ones : nullptr, s);
    else
      e = stage<float>(nc, planes, Tn, O, dY, dYt, ones_needed ? ones : nullptr, s);
    if (e != hipSuccess) return e;
  }
  if (fused) {
    void *xo = ones, *Cw = (char *)ones + align256(Tn * (I + 1) * es_of(dtype));
    const unsigned gx = stride_grid(Tn * (I + 1)), gc = stride_grid(nc * O * (I + 1));
    if (dtype == 0)
      hipLaunchKernelGGL((append_ones_kernel<_Float16>), dim3(gx), dim3(256), 0, s, (const _Float16 *)x,
                         (_Float16 *)xo, Tn, I);
    else if (dtype == 2)
      hipLaunchKernelGGL((append_ones_kernel<double>), dim3(gx), dim3(256), 0, s, (const double *)x, (double *)xo, Tn,
                         I);
    else
      hipLaunchKernelGGL((append_ones_kernel<float>), dim3(gx), dim3(256), 0, s, (const float *)x, (float *)xo, Tn, I);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    e = launch_matmul(dtype, nc, O, I + 1, Tn, dYt, 1, xo, 0, 0, nullptr, Cw, s);
    if (e != hipSuccess) return e;
    if (dtype == 0)
      hipLaunchKernelGGL((split_last_column_kernel<_Float16>), dim3(gc), dim3(256), 0, s, (const _Float16 *)Cw,
                         (_Float16 *)dW, (_Float16 *)db, nc * O, I);
    else if (dtype == 2)
      hipLaunchKernelGGL((split_last_column_kernel<double>), dim3(gc), dim3(256), 0, s, (const double *)Cw,
                         (double *)dW, (double *)db, nc * O, I);
    else
      hipLaunchKernelGGL((split_last_column_kernel<float>), dim3(gc), dim3(256), 0, s, (const float *)Cw,
                         (float *)dW, (float *)db, nc * O, I);
    return hipGetLastError();
  }
  if (dW != nullptr) {
    e = launch_matmul(dtype, nc, O, I, Tn, dYt, 1, x, 0, 0, nullptr, dW, s);
    if (e != hipSuccess) return e;
  }
  if (db != nullptr) e = launch_matmul(dtype, nc, O, 1, Tn, dYt, 1, ones, 0, 0, nullptr, db, s);
  return e;
}

}  // namespace mcf
