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
// the promotion of a plain dY) in the caller's workspace.
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

int64_t linear_bwd_workspace_bytes(int dtype, int nc, int64_t Tn, int64_t O) {
  return align256(nc * O * Tn * es_of(dtype)) + align256(Tn * es_of(dtype));
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
  if (Tn > 0) {
    if (dtype == 0)
      e = stage<_Float16>(nc, planes, Tn, O, dY, dYt, db ? ones : nullptr, s);
    else if (dtype == 2)
      e = stage<double>(nc, planes, Tn, O, dY, dYt, db ? ones : nullptr, s);
    else
      e = stage<float>(nc, planes, Tn, O, dY, dYt, db ? ones : nullptr, s);
    if (e != hipSuccess) return e;
  }
  if (dW != nullptr) {
    e = launch_matmul(dtype, nc, O, I, Tn, dYt, 1, x, 0, 0, nullptr, dW, s);
    if (e != hipSuccess) return e;
  }
  if (db != nullptr) e = launch_matmul(dtype, nc, O, 1, Tn, dYt, 1, ones, 0, 0, nullptr, db, s);
  return e;
}

}  // namespace mcf
