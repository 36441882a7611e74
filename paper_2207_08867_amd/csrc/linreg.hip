// linreg.hip -- one gradient-descent step of MC-Linear regression with the mean-squared
// error, the paper's precision experiment (Section 2.4): a single MC-Linear layer
// without bias fitted by gradient descent to y = X W*^T.
//
// The step (in stream order, all on the device):
//   1. yhat = MC-Linear(X, W)                   MM-MCN order (Section 2.3)
//   2. r    = Grow-ExpN(yhat, -y)               the MC residual, in place of yhat
//   3. G    = r^T X                             K-split product, default slice count
//   4. RR   = r . r                             K-split product, default slice count
//   5. per weight j: g = ScalingN(G_j, fl(2/n)); the gradient is g's leading component
//      (the paper keeps the gradient of an MC value as the plain gradient of its
//      leading component, Section 2.1); W_j = Grow-ExpN(W_j, fl(-lr * grad));
//      loss = ScalingN(RR, fl(1/n)), the mean-squared error at the weights before the
//      update.
// fl(2/n), fl(1/n) and fl(-lr) are the component-format roundings of the binary64
// quotient or value (one rounding each, done on the host); fl(-lr * grad) is one
// rounding of the product in the component format.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mcf_arith.hpp"
#include "mcf_internal.hpp"

namespace mcf {

namespace {

template <typename T, int NC>
__global__ void lr_update_kernel(const T *G, const T *RR, T *W, int64_t d, T s2n, T s1n, T neg_lr, T *loss) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < d) {
    T g[NC], gs[NC], w[NC], wn[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      g[c] = G[c * d + j];
      w[c] = W[c * d + j];
    }
    scaling_n<T, NC, NC>(g, s2n, gs);
    const T step = neg_lr * gs[0];  // one rounding in the component format
    grow_expn<T, NC>(w, step, wn);
#pragma unroll
    for (int c = 0; c < NC; ++c) W[c * d + j] = wn[c];
  }
  if (j == 0 && loss != nullptr) {
    T rr[NC], l[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) rr[c] = RR[c];
    scaling_n<T, NC, NC>(rr, s1n, l);
#pragma unroll
    for (int c = 0; c < NC; ++c) loss[c] = l[c];
  }
}

template <typename T>
hipError_t lr_update(int nc, const void *G, const void *RR, void *W, int64_t d, T s2n, T s1n, T neg_lr, void *loss,
                     hipStream_t s) {
  const dim3 grid((unsigned)((d + 255) / 256)), block(256);
  const T *g = (const T *)G, *rr = (const T *)RR;
  T *w = (T *)W, *l = (T *)loss;
  switch (nc) {
    case 1: hipLaunchKernelGGL((lr_update_kernel<T, 1>), grid, block, 0, s, g, rr, w, d, s2n, s1n, neg_lr, l); break;
    case 2: hipLaunchKernelGGL((lr_update_kernel<T, 2>), grid, block, 0, s, g, rr, w, d, s2n, s1n, neg_lr, l); break;
    case 3: hipLaunchKernelGGL((lr_update_kernel<T, 3>), grid, block, 0, s, g, rr, w, d, s2n, s1n, neg_lr, l); break;
    case 4: hipLaunchKernelGGL((lr_update_kernel<T, 4>), grid, block, 0, s, g, rr, w, d, s2n, s1n, neg_lr, l); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

struct LrLayout {
  int64_t r, g, rr, sk, total;
};

LrLayout lr_layout(int dtype, int nc, int64_t n, int64_t d) {
  const int64_t es = dtype == 0 ? 2 : (dtype == 2 ? 8 : 4);
  LrLayout L;
  L.r = 0;
  L.g = align256(nc * n * es);
  L.rr = L.g + align256(nc * d * es);
  L.sk = L.rr + align256(nc * es);
  // K-split workspaces of r^T X (M = 1, N = d, MC x plain) and r . r (M = N = 1, MC x MC)
  const int64_t w1 = splitk_roots(splitk_default_slices(1, d, n)) * nc * d * es;
  const int64_t w2 = splitk_roots(splitk_default_slices(1, 1, n)) * nc * nc * es;
  L.total = L.sk + align256(w1 > w2 ? w1 : w2);
  return L;
}

}  // namespace

int64_t linreg_workspace_bytes(int dtype, int nc, int64_t n, int64_t d) { return lr_layout(dtype, nc, n, d).total; }

hipError_t launch_linreg_step(int dtype, int nc, int64_t n, int64_t d, const void *X, const void *y_neg, void *W,
                              double s2n, double s1n, double neg_lr, void *ws, void *loss, hipStream_t s) {
  const LrLayout L = lr_layout(dtype, nc, n, d);
  char *w = (char *)ws;
  void *R = w + L.r, *G = w + L.g, *RR = w + L.rr, *SK = w + L.sk;
  hipError_t e = launch_matmul(dtype, nc, n, 1, d, X, 0, W, 1, 1, nullptr, R, s);
  if (e != hipSuccess) return e;
  e = launch_elementwise(dtype, EW_ADD, nc, nc, n, R, 1, y_neg, 0, R, s);
  if (e != hipSuccess) return e;
  e = launch_matmul_splitk(dtype, nc, 1, d, n, R, 1, X, 0, splitk_default_slices(1, d, n), SK, G, s);
  if (e != hipSuccess) return e;
  e = launch_matmul_splitk(dtype, nc, 1, 1, n, R, 1, R, 1, splitk_default_slices(1, 1, n), SK, RR, s);
  if (e != hipSuccess) return e;
  if (dtype == 0)
    return lr_update<_Float16>(nc, G, RR, W, d, (_Float16)(float)s2n, (_Float16)(float)s1n, (_Float16)(float)neg_lr,
                               loss, s);
  if (dtype == 2) return lr_update<double>(nc, G, RR, W, d, s2n, s1n, neg_lr, loss, s);
  return lr_update<float>(nc, G, RR, W, d, (float)s2n, (float)s1n, (float)neg_lr, loss, s);
}

}  // namespace mcf
