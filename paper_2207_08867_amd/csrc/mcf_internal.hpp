// mcf_internal.hpp -- launchers shared between the ABI layer and the kernel files.
// Arguments are already validated by the ABI layer; every launcher returns a
// hipError_t from the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mcf {

enum EwOp { EW_ADD = 0, EW_MUL = 1, EW_DIV = 2, EW_RENORM = 3, EW_SIMPLE_RENORM = 4, EW_EXP = 5, EW_MUL_SLOW = 6,
            EW_SQUARE = 7 };

// Elementwise binary (add/mul/div/Mult-MCN-Slow), Square-MCN and renormalization
// launchers.  dtype 0 = binary16, 1 = binary32.  For the unary ones y is unused; for
// renormalization nc is nc_in.
hipError_t launch_elementwise(int dtype, int op, int nc, int nc_out, int64_t n, const void *x, int x_mc,
                              const void *y, int y_mc, void *out, hipStream_t stream);

// Exp-MCN over binary16 components; builds the per-device exponential table on the
// first call on a device.
hipError_t launch_exp_f16(int nc, int64_t n, const void *x, void *out, hipStream_t stream);

// Exp-MCN over binary32 components (correctly rounded component exponential).
hipError_t launch_exp_f32(int nc, int64_t n, const void *x, void *out, hipStream_t stream);

// Exp-MCN over binary64 components (correctly rounded component exponential, exp64.hip).
hipError_t launch_exp_f64(int nc, int64_t n, const void *x, void *out, hipStream_t stream);

// A product launch in full generality (validated by the ABI layer): batches
// B1 x B2 with per-operand batch strides (0 broadcasts) and plane strides; C dense
// [nc][B1][B2][M][N]; b_trans: B stored [planes][N][K]; epilogue mode 0 none, 1
// Add-MCN with y, 2 AddMM (Add-MCN(ScalingN(C, alpha), ScalingN(y, beta))); alpha and
// beta are exactly representable in the component format.
struct MmLaunch {
  int dtype = 1, nc = 1;
  int64_t M = 0, N = 0, K = 0, B1 = 1, B2 = 1;
  const void *A = nullptr, *B = nullptr;
  void *C = nullptr;
  int a_mc = 1, b_mc = 1, b_trans = 0;
  int64_t a_plane = 0, b_plane = 0, a_s1 = 0, a_s2 = 0, b_s1 = 0, b_s2 = 0;
  int mode = 0;
  const void *y = nullptr;
  int64_t y_plane = 0, y_ld = 0;
  double alpha = 1.0, beta = 1.0;
  int prune = 0;  // 1: the pruned MC x MC product (both operands MC, no epilogue)
};
hipError_t launch_matmul_general(const MmLaunch &L, hipStream_t stream);

// C[nc][M][N] = A x B.  b_trans: B is stored as [planes][N][K] (a linear layer's
// weight) instead of [planes][K][N].  bias: [nc][N] MC bias added with Add-MCN, or
// NULL.
hipError_t launch_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                         const void *B, int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream);

// K-split product (splitk.hip).  S slices (1 <= S <= min(K, SPLITK_MAX_SLICES)); W is
// a workspace of splitk_roots(S) entries when S exceeds one workgroup's slice group,
// else unused.  The default slice count aims at SPLITK_TARGET_LANES lanes in all
// and keeps at least SPLITK_MIN_STEPS reduction steps per slice.
constexpr int64_t SPLITK_TARGET_LANES = (int64_t)1 << 20;
constexpr int64_t SPLITK_MIN_STEPS = 64;
constexpr int64_t SPLITK_MAX_SLICES = (int64_t)1 << 20;
int64_t splitk_default_slices(int64_t M, int64_t N, int64_t K);
void splitk_shape(int64_t S, int *KS, int *G);
// Workspace entries (each NP x nc components per output) for S slices: the G slice
// group roots when G > 1, else none.
int64_t splitk_roots(int64_t S);
hipError_t launch_matmul_splitk(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                                const void *B, int b_mc, int64_t S, void *W, void *C, hipStream_t stream);
// Size of the static per-device scratch that mc_matmul_splitk_noalloc uses in place of
// a workspace, and its device address on the device of `stream` (looked up once per
// device).
constexpr int64_t SPLITK_SCRATCH_BYTES = (int64_t)8 << 20;
hipError_t splitk_scratch(hipStream_t stream, void **ptr);

// Exact binary16 product on the int8 matrix cores (exact.hip).  b_trans: B stored as
// [planes][N][K].  bias: [nc][N] MC row added exactly before the split, or null.  W: a
// workspace of exact_workspace_bytes(M, N, K) bytes.
int64_t exact_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_matmul_exact(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                               int b_mc, int b_trans, const void *bias, void *W, void *C, hipStream_t stream);

// binary16 with scaled low components (scaled.hip): component c stands for 2^(-11 c)
// times its stored value.  Elementwise: op EW_ADD = Add-MCN of two MC operands, EW_MUL
// = ScalingN of the MC operand x by the plain operand y.  Product: kinds as
// launch_matmul (b_trans with a plain A only: MC-Linear), bias [nc][N] or null.
hipError_t launch_scaled_elementwise(int op, int nc, int64_t n, const void *x, const void *y, void *out,
                                     hipStream_t stream);
hipError_t launch_scaled_matmul(int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc, const void *B,
                                int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream);

// MC-Linear backward (linear_bwd.hip): dX = dY W, dW = dY^T x, db = column sums of dY
// (each output optional); dY is [nc or 1][batch][out] (dy_mc).  ws holds
// linear_bwd_workspace_bytes(...) bytes (dY^T promoted to nc planes; then a column of
// ones, or x with a column of ones appended and the [dW | db] product).
int64_t linear_bwd_workspace_bytes(int dtype, int nc, int64_t batch, int64_t in, int64_t out);
hipError_t launch_linear_bwd(int dtype, int nc, int64_t batch, int64_t in, int64_t out, const void *x, const void *W,
                             const void *dY, int dy_mc, void *dX, void *dW, void *db, void *ws, hipStream_t stream);

// One gradient-descent step of MC-Linear regression (linreg.hip).  s2n, s1n and neg_lr
// are fl(2/n), fl(1/n) and fl(-lr), already values of the component format.  ws holds
// linreg_workspace_bytes(...) bytes.
int64_t linreg_workspace_bytes(int dtype, int nc, int64_t n, int64_t d);
hipError_t launch_linreg_step(int dtype, int nc, int64_t n, int64_t d, const void *X, const void *y_neg, void *W,
                              double s2n, double s1n, double neg_lr, void *ws, void *loss, hipStream_t stream);

}  // namespace mcf
