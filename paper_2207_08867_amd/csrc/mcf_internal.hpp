// mcf_internal.hpp -- launchers shared between the ABI layer and the kernel files.
// Arguments are already validated by the ABI layer; every launcher returns a
// hipError_t from the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mcf {

enum EwOp { EW_ADD = 0, EW_MUL = 1, EW_DIV = 2, EW_RENORM = 3, EW_SIMPLE_RENORM = 4, EW_EXP = 5 };

// Elementwise binary (add/mul/div) and renormalization launchers.  dtype 0 = binary16,
// 1 = binary32.  For renormalization y is unused, nc is nc_in.
hipError_t launch_elementwise(int dtype, int op, int nc, int nc_out, int64_t n, const void *x, int x_mc,
                              const void *y, int y_mc, void *out, hipStream_t stream);

// Exp-MCN over binary16 components; builds the per-device exponential table on the
// first call on a device.
hipError_t launch_exp_f16(int nc, int64_t n, const void *x, void *out, hipStream_t stream);

// Exp-MCN over binary32 components (correctly rounded component exponential).
hipError_t launch_exp_f32(int nc, int64_t n, const void *x, void *out, hipStream_t stream);

// C[nc][M][N] = A x B.  b_trans: B is stored as [planes][N][K] (a linear layer's
// weight) instead of [planes][K][N].  bias: [nc][N] MC bias added with Add-MCN, or
// NULL.
hipError_t launch_matmul(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                         const void *B, int b_mc, int b_trans, const void *bias, void *C, hipStream_t stream);

// K-split product (splitk.hip).  S slices (1 <= S <= min(K, SPLITK_MAX_SLICES)); W is
// a workspace of splitk_workspace_elems(...) components when S exceeds one
// workgroup's slice group, else unused.
constexpr int64_t SPLITK_TARGET_LANES = (int64_t)1 << 18;
constexpr int64_t SPLITK_MAX_SLICES = 65536;
int64_t splitk_default_slices(int64_t M, int64_t N, int64_t K);
void splitk_shape(int64_t S, int *KS, int *G);
hipError_t launch_matmul_splitk(int dtype, int nc, int64_t M, int64_t N, int64_t K, const void *A, int a_mc,
                                const void *B, int b_mc, int64_t S, void *W, void *C, hipStream_t stream);

}  // namespace mcf
