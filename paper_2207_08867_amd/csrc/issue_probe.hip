// issue_probe.hip -- VALU issue-rate probe, the measurement behind the VALU roofline
// that the product kernels are reported against.  Built into its own library
// (libmcf_probe.so); nothing in libmcf.so uses it.
//
// Each probe kernel runs CH independent dependency chains per lane of ONE instruction
// kind, UN-fold unrolled, so the issue rate -- not the latency of a chain -- limits
// it.  2048 workgroups of 256 lanes put 8 wavefronts on every SIMD of the 256 CUs.
// Every wavefront also reads the shader clock (clock64) and the constant-rate wall
// clock (wall_clock64) around its loop, so the host can state the clock the rates were
// measured at.  The result is only written when it equals an impossible value, which
// keeps the chains live without memory traffic.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int CH = 8;   // independent chains per lane
constexpr int UN = 16;  // unrolled instructions per chain per loop iteration

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

enum ProbeOp {
  P_ADD_F32 = 0, P_MUL_F32, P_FMA_F32, P_ADD_F16, P_MUL_F16, P_FMA_F16, P_PK_ADD_F16, P_MIN3_F32, P_CVT_F16_F32,
  P_CVT_F32_F16, P_FMA_MIX_F32, P_FMA_MIXLO_F16, P_ADD_F64, P_FMA_F64, P_ADD_U32, P_AND_B32, P_ADD3_U32,
  P_BFE_U32, P_LDEXP_F16, P_MUL_F64, P_LDEXP_F64, P_RNDNE_F64, P_CVT_I32_F64, P_CMP_LT_F64, P_MOV_B64,
  P_LSHL_ADD_U64, P_COUNT
};

template <int OP>
__global__ __launch_bounds__(256) void probe_kernel(float *out, uint64_t *clocks, int iters, float seed) {
  float f[CH];
  _Float16 h[CH];
  double d[CH];
  half2_t p[CH];
  unsigned u[CH];
  uint64_t q[CH];
  uint64_t sc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    f[c] = seed + (float)c + (float)threadIdx.x;
    h[c] = (_Float16)(seed + (float)c);
    d[c] = (double)seed + c;
    p[c] = half2_t{h[c], h[c]};
    u[c] = threadIdx.x + c;
    q[c] = threadIdx.x + 7 * c;
    sc[c] = 0;
  }
  const float g = seed * 0.5f;
  const _Float16 hg = (_Float16)g;
  const double dg = g;
  const half2_t pg = half2_t{hg, hg};
  const unsigned ug = 3u;
  const uint64_t qg = 5u;
  const int ig = -1;
  const uint64_t t0 = clock64(), w0 = wall_clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < UN; ++r) {
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        if constexpr (OP == P_ADD_F32) asm volatile("v_add_f32 %0, %0, %1" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_MUL_F32) asm volatile("v_mul_f32 %0, %0, %1" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_FMA_F32) asm volatile("v_fma_f32 %0, %0, %1, %1" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_ADD_F16) asm volatile("v_add_f16 %0, %0, %1" : "+v"(h[c]) : "v"(hg));
        if constexpr (OP == P_MUL_F16) asm volatile("v_mul_f16 %0, %0, %1" : "+v"(h[c]) : "v"(hg));
        if constexpr (OP == P_FMA_F16) asm volatile("v_fma_f16 %0, %0, %1, %1" : "+v"(h[c]) : "v"(hg));
        if constexpr (OP == P_PK_ADD_F16) asm volatile("v_pk_add_f16 %0, %0, %1" : "+v"(p[c]) : "v"(pg));
        if constexpr (OP == P_MIN3_F32) asm volatile("v_min3_f32 %0, %0, %1, %1" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_CVT_F16_F32) asm volatile("v_cvt_f16_f32 %0, %0" : "+v"(f[c]));
        if constexpr (OP == P_CVT_F32_F16) asm volatile("v_cvt_f32_f16 %0, %1" : "=v"(f[c]) : "v"(h[c]));
        if constexpr (OP == P_FMA_MIX_F32)
          asm volatile("v_fma_mix_f32 %0, %0, %1, %1 op_sel_hi:[1,1,1]" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_FMA_MIXLO_F16)
          asm volatile("v_fma_mixlo_f16 %0, %0, %1, %1 op_sel_hi:[0,0,0]" : "+v"(f[c]) : "v"(g));
        if constexpr (OP == P_ADD_F64) asm volatile("v_add_f64 %0, %0, %1" : "+v"(d[c]) : "v"(dg));
        if constexpr (OP == P_FMA_F64) asm volatile("v_fma_f64 %0, %0, %1, %1" : "+v"(d[c]) : "v"(dg));
        if constexpr (OP == P_ADD_U32) asm volatile("v_add_u32 %0, %0, %1" : "+v"(u[c]) : "v"(ug));
        if constexpr (OP == P_AND_B32) asm volatile("v_and_b32 %0, %0, %1" : "+v"(u[c]) : "v"(ug));
        if constexpr (OP == P_ADD3_U32) asm volatile("v_add3_u32 %0, %0, %1, %1" : "+v"(u[c]) : "v"(ug));
        if constexpr (OP == P_BFE_U32) asm volatile("v_bfe_u32 %0, %0, %1, %1" : "+v"(u[c]) : "v"(ug));
        if constexpr (OP == P_LDEXP_F16) asm volatile("v_ldexp_f16 %0, %0, %1" : "+v"(h[c]) : "v"(ig));
        if constexpr (OP == P_MUL_F64) asm volatile("v_mul_f64 %0, %0, %1" : "+v"(d[c]) : "v"(dg));
        if constexpr (OP == P_LDEXP_F64) asm volatile("v_ldexp_f64 %0, %0, %1" : "+v"(d[c]) : "v"(ig));
        if constexpr (OP == P_RNDNE_F64) asm volatile("v_rndne_f64 %0, %0" : "+v"(d[c]));
        if constexpr (OP == P_CVT_I32_F64) asm volatile("v_cvt_i32_f64 %0, %1" : "=v"(u[c]) : "v"(d[c]));
        if constexpr (OP == P_CMP_LT_F64) asm volatile("v_cmp_lt_f64_e64 %0, %1, %2" : "=s"(sc[c]) : "v"(d[c]), "v"(dg));
        if constexpr (OP == P_MOV_B64) asm volatile("v_mov_b64 %0, %0" : "+v"(d[c]));
        if constexpr (OP == P_LSHL_ADD_U64) asm volatile("v_lshl_add_u64 %0, %0, 1, %1" : "+v"(q[c]) : "v"(qg));
      }
    }
  }
  const uint64_t t1 = clock64(), w1 = wall_clock64();
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < CH; ++c) s += f[c] + (float)h[c] + (float)d[c] + (float)p[c].x + (float)u[c] + (float)q[c] + (float)sc[c];
  if (s == 1234.5f) out[blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    clocks[2 * blockIdx.x] = t1 - t0;
    clocks[2 * blockIdx.x + 1] = w1 - w0;
  }
}

template <int OP>
hipError_t launch(int blocks, int iters, float *out, uint64_t *clocks) {
  hipLaunchKernelGGL(probe_kernel<OP>, dim3(blocks), dim3(256), 0, 0, out, clocks, iters, 1.0f);
  return hipGetLastError();
}

template <int OP = 0>
hipError_t launch_op(int op, int blocks, int iters, float *out, uint64_t *clocks) {
  if constexpr (OP < P_COUNT) {
    if (op == OP) return launch<OP>(blocks, iters, out, clocks);
    return launch_op<OP + 1>(op, blocks, iters, out, clocks);
  }
  return hipErrorInvalidValue;
}

const char *const NAMES[P_COUNT] = {
    "v_add_f32", "v_mul_f32", "v_fma_f32", "v_add_f16", "v_mul_f16", "v_fma_f16", "v_pk_add_f16", "v_min3_f32",
    "v_cvt_f16_f32", "v_cvt_f32_f16", "v_fma_mix_f32", "v_fma_mixlo_f16", "v_add_f64", "v_fma_f64", "v_add_u32",
    "v_and_b32", "v_add3_u32", "v_bfe_u32", "v_ldexp_f16", "v_mul_f64", "v_ldexp_f64", "v_rndne_f64",
    "v_cvt_i32_f64", "v_cmp_lt_f64", "v_mov_b64", "v_lshl_add_u64"};

}  // namespace

extern "C" {

// Number of probe kinds and the name of kind `op` (NULL when out of range).
int mcf_probe_count(void) { return P_COUNT; }
const char *mcf_probe_name(int op) { return (op >= 0 && op < P_COUNT) ? NAMES[op] : nullptr; }

// Runs probe `op` on `blocks` workgroups of 256 lanes with `iters` loop iterations
// (after one short warm-up launch) on the null stream of the current device.
// Outputs: *ms, the launch's duration (HIP events); *lane_instr, the probed VALU
// instructions issued times 64 lanes; *clock_ghz, the mean shader clock of the
// wavefronts' loops (clock64 cycles over wall_clock64 time).  Returns 0 or a
// hipError_t.
int mcf_probe_issue(int op, int blocks, int iters, double *ms, double *lane_instr, double *clock_ghz) {
  if (op < 0 || op >= P_COUNT || blocks < 1 || iters < 1 || !ms || !lane_instr || !clock_ghz)
    return (int)hipErrorInvalidValue;
  float *out = nullptr;
  uint64_t *clocks = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  int wall_khz = 0;
  hipError_t e = hipMalloc(&out, (size_t)blocks * 256 * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&clocks, (size_t)blocks * 2 * sizeof(uint64_t));
  if (e == hipSuccess) e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) {
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev);
  }
  if (e == hipSuccess) e = launch_op(op, blocks, iters < 16 ? iters : 16, out, clocks);
  if (e == hipSuccess) e = hipEventRecord(a, 0);
  if (e == hipSuccess) e = launch_op(op, blocks, iters, out, clocks);
  if (e == hipSuccess) e = hipEventRecord(b, 0);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float t = 0.0f;
  if (e == hipSuccess) e = hipEventElapsedTime(&t, a, b);
  uint64_t *host = nullptr;
  if (e == hipSuccess) {
    host = new uint64_t[(size_t)blocks * 2];
    e = hipMemcpy(host, clocks, (size_t)blocks * 2 * sizeof(uint64_t), hipMemcpyDeviceToHost);
  }
  if (e == hipSuccess) {
    double cyc = 0.0, wall = 0.0;
    for (int i = 0; i < blocks; ++i) {
      cyc += (double)host[2 * i];
      wall += (double)host[2 * i + 1];
    }
    *ms = t;
    *lane_instr = (double)blocks * 256.0 * iters * UN * CH;
    *clock_ghz = (wall > 0.0 && wall_khz > 0) ? cyc / (wall / (wall_khz * 1e3)) / 1e9 : 0.0;
  }
  delete[] host;
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (clocks) (void)hipFree(clocks);
  if (out) (void)hipFree(out);
  return (int)e;
}

}  // extern "C"
