// Measured matrix-core peak of gfx950 for the instructions the tile kernel
// issues (v_mfma_f32_32x32x2_f32, v_mfma_f64_16x16x4_f64), so that the tile
// kernel's rate can be set against a sustained rather than only a published
// peak. No memory traffic: every wave runs four independent accumulation
// chains (enough to cover the instruction's dependency latency) and stores
// one value per lane at the end so the work is kept. Two waves per SIMD, as
// in the tile kernel; the register budget that comes with it also keeps the
// accumulators in place across loop trips (checked in the assembly).
#include "lssvm.h"
#include "lssvm_error.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

namespace lssvm {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef double doublex4 __attribute__((ext_vector_type(4)));

// Exactly one resident round: two workgroups of four waves per CU (two waves
// per SIMD, as in the tile kernel). A grid larger than what is resident at
// once would end in a partial round and report a lower rate.
constexpr int kProbeBlocks = 2 * 256;
constexpr int kProbeThreads = 256;
constexpr int kProbeIters = 32768;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_mfma_loop_f32(
    int iters, float seed, float* sink) {
  floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  const float a = seed * (float)(threadIdx.x & 7), b = seed;
  for (int k = 0; k < iters; ++k) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(b, a, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, a, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(b, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int v = 0; v < 16; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_mfma_loop_f64(
    int iters, double seed, double* sink) {
  doublex4 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  const double a = seed * (double)(threadIdx.x & 7), b = seed;
  for (int k = 0; k < iters; ++k) {
    c0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f64_16x16x4f64(b, a, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f64_16x16x4f64(a, a, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f64_16x16x4f64(b, b, c3, 0, 0, 0);
  }
  double s = 0.0;
#pragma unroll
  for (int v = 0; v < 4; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Flops of one wave's loop: 4 chains x iters x (M M K x 2).
double loop_flops(int32_t dtype) {
  const double per = dtype == LSSVM_F32 ? 32.0 * 32.0 * 2.0 * 2.0 : 16.0 * 16.0 * 4.0 * 2.0;
  const double waves = (double)kProbeBlocks * (kProbeThreads / 64);
  return waves * 4.0 * kProbeIters * per;
}

hipError_t launch(int32_t dtype, void* sink, hipStream_t s) {
  if (dtype == LSSVM_F32)
    hipLaunchKernelGGL(k_mfma_loop_f32, dim3(kProbeBlocks), dim3(kProbeThreads), 0, s,
                       kProbeIters, 1e-3f, static_cast<float*>(sink));
  else
    hipLaunchKernelGGL(k_mfma_loop_f64, dim3(kProbeBlocks), dim3(kProbeThreads), 0, s,
                       kProbeIters, 1e-3, static_cast<double*>(sink));
  return hipGetLastError();
}

}  // namespace
}  // namespace lssvm

using namespace lssvm;

extern "C" {

size_t lssvm_mfma_peak_workspace_bytes(void) {
  return (size_t)kProbeBlocks * kProbeThreads * sizeof(double);
}

int lssvm_mfma_peak(int32_t dtype, void* workspace, size_t workspace_bytes, double* tflops_out,
                    void* stream) {
  clear_error();
  if (dtype != LSSVM_F32 && dtype != LSSVM_F64)
    return fail(LSSVM_EINVAL, "unknown dtype %d", (int)dtype);
  if (!workspace || !tflops_out) return fail(LSSVM_EINVAL, "NULL argument");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0)
    return fail(LSSVM_EINVAL, "workspace must be 256-byte aligned");
  if (workspace_bytes < lssvm_mfma_peak_workspace_bytes())
    return fail(LSSVM_EINVAL, "workspace too small: %zu bytes given, %zu needed", workspace_bytes,
                lssvm_mfma_peak_workspace_bytes());
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  auto done = [&](int code) {
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    return code;
  };
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess)
    return done(fail(LSSVM_EHIP, "hipEventCreate failed"));
  // one untimed launch (clock ramp), then the median of three timed ones
  if (launch(dtype, workspace, s) != hipSuccess) return done(fail(LSSVM_EHIP, "launch failed"));
  float ms[3];
  for (int k = 0; k < 3; ++k) {
    if (hipEventRecord(e0, s) != hipSuccess || launch(dtype, workspace, s) != hipSuccess ||
        hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
        hipEventElapsedTime(&ms[k], e0, e1) != hipSuccess)
      return done(fail(LSSVM_EHIP, "timed launch failed"));
  }
  std::sort(ms, ms + 3);
  *tflops_out = loop_flops(dtype) / ((double)ms[1] * 1e-3) / 1e12;
  return done(LSSVM_OK);
}

}  // extern "C"
