// Measurement aid, not part of the operator: a dense bf16 matrix-core kernel
// whose throughput is the achievable MFMA peak of the chip at the clock it
// sustains under that load, and a reading of that clock.
//
// Every wave runs 8 independent chains of v_mfma_f32_32x32x16_bf16 (32768
// flop each), so the matrix pipe of each SIMD never waits on a result. Wave 0
// of workgroup 0 reads the shader timestamp (s_memtime) and the fixed-rate
// real-time counter (s_memrealtime) before and after its loop; their ratio,
// times the real-time counter's rate, is the clock the loop ran at.
#include "kernels.h"

namespace rel {

namespace {

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, float* sink, unsigned long long* clocks) {
  const int tid = threadIdx.x;
  // operands that depend on the lane, so nothing is folded at compile time
  bf16x8 a, b;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    a[t] = (bf16)(1.0f + 1e-3f * (float)((tid + t) & 7));
    b[t] = (bf16)(1.0f - 1e-3f * (float)((tid * 3 + t) & 7));
  }
  floatx16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = floatx16{};
  const bool timer = blockIdx.x == 0 && tid == 0;
  unsigned long long t0 = 0, r0 = 0;
  if (timer) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = mfma32(a, b, acc[c]);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (timer) {
    const unsigned long long t1 = __builtin_amdgcn_s_memtime();
    const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
    clocks[0] = t1 - t0;
    clocks[1] = r1 - r0;
  }
  sink[(size_t)blockIdx.x * blockDim.x + tid] = s;
}

}  // namespace

int64_t mfma_peak_flops_per_launch(int workgroups, int iters) {
  return (int64_t)workgroups * 4 * iters * kChains * 32768;
}

hipError_t launch_mfma_peak(int workgroups, int iters, float* sink, unsigned long long* clocks, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_peak_kernel, dim3((unsigned)workgroups), dim3(256), 0, stream, iters, sink, clocks);
  return hipGetLastError();
}

}  // namespace rel
