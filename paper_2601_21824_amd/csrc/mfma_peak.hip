// mfma_peak.hip -- measured bf16 dense MFMA throughput of the device, the
// measured counterpart of the published peak in the main kernel's roofline.
// Every wave keeps kChains independent accumulation chains of
// v_mfma_f32_32x32x16_bf16 (32768 FLOP each) busy on register operands, so
// the matrix cores, not issue or memory, set the rate.
#include "common.h"
#include "kernels.h"

namespace dash {
namespace {

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, float* sink) {
  // operands that depend on the lane, so the compiler cannot fold them
  const float x = (float)(threadIdx.x & 7) * 0.0625f;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(x + (float)i);
    b[i] = (__bf16)(x - (float)i);
  }
  f32x16 c[kChains];
#pragma unroll
  for (int k = 0; k < kChains; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) c[k][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < kChains; ++k) c[k] = mfma32(a, b, c[k]);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kChains; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[k][r];
  sink[blockIdx.x * blockDim.x + threadIdx.x] = s;  // keeps the chains alive
}

}  // namespace

double mfma_peak_flops_per_launch(int grid, int iters) { return (double)grid * 4.0 * iters * kChains * 32768.0; }

void launch_mfma_peak(int grid, int iters, float* sink, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(grid), dim3(256), 0, stream, iters, sink);
}

}  // namespace dash
