// Measurement aid: the MFMA rate the chip sustains on a register-only loop of bf16 32x32x16
// MFMAs (no memory traffic), as a reference beside the dense bf16 peak.  Not part of the step.
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kProbeChains = 8;  // independent accumulators per wave

__global__ __launch_bounds__(256, 2) void mfma_probe_kernel(float* __restrict__ out, int iters,
                                                         float seed) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(seed + 1e-3f * static_cast<float>(threadIdx.x) + i);
    b[i] = static_cast<__bf16>(seed - i);
  }
  f32x16 acc[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) acc[j] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j) acc[j] = mfma32(a, b, acc[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  out[blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

double mfma_probe_flops(int groups, int iters) {
  return 2.0 * 32 * 32 * 16 * kProbeChains * static_cast<double>(iters) * 4.0 * groups;
}

hipError_t mfma_probe(float* out, int groups, int iters, hipStream_t s) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(groups), dim3(256), 0, s, out, iters, 0.5f);
  return hipGetLastError();
}

}  // namespace eb
