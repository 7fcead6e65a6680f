// Measurement probes for the benchmark (not part of the tick): achievable
// dense bf16 MFMA throughput on this device.
//
// Every wave keeps 8 independent 32x32 fp32 accumulators and issues
// v_mfma_f32_32x32x16_bf16 back to back on register-resident operands
// loaded once from a buffer (random bits give the power draw of real data,
// zeros the best case). Nothing is stored but one value per wave, so the
// loop is bound by the matrix cores alone.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void mfma_peak_kernel(const u32x4* __restrict__ src, int iters,
                                                        float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const u32x4 a = src[lane];
  const u32x4 b = src[64 + lane];
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  const bf16x8 av = __builtin_bit_cast(bf16x8, a), bv = __builtin_bit_cast(bf16x8, b);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  if (lane == 0) sink[blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6)] = s;
}

}  // namespace

extern "C" {

// Runs the probe on `stream`: `blocks` blocks of 4 waves, `iters` iterations
// of kChains MFMAs per wave. src: device, 128 x 16 bytes of operand bits;
// sink: device, one float per wave. Returns the FLOPs issued (for the caller's
// timing), or -1 on a launch error.
double im_probe_mfma_bf16(const void* src, float* sink, int blocks, int iters, void* stream) {
  hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (const u32x4*)src, iters, sink);
  if (hipGetLastError() != hipSuccess) return -1.0;
  return (double)blocks * 4 * iters * kChains * 2.0 * 32 * 32 * 16;
}

}  // extern "C"
