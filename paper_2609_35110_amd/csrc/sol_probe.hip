// The dense matrix rate the chip sustains under the attention kernels' launch
// shape: one wave per SIMD issuing only fp16 32x32x16 MFMAs (the operation
// both products of the prepared path use) with fp32 accumulation.  The
// datasheet peak assumes 2.4 GHz; under a long dense launch the clock is
// power-limited, so this is the ceiling a kernel can be held to on the box it
// runs on.  Operands are real (seeded) fp16 values: the power draw, and so the
// clock, depends on them.
#include "sol_device.h"

namespace sol {
namespace {

constexpr int kProbeChains = 4;  // independent accumulators per wave

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void mfma_probe_kernel(const uint4* __restrict__ operands, float* __restrict__ out, int iters) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // wave w: A fragments from uint4 [128w, 128w + 128), B fragments from
  // [128w + 512, 128w + 640) of the 1024 (16 KB of operands)
  const int base = wave * 128;
  f16x8 a[2], b[2];
  a[0] = __builtin_bit_cast(f16x8, operands[base + lane]);
  a[1] = __builtin_bit_cast(f16x8, operands[base + 64 + lane]);
  b[0] = __builtin_bit_cast(f16x8, operands[base + 512 + lane]);
  b[1] = __builtin_bit_cast(f16x8, operands[base + 576 + lane]);
  f32x16 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.0f;
#pragma unroll 1
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < kProbeChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[(r + c) & 1], b[(r >> 1) & 1], acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

// 16 MFMAs of 32x32x16 (32,768 flops each) per wave and iteration.
hipError_t launch_mfma_probe(const uint16_t* operands, float* out, int workgroups, int iters,
                             hipStream_t stream) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)workgroups), dim3(256), 0, stream,
                     reinterpret_cast<const uint4*>(operands), out, iters);
  return hipGetLastError();
}

}  // namespace sol
