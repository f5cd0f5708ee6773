// Diagnostic kernel: the achievable dense bf16 MFMA rate of the device.  Each
// wave keeps four independent v_mfma_f32_32x32x16_bf16 accumulation chains
// busy on register operands (no memory traffic in the loop), so the measured
// rate is the matrix-core issue rate the attention kernels are compared with.
#include "pd_common.h"
#include "pd_kernels.h"

namespace pd {

__global__ __launch_bounds__(256) void mfma_rate_kernel(int iters, float* sink) {
  const unsigned lane = threadIdx.x & 63;
  const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u ^ lane, 0x3f80u, 0x3f800000u, lane});
  const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u, lane, 0x3f803f80u ^ (lane << 16), 0u});
  f32x16 c[4] = {f32x16{0}, f32x16{0}, f32x16{0}, f32x16{0}};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = mfma32x32x16(a, b, c[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[j][e];
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

hipError_t launch_mfma_rate(int n_workgroups, int iters, float* sink, hipStream_t s) {
  hipLaunchKernelGGL(mfma_rate_kernel, dim3(n_workgroups), dim3(256), 0, s, iters, sink);
  return hipGetLastError();
}

}  // namespace pd
