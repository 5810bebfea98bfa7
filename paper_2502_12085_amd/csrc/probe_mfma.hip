// Matrix-core ceiling probe for gfx950: back-to-back 32x32x16 bf16 MFMAs on
// operands loaded from memory, no other work.  Measurement infrastructure
// beside the library, not a step of the attention path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "apb_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kPairs = 8;   // operand pairs each wave rotates through
constexpr int kChains = 4;  // independent accumulators per wave

__global__ void __launch_bounds__(64 * kWaves, 1)
mfma_loop_kernel(const uint16_t* __restrict__ operands, float* __restrict__ sink, int iters) {
  const int lane = threadIdx.x & 63;
  // every wave reads the same 16 KiB: pair j's A and B operands of lane l are
  // the 16-byte chunks 2*(64 j + l) and 2*(64 j + l) + 1
  bf16x8 a[kPairs], b[kPairs];
#pragma unroll
  for (int j = 0; j < kPairs; ++j) {
    const u32x4* src = reinterpret_cast<const u32x4*>(operands) + 2 * (64 * j + lane);
    a[j] = __builtin_bit_cast(bf16x8, src[0]);
    b[j] = __builtin_bit_cast(bf16x8, src[1]);
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int it = 0; it < iters; it += kPairs) {
#pragma unroll
    for (int u = 0; u < kPairs; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(u + 2 * c) % kPairs],
                                                         b[(u + 3 * c + 1) % kPairs], acc[c], 0,
                                                         0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

extern "C" int32_t apb_probe_mfma_bf16(const uint16_t* operands, float* sink,
                                       int32_t n_workgroups, int32_t iters, void* stream) {
  if (!operands || !sink || n_workgroups < 1 || n_workgroups > (1 << 20) || iters < 1 ||
      iters > (1 << 20) || iters % kPairs != 0 || ((uintptr_t)operands & 15u) != 0 ||
      ((uintptr_t)sink & 3u) != 0)
    return 1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)n_workgroups), dim3(64 * kWaves), 0,
                     (hipStream_t)stream, operands, sink, iters);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" double apb_probe_mfma_flops(int32_t n_workgroups, int32_t iters) {
  return (double)n_workgroups * kWaves * kChains * (double)iters * 32768.0;  // 2*32*32*16 per MFMA
}
