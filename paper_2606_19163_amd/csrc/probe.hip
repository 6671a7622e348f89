// Matrix-core throughput probe: chains of bf16 MFMAs on register operands,
// no memory traffic in the loop.  It measures the MFMA rate the GPU sustains
// (clock, issue) as the ceiling the implicit-GEMM kernels are compared with.
#include "common.hpp"
#include "kernels.hpp"
#include "pulse_stage.h"

namespace pulse {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

// keeps the operands in registers without letting the compiler fold the chain
__device__ __forceinline__ void opaque(bf16x8_t& v) { asm volatile("" : "+v"(v)); }

// 32x32x16: each wave keeps 2 x 3 independent accumulators; one iteration is
// 6 MFMAs of 32*32*16*2 FLOPs
__global__ __launch_bounds__(256) void k_mfma32(int iters, float* out) {
  const int lane = threadIdx.x & 63;
  f32x16_t acc[2][3];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 3; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  bf16x8_t a[2], b[3];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[0][e] = a[1][e] = (__bf16)(1e-3f * (lane + e));
    b[0][e] = b[1][e] = b[2][e] = (__bf16)(1e-3f * (lane - e));
  }
  for (int it = 0; it < iters; ++it) {
    opaque(a[0]);
    opaque(a[1]);
    opaque(b[0]);
    opaque(b[1]);
    opaque(b[2]);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 3; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 3; ++j) s += acc[i][j][0] + acc[i][j][15];
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// 16x16x32 (the shape of the stage GEMMs): 4 x 5 accumulators; one iteration
// is 20 MFMAs of 16*16*32*2 FLOPs
__global__ __launch_bounds__(256) void k_mfma16(int iters, float* out) {
  const int lane = threadIdx.x & 63;
  f32x4_t acc[4][5];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 5; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  bf16x8_t a[4], b[5];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i][e] = (__bf16)(1e-3f * (lane + e + i));
#pragma unroll
    for (int j = 0; j < 5; ++j) b[j][e] = (__bf16)(1e-3f * (lane - e + j));
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 4; ++i) opaque(a[i]);
#pragma unroll
    for (int j = 0; j < 5; ++j) opaque(b[j]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 5; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 5; ++j) s += acc[i][j][0] + acc[i][j][3];
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace
}  // namespace pulse

extern "C" pulse_status pulse_mfma_probe(int32_t shape, int32_t blocks, int32_t iters, float* out,
                                         double* flops, void* stream) {
  if (shape != 16 && shape != 32) return PULSE_E_INVALID_ARG;
  if (blocks < 1 || iters < 1 || !out) return PULSE_E_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (shape == 32)
    hipLaunchKernelGGL(pulse::k_mfma32, dim3(blocks), dim3(256), 0, st, iters, out);
  else
    hipLaunchKernelGGL(pulse::k_mfma16, dim3(blocks), dim3(256), 0, st, iters, out);
  if (hipGetLastError() != hipSuccess) return PULSE_E_HIP;
  if (flops) {
    const double per_iter = shape == 32 ? 6.0 * 32 * 32 * 16 * 2 : 20.0 * 16 * 16 * 32 * 2;
    *flops = per_iter * iters * 4.0 * blocks;  // 4 waves per block
  }
  return PULSE_OK;
}
