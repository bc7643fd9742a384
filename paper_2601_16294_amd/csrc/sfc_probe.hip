// MFMA throughput probe: the GPU counterpart of the compute micro-benchmark the
// paper uses to set its roofline's gamma (Section III.B, Eq. 1-4).
//
// Every wave of 256 workgroups x 4 waves holds 8 A and 8 B operand fragments in
// registers and runs `iters` rounds of the 64 MFMA 16x16x32 bf16 products (the
// GEMM kernel's instruction) a 128x128 wave tile needs per 32-deep step
// (acc[i][j] += B_j * A_i), with no memory traffic.  With random operands the bits seen by the matrix cores
// change from one MFMA to the next as they do in the GEMM; with constant
// operands they do not.  Wave 0 of every workgroup samples the shader clock
// (s_memtime) against the 100 MHz constant clock (s_memrealtime).
#include "sfc_params.h"

namespace sfc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float hash_unit(uint32_t x) {
  x ^= x >> 16; x *= 0x7feb352du; x ^= x >> 15; x *= 0x846ca68bu; x ^= x >> 16;
  return (float)(x & 0xFFFFFF) * (2.0f / 16777216.0f) - 1.0f;    // [-1, 1)
}

__global__ __launch_bounds__(256, 1) void mfma_probe_kernel(int random_operands, int iters, float* out) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  bf16x8 a[8], b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t key = ((blockIdx.x * 4 + wave) * 64 + lane) * 64 + i * 8 + e;
      a[i][e] = (__bf16)(random_operands ? hash_unit(key * 2 + 1) : 0.25f);
      b[i][e] = (__bf16)(random_operands ? hash_unit(key * 2 + 2) : 0.5f);
    }
  f32x4 acc[8][8] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += acc[i][j][e];
  out[blockIdx.x * 256 + threadIdx.x] = s;    // keeps the products live
  const uint64_t c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  if (threadIdx.x == 0)
    out[256 * 256 + blockIdx.x] = (float)((double)(c1 - c0) / (double)(r1 - r0) * 100.0);   // MHz
}

hipError_t run_mfma_probe(int random_operands, int iters, float* dev_out, double* ms) {
  hipEvent_t e0, e1;
  hipError_t err = hipEventCreate(&e0);
  if (err != hipSuccess) return err;
  err = hipEventCreate(&e1);
  if (err != hipSuccess) { (void)hipEventDestroy(e0); return err; }
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(256), dim3(256), 0, nullptr, random_operands, 16, dev_out);
  err = hipGetLastError();
  if (err == hipSuccess) err = hipEventRecord(e0, nullptr);
  if (err == hipSuccess) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(256), dim3(256), 0, nullptr, random_operands, iters, dev_out);
    err = hipGetLastError();
  }
  if (err == hipSuccess) err = hipEventRecord(e1, nullptr);
  if (err == hipSuccess) err = hipEventSynchronize(e1);
  float f = 0.f;
  if (err == hipSuccess) err = hipEventElapsedTime(&f, e0, e1);
  *ms = f;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return err;
}

}  // namespace sfc
