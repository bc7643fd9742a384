// Reduction of the communication-avoiding layer copies (Listing 1's final
// add-reduce over K_layers, Section II.D): C[i][j] = W[0][i][j] + ... +
// W[c-1][i][j], summed in fp32 in ascending layer order (fixed, so the result
// is reproducible), then stored as fp32 or bf16 (round to nearest even).
//
// A streaming, HBM-bound kernel: each thread owns 4 consecutive columns of one
// row and reads them from every layer with 128-bit loads; grid-stride loop.
#include "sfc_params.h"

namespace sfc {

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <bool OUT_BF16, bool VEC>
__global__ __launch_bounds__(256) void sfc_reduce_kernel(const float* __restrict__ W, int layers,
                                                         int64_t M, int64_t N, void* C,
                                                         int64_t ldc) {
  const int64_t layer_stride = M * N;
  if (VEC) {
    // N % 4 == 0: groups of 4 never straddle a row.
    const int64_t groups = layer_stride / 4;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < groups;
         g += (int64_t)gridDim.x * blockDim.x) {
      const int64_t idx = g * 4;
      f32x4 s = *reinterpret_cast<const f32x4*>(W + idx);
      for (int l = 1; l < layers; ++l) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(W + (int64_t)l * layer_stride + idx);
        s[0] += v[0]; s[1] += v[1]; s[2] += v[2]; s[3] += v[3];
      }
      const int64_t row = idx / N, col = idx - row * N;
      if (OUT_BF16) {
        __bf16* c = reinterpret_cast<__bf16*>(C) + row * ldc + col;
        c[0] = (__bf16)s[0]; c[1] = (__bf16)s[1]; c[2] = (__bf16)s[2]; c[3] = (__bf16)s[3];
      } else {
        float* c = reinterpret_cast<float*>(C) + row * ldc + col;
        c[0] = s[0]; c[1] = s[1]; c[2] = s[2]; c[3] = s[3];
      }
    }
  } else {
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < layer_stride;
         idx += (int64_t)gridDim.x * blockDim.x) {
      float s = W[idx];
      for (int l = 1; l < layers; ++l) s += W[(int64_t)l * layer_stride + idx];
      const int64_t row = idx / N, col = idx - row * N;
      if (OUT_BF16) reinterpret_cast<__bf16*>(C)[row * ldc + col] = (__bf16)s;
      else reinterpret_cast<float*>(C)[row * ldc + col] = s;
    }
  }
}

__global__ __launch_bounds__(256) void sfc_fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(sfc_fill_i32_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, n, v);
  return hipGetLastError();
}

hipError_t launch_reduce(const float* W, int layers, int64_t M, int64_t N, void* C, int64_t ldc,
                         bool out_bf16, hipStream_t stream) {
  const int64_t total = M * N;
  if (total == 0) return hipSuccess;
  const bool vec = (N % 4) == 0;
  const int64_t work = vec ? total / 4 : total;
  int64_t blocks = (work + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  const dim3 g((unsigned)blocks), b(256);
  if (out_bf16) {
    if (vec) hipLaunchKernelGGL((sfc_reduce_kernel<true, true>), g, b, 0, stream, W, layers, M, N, C, ldc);
    else hipLaunchKernelGGL((sfc_reduce_kernel<true, false>), g, b, 0, stream, W, layers, M, N, C, ldc);
  } else {
    if (vec) hipLaunchKernelGGL((sfc_reduce_kernel<false, true>), g, b, 0, stream, W, layers, M, N, C, ldc);
    else hipLaunchKernelGGL((sfc_reduce_kernel<false, false>), g, b, 0, stream, W, layers, M, N, C, ldc);
  }
  return hipGetLastError();
}

}  // namespace sfc
