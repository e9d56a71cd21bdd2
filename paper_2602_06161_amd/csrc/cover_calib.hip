// Calibration kernel for the MFMA counters (measurement build of the library only): every wave
// issues a fixed number of v_mfma_f32_32x32x16_bf16 on four independent accumulators and
// nothing else, so the matrix pipes run near their peak and the counters it produces
// (MFMA-busy cycles, MFMA operations) give the scale against which the attention kernel's
// readings are read.  One output float per thread keeps the results live.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256, 1) void cover_calib_mfma_kernel(float* out, int iters, float x) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(x * (float)(threadIdx.x + i));
    b[i] = (__bf16)(x - (float)i);
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

// grid workgroups of 256 threads, each wave 4 * iters MFMAs of 32x32x16 (32768 flops each);
// out holds grid * 256 floats.  Returns the launch status.
extern "C" int cover_calib_mfma(float* out, int grid, int iters, hipStream_t stream) {
  if (!out || grid < 1 || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(cover_calib_mfma_kernel, dim3((unsigned)grid), dim3(256), 0, stream, out, iters,
                     0.001f);
  return (int)hipGetLastError();
}
