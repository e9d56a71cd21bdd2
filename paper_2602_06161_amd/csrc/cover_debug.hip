// Checks of the device-data contracts, enabled per call by the environment variable
// COVER_DEBUG=1: small kernels enqueued ahead of the checked kernel on the same stream.  Each
// violation sets a bit of one device status word (per GPU), which cover_debug_status reads
// back.  The checked kernels themselves are unchanged: they tolerate every violation listed
// here without out-of-bounds accesses (bad values only give unspecified results).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

__device__ int32_t g_debug_status;

// One workgroup per batch row: the seed count against [0, max_seeds], every listed position
// against [0, L), and repeats through a bitmap of the sequence in LDS.
__global__ __launch_bounds__(256) void check_seeds_kernel(const int32_t* seed_idx, const int32_t* n_seed,
                                                          int max_seeds, int L) {
  __shared__ uint32_t seen[COVER_MAX_L / 32];
  const int b = blockIdx.x;
  for (int w = threadIdx.x; w < (L + 31) / 32; w += blockDim.x) seen[w] = 0u;
  __syncthreads();
  const int n = n_seed[b];
  int bits = 0;
  if (n < 0 || n > max_seeds) bits |= COVER_DEBUG_SEED_COUNT;
  const int nn = n < 0 ? 0 : (n > max_seeds ? max_seeds : n);
  for (int t = threadIdx.x; t < nn; t += blockDim.x) {
    const int j = seed_idx[(int64_t)b * max_seeds + t];
    if (j < 0 || j >= L) {
      bits |= COVER_DEBUG_SEED_RANGE;
      continue;
    }
    const uint32_t m = 1u << (j & 31);
    if (atomicOr(&seen[j >> 5], m) & m) bits |= COVER_DEBUG_SEED_DUPLICATE;
  }
  if (bits) atomicOr(&g_debug_status, bits);
}

// Selection inputs on U_t (flags bit 0): finite, and d_in, d_out >= 0.
__global__ __launch_bounds__(256) void check_select_kernel(const float* logp, const float* d_in,
                                                           const float* d_out, const uint8_t* flags,
                                                           int64_t n) {
  int bits = 0;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    if (!(flags[e] & 1u)) continue;
    const float a = logp[e], x = d_in[e], y = d_out[e];
    if (!__builtin_isfinite(a) || !__builtin_isfinite(x) || !__builtin_isfinite(y))
      bits |= COVER_DEBUG_SELECT_NONFINITE;
    if (x < 0.0f || y < 0.0f) bits |= COVER_DEBUG_SELECT_NEGATIVE;
  }
  if (bits) atomicOr(&g_debug_status, bits);
}

}  // namespace

bool debug_enabled() {
  const char* e = getenv("COVER_DEBUG");
  return e != nullptr && e[0] == '1' && e[1] == '\0';
}

hipError_t launch_check_seeds(const int32_t* seed_idx, const int32_t* n_seed, int B, int max_seeds,
                              int L, hipStream_t stream) {
  if (B <= 0 || max_seeds <= 0) return hipSuccess;
  hipLaunchKernelGGL(check_seeds_kernel, dim3((unsigned)B), dim3(256), 0, stream, seed_idx, n_seed,
                     max_seeds, L);
  return hipGetLastError();
}

hipError_t launch_check_select(const float* logp, const float* d_in, const float* d_out,
                               const uint8_t* flags, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(check_select_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)), dim3(256), 0,
                     stream, logp, d_in, d_out, flags, n);
  return hipGetLastError();
}

hipError_t debug_status(int32_t* status, bool clear, hipStream_t stream) {
  hipError_t e = hipMemcpyFromSymbolAsync(status, HIP_SYMBOL(g_debug_status), sizeof(int32_t), 0,
                                          hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess && clear) {
    static const int32_t zero = 0;
    e = hipMemcpyToSymbolAsync(HIP_SYMBOL(g_debug_status), &zero, sizeof(int32_t), 0,
                               hipMemcpyHostToDevice, stream);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  return e;
}

}  // namespace cover
