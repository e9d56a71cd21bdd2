// Temperature sampling of the draft tokens on gfx950 (the stochastic decoding the paper tests
// in its appendix on robustness, T in {0.1, 0.2, 0.3}).
//
// Per row of logits x (one workgroup of 1024 threads per row, one pass over the row):
//   token = argmax_v (x_v / T + g_v),  g_v = -ln(-ln u_v)   (Gumbel-max: token ~ softmax(x/T))
//   p     = softmax(x / T) at the token (the confidence the drafting threshold compares)
// u_v is word v % 4 of Philox4x32-10 (Salmon et al., SC 2011) at counter (v / 4, row, step, 0)
// and key (seed mod 2^32, seed / 2^32), mapped to ((w >> 9) + 1/2) 2^-23, so every (row,
// token, step) has its own fixed random number whatever the launch shape.  The argmax is
// taken as the equivalent exponential race (below).  Each thread keeps its best token (with
// its logit) and an online (max, sum of exp) of x/T; the workgroup merges them (ties: smaller
// index).  HBM-bound in principle (one read of the logits); in practice bound by the vector
// ALU: per 4 tokens ten Philox rounds of two 32x32 -> 64-bit products (one v_mad_u64_u32
// each) and their mixing, per token one logarithm and one exponential.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 gu32x4;

constexpr int kThreads = 1024;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;

struct SampleParams {
  const char* logits;
  int32_t* token;
  float* prob;
  int64_t row_stride_bytes;
  int V, bf16;
  float inv_t;  // 1 / T
  uint32_t k0, k1, step;
};

// Philox4x32-10: ten rounds; each multiplies counter words 0 and 2 by the two round
// constants and mixes the 64-bit products' halves with words 1 and 3 and the key, which is
// advanced by the Weyl constants between rounds.
__device__ __forceinline__ u32x4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                        uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return u32x4{c0, c1, c2, c3};
}

// The Gumbel-max draw argmax_v (z_v - ln(-ln u_v)), z = x / T, as an exponential race:
// with e_v = exp(z_v - m) (any common m) and E_v = -log2 u_v (ln 2 times an Exp(1) variable),
// it is argmax_v e_v / E_v, compared by cross-multiplication; e_v is also the term of the
// softmax sum, so a token costs one logarithm and one exponential.
__device__ __forceinline__ float race_e(uint32_t w) {  // -log2 u > 0
  const float u = __builtin_fmaf((float)(w >> 9), 1.1920928955078125e-7f, 5.9604644775390625e-8f);  // ((w >> 9) + 1/2) 2^-23
  return -__builtin_amdgcn_logf(u);
}

struct Acc {
  float be;  // e of the best token so far (relative to m)
  float bE;  // its E
  int i;     // its index
  float z;   // its x / T
  float m;   // max of x / T
  float s;   // sum of exp(x / T - m)
};

// tokens reach a thread in increasing order: a tie keeps the earlier (smaller) index
__device__ __forceinline__ void add(Acc& a, float z, float E, int v) {
  if (z > a.m) {
    const float r = __builtin_amdgcn_exp2f((a.m - z) * kLog2e);
    a.s *= r;
    a.be *= r;
    a.m = z;
  }
  const float e = __builtin_amdgcn_exp2f((z - a.m) * kLog2e);
  a.s += e;
  if (e * a.bE > a.be * E) {
    a.be = e;
    a.bE = E;
    a.i = v;
    a.z = z;
  }
}

__device__ __forceinline__ Acc merge(Acc a, Acc b) {
  const float m = fmaxf(a.m, b.m);
  const float ra = a.m == m ? 1.0f : __builtin_amdgcn_exp2f((a.m - m) * kLog2e);
  const float rb = b.m == m ? 1.0f : __builtin_amdgcn_exp2f((b.m - m) * kLog2e);
  a.s = a.s * ra + b.s * rb;
  a.be *= ra;
  b.be *= rb;
  a.m = m;
  const float l = b.be * a.bE, rgt = a.be * b.bE;  // b better: b.be / b.bE > a.be / a.bE
  if (l > rgt || (l == rgt && b.i < a.i)) {
    a.be = b.be;
    a.bE = b.bE;
    a.i = b.i;
    a.z = b.z;
  }
  return a;
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__global__ __launch_bounds__(kThreads) void cover_token_sample_kernel(const SampleParams p) {
  __shared__ Acc red[kThreads / 64];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const char* row = p.logits + (int64_t)r * p.row_stride_bytes;
  const int per = p.bf16 ? 8 : 4;  // elements per 16-byte chunk
  const int nfull = p.V / per;
  Acc acc = {0.0f, 1.0f, 0x7fffffff, 0.0f, -INFINITY, 0.0f};
  for (int c = tid; c < nfull; c += kThreads) {
    const u32x4 raw = *(gu32x4*)((__attribute__((address_space(1))) const char*)row + (int64_t)c * 16);
    if (p.bf16) {
      const u32x4 w0 = philox(2u * c, r, p.step, 0u, p.k0, p.k1);
      const u32x4 w1 = philox(2u * c + 1u, r, p.step, 0u, p.k0, p.k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 8 * c + 2 * e;
        add(acc, bf_lo(raw[e]) * p.inv_t, race_e(e < 2 ? w0[2 * e] : w1[2 * e - 4]), v);
        add(acc, bf_hi(raw[e]) * p.inv_t, race_e(e < 2 ? w0[2 * e + 1] : w1[2 * e - 3]), v + 1);
      }
    } else {
      const u32x4 w = philox((uint32_t)c, r, p.step, 0u, p.k0, p.k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) add(acc, __uint_as_float(raw[e]) * p.inv_t, race_e(w[e]), 4 * c + e);
    }
  }
  // the tail: one element per thread, read at its own width
  if (tid < p.V - nfull * per) {
    const int v = nfull * per + tid;
    const float x = p.bf16 ? __uint_as_float((uint32_t)((const uint16_t*)row)[v] << 16) : ((const float*)row)[v];
    const u32x4 w = philox((uint32_t)(v >> 2), r, p.step, 0u, p.k0, p.k1);
    add(acc, x * p.inv_t, race_e(w[v & 3]), v);
  }
  // merge: across the wave, then the waves
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    Acc b;
    b.be = __shfl_xor(acc.be, o);
    b.bE = __shfl_xor(acc.bE, o);
    b.i = __shfl_xor(acc.i, o);
    b.z = __shfl_xor(acc.z, o);
    b.m = __shfl_xor(acc.m, o);
    b.s = __shfl_xor(acc.s, o);
    acc = merge(acc, b);
  }
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  if (tid == 0) {
    Acc a = red[0];
    for (int w = 1; w < kThreads / 64; ++w) a = merge(a, red[w]);
    p.token[r] = a.i;
    if (p.prob) p.prob[r] = __builtin_amdgcn_exp2f((a.z - a.m) * kLog2e) / a.s;
  }
}

}  // namespace

hipError_t launch_token_sample(const SampleArgs& a, hipStream_t stream) {
  SampleParams p;
  p.logits = (const char*)a.logits;
  p.token = a.token;
  p.prob = a.prob;
  p.row_stride_bytes = a.row_stride * (a.bf16 ? 2 : 4);
  p.V = a.V;
  p.bf16 = a.bf16;
  p.inv_t = 1.0f / a.temperature;
  p.k0 = (uint32_t)(a.seed & 0xffffffffu);
  p.k1 = (uint32_t)(a.seed >> 32);
  p.step = a.step;
  hipLaunchKernelGGL(cover_token_sample_kernel, dim3((unsigned)a.R), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
