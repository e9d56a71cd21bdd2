// COVER stability-aware seed selection with an adaptive revision rate on gfx950
// (arXiv 2602.06161, Sec. 5.3).
//
// One workgroup per batch row.  Per region position j (flags bit 0 = unmasked, bit 1 =
// excluded):
//   score s_j  = (-logp_j) (1 + d_in_j) / (1 + d_out_j)       in IEEE fp64, this association
//   mean       = canonical stride-halving tree sum over U_t (region zero-padded to a power of
//                two) divided by |U_t|
//   budget k   = least k with k*k >= #{j in U_t : s_j > mean}  (= ceil(sqrt(n_t pi_t)))
//   seeds      = the k best eligible positions by (score desc, position asc), emitted ascending
// Every floating-point step is a single IEEE operation in a fixed order (no contraction, see
// the pragma below), so the result is bit-identical to any other implementation that follows
// the same order -- which is what makes the selection reproducible across devices.
//
// Regions of up to 1024 positions run on one wave (scores in registers, DPP reductions, no
// barriers); larger regions use one workgroup of up to 1024 threads with the tree in LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

#pragma clang fp contract(off)

namespace cover {
namespace {

constexpr int kMaxThreads = 1024;
constexpr int kMaxPer = COVER_MAX_LR / kMaxThreads;  // register-resident scores per thread
constexpr int kMaxWinners = 128;                     // ceil(sqrt(COVER_MAX_LR))
static_assert(kMaxWinners * kMaxWinners >= COVER_MAX_LR, "winner list too small");

struct SelParams {
  const float* logp;
  const float* d_in;
  const float* d_out;
  const uint8_t* flags;
  int32_t* seed_idx;
  int32_t* n_seed;
  double* score;
  int Lr, P, per, max_seeds, pos_offset;
};

// (score desc, position asc); position < 0 marks "no candidate"
__device__ __forceinline__ bool better(double sa, int ja, double sb, int jb) {
  if (ja < 0) return false;
  if (jb < 0) return true;
  return sa > sb || (sa == sb && ja < jb);
}

__device__ __forceinline__ int ceil_isqrt(int c) {
  int r = (int)sqrt((double)c);
  while (r * r < c) ++r;
  while (r > 0 && (r - 1) * (r - 1) >= c) --r;
  return r;
}

__global__ __launch_bounds__(kMaxThreads) void cover_select_kernel(const SelParams p) {
  extern __shared__ double tree[];  // P doubles
  __shared__ int cnt[3];
  __shared__ double red_s[kMaxThreads / 64];
  __shared__ int red_j[kMaxThreads / 64];
  __shared__ int winners[kMaxWinners];
  __shared__ int win_now;

  const int b = blockIdx.x, tid = threadIdx.x, nth = blockDim.x;
  const int lane = tid & 63, wv = tid >> 6, nwv = nth >> 6;
  const int64_t base = (int64_t)b * p.Lr;
  if (tid < 3) cnt[tid] = 0;
  __syncthreads();

  // scores (positions tid + m * nth)
  double sc[kMaxPer];
  uint32_t emask = 0, umask = 0;
  int nu = 0, ne = 0;
#pragma unroll
  for (int m = 0; m < kMaxPer; ++m) {
    sc[m] = 0.0;
    if (m < p.per) {
      const int j = tid + m * nth;
      if (j < p.Lr) {
        const uint8_t f = p.flags[base + j];
        if (f & 1u) {
          const double u = -(double)p.logp[base + j];
          const double num = u * (1.0 + (double)p.d_in[base + j]);
          sc[m] = num / (1.0 + (double)p.d_out[base + j]);
          umask |= 1u << m;
          ++nu;
          if (!(f & 2u)) {
            emask |= 1u << m;
            ++ne;
          }
        }
        if (p.score) p.score[base + j] = sc[m];
      }
      if (j < p.P) tree[j] = sc[m];
    }
  }
  if (nu) atomicAdd(&cnt[0], nu);
  if (ne) atomicAdd(&cnt[1], ne);
  __syncthreads();

  // canonical tree: a[i] += a[i + stride] for stride = P/2, P/4, ..., 1
  for (int stride = p.P >> 1; stride >= 1; stride >>= 1) {
    for (int i = tid; i < stride; i += nth) tree[i] = tree[i] + tree[i + stride];
    __syncthreads();
  }
  const int n = cnt[0];
  int c = 0;
  if (n > 0) {
    const double mean = tree[0] / (double)n;
#pragma unroll
    for (int m = 0; m < kMaxPer; ++m)
      if (((umask >> m) & 1u) && sc[m] > mean) ++c;
  }
  if (c) atomicAdd(&cnt[2], c);
  __syncthreads();
  int k = ceil_isqrt(cnt[2]);
  k = min(k, cnt[1]);
  k = min(k, p.max_seeds);

  for (int t = 0; t < k; ++t) {
    double bs = 0.0;
    int bj = -1;
#pragma unroll
    for (int m = 0; m < kMaxPer; ++m) {
      if ((emask >> m) & 1u) {
        const int j = tid + m * nth;
        if (better(sc[m], j, bs, bj)) { bs = sc[m]; bj = j; }
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const double os = __shfl_xor(bs, off);
      const int oj = __shfl_xor(bj, off);
      if (better(os, oj, bs, bj)) { bs = os; bj = oj; }
    }
    if (lane == 0) { red_s[wv] = bs; red_j[wv] = bj; }
    __syncthreads();
    if (tid == 0) {
      double s0 = red_s[0];
      int j0 = red_j[0];
      for (int w = 1; w < nwv; ++w)
        if (better(red_s[w], red_j[w], s0, j0)) { s0 = red_s[w]; j0 = red_j[w]; }
      winners[t] = j0;
      win_now = j0;
    }
    __syncthreads();
    const int w = win_now;
    if (w >= 0 && w % nth == tid) emask &= ~(1u << (w / nth));
  }
  __syncthreads();

  int32_t* out = p.seed_idx + (int64_t)b * p.max_seeds;
  if (tid < k) {
    const int w = winners[tid];
    int rank = 0;
    for (int u = 0; u < k; ++u) rank += winners[u] < w;
    out[rank] = w + p.pos_offset;
  }
  for (int t = k + tid; t < p.max_seeds; t += nth) out[t] = -1;
  if (tid == 0) p.n_seed[b] = k;
}

// ---------------------------------------------------------------------------------------
// Single-wave variant for regions of up to 1024 positions (the paper's generation lengths
// are 256 and 512): no barriers and no LDS.  Lane l holds positions l + 64 m, m < E.  The
// tree, the counts and the ordering are the same operations as above, so the results are
// the same bits.  E is a template argument so that every per-lane loop is fully unrolled
// to its real length, and all global loads are issued before the first one is consumed
// (the kernel is latency bound: one wave, a few hundred positions).
// ---------------------------------------------------------------------------------------
constexpr int kWaveMaxPer = 16;  // 64 lanes x 16 = 1024 positions

// DPP full-wave reductions (result valid in lane 63): quad xor 1 and 2, half-row and row
// mirrors, then row broadcasts 15 and 31.
template <int CTRL, int RMASK>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)u, (int)(uint32_t)u, CTRL, RMASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(u >> 32), (int)(uint32_t)(u >> 32), CTRL, RMASK, 0xF, false);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
// max over the wave of fp64 values (no NaN): result in lane 63
__device__ __forceinline__ double wave_max_f64(double x) {
  x = fmax(x, dpp_f64<0xB1, 0xF>(x));
  x = fmax(x, dpp_f64<0x4E, 0xF>(x));
  x = fmax(x, dpp_f64<0x141, 0xF>(x));
  x = fmax(x, dpp_f64<0x140, 0xF>(x));
  x = fmax(x, dpp_f64<0x142, 0xA>(x));
  x = fmax(x, dpp_f64<0x143, 0xC>(x));
  return x;
}
__device__ __forceinline__ double lane63_f64(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)u, 63);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double first_lane_f64(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((int)(uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((int)(uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int E>
__global__ __launch_bounds__(64) void cover_select_wave_kernel(const SelParams p) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int64_t base = (int64_t)b * p.Lr;

  // 1. loads: every lane loads all of its E positions (clamped into the row, masked below)
  //    before any value is used, so the wave waits for one memory round trip, not E.
  //    An empty region (Lr == 0, input pointers may be null) loads nothing.
  uint32_t f[E] = {};
  float lp[E] = {}, di[E] = {}, dq[E] = {};
  if (p.Lr > 0) {
#pragma unroll
    for (int m = 0; m < E; ++m) {
      const int j = min(lane + 64 * m, p.Lr - 1);
      f[m] = p.flags[base + j];
      lp[m] = p.logp[base + j];
      di[m] = p.d_in[base + j];
      dq[m] = p.d_out[base + j];
    }
  }
  // 2. scores on U_t, and the masks of U_t and of the eligible positions
  double sc[E];
  uint32_t umask = 0, emask = 0;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const bool in = lane + 64 * m < p.Lr;
    const bool u = in && (f[m] & 1u);
    const double num = -(double)lp[m] * (1.0 + (double)di[m]);
    const double s = num / (1.0 + (double)dq[m]);
    sc[m] = u ? s : 0.0;
    umask |= (uint32_t)u << m;
    emask |= (uint32_t)(u && !(f[m] & 2u)) << m;
  }
  if (p.score) {
#pragma unroll
    for (int m = 0; m < E; ++m)
      if (lane + 64 * m < p.Lr) p.score[base + lane + 64 * m] = sc[m];
  }
  int n = 0, n_elig = 0;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    n += __builtin_popcountll(__builtin_amdgcn_ballot_w64((umask >> m) & 1u));
    n_elig += __builtin_popcountll(__builtin_amdgcn_ballot_w64((emask >> m) & 1u));
  }
  // 3. canonical tree over P positions: strides of 64 and more stay inside a lane (position
  //    lane + 64 m pairs with lane + 64 (m + half)), the last six halvings cross lanes.
  double a[E];
#pragma unroll
  for (int m = 0; m < E; ++m) a[m] = sc[m];
#pragma unroll
  for (int half = E / 2; half >= 1; half >>= 1)
#pragma unroll
    for (int m = 0; m < half; ++m) a[m] = a[m] + a[m + half];
  double acc = a[0];
  for (int stride = (p.P < 64 ? p.P : 64) >> 1; stride >= 1; stride >>= 1) {
    const double o = __shfl_down(acc, stride);
    acc = acc + o;  // lanes >= stride compute values that are never used
  }
  const double total = first_lane_f64(acc);
  // 4. budget: c = #{ s_j > mean } over U_t, k = ceil(sqrt(c)), clamped
  int c = 0;
  if (n > 0) {
    const double mean = total / (double)n;
#pragma unroll
    for (int m = 0; m < E; ++m)
      c += __builtin_popcountll(__builtin_amdgcn_ballot_w64(((umask >> m) & 1u) && sc[m] > mean));
  }
  int k = ceil_isqrt(c);
  k = min(k, n_elig);
  k = min(k, p.max_seeds);

  // 5. top-k by (score desc, position asc).  Each lane keeps its own best remaining slot bm
  //    (the smallest m among equal scores, i.e. the smallest position); per round the wave
  //    takes the largest score, then the smallest (m, lane) holding it, and only the winning
  //    lane rescans.
  double bs = 0.0;
  int bm = -1;
  auto rescan = [&]() {
    bm = -1;
#pragma unroll
    for (int m = 0; m < E; ++m)
      if (((emask >> m) & 1u) && (bm < 0 || sc[m] > bs)) { bs = sc[m]; bm = m; }
  };
  rescan();
  int mine = 0x7fffffff;  // lane t keeps the t-th winner (k <= 32 < 64)
  for (int t = 0; t < k; ++t) {
    const double gmax = lane63_f64(wave_max_f64(bm >= 0 ? bs : -INFINITY));
    const bool cand = bm >= 0 && bs == gmax;
    int wm = 0;
    uint64_t wmask = 0;
#pragma unroll
    for (int m = 0; m < E; ++m) {
      if (wmask == 0) {
        wmask = __builtin_amdgcn_ballot_w64(cand && bm == m);
        wm = m;
      }
    }
    const int wl = (int)__builtin_ctzll(wmask);
    if (lane == wl) {
      emask &= ~(1u << wm);
      rescan();
    }
    if (lane == t) mine = wl + 64 * wm;
  }
  int32_t* out = p.seed_idx + (int64_t)b * p.max_seeds;
  if (lane < k) {
    int rank = 0;
    for (int u = 0; u < k; ++u) rank += __builtin_amdgcn_readlane(mine, u) < mine;
    out[rank] = mine + p.pos_offset;
  }
  for (int t = k + lane; t < p.max_seeds; t += 64) out[t] = -1;
  if (lane == 0) p.n_seed[b] = k;
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  SelParams p;
  p.logp = a.logp;
  p.d_in = a.d_in;
  p.d_out = a.d_out;
  p.flags = a.flags;
  p.seed_idx = a.seed_idx;
  p.n_seed = a.n_seed;
  p.score = a.score;
  p.Lr = a.Lr;
  p.max_seeds = a.max_seeds;
  p.pos_offset = a.pos_offset;
  int P = 1;
  while (P < a.Lr) P <<= 1;
  p.P = P;
  if (P <= 64 * kWaveMaxPer) {
    p.per = P > 64 ? P / 64 : 1;
    const dim3 grid((unsigned)a.B), block(64);
    switch (p.per) {
      case 1: hipLaunchKernelGGL(cover_select_wave_kernel<1>, grid, block, 0, stream, p); break;
      case 2: hipLaunchKernelGGL(cover_select_wave_kernel<2>, grid, block, 0, stream, p); break;
      case 4: hipLaunchKernelGGL(cover_select_wave_kernel<4>, grid, block, 0, stream, p); break;
      case 8: hipLaunchKernelGGL(cover_select_wave_kernel<8>, grid, block, 0, stream, p); break;
      default: hipLaunchKernelGGL(cover_select_wave_kernel<16>, grid, block, 0, stream, p); break;
    }
    return hipGetLastError();
  }
  int nth = P < 64 ? 64 : (P > kMaxThreads ? kMaxThreads : P);
  p.per = (P + nth - 1) / nth;
  const size_t lds = (size_t)P * sizeof(double);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)cover_select_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       COVER_MAX_LR * (int)sizeof(double));
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(cover_select_kernel, dim3((unsigned)a.B), dim3(nth), lds, stream, p);
  return hipGetLastError();
}

}  // namespace cover
