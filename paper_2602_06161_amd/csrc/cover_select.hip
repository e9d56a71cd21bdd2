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

// Full-wave butterflies of 32-bit values (the result in every lane): quad xor 1 and 2,
// half-row and row mirrors (each pairs two groups of equal size), then the row and
// half-wave swaps, which return both directions of the exchange at once.
template <bool MAX>
__device__ __forceinline__ uint32_t pick(uint32_t a, uint32_t b) {
  return MAX ? (a > b ? a : b) : (a < b ? a : b);
}
template <bool MAX, int CTRL>
__device__ __forceinline__ uint32_t dpp_step(uint32_t x) {
  return pick<MAX>(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, true));
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t x) {
  x = dpp_step<MAX, 0xB1>(x);   // quad_perm [1,0,3,2]
  x = dpp_step<MAX, 0x4E>(x);   // quad_perm [2,3,0,1]
  x = dpp_step<MAX, 0x141>(x);  // row_half_mirror
  x = dpp_step<MAX, 0x140>(x);  // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = pick<MAX>(r16[0], r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return pick<MAX>(r32[0], r32[1]);
}
// Order-preserving 64-bit key of an fp64 value that is not NaN: a < b exactly when
// key(a) < key(b), and key(-0) = key(+0) (adding +0 maps -0 to +0 and leaves every other
// value unchanged).
__device__ __forceinline__ uint64_t order_key(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x + 0.0);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}
// the value of lane i + S in lane i (for the lanes i whose i + S stays in their 2S-lane group):
// S = 32 and 16 by the half-wave and row swaps, S <= 8 by a row shift
template <int S>
__device__ __forceinline__ uint32_t from_lane_plus_u32(uint32_t x) {
  if constexpr (S == 32) {
    return __builtin_amdgcn_permlane32_swap(x, x, false, false)[1];
  } else if constexpr (S == 16) {
    return __builtin_amdgcn_permlane16_swap(x, x, false, false)[1];
  } else {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x100 + S, 0xF, 0xF, false);
  }
}
template <int S>
__device__ __forceinline__ double from_lane_plus(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint32_t lo = from_lane_plus_u32<S>((uint32_t)u);
  const uint32_t hi = from_lane_plus_u32<S>((uint32_t)(u >> 32));
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
  // Cross-lane halvings: lane i adds lane i + s for s = 32, 16, ..., 1 (those below
  // min(P, 64)); lanes >= s compute values that are never used.  The partner's value comes
  // from the half-wave and row swaps (s = 32, 16) and row shifts (s <= 8), not through LDS.
  double acc = a[0];
  const int lanes = p.P < 64 ? p.P : 64;
  if (lanes > 32) acc = acc + from_lane_plus<32>(acc);
  if (lanes > 16) acc = acc + from_lane_plus<16>(acc);
  if (lanes > 8) acc = acc + from_lane_plus<8>(acc);
  if (lanes > 4) acc = acc + from_lane_plus<4>(acc);
  if (lanes > 2) acc = acc + from_lane_plus<2>(acc);
  if (lanes > 1) acc = acc + from_lane_plus<1>(acc);
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

  // 5. top-k by (score desc, position asc), on the order keys of the scores.  Each lane
  //    keeps its best remaining slot (bk, bm), the smallest m among equal keys, i.e. the
  //    smallest position.  A round takes the wave maximum of the heads' high words; in the
  //    usual case one lane holds it and wins.  Otherwise the low words decide, and between
  //    equal keys the smallest position m * 64 + lane.  The winner drops its slot and every
  //    lane rescans (only the winner's head can change).
  uint64_t key[E];
#pragma unroll
  for (int m = 0; m < E; ++m) key[m] = order_key(sc[m]);
  uint64_t bk = 0;  // no real key is 0 (it would be a NaN's)
  int bm = -1;
  auto rescan = [&]() {
    bk = 0;
    bm = -1;
#pragma unroll
    for (int m = 0; m < E; ++m) {
      const bool take = ((emask >> m) & 1u) && key[m] > bk;
      bk = take ? key[m] : bk;
      bm = take ? m : bm;
    }
  };
  rescan();
  uint32_t selm = 0;  // slots of this lane taken as seeds
  for (int t = 0; t < k; ++t) {
    // (the cross-lane reductions are statements of their own, so that every lane takes
    // part in them; a lane without a slot contributes the identity)
    const uint32_t hi = bm >= 0 ? (uint32_t)(bk >> 32) : 0u;
    const uint32_t max_hi = wave_reduce_u32<true>(hi);
    const bool top_hi = bm >= 0 && hi == max_hi;
    uint64_t wmask = __builtin_amdgcn_ballot_w64(top_hi);
    if (__builtin_popcountll(wmask) > 1) {  // uniform
      const uint32_t lo = top_hi ? (uint32_t)bk : 0u;
      const uint32_t max_lo = wave_reduce_u32<true>(lo);
      const bool top = top_hi && lo == max_lo;
      const uint32_t pos = top ? (uint32_t)(bm * 64 + lane) : 0xFFFFFFFFu;
      const uint32_t min_pos = wave_reduce_u32<false>(pos);
      wmask = __builtin_amdgcn_ballot_w64(top && pos == min_pos);
    }
    // (no winner only if the data contract is broken, e.g. a NaN score: no lane takes one)
    if (wmask != 0 && lane == (int)__builtin_ctzll(wmask)) {
      selm |= 1u << bm;
      emask &= ~(1u << bm);
    }
    rescan();
  }
  // 6. emit ascending: a taken slot's rank is the number of taken positions below it,
  //    those in lower slots plus those of lower lanes in its own slot
  int32_t* out = p.seed_idx + (int64_t)b * p.max_seeds;
  int below = 0;
#pragma unroll
  for (int m = 0; m < E; ++m) {
    const bool mine = (selm >> m) & 1u;
    const uint64_t sm = __builtin_amdgcn_ballot_w64(mine);
    const int rank = below + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(sm >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)sm, 0u));
    if (mine) out[rank] = lane + 64 * m + p.pos_offset;
    below += __builtin_popcountll(sm);
  }
  // below == k for valid inputs; the list is filled and counted from what was emitted, so
  // that no slot is left unwritten otherwise
  k = below;
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
