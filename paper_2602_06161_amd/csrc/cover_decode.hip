// COVER decoding-state update of one step on gfx950 (arXiv 2602.06161, Sec. 5.2 drafting and
// revision, Sec. 3 state update, Sec. 5.3 ReMask budget and exclusion flags).
//
// One workgroup per batch row, every region position owned by one thread (positions
// tid + m * nthreads, m < per), so all reads and writes are coalesced and the per-position
// work needs no synchronisation.  The steps:
//   1. the previous seeds become a bitmap of the region in LDS (entries outside the region are
//      dropped, repeats collapse; a bit at a masked position is ignored in step 4), loaded
//      while the tokens and confidences are in flight;
//   2. the draft candidates (masked, confidence > tau in fp32) get a 64-bit key: the
//      confidence mapped to an order-preserving unsigned integer in the high half, the
//      bitwise complement of the position in the low half.  Keys are distinct and their
//      order is (confidence descending, position ascending);
//      With min_draft > 0 and fewer candidates than that, every masked position with a
//      confidence becomes a candidate and min_draft of them are drafted instead;
//   3. if more candidates qualify than the cap allows, the cap-th largest key is found by a
//      most-significant-digit radix select (8-bit digits, LDS histogram, one wave scans the
//      256 bins), which stops at the first digit whose bucket is taken whole; the drafts are
//      the keys at or above the prefix found;
//   4. per position: drafting, revision of the seeds, ReMask counters, the next selection's
//      flags, flip-flop events (Sec. 4: a drafted token equal to the position's previous
//      unmasked token) when the caller tracks that token, and the row's counts reduced
//      through LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

constexpr int kMaxThreads = 1024;
constexpr int kMaxPer = COVER_MAX_LR / kMaxThreads;

struct UpdParams {
  int32_t* tokens;
  const int32_t* argmax;
  const float* conf;
  const int32_t* seed_idx;
  const int32_t* n_seed;
  int32_t* remask_count;
  uint8_t* flags;
  uint8_t* drafted;
  int32_t* counts;
  int32_t* last_unmask;
  int32_t* flipflops;
  int Lr, per, max_seeds, pos_offset, mask_id, cap, budget, min_draft;
  float tau;
};

// fp32 -> unsigned integer with the same order over all non-NaN values (-0 taken as +0)
__device__ __forceinline__ uint32_t ordered(float c) {
  uint32_t u = __float_as_uint(c);
  if (c == 0.0f) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// PER: positions per thread the register arrays hold (p.per <= PER).  With PER <= 4 the
// argmax and the counters are requested together with the tokens (one round trip fewer).
template <int PER>
__global__ __launch_bounds__(kMaxThreads) void cover_update_kernel(const UpdParams p) {
  constexpr bool kEarly = PER <= 4;
  __shared__ uint32_t seedbits[COVER_MAX_LR / 32];
  __shared__ uint32_t hist[256];
  // candidates, |D|, kept, replaced, remasked, masked after, flip-flops, forced candidates
  __shared__ int sums[8];
  __shared__ uint64_t s_prefix;
  __shared__ int s_need, s_done, s_shift;

  const int b = blockIdx.x, tid = threadIdx.x, nth = blockDim.x, lane = tid & 63;
  const int64_t base = (int64_t)b * p.Lr;
  for (int w = tid; w < (p.Lr + 31) / 32; w += nth) seedbits[w] = 0u;
  if (tid < 8) sums[tid] = 0;
  __syncthreads();

  // 1. per-position inputs, and the seed bitmap
  int tok[PER], am[kEarly ? PER : 1], rc[kEarly ? PER : 1];
  float cf[PER];
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int j = tid + m * nth;
    tok[m] = 0;
    cf[m] = 0.0f;
    if (m < p.per && j < p.Lr) {
      tok[m] = p.tokens[base + j];
      cf[m] = p.conf[base + j];
      if constexpr (kEarly) {
        am[m] = p.argmax[base + j];
        rc[m] = p.remask_count[base + j];
      }
    }
  }
  int ns = p.max_seeds > 0 ? p.n_seed[b] : 0;
  ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
  for (int t = tid; t < ns; t += nth) {
    const int64_t i = (int64_t)p.seed_idx[(int64_t)b * p.max_seeds + t] - p.pos_offset;
    if (i >= 0 && i < p.Lr) atomicOr(&seedbits[i >> 5], 1u << (i & 31));
  }

  // 2. candidate keys
  uint64_t key[PER];
  uint32_t cand = 0;
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int j = tid + m * nth;
    key[m] = 0;
    if (m < p.per && j < p.Lr && tok[m] == p.mask_id && cf[m] > p.tau) {
      cand |= 1u << m;
      key[m] = ((uint64_t)ordered(cf[m]) << 32) | (uint32_t)~(uint32_t)j;
    }
  }
  const int nc = wave_sum(__builtin_popcount(cand));
  if (lane == 0 && nc) atomicAdd(&sums[0], nc);
  __syncthreads();

  int target = p.cap, total = sums[0];
  if (total < p.min_draft) {  // too few above tau: the min_draft most confident masked ones
    cand = 0;
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int j = tid + m * nth;
      key[m] = 0;
      if (m < p.per && j < p.Lr && tok[m] == p.mask_id && cf[m] == cf[m]) {
        cand |= 1u << m;
        key[m] = ((uint64_t)ordered(cf[m]) << 32) | (uint32_t)~(uint32_t)j;
      }
    }
    const int n2 = wave_sum(__builtin_popcount(cand));
    if (lane == 0 && n2) atomicAdd(&sums[7], n2);
    __syncthreads();
    target = p.min_draft;
    total = sums[7];
  }

  // 3. drafts: every candidate, or the `target` largest keys
  uint64_t keep_mask = 0, prefix = 0;  // drafted <=> candidate and (key & keep_mask) >= prefix
  bool none = target <= 0;
  if (!none && total > target) {
    if (tid == 0) {
      s_prefix = 0;
      s_need = target;  // rank, from the top, of the key still to be located
      s_done = 0;
    }
    for (int shift = 56; shift >= 0; shift -= 8) {
      for (int d = tid; d < 256; d += nth) hist[d] = 0u;
      __syncthreads();
      const uint64_t hi = shift == 56 ? 0ull : (~0ull << (shift + 8));
      const uint64_t pre = s_prefix;
#pragma unroll
      for (int m = 0; m < PER; ++m)
        if (((cand >> m) & 1u) && (key[m] & hi) == pre)
          atomicAdd(&hist[(uint32_t)(key[m] >> shift) & 255u], 1u);
      __syncthreads();
      if (tid < 64) {
        // lane l holds digits 255-4l .. 252-4l (descending); inclusive scan over the lanes
        uint32_t h[4], s = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) s += (h[q] = hist[255 - (lane * 4 + q)]);
        uint32_t incl = s;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t v = __shfl_up(incl, o);
          if (lane >= o) incl += v;
        }
        const uint32_t need = (uint32_t)s_need;
        const uint64_t hit = __ballot(incl >= need);
        if (lane == __builtin_ctzll(hit)) {
          uint32_t acc = incl - s;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (acc + h[q] >= need) {
              const uint32_t digit = 255u - (uint32_t)(lane * 4 + q);
              s_prefix = pre | ((uint64_t)digit << shift);
              s_need = (int)(need - acc);
              s_shift = shift;
              s_done = (need - acc == h[q]) ? 1 : 0;  // the whole bucket is drafted
              break;
            }
            acc += h[q];
          }
        }
      }
      __syncthreads();
      if (s_done) break;
    }
    prefix = s_prefix;
    keep_mask = ~0ull << s_shift;
  }

  // 4. per-position update
  int n_d = 0, n_keep = 0, n_rep = 0, n_rm = 0, n_masked = 0, n_ff = 0;
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int j = tid + m * nth;
    if (m < p.per && j < p.Lr) {
      const int64_t e = base + j;
      const bool dr = !none && ((cand >> m) & 1u) && (key[m] & keep_mask) >= prefix;
      // a listed seed at a masked position is no seed
      const bool seed = ((seedbits[j >> 5] >> (j & 31)) & 1u) && tok[m] != p.mask_id;
      int t = tok[m];
      int cnt;
      if constexpr (kEarly) cnt = rc[m];
      else cnt = p.remask_count[e];
      if (dr || seed) {
        int a;
        if constexpr (kEarly) a = am[m];
        else a = p.argmax[e];
        if (dr) {
          t = a;
          ++n_d;
          if (p.last_unmask) {
            n_ff += p.last_unmask[e] == a ? 1 : 0;
            p.last_unmask[e] = a;
          }
        } else if (a == t) {
          ++n_keep;
        } else if (cf[m] > p.tau) {
          t = a;
          ++n_rep;
        } else {
          t = p.mask_id;
          ++cnt;
          ++n_rm;
          p.remask_count[e] = cnt;
        }
        if (t != tok[m]) p.tokens[e] = t;
      }
      const bool unmasked = t != p.mask_id;
      n_masked += unmasked ? 0 : 1;
      if (p.flags) p.flags[e] = (uint8_t)((unmasked ? 1 : 0) | ((seed || cnt >= p.budget) ? 2 : 0));
      if (p.drafted) p.drafted[e] = dr ? 1 : 0;
    }
  }
  if (p.counts || p.flipflops) {
    const int v[6] = {n_d, n_keep, n_rep, n_rm, n_masked, n_ff};
#pragma unroll
    for (int k = 0; k < 6; ++k) {
      const int s = wave_sum(v[k]);
      if (lane == 0 && s) atomicAdd(&sums[1 + k], s);
    }
    __syncthreads();
    if (p.counts && tid < 5) p.counts[(int64_t)b * 5 + tid] = sums[1 + tid];
    if (p.flipflops && tid == 0) p.flipflops[b] = sums[6];
  }
}

}  // namespace

hipError_t launch_decode_update(const UpdateArgs& a, hipStream_t stream) {
  UpdParams p;
  p.tokens = a.tokens; p.argmax = a.argmax; p.conf = a.conf;
  p.seed_idx = a.seed_idx; p.n_seed = a.n_seed; p.remask_count = a.remask_count;
  p.flags = a.flags; p.drafted = a.drafted; p.counts = a.counts;
  p.last_unmask = a.last_unmask; p.flipflops = a.flipflops;
  p.Lr = a.Lr; p.max_seeds = a.max_seeds; p.pos_offset = a.pos_offset; p.mask_id = a.mask_id;
  p.cap = a.draft_cap; p.budget = a.remask_budget; p.tau = a.tau; p.min_draft = a.min_draft;
  int nth = ((a.Lr + 63) / 64) * 64;
  if (nth < 64) nth = 64;
  if (nth > kMaxThreads) nth = kMaxThreads;
  p.per = (a.Lr + nth - 1) / nth;
  if (p.per > kMaxPer) return hipErrorInvalidValue;
  if (p.per <= 1)
    hipLaunchKernelGGL(cover_update_kernel<1>, dim3((unsigned)a.B), dim3((unsigned)nth), 0, stream, p);
  else if (p.per <= 4)
    hipLaunchKernelGGL(cover_update_kernel<4>, dim3((unsigned)a.B), dim3((unsigned)nth), 0, stream, p);
  else
    hipLaunchKernelGGL(cover_update_kernel<kMaxPer>, dim3((unsigned)a.B), dim3((unsigned)nth), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
