// COVER attention for a block of queries against the whole sequence (the prefix-cache
// decoding combined with COVER in Sec. 6.6: only the current block's rows are recomputed; the
// prompt's keys and values come from the caller's cache), bf16, head size 128, on gfx950.
//
// Per query row i at absolute position p = q_off + r the result is the row p of the square
// COVER attention (Sec. 5.1): keys and values of seed positions come from the cache, every
// other position's from the live tensors, and a seed row sees its own live key and value on
// its diagonal (the leave-one-out view whose closed form App. B.4 gives).
//
// With few query rows the work is bound by reading K and V, not by the MFMAs, and one
// workgroup per (row, 128-query tile) would leave most of the chip idle, so the keys are
// split.  Two forms:
//   * n_split == 1, cover_attn_tile_kernel (the default up to L = 2048): one launch, one
//     workgroup of 8 waves per 32 query rows whose waves split the keys among themselves
//     and merge in LDS (described at the kernel, below).
//   * n_split > 1, two launches through the caller's workspace:
//   kernel 1: one workgroup of 4 waves per (batch, query head, 128-query tile, key split).
//     The waves share the split's K/V in LDS, loaded in groups of up to four 32-key stages
//     (128 keys, 64 KiB) that are all requested at once, so a group costs one memory round
//     trip; wave w owns 32 queries.  The Q rows and the seed list are requested together at
//     the start.  S^T = K Q^T and O^T += V^T P^T
//     on 32x32x16 bf16 MFMAs (Q as the B operand straight from registers, V^T by transposing
//     LDS reads, P^T from the S^T registers), online softmax with the row max, row sums and
//     O^T in fp32.  A seed row's cached diagonal score is dropped where it occurs and its
//     live diagonal term is added by the split that holds the position.  Per row the split
//     leaves its normalised output O / l in bf16 (256 bytes) and its max and sum in fp32 in
//     the caller's workspace: the records are written and read once, so their size is
//     traffic on top of K and V.
//   * kernel 2: one wave per query row merges the splits and writes O and the lse.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_t;
typedef __attribute__((address_space(1))) const char gmem_t;

constexpr int kD = 128;
constexpr int kRow = 2 * kD;            // bytes per K/V row
constexpr int kStage = 32;              // keys per stage
constexpr int kGroup = 4;               // stages loaded together
constexpr int kThreads = 256;           // 4 waves
constexpr int kQT = 128;                // queries per workgroup
constexpr int kMaxWords = COVER_MAX_L / 32;
constexpr float kInit = -1.0e30f;       // finite "nothing seen yet" max
constexpr float kLn2 = 0.693147180559945309f;

struct RectParams {
  const __bf16* q;
  const __bf16* kl;
  const __bf16* vl;
  const __bf16* kc;
  const __bf16* vc;
  const int32_t* seed_idx;
  const int32_t* n_seed;
  float* ws;
  __bf16* out;
  float* lse;
  int B, Hq, Hkv, L, Lq, q_off, max_seeds, group, n_qt, n_split, split_stages;
  int n_wg, xcd_slots;  // single-launch form: workgroups, logical tiles per XCD
  float c2;  // scale * log2(e)
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

// LDS layouts: K rows with the 16-byte chunk index XOR-ed by row % 16 (a b128 operand read of
// 32 rows covers all banks); V rows with the chunk index XOR-ed by 4 (row % 4) (a transposing
// read of 8 rows x 64 bytes covers every bank twice).
__device__ __forceinline__ uint32_t k_off(int row, int c) { return row * kRow + ((c ^ (row & 15)) << 4); }
__device__ __forceinline__ uint32_t v_chunk(int row, int c) { return row * kRow + ((c ^ ((row & 3) << 2)) << 4); }
__device__ __forceinline__ uint32_t v_elem(int row, int col) { return v_chunk(row, col >> 3) + ((col & 7) << 1); }

// max / sum of x over a query row's lane pair (lanes l and l ^ 32), on the VALU: the swap
// leaves one copy of each lane's own value and one of its partner's in the two results
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ i16x4 v_tr(const lds_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
}

__global__ __launch_bounds__(kThreads, 2) void cover_attn_rect_kernel(const RectParams p) {
  __shared__ __attribute__((aligned(16))) char sK[kGroup][kStage * kRow];
  __shared__ __attribute__((aligned(16))) char sV[kGroup][kStage * kRow];
  __shared__ uint32_t bm[kMaxWords];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hl = lane >> 5;
  int id = blockIdx.x;
  const int qt = id % p.n_qt;
  id /= p.n_qt;
  const int split = id % p.n_split;
  const int bh = id / p.n_split;
  const int b = bh / p.Hq, h = bh % p.Hq, hk = h / p.group;

  // this wave's queries (requested first: nothing below depends on them until the MFMAs)
  const int qrow0 = qt * kQT + wave * 32;
  const bool active = qrow0 < p.Lq;
  const int qrow = min(qrow0 + l32, p.Lq - 1);
  const int pos = p.q_off + qrow;
  const __bf16* qp = p.q + b * p.q_sb + h * p.q_sh + (int64_t)qrow * p.q_sl;
  bf16x8 qreg[kD / 16];
#pragma unroll
  for (int ks = 0; ks < kD / 16; ++ks)
    qreg[ks] = *(const bf16x8*)(qp + (2 * ks + hl) * 8);

  // seed bitmap of the whole sequence; the count and the list are requested together
  const int nW = (p.L + 31) >> 5;
  for (int w = tid; w < nW; w += kThreads) bm[w] = 0u;
  __syncthreads();
  if (p.max_seeds > 0) {
    int ns = p.n_seed[b];
    ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
    for (int t = tid; t < p.max_seeds; t += kThreads) {
      const int j = p.seed_idx[(int64_t)b * p.max_seeds + t];
      if (t < ns && j >= 0 && j < p.L) atomicOr(&bm[j >> 5], 1u << (j & 31));
    }
  }
  __syncthreads();
  auto is_seed = [&](int j) { return (bm[j >> 5] >> (j & 31)) & 1u; };
  const bool row_seed = is_seed(pos);

  // key range of this split
  const int k_begin = split * p.split_stages * kStage;
  const int k_end = min(p.L, k_begin + p.split_stages * kStage);
  const int n_st = k_end > k_begin ? (k_end - k_begin + kStage - 1) / kStage : 0;

  // cooperative group loads: per stage 512 chunks of 16 bytes of K (and of V), two per
  // thread; every stage of a group is requested before the first is stored
  const int64_t kvbase = b * p.kv_sb + hk * p.kv_sh;
  auto load_group = [&](int st0, int n) {
    u32x4 kr[kGroup][2], vr[kGroup][2];
#pragma unroll
    for (int g = 0; g < kGroup; ++g)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = tid * 2 + u, row = c >> 4, ch = c & 15;
        const int key = k_begin + (st0 + g) * kStage + row;
        kr[g][u] = vr[g][u] = u32x4{0u, 0u, 0u, 0u};
        if (g < n && key < k_end) {
          const int64_t off = kvbase + (int64_t)key * p.kv_sl + ch * 8;
          const bool sd = is_seed(key);
          kr[g][u] = *(const u32x4*)((sd ? p.kc : p.kl) + off);
          vr[g][u] = *(const u32x4*)((sd ? p.vc : p.vl) + off);
        }
      }
#pragma unroll
    for (int g = 0; g < kGroup; ++g)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = tid * 2 + u, row = c >> 4, ch = c & 15;
        if (g < n) {
          *(u32x4*)(sK[g] + k_off(row, ch)) = kr[g][u];
          *(u32x4*)(sV[g] + v_chunk(row, ch)) = vr[g][u];
        }
      }
  };

  // V^T operand addresses: lane (G = lane / 16, i = lane % 16) reads keys
  // 16 kk + {0..3, 8..11} + 4 (G / 2) of d-block db, the key order of the S^T registers
  uint32_t vaddr[kD / 32];
  {
    const int G = lane >> 4, ii = lane & 15;
    const int row = 4 * (G >> 1) + (ii >> 2);
#pragma unroll
    for (int db = 0; db < kD / 32; ++db) vaddr[db] = v_elem(row, db * 32 + 16 * (G & 1) + 4 * (ii & 3));
  }

  f32x16 o[kD / 32];
#pragma unroll
  for (int db = 0; db < kD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m = kInit, l = 0.0f;

  // Two 32-key stages per pass (they are in the same group: groups start at multiples of
  // four stages): two independent S^T chains, one softmax over both, and every LDS operand of
  // the pass requested before its first MFMA (one LDS latency per pass).  The running max is
  // raised lazily, once some row's scores exceed it by 2^8 (weights up to 256 stay exact
  // enough in bf16 and far from fp32 overflow), so O is rarely rescaled; the first pass sets
  // it while O and the sums are still zero.
  constexpr float kLazy = 8.0f;
  for (int st = 0; st < n_st; st += 2) {
    const int buf = st % kGroup;
    if (buf == 0) {
      if (st > 0) __syncthreads();  // every wave is done with the previous group
      load_group(st, min(kGroup, n_st - st));
      __syncthreads();
    }
    const bool two = st + 1 < n_st;
    if (active) {
      bf16x8 ka[2][kD / 16], va[2][2][kD / 32];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const lds_t* kb = (const lds_t*)sK[buf + (two ? kt : 0)];
        const lds_t* vb = (const lds_t*)sV[buf + (two ? kt : 0)];
#pragma unroll
        for (int ks = 0; ks < kD / 16; ++ks)
          ka[kt][ks] = *(const __attribute__((address_space(3))) bf16x8*)(kb + k_off(l32, 2 * ks + hl));
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < kD / 32; ++db) {
            const lds_t* base = vb + vaddr[db] + kk * 16 * kRow;
            va[kt][kk][db] = __builtin_bit_cast(
                bf16x8, __builtin_shufflevector(v_tr(base), v_tr(base + 8 * kRow), 0, 1, 2, 3, 4, 5, 6, 7));
          }
      }
      f32x16 sc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[kt][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < kD / 16; ++ks)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          sc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[kt][ks], qreg[ks], sc[kt], 0, 0, 0);
      // register r of stage kt holds key k0 + 32 kt + 8 (r / 4) + 4 hl + r % 4 of row qrow
      const int k0 = k_begin + st * kStage;
      const bool edge = k0 + 2 * kStage > k_end;  // keys past the split's end (or no stage 2)
      const bool diag = row_seed && pos >= k0 && pos < k0 + 2 * kStage;
      float mx = kInit;
      if (__builtin_amdgcn_ballot_w64(diag) != 0 || edge) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * kt + 8 * (r >> 2) + 4 * hl + (r & 3);
            float t = sc[kt][r] * p.c2;
            if (key >= k_end || (diag && key == pos)) t = -INFINITY;
            sc[kt][r] = t;
            mx = __builtin_fmaxf(mx, t);
          }
      } else {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            sc[kt][r] *= p.c2;
            mx = __builtin_fmaxf(mx, sc[kt][r]);
          }
      }
      mx = pair_max(mx);
      if (st == 0) {
        m = mx;
      } else if (__builtin_amdgcn_ballot_w64(mx > m + kLazy)) {
        const float mn = __builtin_fmaxf(m, mx);
        const float alpha = __builtin_amdgcn_exp2f(m - mn);
        l *= alpha;
#pragma unroll
        for (int db = 0; db < kD / 32; ++db) o[db] *= alpha;
        m = mn;
      }
      bf16x8 pk[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pr = __builtin_amdgcn_exp2f(sc[kt][8 * kk + e] - m);
            l += pr;
            pk[kt][kk][e] = (__bf16)pr;
          }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int db = 0; db < kD / 32; ++db)
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[0][kk][db], pk[0][kk], o[db], 0, 0, 0);
      if (two) {  // (a lone last stage: its second half is all masked, and its buffer stale)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int db = 0; db < kD / 32; ++db)
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[1][kk][db], pk[1][kk], o[db], 0, 0, 0);
      }
    }
  }

  if (!active) return;
  // the live diagonal term of a seed row, in the split that holds its position
  if (row_seed && pos >= k_begin && pos < k_end) {
    const __bf16* kp = p.kl + kvbase + (int64_t)pos * p.kv_sl;
    float dot = 0.0f;
#pragma unroll
    for (int ks = 0; ks < kD / 16; ++ks) {
      const bf16x8 kv8 = *(const bf16x8*)(kp + (2 * ks + hl) * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) dot = __builtin_fmaf((float)qreg[ks][e], (float)kv8[e], dot);
    }
    dot = pair_sum(dot);
    const float t = dot * p.c2;
    const float mn = __builtin_fmaxf(m, t);
    const float alpha = __builtin_amdgcn_exp2f(m - mn);
    m = mn;
    const float pd = __builtin_amdgcn_exp2f(t - m);
    l = l * alpha + (hl == 0 ? pd : 0.0f);
    const __bf16* vp = p.vl + kvbase + (int64_t)pos * p.kv_sl;
#pragma unroll
    for (int db = 0; db < kD / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dim = 32 * db + 8 * g + 4 * hl;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[db][4 * g + e] = __builtin_fmaf(pd, (float)vp[dim + e], o[db][4 * g + e] * alpha);
      }
  }
  const float lt = pair_sum(l);
  if (qrow0 + l32 >= p.Lq) return;
  float* rec = p.ws + (((int64_t)bh * p.n_split + split) * p.Lq + qrow0 + l32) * COVER_RECT_RECORD;
  const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
#pragma unroll
  for (int db = 0; db < kD / 32; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *(bf16x4*)((__bf16*)rec + 32 * db + 8 * g + 4 * hl) =
          bf16x4{(__bf16)(o[db][4 * g] * inv), (__bf16)(o[db][4 * g + 1] * inv),
                 (__bf16)(o[db][4 * g + 2] * inv), (__bf16)(o[db][4 * g + 3] * inv)};
  if (hl == 0) {
    rec[kD / 2] = m;
    rec[kD / 2 + 1] = lt;
  }
}

// One wave per query row: merge the splits' (max, sum, O / sum), write O (bf16) and the lse.
__global__ __launch_bounds__(256) void cover_attn_rect_merge_kernel(const RectParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // over B * Hq * Lq
  if (row >= (int64_t)p.B * p.Hq * p.Lq) return;
  const int64_t bh = row / p.Lq;
  const int r = (int)(row % p.Lq);
  const int b = (int)(bh / p.Hq), h = (int)(bh % p.Hq);
  const float* rec0 = p.ws + (bh * p.n_split * p.Lq + r) * COVER_RECT_RECORD;
  const int64_t sstride = (int64_t)p.Lq * COVER_RECT_RECORD;
  // splits in chunks of 8 whose loads are all issued before the first is used; the running
  // (max, sum, O) is rescaled between chunks
  constexpr int kChunk = 8;
  float M = kInit, den = 0.0f, o0 = 0.0f, o1 = 0.0f;
  for (int s0 = 0; s0 < p.n_split; s0 += kChunk) {
    float ms[kChunk], ls[kChunk];
    uint32_t pr[kChunk];
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      ms[u] = kInit;
      ls[u] = 0.0f;
      pr[u] = 0u;
      if (s0 + u < p.n_split) {
        const float* rec = rec0 + (s0 + u) * sstride;
        ms[u] = rec[kD / 2];
        ls[u] = rec[kD / 2 + 1];
        pr[u] = ((const uint32_t*)rec)[lane];  // bf16 O of dims 2 lane, 2 lane + 1
      }
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) Mn = __builtin_fmaxf(Mn, ms[u]);
    const float a = __builtin_amdgcn_exp2f(M - Mn);
    den *= a;
    o0 *= a;
    o1 *= a;
    M = Mn;
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const float w = ls[u] * __builtin_amdgcn_exp2f(ms[u] - M);
      den += w;
      o0 = __builtin_fmaf(__uint_as_float(pr[u] << 16), w, o0);
      o1 = __builtin_fmaf(__uint_as_float(pr[u] & 0xffff0000u), w, o1);
    }
  }
  const float inv = 1.0f / den;
  __bf16* op = p.out + b * p.q_sb + h * p.q_sh + (int64_t)r * p.q_sl + 2 * lane;
  op[0] = (__bf16)(o0 * inv);
  op[1] = (__bf16)(o1 * inv);
  if (p.lse && lane == 0) p.lse[row] = (M + __builtin_amdgcn_logf(den)) * kLn2;
}


// ---------------------------------------------------------------------------------------
// Single-launch form (n_split == 1): one workgroup of 8 waves per (batch, query head,
// 32-query tile).  A CU's load path, not HBM, bounds a short block (about 100 GB/s per CU),
// and the merge of key splits held by different workgroups costs a second launch; so the
// key split stays inside the workgroup: wave w takes a contiguous share of the 32-key
// stages (the first four waves more than the other four, which issue their loads after
// them) and streams them through a K slot and a V slot of its own by global-to-LDS loads (no
// barrier in the loop), each slot refilled as soon as it has been read.  The eight partial
// (max, sum, O) states and a seed row's live diagonal term are merged through LDS at the end.
// Workgroups that share a KV head are placed on one XCD, so its L2 serves their re-reads.
// ---------------------------------------------------------------------------------------
constexpr int kTW = 8;             // waves per workgroup
constexpr int kTQ = 32;            // queries per workgroup
constexpr int kSB = kStage * kRow; // bytes of one stage of K (or V)
constexpr int kTSeeds = 64 * kTW;  // seed positions fetched into LDS (the rest: plain loads)
constexpr float kLazyT = 8.0f;

// s_waitcnt immediate that waits for vmcnt <= n only
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xf00; }

// Global -> LDS loads: lane l's 16 bytes (4 for the dword form) land at LDS byte lds + 16 l
// (+ 4 l); lds is wave-uniform.  The compiler does not track them: every read of their data
// follows an explicit vmcnt wait of the issuing wave.  A wave's loads land in issue order.
__device__ __forceinline__ uint32_t lds_addr(const void* ptr) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const lds_t*)ptr);
}
__device__ __forceinline__ void dma16(uint32_t lds, gmem_t* addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(lds), "v"((uint64_t)addr) : "memory", "m0");
}
__device__ __forceinline__ void dma16s(uint32_t lds, gmem_t* base, uint32_t voff) {  // uniform base
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
// the uniform-base load for the lanes of `mask` only (exec set and restored inside the
// statement; the scalar moves and the nop keep the load behind any VALU write of its operands)
__device__ __forceinline__ void dma16m(uint32_t lds, gmem_t* base, uint32_t voff, uint64_t mask) {
  uint64_t save;
  asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %1\n\ts_mov_b32 m0, %2\n\ts_nop 1\n\t"
               "global_load_lds_dwordx4 %3, %4\n\ts_mov_b64 exec, %0"
               : "=&s"(save) : "s"(mask), "s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
__device__ __forceinline__ void dma4(uint32_t lds, gmem_t* addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off"
               :: "s"(lds), "v"((uint64_t)addr) : "memory", "m0");
}
// lanes 16 k .. 16 k + 15 for each set bit k of a 4-bit value
__device__ __forceinline__ uint64_t lane_quads(uint32_t n) {
  const uint64_t m = (uint64_t)(n & 1u) | ((uint64_t)(n & 2u) << 15) | ((uint64_t)(n & 4u) << 30) |
                     ((uint64_t)(n & 8u) << 45);
  return (m << 16) - m;
}
__device__ __forceinline__ gmem_t* uniform_ptr(const void* ptr) {
  const uint64_t v = (uint64_t)ptr;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (gmem_t*)(((uint64_t)hi << 32) | lo);
}

// Phase timing (a separate build of the library, -DCOVER_RECT_TIMING=1, used only to measure
// where a workgroup's time goes): lane 0 of every wave of the first kTimeWG logical
// workgroups stores the shader-clock counter at fixed points.  Slots: 0 start, 1 seed list
// and Q landed, 2 seed bitmap built, 3 first stage landed, 4 + i top of the wave's stage i
// (i < 16), 20 loop done, 21 partial states in LDS (after the barrier), 22 end.
#ifndef COVER_RECT_TIMING
#define COVER_RECT_TIMING 0
#endif
#if COVER_RECT_TIMING
constexpr int kTimeWG = 1024, kTimeSlots = 32;
__device__ uint64_t g_rect_times[kTimeWG * kTW * kTimeSlots];
#define RECT_TSTAMP(slot)                                                                        \
  do {                                                                                           \
    if (li < kTimeWG && lane == 0)                                                               \
      g_rect_times[((int64_t)li * kTW + wave) * kTimeSlots + (slot)] = __builtin_readcyclecounter(); \
  } while (0)
#else
#define RECT_TSTAMP(slot) do {} while (0)
#endif

__global__ __launch_bounds__(64 * kTW, 1) void cover_attn_tile_kernel(const RectParams p) {
  // per wave: a K slot and a V slot (at the end: its partial O, 32 rows of 128 fp32);
  // the tile's Q; the seed bitmap of the sequence; the seed list; the partial maxima and sums
  __shared__ __attribute__((aligned(1024))) char sKV[kTW][2][kSB];
  __shared__ __attribute__((aligned(1024))) char sQ[kTQ * kRow];
  __shared__ uint32_t bits[kMaxWords];
  __shared__ __attribute__((aligned(16))) int32_t sSeeds[kTSeeds];
  __shared__ __attribute__((aligned(16))) int32_t sNs[4];
  __shared__ float sM[kTW][kTQ], sL[kTW][kTQ];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hl = lane >> 5;

  // workgroup -> (b, h, tile); consecutive logical tiles (those of one KV head) share an XCD
  const int li = (blockIdx.x & 7) * p.xcd_slots + (blockIdx.x >> 3);
  if (li >= p.n_wg) return;
  RECT_TSTAMP(0);
  const int qt = li % p.n_qt, bh = li / p.n_qt;
  const int h = bh % p.Hq, b = bh / p.Hq, g = h / p.group;
  const int L = p.L;
  const int nst = (L + kStage - 1) / kStage;
  // this wave's stages: waves 0-3 take 10/64 of them each, waves 4-7 (the second wave of
  // each SIMD, which loses the load path's arbitration to the first) 6/64: the measured
  // split that lets the waves finish together
  const int cw0 = wave < 4 ? 10 * wave : 40 + 6 * (wave - 4);
  const int cw1 = wave < 3 ? 10 * (wave + 1) : 40 + 6 * (wave - 3);
  const int s0 = nst * cw0 / 64, s1 = nst * cw1 / 64;
  const int ragged = L % kStage ? nst - 1 : -1;
  const int nW = (L + 31) >> 5;
  for (int w = tid; w < nW; w += 64 * kTW) bits[w] = 0u;

  // load geometry: load j of a stage covers stage rows 4 j + lane / 16 at physical chunk
  // lane % 16, i.e. LDS byte 1024 j + 16 lane of the slot; the source chunk is the one the
  // slot's swizzle puts there (K: chunk ^ row % 16; V: chunk ^ 4 (row % 4))
  const int64_t row_bytes = p.kv_sl * 2, stage_bytes = kStage * row_bytes;
  uint32_t offK[8], offV[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = 4 * j + (lane >> 4), pc = lane & 15;
    offK[j] = (uint32_t)(row * row_bytes) + ((pc ^ (row & 15)) << 4);
    offV[j] = (uint32_t)(row * row_bytes) + ((pc ^ ((row & 3) << 2)) << 4);
  }
  const int64_t kvoff = b * p.kv_sb + g * p.kv_sh;
  const char* const klc = (const char*)(p.kl + kvoff);
  const char* const kcc = (const char*)(p.kc + kvoff);
  const char* const vlc = (const char*)(p.vl + kvoff);
  const char* const vcc = (const char*)(p.vc + kvoff);
  const uint32_t slotK = lds_addr(sKV[wave][0]), slotV = lds_addr(sKV[wave][1]);
  // one stage: every row from the live tensor, or (with seeds = the stage's seed word) a seed
  // row from the cache; rows past L clamped into the sequence
  auto ld_stage = [&](uint32_t slot, const char* live, const char* cache, const uint32_t* off, int st,
                      uint32_t seeds) __attribute__((always_inline)) {
    if (st == ragged || seeds != 0u) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int row = 4 * j + (lane >> 4);
        const int key = min(st * kStage + row, L - 1);
        const char* src = ((seeds >> row) & 1u) ? cache : live;
        dma16(slot + 1024 * j, (gmem_t*)(src + key * row_bytes + (off[j] - (uint32_t)(row * row_bytes))));
      }
    } else {
      gmem_t* base = uniform_ptr(live + st * stage_bytes);
#pragma unroll
      for (int j = 0; j < 8; ++j) dma16s(slot + 1024 * j, base, off[j]);
    }
  };
  auto seed_word = [&](int st) __attribute__((always_inline)) -> uint32_t {
    return __builtin_amdgcn_readfirstlane(bits[st]);
  };
  // the seed rows of the first stage again (its loads went out before the seeds were known),
  // from the cache, issued after the live loads of the same slot so that they land last; a
  // load with no seed row among its four is skipped
  auto patch = [&](uint32_t slot, const char* cache, const uint32_t* off, int st)
                   __attribute__((always_inline)) {
    const uint32_t w = seed_word(st);
    if (w == 0u) return;
    gmem_t* base = uniform_ptr(cache + st * stage_bytes);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t nib = (w >> (4 * j)) & 15u;
      if (nib) dma16m(slot + 1024 * j, base, off[j], lane_quads(nib));
    }
  };

  // ---- prologue: the seed list, Q, and this wave's first stage from the live tensors ------
  const int64_t sbase = (int64_t)b * p.max_seeds;
  if (p.max_seeds > 0) {
    if (tid == 0) dma4(lds_addr(sNs), (gmem_t*)(p.n_seed + b));
    const int e = 64 * wave + lane;
    if (e < p.max_seeds) dma4(lds_addr((const char*)sSeeds + 256 * wave), (gmem_t*)(p.seed_idx + sbase + e));
  }
  const __bf16* qbase = p.q + b * p.q_sb + h * p.q_sh;
  {
    const int row = 4 * wave + (lane >> 4), pc = lane & 15;
    const int qi = min(qt * kTQ + row, p.Lq - 1);
    dma16(lds_addr(sQ + 1024 * wave), (gmem_t*)((const char*)(qbase + (int64_t)qi * p.q_sl) + ((pc ^ (row & 15)) << 4)));
  }
  if (s0 < s1) {
    ld_stage(slotK, klc, kcc, offK, s0, 0u);
    ld_stage(slotV, vlc, vcc, offV, s0, 0u);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(16));  // the seed list and Q have landed
  } else {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  }
  RECT_TSTAMP(1);
  __syncthreads();
  if (p.max_seeds > 0) {
    int ns = sNs[0];
    ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
    if (tid < ns && tid < kTSeeds) {
      const int j = sSeeds[tid];
      if ((unsigned)j < (unsigned)L) atomicOr(&bits[j >> 5], 1u << (j & 31));
    }
    for (int t = tid + kTSeeds; t < ns; t += 64 * kTW) {  // long seed lists
      const int j = p.seed_idx[sbase + t];
      if ((unsigned)j < (unsigned)L) atomicOr(&bits[j >> 5], 1u << (j & 31));
    }
  }
  __syncthreads();
  RECT_TSTAMP(2);
  auto is_seed = [&](int j) __attribute__((always_inline)) -> bool { return (bits[j >> 5] >> (j & 31)) & 1u; };
  if (s0 < s1) {
    patch(slotK, kcc, offK, s0);
    patch(slotV, vcc, offV, s0);
  }

  // Q fragments (B operand of S^T = K Q^T): query l32, d-chunk 2 ks + hl
  bf16x8 qreg[kD / 16];
#pragma unroll
  for (int ks = 0; ks < kD / 16; ++ks)
    qreg[ks] = *(const __attribute__((address_space(3))) bf16x8*)((const lds_t*)sQ + k_off(l32, 2 * ks + hl));
  const int qrow = min(qt * kTQ + l32, p.Lq - 1);
  const int pos = p.q_off + qrow;
  const bool row_seed = is_seed(pos);

  // the live key and value rows of the seed rows this wave finishes: lane group fq = lane / 16
  // takes query kFin wave + fq, dims 8 (lane % 16) .. + 7, requested now and used in the merge
  constexpr int kFin = kTQ / kTW;
  const int fq = lane >> 4, fj = lane & 15;
  const int qfin = qt * kTQ + kFin * wave + fq;
  const bool fin_ok = qfin < p.Lq;
  const bool fseed = fin_ok && is_seed(p.q_off + qfin);
  u32x4 kd = {0u, 0u, 0u, 0u}, vd = {0u, 0u, 0u, 0u};
  if (fseed) {
    const int64_t ro = kvoff + (int64_t)(p.q_off + qfin) * p.kv_sl + 8 * fj;
    kd = *(const u32x4*)(p.kl + ro);
    vd = *(const u32x4*)(p.vl + ro);
  }

  // V^T operand addresses (as in the split kernel)
  uint32_t vaddr[kD / 32];
  {
    const int G = lane >> 4, ii = lane & 15;
    const int row = 4 * (G >> 1) + (ii >> 2);
#pragma unroll
    for (int db = 0; db < kD / 32; ++db) vaddr[db] = v_elem(row, db * 32 + 16 * (G & 1) + 4 * (ii & 3));
  }
  f32x16 o[kD / 32];
#pragma unroll
  for (int db = 0; db < kD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m = kInit, l = 0.0f;
  const lds_t* const kb = (const lds_t*)sKV[wave][0];
  const lds_t* const vb = (const lds_t*)sKV[wave][1];

  for (int st = s0; st < s1; ++st) {
    const bool more = st + 1 < s1;
    // K(st) has landed: younger are V(st)'s 8 loads; at the first stage everything is waited
    // for (the patches of the prologue are counted nowhere)
    if (st == s0) __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(8));
    if (st == s0) RECT_TSTAMP(3);
    if (st - s0 < 16) RECT_TSTAMP(4 + st - s0);
    bf16x8 ka[kD / 16];
#pragma unroll
    for (int ks = 0; ks < kD / 16; ++ks)
      ka[ks] = *(const __attribute__((address_space(3))) bf16x8*)(kb + k_off(l32, 2 * ks + hl));
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the K slot is read: refill it
    if (more) ld_stage(slotK, klc, kcc, offK, st + 1, seed_word(st + 1));
    f32x16 sc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[r] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < kD / 16; ++ks) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[ks], qreg[ks], sc, 0, 0, 0);
    // register r holds key k0 + 8 (r / 4) + 4 hl + r % 4 of query qrow
    const int k0 = st * kStage;
    const bool edge = k0 + kStage > L;
    const bool diag = row_seed && pos >= k0 && pos < k0 + kStage;
    float mx = kInit;
    if (__builtin_amdgcn_ballot_w64(diag) != 0 || edge) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + 8 * (r >> 2) + 4 * hl + (r & 3);
        float t = sc[r] * p.c2;
        if (key >= L || (diag && key == pos)) t = -INFINITY;
        sc[r] = t;
        mx = __builtin_fmaxf(mx, t);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sc[r] *= p.c2;
        mx = __builtin_fmaxf(mx, sc[r]);
      }
    }
    mx = pair_max(mx);
    if (st == s0) {
      m = mx;
    } else if (__builtin_amdgcn_ballot_w64(mx > m + kLazyT)) {
      const float mn = __builtin_fmaxf(m, mx);
      const float alpha = __builtin_amdgcn_exp2f(m - mn);
      l *= alpha;
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) o[db] *= alpha;
      m = mn;
    }
    bf16x8 pk[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pr = __builtin_amdgcn_exp2f(sc[8 * kk + e] - m);
        l += pr;
        pk[kk][e] = (__bf16)pr;
      }
    // V(st) has landed: younger are K(st + 1)'s 8 loads, if there is a stage st + 1
    if (more) __builtin_amdgcn_s_waitcnt(vmcnt_imm(8));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    bf16x8 va[2][kD / 32];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int db = 0; db < kD / 32; ++db) {
        const lds_t* base = vb + vaddr[db] + kk * 16 * kRow;
        va[kk][db] = __builtin_bit_cast(
            bf16x8, __builtin_shufflevector(v_tr(base), v_tr(base + 8 * kRow), 0, 1, 2, 3, 4, 5, 6, 7));
      }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the V slot is read: refill it
    if (more) {
      ld_stage(slotV, vlc, vcc, offV, st + 1, seed_word(st + 1));
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int db = 0; db < kD / 32; ++db)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[kk][db], pk[kk], o[db], 0, 0, 0);
  }

  // ---- merge: every wave's (max, sum, O) through LDS ---------------------------------------
  // O goes to this wave's own slots (its loads have all landed and been read): row l32, 16-byte
  // chunk c (dims 4 c .. 4 c + 3) at byte 512 l32 + 16 (c ^ l32)
  RECT_TSTAMP(20);
  const float lt = pair_sum(l);
  if (hl == 0) {
    sM[wave][l32] = m;
    sL[wave][l32] = lt;
  }
  {
    lds_t* const ob = (lds_t*)sKV[wave][0] + 512 * l32;
#pragma unroll
    for (int db = 0; db < kD / 32; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int c = 8 * db + 2 * gq + hl;
        *(__attribute__((address_space(3))) f32x4*)(ob + ((c ^ l32) << 4)) =
            f32x4{o[db][4 * gq], o[db][4 * gq + 1], o[db][4 * gq + 2], o[db][4 * gq + 3]};
      }
  }
  __syncthreads();
  RECT_TSTAMP(21);
  // wave w finishes queries kFin w + fq (lane group fq), lane dims 8 fj .. 8 fj + 7; every
  // LDS read of the merge is requested before the first is used
  {
    const int f = kFin * wave + fq;
    float mw[kTW], lw[kTW];
    f32x4 ow[kTW][2];
#pragma unroll
    for (int w = 0; w < kTW; ++w) {
      mw[w] = sM[w][f];
      lw[w] = sL[w][f];
      const lds_t* rb = (const lds_t*)sKV[w][0] + 512 * f;
      ow[w][0] = *(const __attribute__((address_space(3))) f32x4*)(rb + (((2 * fj) ^ f) << 4));
      ow[w][1] = *(const __attribute__((address_space(3))) f32x4*)(rb + (((2 * fj + 1) ^ f) << 4));
    }
    const u32x4 qv = *(const __attribute__((address_space(3))) u32x4*)((const lds_t*)sQ + k_off(f, fj));
    float M = kInit;
#pragma unroll
    for (int w = 0; w < kTW; ++w) M = __builtin_fmaxf(M, mw[w]);
    // the live diagonal score q . k_live(pos) of a seed row (App. B.4), summed over the
    // group's 16 lanes
    float dot = 0.0f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      dot = __builtin_fmaf(__uint_as_float(qv[e] << 16), __uint_as_float(kd[e] << 16), dot);
      dot = __builtin_fmaf(__uint_as_float(qv[e] & 0xffff0000u), __uint_as_float(kd[e] & 0xffff0000u), dot);
    }
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1) dot += __shfl_xor(dot, off);
    const float t = dot * p.c2;
    if (fseed) M = __builtin_fmaxf(M, t);
    float den = 0.0f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int w = 0; w < kTW; ++w) {
      const float a = __builtin_amdgcn_exp2f(mw[w] - M);
      den = __builtin_fmaf(lw[w], a, den);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[e] = __builtin_fmaf(a, ow[w][0][e], acc[e]);
        acc[4 + e] = __builtin_fmaf(a, ow[w][1][e], acc[4 + e]);
      }
    }
    if (fseed) {
      const float pd = __builtin_amdgcn_exp2f(t - M);
      den += pd;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = __builtin_fmaf(pd, __uint_as_float(vd[e] << 16), acc[2 * e]);
        acc[2 * e + 1] = __builtin_fmaf(pd, __uint_as_float(vd[e] & 0xffff0000u), acc[2 * e + 1]);
      }
    }
    if (fin_ok) {
      const float inv = 1.0f / den;
      bf16x8 ob;
#pragma unroll
      for (int e = 0; e < 8; ++e) ob[e] = (__bf16)(acc[e] * inv);
      *(bf16x8*)(p.out + b * p.q_sb + h * p.q_sh + (int64_t)qfin * p.q_sl + 8 * fj) = ob;
      if (p.lse && fj == 0) p.lse[(int64_t)bh * p.Lq + qfin] = (M + __builtin_amdgcn_logf(den)) * kLn2;
    }
  }
  RECT_TSTAMP(22);
}

}  // namespace

#if COVER_RECT_TIMING
// Copies the timing slots of the last launch of the single-launch kernel (layout
// [workgroup][wave][slot], 1024 x 8 x 32 values) to host memory; waits for the device.  Only
// in the timing build of the library.
extern "C" int cover_rect_timing_read(uint64_t* host, int64_t n) {
  const int64_t cap = (int64_t)kTimeWG * kTW * kTimeSlots;
  return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(g_rect_times), sizeof(uint64_t) * (n < cap ? n : cap),
                                  0, hipMemcpyDeviceToHost);
}
#endif

hipError_t launch_attn_rect(const RectArgs& a, hipStream_t stream) {
  RectParams p;
  p.q = (const __bf16*)a.q; p.kl = (const __bf16*)a.k_live; p.vl = (const __bf16*)a.v_live;
  p.kc = (const __bf16*)a.k_cache; p.vc = (const __bf16*)a.v_cache;
  p.seed_idx = a.seed_idx; p.n_seed = a.n_seed; p.ws = a.workspace;
  p.out = (__bf16*)a.out; p.lse = a.lse;
  p.B = a.B; p.Hq = a.Hq; p.Hkv = a.Hkv; p.L = a.L; p.Lq = a.Lq; p.q_off = a.q_off;
  p.max_seeds = a.max_seeds; p.group = a.Hq / a.Hkv;
  p.n_qt = (a.Lq + kQT - 1) / kQT;
  p.n_split = a.n_split;
  const int stages = (a.L + kStage - 1) / kStage;
  p.split_stages = (stages + a.n_split - 1) / a.n_split;
  p.c2 = a.scale * 1.44269504088896341f;
  p.q_sb = a.q_sb; p.q_sh = a.q_sh; p.q_sl = a.q_sl;
  p.kv_sb = a.kv_sb; p.kv_sh = a.kv_sh; p.kv_sl = a.kv_sl;
  if (a.n_split == 1) {  // single launch, no workspace (kv_sl < 2^26: 32-bit in-stage offsets)
    p.n_qt = (a.Lq + kTQ - 1) / kTQ;
    const int64_t n = (int64_t)a.B * a.Hq * p.n_qt;
    p.n_wg = (int)n;
    p.xcd_slots = (int)((n + 7) / 8);
    hipLaunchKernelGGL(cover_attn_tile_kernel, dim3((unsigned)(8 * (int64_t)p.xcd_slots)), dim3(64 * kTW), 0,
                       stream, p);
    return hipGetLastError();
  }
  const int64_t nwg = (int64_t)a.B * a.Hq * p.n_qt * a.n_split;
  hipLaunchKernelGGL(cover_attn_rect_kernel, dim3((unsigned)nwg), dim3(kThreads), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t rows = (int64_t)a.B * a.Hq * a.Lq;
  hipLaunchKernelGGL(cover_attn_rect_merge_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
