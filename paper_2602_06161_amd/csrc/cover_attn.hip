// COVER attention on gfx950: bidirectional attention over the KV-cache-overridden memory
// with the diagonal correction for seed rows (arXiv 2602.06161, Sec. 5.1 and App. B).
//
// What every query row i of batch row b computes (S_b = seed set of b):
//   K'_j = k_cache_j if j in S_b else k_live_j          (override memory, Sec. 5.1)
//   row view: K'_j for j != i;  k_live_i at j == i when i in S_b   (leave-one-out view)
//   out_i = softmax_j(scale <q_i, K^(i)_j>) V^(i),  lse_i = log sum_j exp(...)
// The paper derives the seed-row result as a post-hoc rescaling of the overridden row
// (Lemma B.1, closed form of App. B.4).  Here the same quantity is formed inside the
// online softmax instead: the overridden diagonal score is replaced by the live one before
// the row max/exponentials, so the normaliser already holds exp(q.k_live) in place of
// exp(q.k_cache) and no division by r_i is needed (by Lemma B.1 the two are equal in exact
// arithmetic; this form has no cancellation when the cached diagonal dominates the row).
// The value side is done with a second, tiny PV product: the diagonal probability is
// removed from the P fed to the main PV product and multiplied by the live value row
// instead.
//
// bf16 kernel for head size 64 (head size 128 has its own four-wave kernel, cover_attn_w4.hip);
// design (one workgroup = 8 waves, two per SIMD = 128 queries of one (b, h)):
//   * Transposed products keep every query row inside one lane pair:
//       S^T = K Q^T   (v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q from registers)
//       O^T += V^T P^T (A = V^T read with ds_read_b64_tr_b16, B = P straight from the S^T
//                       registers after exp2 and bf16 packing)
//     so row max / row sum / rescale are lane-local plus one v_permlane32_swap.
//   * Wave w owns the 32 queries of block w%4 and the 32-key half w/4 of every 64-key
//     stage; the two key halves of a query block are merged through LDS at the end.  With
//     256 registers per wave (two waves per SIMD) every MFMA keeps its accumulator in
//     VGPRs, so the softmax reads S without copies.
//   * K/V stages of 64 keys: each wave loads an eighth of a stage into registers one step
//     ahead and stores it to LDS (double-buffered), choosing each row's source (live or
//     cache) from a per-sequence seed bitmap in LDS; the first stages are loaded from the
//     live tensors before the bitmap is known and reloaded only if they hold seeds.
//   * Stages are walked in order; S of the next stage is computed while the softmax and the
//     PV product of the current one run, with one barrier per stage.
//   * Lazy softmax rescaling: a row's reference max moves only when the row max grows by
//     more than 2^20, so most stages skip the O rescale (exact: O and l share the
//     reference).
//   * Workgroups sharing one (b, key/value head) are placed on the same XCD so its K/V
//     stays resident in that XCD's L2.
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
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) char lds_t;
typedef __attribute__((address_space(1))) const char gmem_t;  // global memory, read-only here

constexpr int kWaves = 8;             // waves per workgroup: two per SIMD
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = 128;             // queries per workgroup
constexpr int kStageKeys = 64;       // keys per pipeline stage = two 32-key wave tiles
constexpr float kSlack = 20.0f;      // rescale only when a row max grows by > 2^20
constexpr float kInitMax = -1.0e30f; // finite "no key seen yet" reference max
constexpr float kLn2 = 0.693147180559945309f;

// s_waitcnt immediates waiting for vmcnt <= n only, or for lgkmcnt <= n only
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xf00; }
constexpr int lgkmcnt_imm(int n) { return 0xf | (3 << 14) | 0x70 | ((n & 15) << 8); }

template <int D>
struct Tile {
  static constexpr int CH = D / 8;                     // 16-byte chunks per bf16 row
  static constexpr int KS = D / 16;                    // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;                    // 32-row blocks of O^T
  static constexpr int ROW = D * 2;                    // bytes per row
  static constexpr int SBYTES = kStageKeys * ROW;      // one K or V stage of 64 rows
  static constexpr int RPI = 1024 / ROW;               // rows per 1-KiB wave load
  static constexpr int IPW = SBYTES / 1024 / kWaves;   // such loads per wave per stage
  static constexpr int NJH = DB / 2 * 16;              // O^T values per lane in half of d
  static constexpr int kWaitPrev = vmcnt_imm(2 * IPW);
  static_assert(IPW >= 1, "a stage must give every wave at least one load");
  static_assert(2 * NJH * 64 * 4 <= SBYTES, "two merge slots must fit one stage buffer");
};

struct Params {
  const __bf16* q;
  const __bf16* kl;
  const __bf16* vl;
  const __bf16* kc;
  const __bf16* vc;
  const int32_t* seed_idx;
  const int32_t* n_seed;
  __bf16* out;
  float* lse;
  int B, Hq, Hkv, L, max_seeds, group, n_qt, xcd_slots;
  float c2;  // scale * log2(e)
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

// LDS swizzles (64 banks of 4 bytes: one 256-byte window per cycle).  K rows are read 16
// rows per LDS cycle at one logical chunk (b128 reads), so the chunk index is XOR-ed with
// the row (D = 128) or with row/2 (D = 64, two rows per 256-byte window).  A V transpose
// read covers 8 rows x 64 bytes (one 32-column block); the chunk XOR (4*(r%4) for D = 128,
// 2*(r%4) for D = 64) places the rows' segments so that the 512 bytes fill every bank
// exactly twice.
template <int ROW>
__device__ __forceinline__ int k_swz(int row) {
  return (ROW == 256) ? (row & 15) : ((row >> 1) & 7);
}
template <int ROW>
__device__ __forceinline__ int v_swz(int row) {
  return (ROW == 256) ? ((row & 3) << 2) : ((row & 3) << 1);
}
template <int ROW>
__device__ __forceinline__ uint32_t k_off(int row, int c) {
  return row * ROW + ((c ^ k_swz<ROW>(row)) << 4);
}
// byte address of element `col` of V row `row`
template <int ROW>
__device__ __forceinline__ uint32_t v_elem(int row, int col) {
  return row * ROW + (((col >> 3) ^ v_swz<ROW>(row)) << 4) + ((col & 7) << 1);
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 lds_read16(const lds_t* p) { return *(const __attribute__((address_space(3))) u32x4*)p; }

// Half of the A operand of O^T += V^T P^T: transpose read of 4 V rows x 4 columns per lane.
__device__ __forceinline__ i16x4 v_tr(const lds_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
}

__device__ __forceinline__ float swap_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float swap_add(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float fmax2(float a, float b) { return __builtin_fmaxf(a, b); }
__device__ __forceinline__ float fmax3(float a, float b, float c) { return __builtin_fmaxf(__builtin_fmaxf(a, b), c); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int N>
struct IC {
  static constexpr int value = N;
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void cover_attn_bf16_kernel(const Params p) {
  using T = Tile<D>;
  // Two K and two V stage buffers (the loads of a stage are staged in registers one step
  // ahead), the live value rows of the seed rows' diagonals, merge scalars, seed bitmap.
  __shared__ __attribute__((aligned(1024))) char sK0[T::SBYTES];
  __shared__ __attribute__((aligned(1024))) char sK1[T::SBYTES];
  __shared__ __attribute__((aligned(1024))) char sV0[T::SBYTES];
  __shared__ __attribute__((aligned(1024))) char sV1[T::SBYTES];
  __shared__ __attribute__((aligned(1024))) char sDiag[4 * 32 * T::ROW];
  __shared__ __attribute__((aligned(16))) float sML[kWaves * 2 * 64];
  __shared__ uint32_t bits[COVER_MAX_L / 32];
  __shared__ uint32_t sdirty[COVER_MAX_L / kStageKeys / 32];  // stages holding a seed
  auto kbuf = [&](int n) -> lds_t* { return (lds_t*)(n == 0 ? sK0 : sK1); };
  auto vbuf = [&](int n) -> lds_t* { return (lds_t*)(n == 0 ? sV0 : sV1); };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qq = wave & 3;   // 32-query block of the workgroup tile
  const int kp = wave >> 2;  // key half: 32-key tile kp of every 64-key stage
  const int hl = lane >> 5, l32 = lane & 31;

  // ---- workgroup -> (b, h, query tile); consecutive logical tiles share an XCD --------
  int li = blockIdx.x;
  if (p.xcd_slots > 0) li = (li & 7) * p.xcd_slots + (li >> 3);
  const int qt = li % p.n_qt;
  const int bh = li / p.n_qt;
  const int h = bh % p.Hq, b = bh / p.Hq;
  const int g = h / p.group;
  const int L = p.L;
  const int q0 = qt * kBM;
  const int qw = q0 + qq * 32;  // this wave's first query
  const __bf16* qbase = p.q + b * p.q_sb + h * p.q_sh;
  const int64_t kvoff = b * p.kv_sb + g * p.kv_sh;
  const float c2 = p.c2;

  // ---- Q fragments (B operand of S^T = K Q^T): query qw + l32, d-chunk 2*ks + hl ---------
  bf16x8 qreg[T::KS];
  {
    const int qi = min(qw + l32, L - 1);
    const __bf16* qrow = qbase + (int64_t)qi * p.q_sl + hl * 8;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) qreg[ks] = *(const bf16x8*)(qrow + ks * 16);
  }

  // ---- stage loads -------------------------------------------------------------------------
  // A stage is 64 rows; each wave moves IPW KiB of it, 16 bytes per lane per KiB, through
  // registers: load j of this wave holds row (wave*IPW + j)*RPI + lane/CH, physical chunk
  // lane%CH, which is the row's logical chunk (physical ^ swizzle), and is stored to LDS at
  // (wave*IPW + j)*1024 + 16*lane.  A row comes from the cache when its position is a seed;
  // rows past L (ragged last stage) repeat row L-1 (their scores are masked).
  auto ld_row = [&](int j) { return (wave * T::IPW + j) * T::RPI + lane / T::CH; };
  auto ld_chunk = [&](int j, bool is_v) -> uint32_t {
    const int row = ld_row(j), pc = lane % T::CH;
    return (uint32_t)((pc ^ (is_v ? (v_swz<T::ROW>(row) & (T::CH - 1)) : k_swz<T::ROW>(row))) << 4);
  };
  const int64_t row_bytes = p.kv_sl * 2;
  const int64_t stage_bytes = kStageKeys * row_bytes;
  uint32_t offK[T::IPW], offV[T::IPW];
#pragma unroll
  for (int j = 0; j < T::IPW; ++j) {
    offK[j] = (uint32_t)(ld_row(j) * row_bytes) + ld_chunk(j, false);
    offV[j] = (uint32_t)(ld_row(j) * row_bytes) + ld_chunk(j, true);
  }
  auto uniform_ptr = [](const void* ptr) -> gmem_t* {
    const uint64_t v = (uint64_t)ptr;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (gmem_t*)(((uint64_t)hi << 32) | lo);
  };
  gmem_t* const klb = uniform_ptr(p.kl + kvoff);
  gmem_t* const kcb = uniform_ptr(p.kc + kvoff);
  gmem_t* const vlb = uniform_ptr(p.vl + kvoff);
  gmem_t* const vcb = uniform_ptr(p.vc + kvoff);
  typedef __attribute__((address_space(1))) const u32x4 gu32x4;

  // The first stages are loaded speculatively from the live tensors (rows past L clamped),
  // in the shadow of the seed list's latency; stages that turn out to hold seeds are loaded
  // again once the bitmap is known.  K(0), V(0), K(1) go to pre[], K(2), V(1) to staging.
  const int n_it = (L + kStageKeys - 1) / kStageKeys;
  auto clamp_stage = [=](int i) -> int { return i < n_it ? i : n_it - 1; };
  auto ld_live = [&](u32x4* st, gmem_t* live, bool is_v, int stage) {
    const int kb = stage * kStageKeys;
#pragma unroll
    for (int j = 0; j < T::IPW; ++j) {
      const int key = min(kb + ld_row(j), L - 1);
      st[j] = *(gu32x4*)(live + key * row_bytes + ld_chunk(j, is_v));
    }
  };
  u32x4 pre[3][T::IPW], stgK[T::IPW], stgV[T::IPW];
  ld_live(pre[0], klb, false, 0);
  ld_live(pre[1], vlb, true, 0);
  ld_live(pre[2], klb, false, clamp_stage(1));
  ld_live(stgK, klb, false, clamp_stage(2));
  ld_live(stgV, vlb, true, clamp_stage(1));

  // ---- seed bitmap of this sequence ---------------------------------------------------
  // The seed list is read speculatively (the first kThreads entries) with its length.
  const int nwords = (L + 31) >> 5;
  const int64_t sbase = (int64_t)b * p.max_seeds;
  int ns = 0;
  if (p.max_seeds > 0) ns = p.n_seed[b];
  const int sj0 = tid < p.max_seeds ? p.seed_idx[sbase + tid] : -1;
  // words past the sequence are cleared too: per-stage lookups read two words per stage
  for (int w = tid; w < 2 * n_it; w += kThreads) bits[w] = 0u;
  if (tid < COVER_MAX_L / kStageKeys / 32) sdirty[tid] = 0u;
  __syncthreads();
  ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
  auto mark = [&](int j) {
    atomicOr(&bits[j >> 5], 1u << (j & 31));
    atomicOr(&sdirty[j >> 11], 1u << ((j >> 6) & 31));
  };
  if (tid < ns && (unsigned)sj0 < (unsigned)L) mark(sj0);
  for (int t = tid + kThreads; t < ns; t += kThreads) {
    const int j = p.seed_idx[sbase + t];
    if ((unsigned)j < (unsigned)L) mark(j);
  }
  __syncthreads();
  auto is_seed = [&](int j) -> bool { return (bits[j >> 5] >> (j & 31)) & 1u; };

  // ---- stages ----------------------------------------------------------------------------
  // Stages of 64 keys are processed in order.  Up to three need per-element care: the two
  // holding this tile's diagonal when the tile has seeds, and a ragged last stage.
  uint32_t tile_bits = 0;
#pragma unroll
  for (int w = 0; w < kBM / 32; ++w) tile_bits |= (q0 / 32 + w < nwords) ? bits[q0 / 32 + w] : 0u;
  const bool tile_seeded = __builtin_amdgcn_readfirstlane(tile_bits) != 0u;
  const int spA = tile_seeded ? 2 * qt : -1;
  const int spB = tile_seeded ? 2 * qt + 1 : -1;
  const int spC = L % kStageKeys != 0 ? n_it - 1 : -1;  // ragged
  auto is_special = [=](int i) -> bool { return (i == spA) | (i == spB) | (i == spC); };
  // Lane l holds the seed flags of stages 64l .. 64l+63 (two words); a stage's flag is read
  // back with a lane read, no memory access.
  const uint32_t dirty_lo = sdirty[(2 * lane) & (COVER_MAX_L / kStageKeys / 32 - 1)];
  const uint32_t dirty_hi = sdirty[(2 * lane + 1) & (COVER_MAX_L / kStageKeys / 32 - 1)];
  auto dirty = [&](int stage) -> bool {
    const uint32_t w = ((stage >> 5) & 1) ? __builtin_amdgcn_readlane(dirty_hi, stage >> 6)
                                          : __builtin_amdgcn_readlane(dirty_lo, stage >> 6);
    return (w >> (stage & 31)) & 1u;
  };

  // Issue the loads of one stage of K or V into st[0..IPW).  Stages without seeds and within
  // L use a scalar base and per-lane 32-bit offsets; the others choose each row's source and
  // clamp rows past L.
  auto ld = [&](u32x4* st, gmem_t* live, gmem_t* cache, const uint32_t* off, bool is_v,
                int stage_in) {
    const int stage = __builtin_amdgcn_readfirstlane(stage_in);
    const int kb = stage * kStageKeys;
    if (stage != spC && !dirty(stage)) {
      gmem_t* lb = uniform_ptr((const void*)(live + stage * stage_bytes));
#pragma unroll
      for (int j = 0; j < T::IPW; ++j) st[j] = *(gu32x4*)(lb + off[j]);
    } else {
#pragma unroll
      for (int j = 0; j < T::IPW; ++j) {
        const int key = min(kb + ld_row(j), L - 1);
        gmem_t* src = is_seed(key) ? cache : live;
        st[j] = *(gu32x4*)(src + key * row_bytes + ld_chunk(j, is_v));
      }
    }
  };
  const uint32_t lds_slot = wave * (T::IPW * 1024) + lane * 16;  // within a stage buffer
  auto st = [&](const u32x4* stg, lds_t* buf) {
#pragma unroll
    for (int j = 0; j < T::IPW; ++j) *(__attribute__((address_space(3))) u32x4*)(buf + lds_slot + j * 1024) = stg[j];
  };

  // ---- diagonal set-up ------------------------------------------------------------------
  // Query c of this wave (position qw + c) has its diagonal key at position qw + c, which
  // lies in this wave's key tile exactly when kp == qq % 2, in stage itd = qw / 64.  In S^T
  // the diagonal entry of query c sits in lane half (c/4)%2, register (c/8)*4 + c%4.
  const bool diag_wave = kp == (qq & 1);
  const int itd = qw / kStageKeys;
  const bool holds_diag = hl == ((l32 >> 2) & 1);
  const int rd = ((l32 >> 3) << 2) | (l32 & 3);
  const bool qd_seed = (qw + l32) < L && is_seed(qw + l32);  // this lane's query is a seed
  const bool diag_seed = diag_wave && holds_diag && qd_seed;
  const bool block_seeded = __builtin_amdgcn_ballot_w64(qd_seed) != 0;
  // Seed rows need the live value row of their own position in the epilogue: the 32 rows
  // of each query block go to its sDiag slot (K swizzle), loaded by the block's diagonal wave.
  lds_t* const dg = (lds_t*)sDiag + qq * (32 * T::ROW);
  if (block_seeded && diag_wave) {
    constexpr int NL = 32 * T::ROW / 1024;
    u32x4 dv[NL];
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int row = j * T::RPI + lane / T::CH, pc = lane % T::CH;
      const int vr = min(qw + row, L - 1);
      dv[j] = *(gu32x4*)(vlb + vr * row_bytes + ((pc ^ k_swz<T::ROW>(row)) << 4));
    }
#pragma unroll
    for (int j = 0; j < NL; ++j) *(__attribute__((address_space(3))) u32x4*)(dg + j * 1024 + lane * 16) = dv[j];
  }
  // Seed rows: raw live diagonal score q_i . k_live_i (both waves of the block need it).
  float s_live = 0.0f;
  if (block_seeded) {
    const int qr = min(qw + l32, L - 1);
    const uint32_t* krow = (const uint32_t*)(p.kl + kvoff + (int64_t)qr * p.kv_sl + hl * 8);
    float acc = 0.0f;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) {
      const u32x4 kv = *(const u32x4*)(krow + ks * 8);
      const u32x4 qv = __builtin_bit_cast(u32x4, qreg[ks]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc = __builtin_fmaf(bf16_lo(qv[e]), bf16_lo(kv[e]), acc);
        acc = __builtin_fmaf(bf16_hi(qv[e]), bf16_hi(kv[e]), acc);
      }
    }
    s_live = swap_add(acc);
  }

  // ---- per-lane LDS read addresses (relative to a stage buffer) ---------------------------
  uint32_t kaddr[T::KS];
#pragma unroll
  for (int ks = 0; ks < T::KS; ++ks) kaddr[ks] = k_off<T::ROW>(kp * 32 + l32, 2 * ks + hl);
  // A operand of O^T += V^T P^T for keys kp*32 + 16*kk + {0..3, 8..11} + 4*(G/2), d-block db:
  // lane (G = lane/16, i = lane%16) reads V[row][db*32 + 16*(G%2) + 4*(i%4) ..+3] with
  // row = kp*32 + 16*kk + 4*(G/2) + i/4 (+8 for the upper half).  The same key order is
  // what the S^T registers give the P^T operand.  kk and the +8 move the row by multiples
  // of 4, which leaves the swizzle unchanged: they are constant offsets.
  uint32_t vaddr[T::DB];
  {
    const int G = lane >> 4, ii = lane & 15;
    const int row = kp * 32 + 4 * (G >> 1) + (ii >> 2);
#pragma unroll
    for (int db = 0; db < T::DB; ++db) vaddr[db] = v_elem<T::ROW>(row, db * 32 + 16 * (G & 1) + 4 * (ii & 3));
  }

  auto qk = [&](const lds_t* kb, f32x16& s) {
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, lds_read16(kb + kaddr[ks]));
      s = mfma(a, qreg[ks], ks == 0 ? (f32x16){} : s);
    }
  };
  // keys of this wave's tile of `stage` past L, and the seed rows' own (cached) column, get
  // no weight; the live diagonal term is added in the epilogue
  auto special_fix = [&](int stage, f32x16& s) {
    if (stage * kStageKeys + kStageKeys > L) {
      const int kbase = stage * kStageKeys + kp * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool ok = kbase + ((r >> 2) << 3) + hl * 4 + (r & 3) < L;
        s[r] = ok ? s[r] : -INFINITY;
      }
    }
    if (diag_wave && block_seeded && stage == itd) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = (diag_seed && r == rd) ? -INFINITY : s[r];
    }
  };
  // a tree of depth 3 (independent max3 operations first), not a chain of 8
  auto lane_max = [&](const f32x16& s) -> float {
    const float a = fmax3(s[0], s[1], s[2]), b = fmax3(s[3], s[4], s[5]);
    const float c = fmax3(s[6], s[7], s[8]), d = fmax3(s[9], s[10], s[11]);
    const float e = fmax3(s[12], s[13], s[14]);
    return fmax3(fmax3(a, b, c), fmax2(d, e), s[15]);
  };

  float m, lsum = 0.0f, thr;
  f32x16 o[T::DB];
#pragma unroll
  for (int db = 0; db < T::DB; ++db) o[db] = (f32x16){};
  // raw score above which a row leaves the branch-free steps: (m + slack) / c2 (c2 > 0)
  const float inv_c2 = 1.0f / c2;

  // softmax of S into bf16 P (row sums of the bf16 weights, as the MFMA sees them), then
  // O^T += V^T P^T
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  auto softmax_pv = [&](const f32x16& s, const lds_t* vcur) {
    const float nm = -m;
    f32x16 pr;
#pragma unroll
    for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], c2, nm));
    bf16x8 pk[2];
    pk[0] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 0, 1, 2, 3, 4, 5, 6, 7), bf16x8);
    pk[1] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 8, 9, 10, 11, 12, 13, 14, 15), bf16x8);
    // row sums in two independent chains of four
    float ls[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const bf16x8 w = pk[kk];
      float a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 0, 1), ones, 0.0f, false);
      a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 2, 3), ones, a, false);
      a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 4, 5), ones, a, false);
      ls[kk] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 6, 7), ones, a, false);
    }
    lsum += ls[0] + ls[1];
    typedef short i16x8 __attribute__((ext_vector_type(8)));
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int db = 0; db < T::DB; ++db) {
        const lds_t* base = vcur + vaddr[db] + kk * 16 * T::ROW;
        const i16x8 v = __builtin_shufflevector(v_tr(base), v_tr(base + 8 * T::ROW), 0, 1, 2, 3, 4, 5, 6, 7);
        o[db] = mfma(__builtin_bit_cast(bf16x8, v), pk[kk], o[db]);
      }
    }
  };

  // ---- prologue ------------------------------------------------------------------------------
  // K(0), V(0), K(1) go straight to their buffers; K(2) and V(1) wait in the staging
  // registers for the first step (all loaded before the bitmap, again here if they hold
  // seeds).  Then S(0) and the reference row max.
  {
    if (dirty(0) || dirty(clamp_stage(1)) || dirty(clamp_stage(2))) {
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // the speculative loads are replaced
      ld(pre[0], klb, kcb, offK, false, 0);
      ld(pre[1], vlb, vcb, offV, true, 0);
      ld(pre[2], klb, kcb, offK, false, clamp_stage(1));
      ld(stgK, klb, kcb, offK, false, clamp_stage(2));
      ld(stgV, vlb, vcb, offV, true, clamp_stage(1));
    }
    __builtin_amdgcn_s_waitcnt(T::kWaitPrev);  // the first three stages landed
    st(pre[0], kbuf(0));
    st(pre[1], vbuf(0));
    st(pre[2], kbuf(1));
  }
  __syncthreads();
  f32x16 sA, sB;
  qk(kbuf(0), sA);
  if (is_special(0)) special_fix(0, sA);
  {
    const float mt = swap_max(lane_max(sA)) * c2;
    m = mt > kInitMax ? mt : kInitMax;
    thr = (m + kSlack) * inv_c2;
  }
  __builtin_amdgcn_s_barrier();  // every wave has read K(0) before its buffer is refilled

  // ---- steady state ------------------------------------------------------------------------
  // Step i: store the staged K(i+2) and V(i+1) (loaded during step i-1) into the buffers of
  // K(i) and V(i-1), start the loads of K(i+3) and V(i+2); S(i+1) = K(i+1) Q^T; softmax of
  // S(i) and O += P V(i).  Stage i uses K/V buffer i%2 and S buffer i%2, so two steps are
  // unrolled with fixed buffers.  A row whose next scores exceed its reference max by more
  // than 2^kSlack sends the remaining stages to the general step, which rescales before the
  // exponentials.
  int i = 0;
  const int fast_end = n_it - 1;
  auto fast_step = [&](auto ph) -> bool {
    constexpr int P = decltype(ph)::value;
    f32x16& sc = P ? sB : sA;
    f32x16& sn = P ? sA : sB;
    if (is_special(i)) special_fix(i, sc);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // K(i+2), V(i+1) staged
    st(stgK, kbuf(P));
    st(stgV, vbuf(P ^ 1));
    ld(stgK, klb, kcb, offK, false, clamp_stage(i + 3));
    ld(stgV, vlb, vcb, offV, true, clamp_stage(i + 2));
    qk(kbuf(P ^ 1), sn);
    softmax_pv(sc, vbuf(P));
    const bool ok = __builtin_amdgcn_ballot_w64(lane_max(sn) > thr) == 0;
    __builtin_amdgcn_s_waitcnt(lgkmcnt_imm(0));  // this step's LDS stores are complete
    __builtin_amdgcn_s_barrier();
    return ok;
  };
  while (i < fast_end) {
    bool ok;
    ok = fast_step(IC<0>{}); if (++i >= fast_end || !ok) break;
    ok = fast_step(IC<1>{}); ++i;
    if (!ok) break;
  }
  f32x16 s_cur = (i & 1) ? sB : sA, s_nxt;

  // ---- general step: the last stage, and every stage after a rescale ----------------------
  for (; i < n_it; ++i) {
    const int r = i & 1;
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    st(stgK, kbuf(r));
    st(stgV, vbuf(r ^ 1));
    ld(stgK, klb, kcb, offK, false, clamp_stage(i + 3));
    ld(stgV, vlb, vcb, offV, true, clamp_stage(i + 2));
    if (is_special(i)) special_fix(i, s_cur);
    const float mt = swap_max(lane_max(s_cur)) * c2;
    if (__builtin_amdgcn_ballot_w64(mt > m + kSlack) != 0) {
      const float mn = mt > m + kSlack ? mt : m;
      const float alpha = __builtin_amdgcn_exp2f(m - mn);
      m = mn;
      thr = (m + kSlack) * inv_c2;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < T::DB; ++db) o[db] *= alpha;
    }
    if (i + 1 < n_it) qk(kbuf(r ^ 1), s_nxt);
    softmax_pv(s_cur, vbuf(r));
    __builtin_amdgcn_s_waitcnt(lgkmcnt_imm(0));
    __builtin_amdgcn_s_barrier();
    s_cur = s_nxt;
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();

  // ---- merge the two key halves, add the live diagonal term, normalise, store -----------
  // Waves w and w^4 hold the same 32 queries over the two key halves.  Wave kp finalises the
  // d-half kp; the other half of its O^T goes to the partner through LDS (slot per wave,
  // two slots per stage buffer; m and l separately).  Register arrays are indexed with
  // compile-time numbers only.
  lsum = swap_add(lsum);
  constexpr int NJH = T::NJH;
  constexpr int DBH = T::DB / 2;
  auto slot = [&](int w) -> float* {
    char* base = w < 2 ? sK0 : (w < 4 ? sK1 : (w < 6 ? sV0 : sV1));
    return (float*)(base + (w & 1) * (NJH * 64 * 4));
  };
  float* mine = slot(wave);
  const float* theirs = slot(wave ^ 4);
  auto give = [&](auto half) {
    constexpr int HF = decltype(half)::value;  // d-half handed to the partner
#pragma unroll
    for (int j = 0; j < NJH; j += 4) {
      const f32x16& src = o[HF * DBH + (j >> 4)];
      const f32x4 v = {src[(j & 15) + 0], src[(j & 15) + 1], src[(j & 15) + 2], src[(j & 15) + 3]};
      *(f32x4*)(mine + (j >> 2) * 256 + lane * 4) = v;  // four values of a lane are contiguous
    }
  };
  if (kp) give(IC<0>{}); else give(IC<1>{});
  sML[(wave * 2 + 0) * 64 + lane] = m;
  sML[(wave * 2 + 1) * 64 + lane] = lsum;
  __syncthreads();
  // The finished d-half of the wave's 32 rows (bf16), in O^T order: entry dbh*4+g4 holds
  // columns dbh*32 + g4*8 + hl*4 .. +3 of the half for row l32.
  bf16x4 outv[DBH * 4];
  float mm_out = 0.0f, ltot_out = 1.0f;
  auto finish = [&](auto half) {
    constexpr int HF = decltype(half)::value;  // d-half finalised here
    // seed rows: the live diagonal term, one more element of the row's softmax
    const float td = qd_seed ? s_live * c2 : -INFINITY;
    const float mb = sML[((wave ^ 4) * 2 + 0) * 64 + lane], lb = sML[((wave ^ 4) * 2 + 1) * 64 + lane];
    const float mm = fmax3(m, mb, td);
    const float fa = __builtin_amdgcn_exp2f(m - mm), fb = __builtin_amdgcn_exp2f(mb - mm);
    const float fd = __builtin_amdgcn_exp2f(td - mm);
    const float ltot = lsum * fa + lb * fb + fd;
    const float inv = 1.0f / ltot;
    mm_out = mm;
    ltot_out = ltot;
#pragma unroll
    for (int dbh = 0; dbh < DBH; ++dbh) {
      const int db = HF * DBH + dbh;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = db * 32 + g4 * 8 + hl * 4;
        const f32x4 tv = *(const f32x4*)(theirs + (dbh * 4 + g4) * 256 + lane * 4);
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[db][g4 * 4 + e] * fa + tv[e] * fb;
        if (block_seeded) {
          typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
          const u32x2 raw = *(const __attribute__((address_space(3))) u32x2*)(
              dg + l32 * T::ROW + ((((d0 >> 3) ^ k_swz<T::ROW>(l32))) << 4) + (d0 & 7) * 2);
          v[0] += fd * bf16_lo(raw[0]);
          v[1] += fd * bf16_hi(raw[0]);
          v[2] += fd * bf16_lo(raw[1]);
          v[3] += fd * bf16_hi(raw[1]);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] *= inv;
        outv[dbh * 4 + g4] = __builtin_convertvector(v, bf16x4);
      }
    }
  };
  if (kp) finish(IC<1>{}); else finish(IC<0>{});
  if (p.lse && hl == 0 && kp == 0 && qw + l32 < L)
    p.lse[((int64_t)b * p.Hq + h) * L + qw + l32] = (mm_out + __builtin_amdgcn_logf(ltot_out)) * kLn2;
  // Stores: the half-rows go through an LDS tile (rows padded to keep 16-byte alignment and
  // spread banks) so that each global store writes whole 128-byte lines of consecutive
  // columns instead of 8-byte pieces of 32 rows.
  __syncthreads();  // every wave has read its partner's merge slot
  constexpr int TROW = D + 16;                     // bytes per tile row: D/2 columns + pad
  static_assert(32 * TROW <= NJH * 64 * 4, "the output tile must fit a merge slot");
  lds_t* const tile = (lds_t*)slot(wave);          // this wave's slot, now free
#pragma unroll
  for (int dbh = 0; dbh < DBH; ++dbh)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *(__attribute__((address_space(3))) bf16x4*)(tile + l32 * TROW + (dbh * 32 + g4 * 8 + hl * 4) * 2) = outv[dbh * 4 + g4];
  constexpr int CPR = D / 16;          // 16-byte chunks per half-row
  constexpr int NRD = 32 * CPR / 64;   // reads (and stores) per lane
  __bf16* const obase = p.out + b * p.q_sb + h * p.q_sh + kp * (D / 2);
#pragma unroll
  for (int it = 0; it < NRD; ++it) {
    const int idx = it * 64 + lane, row = idx / CPR, ch = idx % CPR;
    const u32x4 v = *(const __attribute__((address_space(3))) u32x4*)(tile + row * TROW + ch * 16);
    if (qw + row < L) *(u32x4*)(obase + (int64_t)(qw + row) * p.q_sl + ch * 8) = v;
  }
}

// ----------------------------------------------------------------------------------------
// fp32 path: one wave per 64 queries of one (b, h); each lane owns one query row and walks
// the keys with an exact online softmax.  Same override / leave-one-out rule as above.
// ----------------------------------------------------------------------------------------
struct ParamsF {
  const float* q;
  const float* kl;
  const float* vl;
  const float* kc;
  const float* vc;
  const int32_t* seed_idx;
  const int32_t* n_seed;
  float* out;
  float* lse;
  int B, Hq, Hkv, L, max_seeds, group, n_qt;
  float c2;
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

template <int D>
__global__ __launch_bounds__(64, 1) void cover_attn_f32_kernel(const ParamsF p) {
  constexpr int TK = 32;  // keys per LDS tile
  __shared__ __attribute__((aligned(16))) float ks[TK][D];
  __shared__ __attribute__((aligned(16))) float vs[TK][D];
  __shared__ uint32_t bits[COVER_MAX_L / 32];
  const int lane = threadIdx.x;
  const int qt = blockIdx.x % p.n_qt;
  const int bh = blockIdx.x / p.n_qt;
  const int h = bh % p.Hq, b = bh / p.Hq;
  const int g = h / p.group;
  const int L = p.L;
  const int64_t kvoff = b * p.kv_sb + g * p.kv_sh;

  const int nwords = (L + 31) >> 5;
  for (int w = lane; w < nwords; w += 64) bits[w] = 0u;
  __syncthreads();
  int ns = 0;
  if (p.max_seeds > 0) {
    ns = p.n_seed[b];
    ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
  }
  for (int t = lane; t < ns; t += 64) {
    const int j = p.seed_idx[(int64_t)b * p.max_seeds + t];
    if ((unsigned)j < (unsigned)L) atomicOr(&bits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();

  const int qi = qt * 64 + lane;
  const int qc = min(qi, L - 1);
  const float* qrow = p.q + b * p.q_sb + h * p.q_sh + (int64_t)qc * p.q_sl;
  float qv[D];
#pragma unroll
  for (int k = 0; k < D; k += 4) *(f32x4*)(qv + k) = *(const f32x4*)(qrow + k);
  const bool seed = qi < L && ((bits[qc >> 5] >> (qc & 31)) & 1u);
  float s_live = 0.0f;
  if (seed) {
    const float* kr = p.kl + kvoff + (int64_t)qc * p.kv_sl;
    for (int k = 0; k < D; ++k) s_live = __builtin_fmaf(qv[k], kr[k], s_live);
  }
  float m = kInitMax, l = 0.0f;
  float o[D];
#pragma unroll
  for (int k = 0; k < D; ++k) o[k] = 0.0f;

  for (int k0 = 0; k0 < L; k0 += TK) {
    __syncthreads();
    for (int idx = lane; idx < TK * D / 4; idx += 64) {
      const int row = idx / (D / 4), c = idx % (D / 4);
      const int key = min(k0 + row, L - 1);
      const bool sd = (bits[key >> 5] >> (key & 31)) & 1u;
      const int64_t off = kvoff + (int64_t)key * p.kv_sl + c * 4;
      *(f32x4*)(&ks[row][c * 4]) = *(const f32x4*)((sd ? p.kc : p.kl) + off);
      *(f32x4*)(&vs[row][c * 4]) = *(const f32x4*)((sd ? p.vc : p.vl) + off);
    }
    __syncthreads();
    const int kn = min(TK, L - k0);
    for (int j = 0; j < kn; ++j) {
      const int key = k0 + j;
      const bool diag = seed && key == qi;
      float s = 0.0f;
      if (diag) {
        s = s_live;
      } else {
#pragma unroll
        for (int k = 0; k < D; ++k) s = __builtin_fmaf(qv[k], ks[j][k], s);
      }
      const float t = s * p.c2;
      if (t > m) {
        const float alpha = __builtin_amdgcn_exp2f(m - t);
        l *= alpha;
#pragma unroll
        for (int k = 0; k < D; ++k) o[k] *= alpha;
        m = t;
      }
      const float pw = __builtin_amdgcn_exp2f(t - m);
      l += pw;
      if (diag) {
        const float* vr = p.vl + kvoff + (int64_t)qi * p.kv_sl;
        for (int k = 0; k < D; ++k) o[k] = __builtin_fmaf(pw, vr[k], o[k]);
      } else {
#pragma unroll
        for (int k = 0; k < D; ++k) o[k] = __builtin_fmaf(pw, vs[j][k], o[k]);
      }
    }
  }
  if (qi < L) {
    const float inv = 1.0f / l;
    float* orow = p.out + b * p.q_sb + h * p.q_sh + (int64_t)qi * p.q_sl;
#pragma unroll
    for (int k = 0; k < D; k += 4) {
      f32x4 v = {o[k] * inv, o[k + 1] * inv, o[k + 2] * inv, o[k + 3] * inv};
      *(f32x4*)(orow + k) = v;
    }
    if (p.lse) p.lse[((int64_t)b * p.Hq + h) * L + qi] = (m + __builtin_amdgcn_logf(l)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t stream) {
  Params p;
  p.q = (const __bf16*)a.q;
  p.kl = (const __bf16*)a.k_live;
  p.vl = (const __bf16*)a.v_live;
  p.kc = (const __bf16*)a.k_cache;
  p.vc = (const __bf16*)a.v_cache;
  p.seed_idx = a.seed_idx;
  p.n_seed = a.n_seed;
  p.out = (__bf16*)a.out;
  p.lse = a.lse;
  p.B = a.B; p.Hq = a.Hq; p.Hkv = a.Hkv; p.L = a.L; p.max_seeds = a.max_seeds;
  p.group = a.Hq / a.Hkv;
  p.n_qt = (a.L + kBM - 1) / kBM;
  const int64_t nwg = (int64_t)a.B * a.Hq * p.n_qt;
  p.xcd_slots = (nwg % 8 == 0) ? (int)(nwg / 8) : 0;
  p.c2 = a.scale * 1.44269504088896341f;
  p.q_sb = a.q_sb; p.q_sh = a.q_sh; p.q_sl = a.q_sl;
  p.kv_sb = a.kv_sb; p.kv_sh = a.kv_sh; p.kv_sl = a.kv_sl;
  if (nwg > 0x7fffffff || a.d != 64) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(cover_attn_bf16_kernel<64>, dim3((unsigned)nwg), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t stream) {
  ParamsF p;
  p.q = (const float*)a.q;
  p.kl = (const float*)a.k_live;
  p.vl = (const float*)a.v_live;
  p.kc = (const float*)a.k_cache;
  p.vc = (const float*)a.v_cache;
  p.seed_idx = a.seed_idx;
  p.n_seed = a.n_seed;
  p.out = (float*)a.out;
  p.lse = a.lse;
  p.B = a.B; p.Hq = a.Hq; p.Hkv = a.Hkv; p.L = a.L; p.max_seeds = a.max_seeds;
  p.group = a.Hq / a.Hkv;
  p.n_qt = (a.L + 63) / 64;
  p.c2 = a.scale * 1.44269504088896341f;
  p.q_sb = a.q_sb; p.q_sh = a.q_sh; p.q_sl = a.q_sl;
  p.kv_sb = a.kv_sb; p.kv_sh = a.kv_sh; p.kv_sl = a.kv_sl;
  const int64_t nwg = (int64_t)a.B * a.Hq * p.n_qt;
  if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (a.d == 128)
    hipLaunchKernelGGL(cover_attn_f32_kernel<128>, dim3((unsigned)nwg), dim3(64), 0, stream, p);
  else
    hipLaunchKernelGGL(cover_attn_f32_kernel<64>, dim3((unsigned)nwg), dim3(64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
