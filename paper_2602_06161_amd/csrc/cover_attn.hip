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
// bf16 kernel design (one workgroup = 4 waves = 128 queries of one (b, h)):
//   * Transposed products keep every query row inside one lane pair:
//       S^T = K Q^T   (v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q from registers)
//       O^T += V^T P^T (A = V^T read with ds_read_b64_tr_b16, B = P straight from the S^T
//                       registers after exp2 and bf16 packing)
//     so row max / row sum / rescale are lane-local plus one v_permlane32_swap.
//   * Wave w owns 64 queries (two 32-query blocks, half (w & 1) of the tile) and the keys
//     of parity (w >> 1): K/V operands read from LDS feed two MFMAs each, halving LDS
//     traffic relative to 32 queries per wave; the two key halves are merged at the end.
//   * K/V stages of 64 keys are double buffered in LDS; each row's source (live or cache)
//     is chosen while loading from a per-sequence seed bitmap in LDS.
//   * Lazy softmax rescaling: a row's reference max moves only when the row max grows by
//     more than 2^8, so most tiles skip the O rescale (exact: O and l share the reference).
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

constexpr int kThreads = 256;
constexpr int kBM = 128;             // queries per workgroup
constexpr int kStageKeys = 64;       // keys per pipeline stage = two 32-key wave tiles
constexpr float kSlack = 20.0f;      // rescale only when a row max grows by > 2^20
constexpr float kInitMax = -1.0e30f; // finite "no key seen yet" reference max
constexpr float kLn2 = 0.693147180559945309f;

template <int D>
struct Tile {
  static constexpr int CH = D / 8;                  // 16-byte chunks per bf16 row
  static constexpr int KS = D / 16;                 // k-steps of S^T = K Q^T
  static constexpr int DB = D / 32;                 // 32-row blocks of O^T
  static constexpr int ROW = D * 2;                 // bytes per row
  static constexpr int SBYTES = kStageKeys * ROW;   // one K or V stage of 64 rows
  static constexpr int LOADS = kStageKeys * CH / kThreads;  // 16-B chunks per thread per tensor
  static constexpr int RPP = kThreads / CH;         // rows per load pass
  static constexpr int OFF_K0 = 0, OFF_K1 = SBYTES, OFF_V0 = 2 * SBYTES, OFF_V1 = 3 * SBYTES;
  static constexpr int MERGE = (DB * 16 + 2) * 64 * 4;  // per-wave merge slot (after the loop)
  static constexpr int OFF_DIAG = ((4 * SBYTES > 4 * MERGE ? 4 * SBYTES : 4 * MERGE) + 1023) / 1024 * 1024;
  static constexpr int DIAG = 32 * ROW;             // per wave: live V rows of its diagonal block
  static constexpr int OFF_BITS = OFF_DIAG + 4 * DIAG;
  static constexpr int BYTES = OFF_BITS + COVER_MAX_L / 8;
  static_assert(LOADS * kThreads == kStageKeys * CH, "stage must split evenly");
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

// LDS swizzles.  K rows are read 16 rows per LDS cycle at one logical chunk (b128 reads), so
// the chunk index is XOR-ed with the row (D = 128) or with row/2 (D = 64, two rows per
// 256-byte bank window).  V rows are read by transpose reads, 4 rows x 2 chunks per 16-lane
// group, spread by XOR-ing with 2*(row%4).
template <int ROW>
__device__ __forceinline__ uint32_t k_off(int row, int c) {
  const int sw = (ROW == 256) ? (row & 15) : ((row >> 1) & 7);
  return row * ROW + ((c ^ sw) << 4);
}
template <int ROW>
__device__ __forceinline__ uint32_t v_off(int row, int c) {
  return row * ROW + ((c ^ ((row & 3) << 1)) << 4);
}
// byte address of element `col` of V row `row`
template <int ROW>
__device__ __forceinline__ uint32_t v_elem(int row, int col) {
  return v_off<ROW>(row, col >> 3) + ((col & 7) << 1);
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 lds_read16(const lds_t* p) { return *(const __attribute__((address_space(3))) u32x4*)p; }
__device__ __forceinline__ void lds_write16(lds_t* p, u32x4 v) { *(__attribute__((address_space(3))) u32x4*)p = v; }

// A operand of O^T += V^T P^T for 16 keys starting at stage row `row0`, d-block `db`:
// lane (G = lane/16, i = lane%16) receives V[row0 + 4*(G/2) + {0..3, 8..11}][db*32 + 16*(G%2) + i].
template <int ROW>
__device__ __forceinline__ bf16x8 v_operand(const lds_t* vbase, int row0, int db, int lane) {
  const int G = lane >> 4, i = lane & 15;
  const int row = row0 + 4 * (G >> 1) + (i >> 2);
  const int col = db * 32 + 16 * (G & 1) + 4 * (i & 3);
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(vbase + v_elem<ROW>(row, col)));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(vbase + v_elem<ROW>(row + 8, col)));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
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
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int N>
struct IC {
  static constexpr int value = N;
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void cover_attn_bf16_kernel(const Params p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(16))) char smem_raw[T::BYTES];
  lds_t* smem = (lds_t*)smem_raw;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qh = wave & 1;   // which 64-query half of the workgroup tile
  const int kp = wave >> 1;  // which key parity (32-key tile kp of every 64-key stage)
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
  const __bf16* qbase = p.q + b * p.q_sb + h * p.q_sh;
  const int64_t kvoff = b * p.kv_sb + g * p.kv_sh;

  // ---- Q fragments (B operand of S^T = K Q^T): query l32 of block qb, d-chunk 2*ks + hl
  bf16x8 qreg[2][T::KS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int qi = min(q0 + qh * 64 + qb * 32 + l32, L - 1);
    const __bf16* qrow = qbase + (int64_t)qi * p.q_sl + hl * 8;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) qreg[qb][ks] = *(const bf16x8*)(qrow + ks * 16);
  }

  // ---- seed bitmap of this sequence ---------------------------------------------------
  // The seed list is read speculatively (all max_seeds entries) together with its length.
  uint32_t* bits = (uint32_t*)(smem_raw + T::OFF_BITS);
  const int nwords = (L + 31) >> 5;
  const int64_t sbase = (int64_t)b * p.max_seeds;
  int ns = 0;
  if (p.max_seeds > 0) ns = p.n_seed[b];
  const int sj0 = tid < p.max_seeds ? p.seed_idx[sbase + tid] : -1;
  for (int w = tid; w < nwords; w += kThreads) bits[w] = 0u;
  __syncthreads();
  ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
  if (tid < ns && (unsigned)sj0 < (unsigned)L) atomicOr(&bits[sj0 >> 5], 1u << (sj0 & 31));
  for (int t = tid + kThreads; t < ns; t += kThreads) {
    const int j = p.seed_idx[sbase + t];
    if ((unsigned)j < (unsigned)L) atomicOr(&bits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  auto is_seed = [&](int j) -> bool { return (bits[j >> 5] >> (j & 31)) & 1u; };

  // ---- stage order --------------------------------------------------------------------
  // The two stages holding this tile's diagonal (2qt, 2qt+1) and a ragged last stage are
  // "special" and processed last, so all earlier stages run through one branch-free loop.
  const int n_it = (L + kStageKeys - 1) / kStageKeys;
  constexpr int kNone = 0x7fffffff;
  // Does any query of this tile (rows q0 .. q0+127) have a seed?  Same answer in every lane.
  uint32_t tile_bits = 0;
#pragma unroll
  for (int w = 0; w < kBM / 32; ++w) tile_bits |= (q0 / 32 + w < nwords) ? bits[q0 / 32 + w] : 0u;
  const bool tile_seeded = __builtin_amdgcn_readfirstlane(tile_bits) != 0u;
  int sp0 = tile_seeded ? 2 * qt : kNone;
  int sp1 = (tile_seeded && 2 * qt + 1 < n_it) ? 2 * qt + 1 : kNone;
  int sp2 = (L % kStageKeys != 0 && (n_it - 1 != sp0) && (n_it - 1 != sp1)) ? n_it - 1 : kNone;
  // sorted: sp0 < sp1 < sp2 whenever present; compact missing entries to the end
  if (sp0 == kNone) { sp0 = sp1; sp1 = sp2; sp2 = kNone; }
  if (sp0 == kNone) { sp0 = sp1; sp1 = kNone; }
  if (sp1 == kNone) { sp1 = sp2; sp2 = kNone; }
  const int nsp = (sp0 != kNone) + (sp1 != kNone) + (sp2 != kNone);
  const int n_reg = n_it - nsp;
  auto seq = [=](int i) -> int {  // i-th stage processed
    if (i >= n_it) i = n_it - 1;
    if (i >= n_reg) {
      const int k = i - n_reg;
      return k == 0 ? sp0 : (k == 1 ? sp1 : sp2);
    }
    int j = i;
    if (j >= sp0) ++j;
    if (j >= sp1) ++j;
    if (j >= sp2) ++j;
    return j;
  };

  // ---- stage loader: 64 rows of K or V (global -> registers -> LDS) --------------------
  // Each row comes from the cache if its position is a seed, else from the live tensor.
  // Thread tid loads chunk (tid % CH) of rows (tid / CH) + RPP * i.  Rows past the end read
  // row L-1 (never used unmasked).
  const int lrow = tid / T::CH, lcol = tid % T::CH;
  const int64_t lane_off = kvoff + (int64_t)lrow * p.kv_sl + lcol * 8;
  u32x4 kst[T::LOADS], vst[T::LOADS];
  auto gload = [&](u32x4* regs, const __bf16* live, const __bf16* cache, int stage) {
    const int kb = stage * kStageKeys;
    // seed bits of the stage's 64 rows, then of this thread's rows lrow + RPP * i
    const uint32_t w0 = __builtin_amdgcn_readfirstlane(bits[kb >> 5]);
    const uint32_t w1 = (kb >> 5) + 1 < nwords ? __builtin_amdgcn_readfirstlane(bits[(kb >> 5) + 1]) : 0u;
    const uint64_t mrow = ((((uint64_t)w1) << 32) | w0) >> lrow;
#pragma unroll
    for (int i = 0; i < T::LOADS; ++i) {
      const int key = min(kb + lrow + T::RPP * i, L - 1);
      const bool sd = (mrow >> (T::RPP * i)) & 1u;  // rows past L: live row L-1, masked later
      const __bf16* src = sd ? cache : live;
      regs[i] = *(const u32x4*)(src + lane_off + (int64_t)(key - lrow) * p.kv_sl);
    }
  };
  auto kstore = [&](lds_t* buf) {
#pragma unroll
    for (int i = 0; i < T::LOADS; ++i) lds_write16(buf + k_off<T::ROW>(lrow + T::RPP * i, lcol), kst[i]);
  };
  auto vstore = [&](lds_t* buf) {
#pragma unroll
    for (int i = 0; i < T::LOADS; ++i) lds_write16(buf + v_off<T::ROW>(lrow + T::RPP * i, lcol), vst[i]);
  };
  lds_t* const K0 = smem + T::OFF_K0;
  lds_t* const K1 = smem + T::OFF_K1;
  lds_t* const V0 = smem + T::OFF_V0;
  lds_t* const V1 = smem + T::OFF_V1;

  u32x4 kst1[T::LOADS];
  gload(kst, p.kl, p.kc, seq(0));
  gload(vst, p.vl, p.vc, seq(0));
  gload(kst1, p.kl, p.kc, seq(1));

  // ---- diagonal set-up ------------------------------------------------------------------
  // Query block kp of this wave (queries qd0 .. qd0+31) has its diagonal in this wave's
  // 32-key tile of stage itd = qd0 / 64.  In S^T the diagonal entry of query nq sits in lane
  // half (nq/4)%2, register (nq/8)*4 + nq%4.
  const int qd0 = q0 + qh * 64 + kp * 32;
  const int itd = qd0 / kStageKeys;
  const bool holds_diag = hl == ((l32 >> 2) & 1);
  const int rd = ((l32 >> 3) << 2) | (l32 & 3);
  const bool qd_seed = (qd0 + l32) < L && is_seed(qd0 + l32);  // this lane's diagonal query
  const bool diag_seed = holds_diag && qd_seed;
  const bool wave_diag = __builtin_amdgcn_ballot_w64(qd_seed) != 0;
  lds_t* const dg = smem + T::OFF_DIAG + wave * T::DIAG;
  float s_live = 0.0f;  // raw score q_i . k_live_i of this lane's diagonal query
  if (wave_diag) {
    const int qr = min(qd0 + l32, L - 1);
    const uint32_t* krow = (const uint32_t*)(p.kl + kvoff + (int64_t)qr * p.kv_sl + hl * 8);
    float acc = 0.0f;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) {
      const u32x4 kv = *(const u32x4*)(krow + ks * 8);
      const u32x4 qv = __builtin_bit_cast(u32x4, kp ? qreg[1][ks] : qreg[0][ks]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc = __builtin_fmaf(bf16_lo(qv[e]), bf16_lo(kv[e]), acc);
        acc = __builtin_fmaf(bf16_hi(qv[e]), bf16_hi(kv[e]), acc);
      }
    }
    s_live = swap_add(acc);
    // live V rows of the block's queries, row-major, for the epilogue
#pragma unroll
    for (int i = 0; i < 32 * T::CH / 64; ++i) {
      const int idx = lane + i * 64;
      const int row = idx / T::CH, c = idx % T::CH;
      const int vr = min(qd0 + row, L - 1);
      lds_write16(dg + row * T::ROW + c * 16, *(const u32x4*)(p.vl + kvoff + (int64_t)vr * p.kv_sl + c * 8));
    }
  }

  // ---- pipeline prologue: K(seq 0), V(seq 0), K(seq 1) resident; S(seq 0) computed ---------
  kstore(K0);
  vstore(V0);
#pragma unroll
  for (int j = 0; j < T::LOADS; ++j) kst[j] = kst1[j];
  kstore(K1);
  __syncthreads();

  const float c2 = p.c2;
  auto qk = [&](const lds_t* kb, f32x16* s) {
    s[0] = (f32x16){};
    s[1] = (f32x16){};
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, lds_read16(kb + k_off<T::ROW>(kp * 32 + l32, 2 * ks + hl)));
      s[0] = mfma(a, qreg[0][ks], s[0]);
      s[1] = mfma(a, qreg[1][ks], s[1]);
    }
  };
  // keys of this wave's tile of `stage` past L, and the seed rows' own (cached) column, get
  // no weight; the live diagonal term is added in the epilogue
  auto special_fix = [&](int stage, f32x16* s) {
    if (stage * kStageKeys + kStageKeys > L) {
      const int kbase = stage * kStageKeys + kp * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool ok = kbase + ((r >> 2) << 3) + hl * 4 + (r & 3) < L;
        s[0][r] = ok ? s[0][r] : -INFINITY;
        s[1][r] = ok ? s[1][r] : -INFINITY;
      }
    }
    if (wave_diag && stage == itd) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool hit = diag_seed && r == rd;
        s[0][r] = (hit && kp == 0) ? -INFINITY : s[0][r];
        s[1][r] = (hit && kp == 1) ? -INFINITY : s[1][r];
      }
    }
  };
  auto rowmax = [&](const f32x16* s, float* mt) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float mx = s[qb][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmax2(mx, s[qb][r]);
      mt[qb] = swap_max(mx) * c2;
    }
  };

  float m[2], lsum[2] = {0.0f, 0.0f};
  f32x16 o[2][T::DB];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int db = 0; db < T::DB; ++db) o[qb][db] = (f32x16){};

  f32x16 s_cur[2], s_nxt[2];
  qk(K0, s_cur);
  special_fix(seq(0), s_cur);
  {
    // the first tile fixes each row's reference max (no accumulator to rescale yet)
    float mt[2];
    rowmax(s_cur, mt);
    m[0] = mt[0] > kInitMax ? mt[0] : kInitMax;
    m[1] = mt[1] > kInitMax ? mt[1] : kInitMax;
  }
  __syncthreads();  // every wave has read K(seq 0) before iteration 0 overwrites its buffer

  // softmax of S(seq i) into bf16 P (row sums accumulated), then O^T += V^T P^T
  auto softmax_pv = [&](const lds_t* vcur) {
    bf16x8 pk[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const float nm = -m[qb];
      f32x16 pr;
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s_cur[qb][r], c2, nm));
      float ls = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) ls += pr[r];
      lsum[qb] += ls;
      pk[qb][0] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 0, 1, 2, 3, 4, 5, 6, 7), bf16x8);
      pk[qb][1] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 8, 9, 10, 11, 12, 13, 14, 15), bf16x8);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int db = 0; db < T::DB; ++db) {
        const bf16x8 a = v_operand<T::ROW>(vcur, kp * 32 + 16 * kk, db, lane);
        o[0][db] = mfma(a, pk[0][kk], o[0][db]);
        o[1][db] = mfma(a, pk[1][kk], o[1][db]);
      }
    }
  };

  // ---- steady state: regular stages, no masking, no diagonal, no rescale ----------------
  // A row whose max grows by more than 2^kSlack over its reference leaves for the general
  // loop below, which rescales.
  int i = 0;
  for (; i < n_reg; ++i) {
    float mt[2];
    rowmax(s_cur, mt);
    if (__builtin_amdgcn_ballot_w64((mt[0] > m[0] + kSlack) || (mt[1] > m[1] + kSlack)) != 0) break;
    gload(kst, p.kl, p.kc, seq(i + 2));
    gload(vst, p.vl, p.vc, seq(i + 1));
    qk((i & 1) ? K0 : K1, s_nxt);
    softmax_pv((i & 1) ? V1 : V0);
    kstore((i & 1) ? K1 : K0);        // K(seq i+2) replaces K(seq i)
    vstore((i & 1) ? V0 : V1);  // V(seq i+1) replaces V(seq i-1)
    __syncthreads();
    s_cur[0] = s_nxt[0];
    s_cur[1] = s_nxt[1];
  }
  // ---- general step: special tiles, and regular tiles after a rescale ------------------
  auto general_step = [&](int i, bool special) {
    const bool more = i + 1 < n_it;
    if (more) {
      gload(kst, p.kl, p.kc, seq(i + 2));
      gload(vst, p.vl, p.vc, seq(i + 1));
    }
    if (special) special_fix(seq(i), s_cur);
    float mt[2];
    rowmax(s_cur, mt);
    if (__builtin_amdgcn_ballot_w64((mt[0] > m[0] + kSlack) || (mt[1] > m[1] + kSlack)) != 0) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const float mn = mt[qb] > m[qb] + kSlack ? mt[qb] : m[qb];
        const float alpha = __builtin_amdgcn_exp2f(m[qb] - mn);
        m[qb] = mn;
        lsum[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < T::DB; ++db) o[qb][db] *= alpha;
      }
    }
    if (more) qk((i & 1) ? K0 : K1, s_nxt);
    softmax_pv((i & 1) ? V1 : V0);
    if (more) {
      kstore((i & 1) ? K1 : K0);
      vstore((i & 1) ? V0 : V1);
    }
    __syncthreads();
    s_cur[0] = s_nxt[0];
    s_cur[1] = s_nxt[1];
  };
  // regular stages left after a rescale (rare)
  for (; i < n_reg; ++i) general_step(i, false);
  // the (at most three) special stages, straight-line
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    if (i < n_it) {
      general_step(i, true);
      ++i;
    }
  }

  // ---- merge the two key parities, add the live diagonal term, normalise, store ---------
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) lsum[qb] = swap_add(lsum[qb]);
  // Wave kp finalises its query block kp; the other block goes to the partner wave (w ^ 2).
  // Register arrays are indexed with compile-time block numbers only.
  float* mine = (float*)(smem_raw + wave * T::MERGE);
  const float* theirs = (const float*)(smem_raw + (wave ^ 2) * T::MERGE);
  constexpr int NJ = T::DB * 16;
  auto give = [&](auto qo) {
    constexpr int QO = decltype(qo)::value;
#pragma unroll
    for (int j = 0; j < NJ; ++j) mine[j * 64 + lane] = o[QO][j >> 4][j & 15];
    mine[NJ * 64 + lane] = m[QO];
    mine[(NJ + 1) * 64 + lane] = lsum[QO];
  };
  if (kp) give(IC<0>{}); else give(IC<1>{});
  __syncthreads();
  auto finish = [&](auto qf_) {
    constexpr int QF = decltype(qf_)::value;
    // seed rows: the live diagonal term, one more element of the row's softmax
    const float td = qd_seed ? s_live * c2 : -INFINITY;
    const float ma = m[QF], la = lsum[QF];
    const float mb = theirs[NJ * 64 + lane], lb = theirs[(NJ + 1) * 64 + lane];
    const float mm = fmax2(fmax2(ma, mb), td);
    const float fa = __builtin_amdgcn_exp2f(ma - mm), fb = __builtin_amdgcn_exp2f(mb - mm);
    const float fd = __builtin_amdgcn_exp2f(td - mm);
    const float ltot = la * fa + lb * fb + fd;
    const float inv = 1.0f / ltot;
    const int qf = qd0 + l32;
    if (qf < L) {
      __bf16* orow = p.out + b * p.q_sb + h * p.q_sh + (int64_t)qf * p.q_sl;
#pragma unroll
      for (int db = 0; db < T::DB; ++db) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int d0 = db * 32 + g4 * 8 + hl * 4;
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int j = db * 16 + g4 * 4 + e;
            v[e] = o[QF][db][g4 * 4 + e] * fa + theirs[j * 64 + lane] * fb;
          }
          if (wave_diag) {
            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
            const u32x2 raw = *(const __attribute__((address_space(3))) u32x2*)(dg + l32 * T::ROW + d0 * 2);
            v[0] += fd * bf16_lo(raw[0]);
            v[1] += fd * bf16_hi(raw[0]);
            v[2] += fd * bf16_lo(raw[1]);
            v[3] += fd * bf16_hi(raw[1]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= inv;
          *(bf16x4*)(orow + d0) = __builtin_convertvector(v, bf16x4);
        }
      }
      if (p.lse && hl == 0)
        p.lse[((int64_t)b * p.Hq + h) * L + qf] = (mm + __builtin_amdgcn_logf(ltot)) * kLn2;
    }
  };
  if (kp) finish(IC<1>{}); else finish(IC<0>{});
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
  if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (a.d == 128)
    hipLaunchKernelGGL(cover_attn_bf16_kernel<128>, dim3((unsigned)nwg), dim3(kThreads), 0, stream, p);
  else
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
