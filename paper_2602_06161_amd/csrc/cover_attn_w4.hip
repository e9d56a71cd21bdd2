// COVER attention on gfx950, head dimension 128, bf16: four waves per workgroup, one per SIMD.
//
// Same operation as the eight-wave kernel (arXiv 2602.06161, Sec. 5.1 "KV cache override" and
// "Diagonal correction"; App. B): for query row i of batch row b with seed set S_b,
//   K'_j = k_cache_j if j in S_b else k_live_j (V' likewise); row i attends to K' except that a
//   seed row sees its own live key/value on the diagonal; out_i = softmax(scale q_i K^(i)) V^(i).
// The diagonal is handled as in the eight-wave kernel: the cached diagonal score of a seed row
// gets no weight in the main loop, and the live diagonal term exp(scale q_i.k_live_i) v_live_i
// joins the row's softmax in the epilogue (exactly the leave-one-out row of App. B.1, with no
// division by the closed form's r_i).
//
// Layout (one workgroup = 128 queries of one (b, h); wave w: query block qb = w & 1 of 64
// queries, key half kh = w >> 1 of every 64-key stage):
//   * S^T = K Q^T per 32-query tile (v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q from
//     AGPRs) and O^T += V^T P^T (A = V^T by ds_read_b64_tr_b16, B = P from the S^T registers).
//     A wave owns two 32-query tiles, so every K or V^T operand read from LDS feeds two MFMAs:
//     a stage costs the workgroup 64 KiB of LDS reads (the transposing V read delivers about a
//     third of the bandwidth of a plain 16-byte read), not 128 KiB.
//   * The 128 O^T accumulators per lane and Q live in AGPRs (one wave per SIMD has 512
//     registers); S, P and the operands read from LDS stay in VGPRs.
//   * Every global load goes straight to LDS (global_load_lds_dwordx4): the seed list, Q (read
//     into registers once), the live rows of a seeded tile's diagonal (with the last step, into
//     the Q area), and K/V stages in three buffers each, issued two stages ahead and
//     spread between the MFMAs (a burst of them stalls the issuing wave on the vector-memory
//     queue).  A stage is loaded from the live tensors through one scalar base; the rows that
//     need another source (seed rows from the cache, rows of a ragged last stage) are loaded
//     again one step later by exec-masked loads, only in the stages that have such rows (a
//     scalar window of per-stage flags decides, with one scalar test per step).
//   * Softmax without a running max: every row keeps the reference max of its first stage.
//     A lane's per-stage probability sum above 2^24 (or not finite) flags the workgroup, which
//     then recomputes its tile with an exact per-stage rescaling pass.  The flag never fires
//     unless a later score exceeds the first stage's maximum by more than 24 in log2 units.
//   * Waves w and w ^ 2 hold the same queries over the two key halves; they exchange one
//     32-query tile each through LDS at the end, so each wave finishes 32 complete rows.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) char lds_t;
typedef __attribute__((address_space(1))) const char gmem_t;

constexpr int kD = 128;
constexpr int kRow = 2 * kD;                 // bytes per K/V/Q row
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = 128;                     // queries per workgroup
constexpr int kStage = 64;                   // keys per stage
constexpr int kSBytes = kStage * kRow;       // one K or V stage buffer (16 KiB)
constexpr int kLoads = kSBytes / 1024 / kWaves;  // 1-KiB loads per wave per stage buffer
constexpr int kKS = kD / 16;                 // k-steps of S^T = K Q^T
constexpr int kDB = kD / 32;                 // 32-row blocks of O^T
constexpr int kSeedsLds = kThreads;          // seed positions staged in LDS (more: read directly)
constexpr float kInitMax = -1.0e30f;         // finite "no key seen yet" reference max
constexpr float kBig = 16777216.0f;          // 2^24
constexpr float kLn2 = 0.693147180559945309f;
static_assert(kLoads == 4, "a stage gives every wave four 1-KiB loads");

// s_waitcnt immediates that wait for vmcnt <= n only (lgkmcnt and expcnt untouched)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xf00; }
// at the top of a step the eight loads of the previous step may stay in flight
constexpr int kWaitStep = vmcnt_imm(2 * kLoads);

struct Params4 {
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

// LDS swizzles (64 banks of 4 bytes).  K and Q rows: the 16-byte chunk index is XOR-ed with
// row % 16, so the 32 rows of one b128 operand read spread over all banks.  V rows: the chunk
// index is XOR-ed with 4 * (row % 4), so one transposing read (8 rows x 64 bytes) covers every
// bank exactly twice.
__device__ __forceinline__ int k_swz(int row) { return row & 15; }
__device__ __forceinline__ int v_swz(int row) { return (row & 3) << 2; }
__device__ __forceinline__ uint32_t k_off(int row, int c) { return row * kRow + ((c ^ k_swz(row)) << 4); }
__device__ __forceinline__ uint32_t v_elem(int row, int col) {
  return row * kRow + (((col >> 3) ^ v_swz(row)) << 4) + ((col & 7) << 1);
}

// The MFMAs are written as inline assembly so that the register class of every operand is
// fixed: S in VGPRs (read by the softmax), O and Q in AGPRs.  The compiler does not see these
// as MFMAs, so the few places where VALU code reads an MFMA result soon after it was written
// wait explicitly (mfma_drain), and VALU-written operands are separated from their MFMA
// (valu_to_mfma).
__device__ __forceinline__ void mfma_first(f32x16& d, bf16x8 a, bf16x8 qb) {  // d = a q
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(qb));
}
__device__ __forceinline__ void mfma_v(f32x16& d, bf16x8 a, bf16x8 qb) {  // d += a q (VGPR)
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "a"(qb));
}
__device__ __forceinline__ void mfma_a(f32x16& d, bf16x8 a, bf16x8 b) {  // d += a b (AGPR)
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(d) : "v"(a), "v"(b));
}
// wait until every issued MFMA has written its result (the 8-pass 32x32x16 MFMA needs at
// most 18 wait states before a dependent VALU read; 3 x 8 are given)
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory"); }
// VALU-written operands need 2 wait states before an MFMA reads them; tying the nop to the
// operand orders it after the write and before the read
__device__ __forceinline__ void valu_to_mfma(bf16x8& x) { asm("s_nop 1" : "+v"(x)); }
__device__ __forceinline__ u32x4 lds_read16(const lds_t* p) {
  return *(const __attribute__((address_space(3))) u32x4*)p;
}
__device__ __forceinline__ i16x4 v_tr(const lds_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
}

// Global -> LDS loads as inline assembly: lane l's bytes land at LDS byte lds + 16 l (or + 4 l
// for the dword form); lds is wave-uniform.  Every global load of this kernel takes this path
// (apart from seed lists longer than 256 entries and the register loads of the live diagonal
// rows of a tile with more than 16 seed rows), so the compiler tracks none of them: every read
// of their data is preceded by an explicit vmcnt wait of the issuing wave (and a barrier where
// other waves' loads are read).
__device__ __forceinline__ uint32_t lds_u32v(const lds_t* ptr) { return (uint32_t)(uintptr_t)ptr; }
__device__ __forceinline__ uint32_t lds_u32(const lds_t* ptr) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)ptr);
}
__device__ __forceinline__ void dma16(uint32_t lds, gmem_t* addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(lds), "v"((uint64_t)addr) : "memory", "m0");
}
__device__ __forceinline__ void dma16s(uint32_t lds, gmem_t* base, uint32_t voff) {  // uniform base
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
// the uniform-base load for the lanes of `mask` only (exec is set and restored inside the
// statement, so the compiler sees straight-line code; with an empty mask nothing moves).  The
// three scalar moves and the nop keep the load five instructions behind any VALU write of the
// scalar operands.
__device__ __forceinline__ void dma16m(uint32_t lds, gmem_t* base, uint32_t voff, uint64_t mask) {
  uint64_t save;
  asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %1\n\ts_mov_b32 m0, %2\n\ts_nop 1\n\t"
               "global_load_lds_dwordx4 %3, %4\n\ts_mov_b64 exec, %0"
               : "=&s"(save) : "s"(mask), "s"(lds), "v"(voff), "s"(base) : "memory", "m0");
}
// lanes 16 k .. 16 k + 15 for each set bit k of a 4-bit value
__device__ __forceinline__ uint64_t lane_quads(uint32_t n) {
  const uint64_t m = (uint64_t)(n & 1u) | ((uint64_t)(n & 2u) << 15) | ((uint64_t)(n & 4u) << 30) |
                     ((uint64_t)(n & 8u) << 45);
  return (m << 16) - m;
}
__device__ __forceinline__ void dma4(uint32_t lds, gmem_t* addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off"
               :: "s"(lds), "v"((uint64_t)addr) : "memory", "m0");
}
__device__ __forceinline__ float swap_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float swap_add(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float fmax3(float a, float b, float c) { return __builtin_fmaxf(__builtin_fmaxf(a, b), c); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float lane_max(const f32x16& s) {
  const float a = fmax3(s[0], s[1], s[2]), b = fmax3(s[3], s[4], s[5]);
  const float c = fmax3(s[6], s[7], s[8]), d = fmax3(s[9], s[10], s[11]);
  const float e = fmax3(s[12], s[13], s[14]);
  return fmax3(fmax3(a, b, c), __builtin_fmaxf(d, e), s[15]);
}
__device__ __forceinline__ gmem_t* uniform_ptr(const void* ptr) {
  const uint64_t v = (uint64_t)ptr;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (gmem_t*)(((uint64_t)hi << 32) | lo);
}

template <int N>
struct IC {
  static constexpr int value = N;
};

// Phase timing (a separate build of the library, -DCOVER_ATTN_TIMING=1, used only to measure
// where a workgroup's time goes): lane 0 of every wave of the first kTimeWG logical
// workgroups stores the shader-clock counter at fixed points of the kernel, plus the 100-MHz
// real-time counter at the start and the end (their ratio is the shader clock under load).
// Slots: 0 start, 1 real time at start, 2 Q and K(0) landed, 3 seed bitmap built, 4 Q in
// registers, 5 S(0) and the reference maxima, 6 + i top of step i (after its barrier, i < 64),
// 70 last stage after its barrier, 71 last stage done, 72 all loads landed, 73 partner tile
// readable, 74 rows finished, 75 stores issued, 94 end, 95 real time at the end.
#ifndef COVER_ATTN_TIMING
#define COVER_ATTN_TIMING 0
#endif
#if COVER_ATTN_TIMING
constexpr int kTimeWG = 4096, kTimeSlots = 96;
__device__ uint64_t g_attn_times[kTimeWG * kWaves * kTimeSlots];
#define COVER_TSTAMP(slot)                                                                      \
  do {                                                                                          \
    if (li < kTimeWG && lane == 0 && (slot) < kTimeSlots)                                       \
      g_attn_times[((int64_t)li * kWaves + wave) * kTimeSlots + (slot)] = __builtin_readcyclecounter(); \
  } while (0)
#define COVER_TREAL(slot)                                                                       \
  do {                                                                                          \
    if (li < kTimeWG && lane == 0)                                                              \
      g_attn_times[((int64_t)li * kWaves + wave) * kTimeSlots + (slot)] = __builtin_amdgcn_s_memrealtime(); \
  } while (0)
#else
#define COVER_TSTAMP(slot) do {} while (0)
#define COVER_TREAL(slot) do {} while (0)
#endif

__global__ __launch_bounds__(kThreads, 1) void cover_attn_w4_kernel(const Params4 p) {
  // Three K and three V stage buffers; Q of the workgroup on its way to registers (later: the
  // live rows of the seed rows' diagonals, then the output tiles); the seed list, the seed
  // bitmap of the sequence and its per-stage summary; merge scalars; the recompute flag.
  __shared__ __attribute__((aligned(1024))) char sK0[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sK1[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sK2[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sV0[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sV1[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sV2[kSBytes];
  __shared__ __attribute__((aligned(1024))) char sQ[kBM * kRow];
  __shared__ uint32_t bits[COVER_MAX_L / 32];
  __shared__ uint32_t sdirty[COVER_MAX_L / kStage / 32];
  __shared__ __attribute__((aligned(16))) int32_t sSeeds[kSeedsLds];
  __shared__ __attribute__((aligned(16))) int32_t sNs[4];
  __shared__ __attribute__((aligned(16))) float sML[kWaves * 2 * 64];
  __shared__ uint32_t sbad;
  auto kbuf = [&](int n) __attribute__((always_inline)) -> lds_t* { return (lds_t*)(n == 0 ? sK0 : (n == 1 ? sK1 : sK2)); };
  auto vbuf = [&](int n) __attribute__((always_inline)) -> lds_t* { return (lds_t*)(n == 0 ? sV0 : (n == 1 ? sV1 : sV2)); };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qb = wave & 1;   // 64-query block
  const int kh = wave >> 1;  // key half of every stage; the wave finishes queries qw + 32 kh
  const int hl = lane >> 5, l32 = lane & 31;

  // ---- workgroup -> (b, h, query tile); consecutive logical tiles share an XCD ------------
  int li = blockIdx.x;
  if (p.xcd_slots > 0) li = (li & 7) * p.xcd_slots + (li >> 3);
  COVER_TSTAMP(0);
  COVER_TREAL(1);
  const int qt = li % p.n_qt;
  const int bh = li / p.n_qt;
  const int h = bh % p.Hq, b = bh / p.Hq;
  const int g = h / p.group;
  const int L = p.L;
  const int q0 = qt * kBM;
  const int qw = q0 + qb * 64;  // first query of this wave's block
  const __bf16* qbase = p.q + b * p.q_sb + h * p.q_sh;
  const int64_t kvoff = b * p.kv_sb + g * p.kv_sh;
  const int n_it = (L + kStage - 1) / kStage;
  const int64_t sbase = (int64_t)b * p.max_seeds;

  // ---- load geometry -------------------------------------------------------------------
  // Load j of this wave covers stage rows (wave * 4 + j) * 4 + lane / 16, physical chunk
  // lane % 16 (logical chunk = physical ^ swizzle), landing at byte (wave * 4 + j) * 1024 +
  // 16 lane of the stage buffer, which is where the swizzled layout wants it.
  auto ld_row = [&](int j) __attribute__((always_inline)) { return (wave * kLoads + j) * 4 + (lane >> 4); };
  auto ld_chunk = [&](int j, bool is_v) __attribute__((always_inline)) -> uint32_t {
    const int row = ld_row(j), pc = lane & 15;
    return (uint32_t)((pc ^ (is_v ? v_swz(row) : k_swz(row))) << 4);
  };
  const int64_t row_bytes = p.kv_sl * 2;
  const int64_t stage_bytes = kStage * row_bytes;
  uint32_t offK[kLoads], offV[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    offK[j] = (uint32_t)(ld_row(j) * row_bytes) + ld_chunk(j, false);
    offV[j] = (uint32_t)(ld_row(j) * row_bytes) + ld_chunk(j, true);
  }
  gmem_t* const klb = uniform_ptr(p.kl + kvoff);
  gmem_t* const kcb = uniform_ptr(p.kc + kvoff);
  gmem_t* const vlb = uniform_ptr(p.vl + kvoff);
  gmem_t* const vcb = uniform_ptr(p.vc + kvoff);
  auto clamp_stage = [=](int i) __attribute__((always_inline)) -> int { return i < n_it ? i : n_it - 1; };
  auto wdst = [&](lds_t* buf, int j) __attribute__((always_inline)) -> uint32_t {
    return lds_u32(buf + (wave * kLoads + j) * 1024);
  };
  // the loads of one stage from the live tensors, rows past L clamped (before the seeds are known)
  auto ld_live = [&](lds_t* buf, gmem_t* live, bool is_v, int stage) __attribute__((always_inline)) {
    const int kb = stage * kStage;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int key = min(kb + ld_row(j), L - 1);
      dma16(wdst(buf, j), live + key * row_bytes + ld_chunk(j, is_v));
    }
  };

  // ---- prologue loads: the seed count and the first 256 seed positions, K(0) and Q; after
  // they have landed, V(0), K(1), V(1), K(2) ------------------------------------------------
  if (p.max_seeds > 0) {
    if (tid == 0) dma4(lds_u32((lds_t*)sNs), (gmem_t*)(p.n_seed + b));
    const int e = 64 * wave + lane;
    if (e < p.max_seeds && e < kSeedsLds)
      dma4(lds_u32((lds_t*)sSeeds + 256 * wave), (gmem_t*)(p.seed_idx + sbase + e));
  }
  ld_live(kbuf(0), klb, false, 0);
  // Q rows q0 + r (r = 32 wave + 4 j + lane / 16), rows past L clamped, K swizzle
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = 32 * wave + 4 * j + (lane >> 4), pc = lane & 15;
    const int qi = min(q0 + r, L - 1);
    dma16(lds_u32((lds_t*)sQ + (32 * wave + 4 * j) * kRow),
          (gmem_t*)(qbase + (int64_t)qi * p.q_sl) + ((pc ^ k_swz(r)) << 4));
  }
  // words past the sequence are cleared too: per-stage lookups read two words per stage
  for (int w = tid; w < 2 * n_it; w += kThreads) bits[w] = 0u;
  if (tid < COVER_MAX_L / kStage / 32) sdirty[tid] = 0u;
  if (tid == 0) sbad = 0u;
  // the O^T accumulators start at zero (written while the loads are in flight)
  f32x16 o[2][kDB];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int db = 0; db < kDB; ++db) asm volatile("; O = 0" : "=a"(o[t][db]) : "0"((f32x16){}));
  // the seed list, K(0) and Q have landed; the next stages go out only now, so that Q and
  // K(0) do not share the vector-memory path with them at the start of the kernel (V(0) and
  // K(1) are first needed at the top of step 0)
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();
  COVER_TSTAMP(2);
  ld_live(vbuf(0), vlb, true, 0);
  ld_live(kbuf(1), klb, false, clamp_stage(1));
  ld_live(vbuf(1), vlb, true, clamp_stage(1));
  ld_live(kbuf(2), klb, false, clamp_stage(2));

  // ---- seed bitmap of this sequence -----------------------------------------------------
  int ns = p.max_seeds > 0 ? sNs[0] : 0;
  ns = ns < 0 ? 0 : (ns > p.max_seeds ? p.max_seeds : ns);
  auto mark = [&](int j) __attribute__((always_inline)) {
    atomicOr(&bits[j >> 5], 1u << (j & 31));
    atomicOr(&sdirty[j >> 11], 1u << ((j >> 6) & 31));
  };
  if (tid < ns && tid < kSeedsLds) {
    const int j = sSeeds[tid];
    if ((unsigned)j < (unsigned)L) mark(j);
  }
  for (int t = tid + kSeedsLds; t < ns; t += kThreads) {  // long seed lists
    const int j = p.seed_idx[sbase + t];
    if ((unsigned)j < (unsigned)L) mark(j);
  }
  __syncthreads();
  COVER_TSTAMP(3);
  auto is_seed = [&](int j) __attribute__((always_inline)) -> bool { return (bits[j >> 5] >> (j & 31)) & 1u; };

  // Lane l holds the seed flags of stages 64 l .. 64 l + 63 (two words); a stage's flag is
  // read back with a lane read.
  const uint32_t dirty_lo = sdirty[(2 * lane) & (COVER_MAX_L / kStage / 32 - 1)];
  const uint32_t dirty_hi = sdirty[(2 * lane + 1) & (COVER_MAX_L / kStage / 32 - 1)];
  auto dirty = [&](int stage) __attribute__((always_inline)) -> bool {
    const uint32_t w = ((stage >> 5) & 1) ? __builtin_amdgcn_readlane(dirty_hi, stage >> 6)
                                          : __builtin_amdgcn_readlane(dirty_lo, stage >> 6);
    return (w >> (stage & 31)) & 1u;
  };
  const int spC = L % kStage != 0 ? n_it - 1 : -1;  // ragged last stage
  // stages 0..63 that need row-by-row loads (seeds, or the ragged end), as a scalar mask, so
  // the per-step check costs no lane reads; later stages use the lane lookup
  // The rows of a stage that this wave loads are rows 16 wave .. 16 wave + 15; their seed flags
  // (a 16-bit chunk of the stage's 64) sit in lane `stage` of seed_chunk_l for stages below 64.
  auto chunk_of = [&](int stage) __attribute__((always_inline)) -> uint32_t {
    return (bits[2 * stage + (wave >> 1)] >> (16 * (wave & 1))) & 0xffffu;
  };
  // lane s holds the chunk of stage s (stages below 64; later ones are read from the bitmap)
  const uint32_t seed_chunk_l = lane < n_it ? chunk_of(lane) : 0u;
  auto seed_chunk = [&](int stage) __attribute__((always_inline)) -> uint32_t {
    if (__builtin_expect(stage < 64, 1)) return __builtin_amdgcn_readlane(seed_chunk_l, stage);
    return __builtin_amdgcn_readfirstlane(chunk_of(stage));
  };
  // Row-by-row flags of stages w0 .. w0 + 63 (w0 a multiple of 32) as one scalar: bit s - w0
  // is set for a stage with seeds, or the ragged last one.
  auto flags_at = [&](int w0) __attribute__((always_inline)) -> uint64_t {
    constexpr int kWords = COVER_MAX_L / kStage / 32;
    const int w = w0 >> 5;
    const uint32_t a = sdirty[w];
    const uint32_t c = w + 1 < kWords ? sdirty[w + 1] : 0u;
    uint64_t f = ((uint64_t)__builtin_amdgcn_readfirstlane(c) << 32) | __builtin_amdgcn_readfirstlane(a);
    if (spC >= w0 && spC < w0 + 64) f |= 1ull << (spC - w0);
    return f;
  };

  // Per-lane source addresses of the loads of one stage: the live row, or the cached row at
  // a seed position, rows past L clamped (stages without seeds inside L: base + offset).
  auto addrs = [&](gmem_t* live, gmem_t* cache, const uint32_t* off, bool is_v, int stage,
                   gmem_t** a) __attribute__((always_inline)) {
    if (stage != spC && !dirty(stage)) {
      gmem_t* lb = uniform_ptr((const void*)(live + stage * stage_bytes));
#pragma unroll
      for (int j = 0; j < kLoads; ++j) a[j] = lb + off[j];
    } else {
      const int kb = stage * kStage;
#pragma unroll
      for (int j = 0; j < kLoads; ++j) {
        const int key = min(kb + ld_row(j), L - 1);
        a[j] = (is_seed(key) ? cache : live) + key * row_bytes + ld_chunk(j, is_v);
      }
    }
  };
  auto ld = [&](lds_t* buf, gmem_t* live, gmem_t* cache, const uint32_t* off, bool is_v,
                int stage) __attribute__((always_inline)) {
    gmem_t* a[kLoads];
    addrs(live, cache, off, is_v, stage, a);
#pragma unroll
    for (int j = 0; j < kLoads; ++j) dma16(wdst(buf, j), a[j]);
  };

  // Uniform base of the in-loop loads of a stage: its rows, or for the ragged last stage the
  // last 64 rows of the sequence (in bounds; the rows below L are then reloaded by patch).
  auto clean_base = [&](gmem_t* live, int stage) __attribute__((always_inline)) -> gmem_t* {
    const int64_t off = stage == spC ? (int64_t)(L - kStage) * row_bytes : stage * stage_bytes;
    return uniform_ptr((const void*)(live + off));
  };
  // Reload the rows of a stage that the uniform loads got wrong: in the ragged last stage the
  // rows below L (from the live tensor), and every seed row (from the cache).  Issued after
  // the uniform loads of the same wave, so these land last; load j takes the lanes of rows
  // 16 wave + 4 j + {0..3} that need it (lane / 16 selects the row), and is skipped if there
  // are none (back-to-back global-to-LDS loads issue slowly, so only the needed ones go out).
  auto patch = [&](lds_t* buf, gmem_t* live, gmem_t* cache, const uint32_t* off, int stage_in)
                   __attribute__((always_inline)) {
    const int st = __builtin_amdgcn_readfirstlane(stage_in);
    if (st == spC) {
      gmem_t* lb = uniform_ptr((const void*)(live + st * stage_bytes));
      const int nv = min(max(L - st * kStage - 16 * wave, 0), 16);  // this wave's rows below L
      const uint32_t vm = (1u << nv) - 1u;
#pragma unroll
      for (int j = 0; j < kLoads; ++j)
        if ((vm >> (4 * j)) & 15u) dma16m(wdst(buf, j), lb, off[j], lane_quads((vm >> (4 * j)) & 15u));
    }
    gmem_t* cb = uniform_ptr((const void*)(cache + st * stage_bytes));
    const uint32_t sc = seed_chunk(st);  // seeds lie below L
#pragma unroll
    for (int j = 0; j < kLoads; ++j)
      if ((sc >> (4 * j)) & 15u) dma16m(wdst(buf, j), cb, off[j], lane_quads((sc >> (4 * j)) & 15u));
  };

  // ---- diagonal set-up --------------------------------------------------------------------
  // A wave's query tile t holds queries qw + 32 (t ^ kh): tile 0 is always the one it finishes
  // (queries qd0 + c), whose diagonal keys lie in stage sd, key half kh, tile row c: lane half
  // (c / 4) % 2, register (c / 8) * 4 + c % 4; tile 1 goes to the partner wave.
  const int qd0 = qw + 32 * kh;
  const int sd = qw / kStage;
  const bool holds_diag = hl == ((l32 >> 2) & 1);
  const int rd = ((l32 >> 3) << 2) | (l32 & 3);
  const bool qd_seed = (qd0 + l32) < L && is_seed(qd0 + l32);
  const bool diag_seed = holds_diag && qd_seed;
  const bool block_seeded = __builtin_amdgcn_ballot_w64(qd_seed) != 0;
  const int spA = block_seeded ? sd : -1;
  auto is_special = [=](int i) __attribute__((always_inline)) -> bool { return (i == spA) | (i == spC); };

  // Stages 0..2 were loaded from the live tensors before the seeds were known; reload the
  // ones that hold seeds (after every wave's first loads have landed).
  if (dirty(0) || dirty(clamp_stage(1)) || dirty(clamp_stage(2))) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    ld(kbuf(0), klb, kcb, offK, false, 0);
    ld(vbuf(0), vlb, vcb, offV, true, 0);
    ld(kbuf(1), klb, kcb, offK, false, clamp_stage(1));
    ld(vbuf(1), vlb, vcb, offV, true, clamp_stage(1));
    ld(kbuf(2), klb, kcb, offK, false, clamp_stage(2));
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * kLoads));  // K(0) back in place
    __syncthreads();
  }

  // ---- Q fragments (B operand of S^T = K Q^T): tile t, query qw + 32 (t ^ kh) + l32,
  // d-chunk 2 ks + hl, from LDS into AGPRs for good -----------------------------------------
  bf16x8 qa[2][kKS];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      const int r = 64 * qb + 32 * (t ^ kh) + l32;
      asm volatile("ds_read_b128 %0, %1" : "=a"(qa[t][ks]) : "v"(lds_u32v((lds_t*)sQ + k_off(r, 2 * ks + hl))));
    }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the Q reads above (not tracked by the compiler)
  COVER_TSTAMP(4);

  // ---- per-lane LDS read addresses (relative to a stage buffer) ---------------------------
  uint32_t kaddr[kKS];
#pragma unroll
  for (int ks = 0; ks < kKS; ++ks) kaddr[ks] = k_off(kh * 32 + l32, 2 * ks + hl);
  // A operand of O^T += V^T P^T for keys kh*32 + 16 kk + {0..3, 8..11} + 4 (G / 2), d-block
  // db: lane (G = lane / 16, i = lane % 16) reads V[row][db*32 + 16 (G % 2) + 4 (i % 4) .. +3]
  // with row = kh*32 + 16 kk + 4 (G / 2) + i / 4 (+8 for the upper half); the same key order
  // the S^T registers give the P^T operand.  kk and the +8 move the row by multiples of 4,
  // which leave the swizzle unchanged: constant offsets.
  uint32_t vaddr[kDB];
  {
    const int G = lane >> 4, ii = lane & 15;
    const int row = kh * 32 + 4 * (G >> 1) + (ii >> 2);
#pragma unroll
    for (int db = 0; db < kDB; ++db) vaddr[db] = v_elem(row, db * 32 + 16 * (G & 1) + 4 * (ii & 3));
  }

  // ---- compute pieces ----------------------------------------------------------------------
  // (operand reads `ahead` k-steps before their MFMAs; the exact pass keeps registers free)
  auto qk = [&](const lds_t* kb, f32x16* s, auto ahead) __attribute__((always_inline)) {
    constexpr int A = decltype(ahead)::value;
    bf16x8 a[kKS];
#pragma unroll
    for (int ks = 0; ks < A; ++ks) a[ks] = __builtin_bit_cast(bf16x8, lds_read16(kb + kaddr[ks]));
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      if (ks + A < kKS) a[ks + A] = __builtin_bit_cast(bf16x8, lds_read16(kb + kaddr[ks + A]));
      if (ks == 0) {
        mfma_first(s[0], a[0], qa[0][ks]);
        mfma_first(s[1], a[0], qa[1][ks]);
      } else {
        mfma_v(s[0], a[ks], qa[0][ks]);
        mfma_v(s[1], a[ks], qa[1][ks]);
      }
    }
  };
  // keys of this wave's half of `stage` past L, and the seed rows' own (cached) column, get no
  // weight; the live diagonal term joins in the epilogue
  // (The per-lane limits pass through an empty asm at each use: otherwise the compiler keeps
  // the 32 element masks of each test alive across the loop as scalar register pairs.)
  auto special_fix = [&](int stage, f32x16* s) __attribute__((always_inline)) {
    if (stage * kStage + kStage > L) {
      // element r holds key stage * 64 + 32 kh + 8 (r / 4) + 4 hl + r % 4
      int lim = L - (stage * kStage + kh * 32) - 4 * hl;
      asm volatile("" : "+v"(lim));
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[t][r] = ((r >> 2) << 3) + (r & 3) < lim ? s[t][r] : -INFINITY;
    }
    if (block_seeded && stage == sd) {  // tile 0 holds the diagonal
      int dsel = diag_seed ? rd : -1;
      asm volatile("" : "+v"(dsel));
#pragma unroll
      for (int r = 0; r < 16; ++r) s[0][r] = r == dsel ? -INFINITY : s[0][r];
    }
  };

  float m[2], lsum[2] = {0.0f, 0.0f};
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // row sums of the bf16 weights (as the MFMA used them) and the range check
  auto rowsums = [&](bf16x8 (*pk)[2]) __attribute__((always_inline)) -> uint64_t {
    uint64_t bad = 0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      float ls[2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 w = pk[t][kk];
        float a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 0, 1), ones, 0.0f, false);
        a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 2, 3), ones, a, false);
        a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 4, 5), ones, a, false);
        ls[kk] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(w, w, 6, 7), ones, a, false);
      }
      const float st = ls[0] + ls[1];
      lsum[t] += st;
      bad |= __builtin_amdgcn_ballot_w64(!(st <= kBig));
    }
    return bad;
  };
  // exp2(c2 s - m) -> bf16 P (both tiles); returns the lanes whose per-stage sum left the
  // safe range
  auto softmax = [&](const f32x16* s, bf16x8 (*pk)[2], float* mref) __attribute__((always_inline)) -> uint64_t {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const float nm = -mref[t];
      f32x16 pr;
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[t][r], p.c2, nm));
      pk[t][0] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 0, 1, 2, 3, 4, 5, 6, 7), bf16x8);
      pk[t][1] = __builtin_convertvector(__builtin_shufflevector(pr, pr, 8, 9, 10, 11, 12, 13, 14, 15), bf16x8);
    }
    return rowsums(pk);
  };
  // (V operands read `ahead` MFMA pairs before use; the exact pass keeps registers free)
  auto pv = [&](const lds_t* vb, bf16x8 (*pk)[2], auto ahead) __attribute__((always_inline)) {
    constexpr int A = decltype(ahead)::value;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) valu_to_mfma(pk[t][kk]);
    bf16x8 va[2 * kDB];  // operand n: kk = n / kDB, db = n % kDB
    auto vread = [&](int n) __attribute__((always_inline)) {
      const lds_t* base = vb + vaddr[n % kDB] + (n / kDB) * 16 * kRow;
      va[n] = __builtin_bit_cast(
          bf16x8, __builtin_shufflevector(v_tr(base), v_tr(base + 8 * kRow), 0, 1, 2, 3, 4, 5, 6, 7));
    };
#pragma unroll
    for (int n = 0; n < A; ++n) vread(n);
#pragma unroll
    for (int n = 0; n < 2 * kDB; ++n) {
      if (n + A < 2 * kDB) vread(n + A);
      mfma_a(o[0][n % kDB], va[n], pk[0][n / kDB]);
      mfma_a(o[1][n % kDB], va[n], pk[1][n / kDB]);
    }
  };

  // The main block of a step: S(i+1) = K(i+1) Q^T, softmax of S(i), O += P(i) V(i), and the
  // loads of K(i+3) and V(i+2), written in issue order (the MFMAs keep their order; LDS reads
  // and global loads stay where they are written): K operands four k-steps ahead, V operands
  // one d-block ahead, one global load between MFMA pairs; the exponentials of the first key
  // half of both tiles go between the S MFMAs (the first PV half needs them), those of the
  // second half between the first PV half's MFMAs.
  auto fused = [&](const lds_t* kb, f32x16* sn, const f32x16* sc, const lds_t* vb, lds_t* kdst,
                   gmem_t* kg, lds_t* vdst, gmem_t* vg) __attribute__((always_inline)) -> uint64_t {
    bf16x8 ka[kKS];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) ka[ks] = __builtin_bit_cast(bf16x8, lds_read16(kb + kaddr[ks]));
    const float nm[2] = {-m[0], -m[1]};
    f32x16 pr[2];
    auto expo = [&](int e) __attribute__((always_inline)) {  // element e of the order below
      const int t = (e >> 3) & 1, r = (e & 7) + ((e >> 4) << 3);
      pr[t][r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[t][r], p.c2, nm[t]));
    };
    bf16x8 va[2][kDB];
    auto vread = [&](int kk, int db) __attribute__((always_inline)) {
      const lds_t* base = vb + vaddr[db] + kk * 16 * kRow;
      va[kk][db] = __builtin_bit_cast(
          bf16x8, __builtin_shufflevector(v_tr(base), v_tr(base + 8 * kRow), 0, 1, 2, 3, 4, 5, 6, 7));
    };
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      if (ks == 0) {
        mfma_first(sn[0], ka[0], qa[0][0]);
        mfma_first(sn[1], ka[0], qa[1][0]);
      } else {
        mfma_v(sn[0], ka[ks], qa[0][ks]);
        mfma_v(sn[1], ka[ks], qa[1][ks]);
      }
      if (ks + 4 < kKS) ka[ks + 4] = __builtin_bit_cast(bf16x8, lds_read16(kb + kaddr[ks + 4]));
      else vread(0, ks - 4);
      if ((ks & 1) == 0) dma16s(wdst(kdst, ks >> 1), kg, offK[ks >> 1]);
      // elements 2 ks, 2 ks + 1 of the order (t0 r0-7, t1 r0-7, t0 r8-15, t1 r8-15)
#pragma unroll
      for (int u = 0; u < 2; ++u) expo(ks * 2 + u);
    }
    bf16x8 pk[2][2];
    auto cvt = [&](int kk) __attribute__((always_inline)) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        pk[t][kk] = kk == 0
            ? __builtin_convertvector(__builtin_shufflevector(pr[t], pr[t], 0, 1, 2, 3, 4, 5, 6, 7), bf16x8)
            : __builtin_convertvector(__builtin_shufflevector(pr[t], pr[t], 8, 9, 10, 11, 12, 13, 14, 15), bf16x8);
        valu_to_mfma(pk[t][kk]);
      }
    };
    cvt(0);
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      mfma_a(o[0][db], va[0][db], pk[0][0]);
      mfma_a(o[1][db], va[0][db], pk[1][0]);
      vread(1, db);
      dma16s(wdst(vdst, db), vg, offV[db]);
#pragma unroll
      for (int u = 0; u < 4; ++u) expo(16 + db * 4 + u);
    }
    cvt(1);
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      mfma_a(o[0][db], va[1][db], pk[0][1]);
      mfma_a(o[1][db], va[1][db], pk[1][1]);
    }
    return rowsums(pk);
  };

  // ---- prologue compute: S(0) and the reference row maxima --------------------------------
  f32x16 sA[2], sB[2];
  qk(kbuf(0), sA, IC<4>{});
  mfma_drain();
  if (is_special(0)) special_fix(0, sA);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const float mt = swap_max(lane_max(sA[t])) * p.c2;
    m[t] = mt > kInitMax ? mt : kInitMax;
  }
  COVER_TSTAMP(5);

  // ---- steady state --------------------------------------------------------------------------
  // Step i (i < n_it - 1): wait for this wave's loads of K(i+1), V(i) (issued two steps
  // before; the eight loads of the previous step may still be in flight), barrier (every
  // wave's loads landed; every wave done with step i-1), then the main block, whose loads go
  // to K buffer i%3 and V buffer (i+2)%3.  Past the end the loads repeat the last stage (they
  // keep the per-step load count, which the waits rely on).  Buffers depend on i mod 3 and S
  // on i mod 2: six steps are unrolled with fixed buffers.
  uint64_t bad = 0;
  int i = 0;
  const int last = n_it - 1;
  // uniform bases of the in-loop loads: K(i+3) and V(i+2) advance a stage per step; the last
  // (possibly ragged) stage has its own
  gmem_t* kgr = uniform_ptr((const void*)(klb + 3 * stage_bytes));
  gmem_t* vgr = uniform_ptr((const void*)(vlb + 2 * stage_bytes));
  gmem_t* const k_last = clean_base(klb, n_it - 1);
  gmem_t* const v_last = clean_base(vlb, n_it - 1);
  // Live key and value rows of the finished tile's queries (qd0 + l32, clamped below L), for
  // the diagonal terms of its seed rows: loaded into registers by seeded waves at the last
  // stage.  Lane half hl takes the d-chunks it also holds of Q (key: 2 ks + hl, 16 bytes
  // each) and of O (value: d = 8 c + 4 hl + 0..3 for c = 0..15, 8 bytes each).
  const int64_t diag_row = kvoff + (int64_t)min(qd0 + l32, L - 1) * p.kv_sl;
  u32x4 dkr[kKS];
  u32x2 dvr[kDB * 4];
  auto load_diag_k = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) dkr[ks] = *(const u32x4*)(p.kl + diag_row + (2 * ks + hl) * 8);
  };
  auto load_diag_v = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kDB * 4; ++c) dvr[c] = *(const u32x2*)(p.vl + diag_row + c * 8 + hl * 4);
  };
  // q_i . k_live_i for the finished tile's query of this lane pair (halves of d summed by
  // a swap)
  auto live_score = [&]() __attribute__((always_inline)) -> float {
    float acc = 0.0f;
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      const bf16x8 kv = __builtin_bit_cast(bf16x8, dkr[ks]);
      const bf16x8 qv = qa[0][ks];
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(qv, qv, 0, 1), __builtin_shufflevector(kv, kv, 0, 1), acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(qv, qv, 2, 3), __builtin_shufflevector(kv, kv, 2, 3), acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(qv, qv, 4, 5), __builtin_shufflevector(kv, kv, 4, 5), acc, false);
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(qv, qv, 6, 7), __builtin_shufflevector(kv, kv, 6, 7), acc, false);
    }
    return swap_add(acc);
  };
  float s_live = 0.0f;
  // The seed rows among the finished tile's queries (its 32 positions are bitmap word qd0 / 32):
  // their live key and value rows go to this wave's 8 KiB of the Q area (free from the first
  // step until the output tile is staged there) by global-to-LDS loads, four rows per load,
  // issued with the last step; slot k holds the k-th seed row (key at 256 k, value at 4096 +
  // 256 k).  A tile with more than 16 seed rows (or a sequence without steps) loads the rows
  // of all its queries into registers instead.
  const uint32_t dmask = block_seeded ? bits[qd0 >> 5] : 0u;
  const bool diag_lds = __builtin_popcount(dmask) <= 16 && last > 0;
  lds_t* const dgA = (lds_t*)sQ + wave * (32 * kRow);
  auto issue_diag = [&]() __attribute__((always_inline)) {
    uint32_t msk = dmask;
    for (int u = 0; msk; ++u) {
      int r = -1;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (msk) {
          const int b = __builtin_ctz(msk);
          msk &= msk - 1;
          if ((lane >> 4) == g) r = b;
        }
      }
      if (r >= 0) {
        const int64_t src = (int64_t)(qd0 + r) * row_bytes + ((lane & 15) << 4);
        dma16(lds_u32(dgA + u * 1024), klb + src);
        dma16(lds_u32(dgA + 4096 + u * 1024), vlb + src);
      }
    }
  };
  // this lane's query's slot (meaningful for seed rows only)
  const int dslot = __builtin_popcount(dmask & ((1u << l32) - 1u));
  auto diag_from_lds = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) dkr[ks] = lds_read16(dgA + dslot * kRow + (2 * ks + hl) * 16);
#pragma unroll
    for (int c = 0; c < kDB * 4; ++c)
      dvr[c] = qd_seed ? *(const __attribute__((address_space(3))) u32x2*)(dgA + 4096 + dslot * kRow + 16 * c + 8 * hl)
                       : (u32x2){0u, 0u};
  };
  uint64_t win = flags_at(0);  // the row-by-row flags of stages (i & ~31) + 0 .. 63
  auto step = [&](auto ph) __attribute__((always_inline)) -> bool {
    constexpr int P = decltype(ph)::value;
    f32x16* sc = (P & 1) ? sB : sA;
    f32x16* sn = (P & 1) ? sA : sB;
    if (i == last) return true;  // finished below, outside the unrolled steps
    if (__builtin_expect((i & 31) == 0 && i > 0, 0)) win = flags_at(i);
    if (__builtin_expect(is_special(i), 0)) special_fix(i, sc);
    gmem_t* const kg = i + 3 < n_it - 1 ? kgr : k_last;
    gmem_t* const vg = i + 2 < n_it - 1 ? vgr : v_last;
    kgr += stage_bytes;
    vgr += stage_bytes;
    __builtin_amdgcn_s_waitcnt(kWaitStep);
    __builtin_amdgcn_s_barrier();
    COVER_TSTAMP(6 + (i < 64 ? i : 63));
    // the stages loaded in the previous step, K(i+2) and V(i+1), get their seed / ragged
    // rows now: after the wait (which would otherwise also wait for the previous step's
    // loads), before this step's loads (so the wait at the top of the next step covers them);
    // neither buffer is read in this step
    if (__builtin_expect(((win >> ((i & 31) + 1)) & 3u) != 0, 0)) {
      if (i + 2 < n_it) patch(kbuf((P + 2) % 3), klb, kcb, offK, i + 2);
      patch(vbuf((P + 1) % 3), vlb, vcb, offV, i + 1);
    }
    // a seeded tile's live diagonal key and value rows go out with the last step, so that
    // they have landed by the last stage and the finish
    if (__builtin_expect(block_seeded && i == last - 1, 0)) {
      if (diag_lds) {
        issue_diag();
      } else {
        load_diag_k();
        load_diag_v();
      }
    }
    bad |= fused(kbuf((P + 1) % 3), sn, sc, vbuf(P % 3), kbuf(P % 3), kg, vbuf((P + 2) % 3), vg);
    ++i;
    return false;
  };
  for (;;) {
    if (step(IC<0>{})) break;
    if (step(IC<1>{})) break;
    if (step(IC<2>{})) break;
    if (step(IC<3>{})) break;
    if (step(IC<4>{})) break;
    if (step(IC<5>{})) break;
  }
  // Last stage: its S is in sA or sB by parity (selected by value: a selected pointer would
  // send the tiles through memory), V in buffer last % 3.  Seeded waves issued their diagonal
  // key and value rows with the last step (here, if there was none).
  {
    f32x16 sc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) sc[t] = (last & 1) ? sB[t] : sA[t];
    if (is_special(last)) special_fix(last, sc);
    // V(last) and its re-loaded rows were issued two steps and one step ago; the eight loads
    // of the previous step (stages past the end) and the diagonal rows issued before them may
    // stay in flight (loads complete in order).  Every load has landed before the buffers are
    // reused after this block.
    if (block_seeded && last == 0) {  // (no steps: the diagonal rows are loaded here)
      load_diag_k();
      load_diag_v();
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    } else if (block_seeded && !diag_lds) {  // the diagonal rows and the previous step's loads may fly
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * kLoads + kKS + kDB * 4));
    } else {  // (the diagonal rows' global-to-LDS loads, issued a step ago, land here too)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * kLoads));
    }
    __builtin_amdgcn_s_barrier();
    COVER_TSTAMP(70);
    bf16x8 pk[2][2];
    bad |= softmax(sc, pk, m);
    const int vb = last % 3;
    pv(vbuf(0) + (vb == 0 ? 0 : (vb == 1 ? (int)(vbuf(1) - vbuf(0)) : (int)(vbuf(2) - vbuf(0)))), pk, IC<4>{});
    if (block_seeded) {
      if (diag_lds) diag_from_lds();
      s_live = live_score();
    }
    COVER_TSTAMP(71);
  }
  if (bad) atomicOr(&sbad, 1u);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // the loads past the end (their buffers are reused)
  __syncthreads();
  COVER_TSTAMP(72);

  // ---- exact pass (only if some row's scores outgrew its first-stage maximum by 2^24) ----
  if (sbad) {
    mfma_drain();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      m[t] = kInitMax;
      lsum[t] = 0.0f;
#pragma unroll
      for (int db = 0; db < kDB; ++db) o[t][db] = (f32x16){};
    }
    for (int it = 0; it < n_it; ++it) {
      __syncthreads();
      ld(kbuf(0), klb, kcb, offK, false, it);
      ld(vbuf(0), vlb, vcb, offV, true, it);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
      __syncthreads();
      f32x16 s[2];
      qk(kbuf(0), s, IC<0>{});
      mfma_drain();
      if (is_special(it)) special_fix(it, s);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const float mt = swap_max(lane_max(s[t])) * p.c2;
        const float mn = mt > m[t] ? mt : m[t];
        const float alpha = __builtin_amdgcn_exp2f(m[t] - mn);
        m[t] = mn;
        lsum[t] *= alpha;
#pragma unroll
        for (int db = 0; db < kDB; ++db) o[t][db] *= alpha;
      }
      bf16x8 pk[2][2];
      (void)softmax(s, pk, m);
      pv(vbuf(0), pk, IC<0>{});
      mfma_drain();
    }
    __syncthreads();
  }

  mfma_drain();
  // ---- merge the two key halves, add the live diagonal term, normalise, store --------------
  // Wave w finishes its tile 0; its tile 1 goes to the partner w ^ 2 (for which it is tile 0)
  // through LDS (16 KiB per wave: buffers V0, V1, V2, K2 are free now), with that tile's m and
  // row sum.
  float* const slot_mine = (float*)(wave == 0 ? sV0 : (wave == 1 ? sV1 : (wave == 2 ? sV2 : sK2)));
  const int pw = wave ^ 2;
  const float* const slot_theirs = (const float*)(pw == 0 ? sV0 : (pw == 1 ? sV1 : (pw == 2 ? sV2 : sK2)));
  const float l_tot0 = swap_add(lsum[0]), l_tot1 = swap_add(lsum[1]);
#pragma unroll
  for (int db = 0; db < kDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; j += 4) {
      const f32x4 v = {o[1][db][j], o[1][db][j + 1], o[1][db][j + 2], o[1][db][j + 3]};
      *(f32x4*)(slot_mine + (db * 4 + (j >> 2)) * 256 + lane * 4) = v;
    }
  sML[(wave * 2 + 0) * 64 + lane] = m[1];
  sML[(wave * 2 + 1) * 64 + lane] = l_tot1;
  __syncthreads();
  COVER_TSTAMP(73);
  // The finished tile: O^T entry (db, j) of lane (l32, hl) is column l32 (query qd0 + l32),
  // d = 32 db + 8 (j / 4) + 4 hl + j % 4.
  bf16x4 outv[kDB * 4];
  float mm_out = 0.0f, ltot_out = 1.0f;
  // The partner's tile is read whole before any use, and the seed term is a separate
  // instantiation, so no branch sits between a read and its use.
  auto finish = [&](auto seeded) __attribute__((always_inline)) {
    constexpr int T = 0;                          // the tile finished here
    constexpr bool SD = decltype(seeded)::value;  // this wave's tile holds seed rows
    f32x4 tv[kDB * 4];
#pragma unroll
    for (int n = 0; n < kDB * 4; ++n) tv[n] = *(const f32x4*)(slot_theirs + n * 256 + lane * 4);
    const float td = qd_seed ? s_live * p.c2 : -INFINITY;
    const float mb = sML[(pw * 2 + 0) * 64 + lane], lb = sML[(pw * 2 + 1) * 64 + lane];
    const float ma = m[T], la = l_tot0;
    const float mm = fmax3(ma, mb, td);
    const float fa = __builtin_amdgcn_exp2f(ma - mm), fb = __builtin_amdgcn_exp2f(mb - mm);
    const float fd = __builtin_amdgcn_exp2f(td - mm);  // 0 for rows that are not seeds
    const float ltot = la * fa + lb * fb + fd;
    const float inv = 1.0f / ltot;
    mm_out = mm;
    ltot_out = ltot;
#pragma unroll
    for (int n = 0; n < kDB * 4; ++n) {  // O^T block n / 4, rows 8 (n % 4) + 4 hl + 0..3
      f32x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = o[T][n >> 2][(n & 3) * 4 + e] * fa + tv[n][e] * fb;
      if constexpr (SD) {
        const u32x2 raw = dvr[n];
        v[0] += fd * bf16_lo(raw[0]);
        v[1] += fd * bf16_hi(raw[0]);
        v[2] += fd * bf16_lo(raw[1]);
        v[3] += fd * bf16_hi(raw[1]);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] *= inv;
      outv[n] = __builtin_convertvector(v, bf16x4);
    }
  };
  if (block_seeded) finish(IC<1>{}); else finish(IC<0>{});
  COVER_TSTAMP(74);
  if (p.lse && hl == 0 && qd0 + l32 < L)
    p.lse[((int64_t)b * p.Hq + h) * L + qd0 + l32] = (mm_out + __builtin_amdgcn_logf(ltot_out)) * kLn2;
  // Rows go out through this wave's own 8-KiB tile in the Q area (idle since Q went to
  // registers; 16-byte chunks XOR-swizzled by row % 16), so that each global store writes
  // whole 256-byte rows and no other wave has to be waited for.  The stores are
  // non-temporal: every workgroup writes its output at about the same time at the end, and
  // streaming it out instead of leaving it dirty in L2 shortens the launch (measured).
  lds_t* const tile = (lds_t*)sQ + wave * (32 * kRow);
#pragma unroll
  for (int n = 0; n < kDB * 4; ++n)
    *(__attribute__((address_space(3))) bf16x4*)(tile + k_off(l32, n) + hl * 8) = outv[n];
  constexpr int CPR = kRow / 16;       // 16-byte chunks per row
  constexpr int NRD = 32 * CPR / 64;   // reads (and stores) per lane
  __bf16* const obase = p.out + b * p.q_sb + h * p.q_sh;
  u32x4 ov[NRD];
#pragma unroll
  for (int it = 0; it < NRD; ++it) {
    const int idx = it * 64 + lane, row = idx / CPR, ch = idx % CPR;
    ov[it] = *(const __attribute__((address_space(3))) u32x4*)(tile + k_off(row, ch));
  }
  if (qd0 + 32 <= L) {
#pragma unroll
    for (int it = 0; it < NRD; ++it) {
      const int idx = it * 64 + lane, row = idx / CPR, ch = idx % CPR;
      __builtin_nontemporal_store(ov[it], (u32x4*)(obase + (int64_t)(qd0 + row) * p.q_sl + ch * 8));
    }
  } else {
#pragma unroll
    for (int it = 0; it < NRD; ++it) {
      const int idx = it * 64 + lane, row = idx / CPR, ch = idx % CPR;
      if (qd0 + row < L) __builtin_nontemporal_store(ov[it], (u32x4*)(obase + (int64_t)(qd0 + row) * p.q_sl + ch * 8));
    }
  }
  COVER_TSTAMP(75);
#if COVER_ATTN_TIMING
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores complete
  COVER_TSTAMP(94);
  COVER_TREAL(95);
#endif
}

}  // namespace

#if COVER_ATTN_TIMING
// Copies the timing slots of the last launches (layout [workgroup][wave][slot], 4096 x 4 x 96
// values) to host memory; waits for the device.  Only in the timing build of the library.
extern "C" int cover_attn_timing_read(uint64_t* host, int64_t n) {
  const int64_t cap = (int64_t)kTimeWG * kWaves * kTimeSlots;
  return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(g_attn_times), sizeof(uint64_t) * (n < cap ? n : cap),
                                  0, hipMemcpyDeviceToHost);
}
#endif

hipError_t launch_attn_bf16_w4(const AttnArgs& a, hipStream_t stream) {
  Params4 p;
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
  if (nwg > 0x7fffffff || a.d != kD) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(cover_attn_w4_kernel, dim3((unsigned)nwg), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
