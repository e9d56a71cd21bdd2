// Producers of the seed-selection signals on gfx950 (arXiv 2602.06161, Sec. 5.3; Sec. 3).
//
// cover_token_stats_kernel: per row of the model's output logits, the log-probability of the
// token currently placed there (u = -log p, Sec. 5.3), the maximum probability (the
// confidence of Sec. 3) and the token attaining it.  One workgroup of 1024 threads per row;
// each thread streams 16-byte chunks with four loads in flight and keeps an online (max, sum
// of exp) pair and the chunk where its max was last raised (the index inside it is found at
// the end), merged across the workgroup.  The placed token and its logit are fetched at the
// start by scalar loads, so no memory round trip is left for the end.
//
// cover_attn_stats_kernel + cover_attn_stats_reduce_kernel: the in/out attention masses of
// Sec. 5.3 over a response region [r0, r0+Lr), from the last layer's corrected weights
// w_qj = exp(scale q.K^(q)_j - lse_q) (the same leave-one-out rows the attention computes,
// normalised over the whole sequence by the forward pass's lse), averaged over query heads:
//   d_in(j)  = (1/Hq) sum_h sum_{q masked} w_qj,    d_out(j) = (1/Hq) sum_h sum_{i drafted} w_ji
// One workgroup per (batch row, query head, group of 32-key tiles), about 256 in all; each of
// its waves takes 32-query blocks of the region and forms both S = Q K^T and S^T = K Q^T over
// the group's key tiles (the same operand registers, swapped), so each mass is a sum inside a
// lane.  A key's d_in is complete inside its group's workgroup; d_out gets one partial per
// key group.  Both go to a caller-provided workspace and a second kernel adds the partials
// and averages over heads; every sum runs in a fixed order, so the results do not depend on
// scheduling.
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace cover {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 gu32x4;

constexpr int kTokThreads = 1024;
constexpr int kTokUnroll = 4;  // 16-byte loads in flight per thread (more measured slower)
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;

struct TokParams {
  const char* logits;
  const int32_t* tokens;
  float* logp;
  float* conf;
  int32_t* argmax;
  int64_t row_stride_bytes;
  int V;
};

// (m, s, i): running max, sum of exp2((x - m) * log2e) over the elements seen, the smallest
// index holding m.  Merging two triples keeps the larger max (smaller index on ties).
struct Acc {
  float m, s;
  int i;
};
__device__ __forceinline__ Acc merge(Acc a, Acc b) {
  const float m = fmaxf(a.m, b.m);
  Acc r;
  r.m = m;
  const float sa = a.s == 0.0f ? 0.0f : a.s * __builtin_amdgcn_exp2f((a.m - m) * kLog2e);
  const float sb = b.s == 0.0f ? 0.0f : b.s * __builtin_amdgcn_exp2f((b.m - m) * kLog2e);
  r.s = sa + sb;
  r.i = a.m > b.m ? a.i : (b.m > a.m ? b.i : min(a.i, b.i));
  return r;
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// the N values of a 16-byte chunk
template <bool BF>
__device__ __forceinline__ void unpack(u32x4 v, float* x) {
  if constexpr (BF) {
#pragma unroll
    for (int e = 0; e < 4; ++e) { x[2 * e] = bf_lo(v[e]); x[2 * e + 1] = bf_hi(v[e]); }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(v[e]);
  }
}

// Per thread: the chunks c = tid + 1024 k in increasing order.  A chunk whose maximum exceeds
// the running one raises it (rescaling the sum) and becomes the thread's best chunk; the
// index inside that chunk is found once at the end, so the common path tracks no indices:
// a max over the chunk, then one exp2 per element into the sum.
template <bool BF>
__global__ __launch_bounds__(kTokThreads) void cover_token_stats_kernel(const TokParams p) {
  constexpr int N = BF ? 8 : 4;  // elements per 16-byte chunk
  __shared__ float sm[kTokThreads / 64], ss[kTokThreads / 64];
  __shared__ int si[kTokThreads / 64];
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const char* row = p.logits + (int64_t)r * p.row_stride_bytes;
  auto chunk = [&](int c) __attribute__((always_inline)) {
    return *(gu32x4*)((__attribute__((address_space(1))) const char*)row + (int64_t)c * 16);
  };
  const int nfull = p.V / N;  // whole chunks; the last V % N elements come after
  // the placed token's logit, requested now (uniform: scalar loads, apart from the stream)
  float xy = __builtin_nanf("");
  if (p.logp) {
    const int y = p.tokens[r];
    if ((unsigned)y < (unsigned)p.V) {
      if constexpr (BF) {
        const uint32_t w = *(const uint32_t*)(row + ((int64_t)y * 2 & ~(int64_t)3));
        xy = (y & 1) ? bf_hi(w) : bf_lo(w);
      } else {
        xy = *(const float*)(row + (int64_t)y * 4);
      }
    }
  }
  float m = -INFINITY, s = 0.0f;
  int cbest = -1;
  auto fold = [&](const float* x, int c) __attribute__((always_inline)) {
    float cm = x[0];
#pragma unroll
    for (int e = 1; e < N; ++e) cm = __builtin_fmaxf(cm, x[e]);
    const float mn = __builtin_fmaxf(m, cm);
    s *= __builtin_amdgcn_exp2f((m - mn) * kLog2e);  // 1 unless the max was raised
    cbest = cm > m ? c : cbest;
    m = mn;
    const float nm = -mn * kLog2e;
    float a[N / 2];
#pragma unroll
    for (int e = 0; e < N / 2; ++e)
      a[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[2 * e], kLog2e, nm)) +
             __builtin_amdgcn_exp2f(__builtin_fmaf(x[2 * e + 1], kLog2e, nm));
    float t = a[0];
#pragma unroll
    for (int e = 1; e < N / 2; ++e) t += a[e];
    s += t;
  };
  // rounds in which every thread's chunks exist: no bounds tests
  constexpr int kRound = kTokThreads * kTokUnroll;
  int c0 = tid;
  for (; c0 - tid + kRound <= nfull; c0 += kRound) {
    u32x4 v[kTokUnroll];
#pragma unroll
    for (int u = 0; u < kTokUnroll; ++u) v[u] = chunk(c0 + u * kTokThreads);
#pragma unroll
    for (int u = 0; u < kTokUnroll; ++u) {
      float x[N];
      unpack<BF>(v[u], x);
      fold(x, c0 + u * kTokThreads);
    }
  }
  {  // the last, partial round
    u32x4 v[kTokUnroll];
#pragma unroll
    for (int u = 0; u < kTokUnroll; ++u) {
      const int c = c0 + u * kTokThreads;
      v[u] = c < nfull ? chunk(c) : (u32x4){};
    }
#pragma unroll
    for (int u = 0; u < kTokUnroll; ++u) {
      const int c = c0 + u * kTokThreads;
      if (c < nfull) {
        float x[N];
        unpack<BF>(v[u], x);
        fold(x, c);
      }
    }
  }
  // index of the maximum: the first element of the best chunk that holds it
  int ibest = 0x7fffffff;
  if (cbest >= 0) {
    float x[N];
    unpack<BF>(chunk(cbest), x);
#pragma unroll
    for (int e = N - 1; e >= 0; --e)
      if (x[e] == m) ibest = cbest * N + e;
  }
  Acc acc = {m, s, ibest};
  // the tail: one element per thread, read at its own width (never past the row's end)
  if (tid < p.V - nfull * N) {
    const int j = nfull * N + tid;
    const float xj = BF ? __uint_as_float((uint32_t)(*(const uint16_t*)(row + (int64_t)j * 2)) << 16)
                        : *(const float*)(row + (int64_t)j * 4);
    acc = merge(acc, Acc{xj, 1.0f, j});
  }
  // wave, then workgroup
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Acc o;
    o.m = __shfl_xor(acc.m, off);
    o.s = __shfl_xor(acc.s, off);
    o.i = __shfl_xor(acc.i, off);
    acc = merge(acc, o);
  }
  if (lane == 0) { sm[wave] = acc.m; ss[wave] = acc.s; si[wave] = acc.i; }
  __syncthreads();
  if (wave == 0) {  // the 16 wave results: a tree over lanes 0..15 of wave 0
    constexpr int W = kTokThreads / 64;
    Acc t = lane < W ? Acc{sm[lane], ss[lane], si[lane]} : Acc{-INFINITY, 0.0f, 0x7fffffff};
#pragma unroll
    for (int off = W / 2; off >= 1; off >>= 1) {
      Acc o;
      o.m = __shfl_xor(t.m, off);
      o.s = __shfl_xor(t.s, off);
      o.i = __shfl_xor(t.i, off);
      t = merge(t, o);
    }
    if (lane == 0) {
      const float lz = t.m + __builtin_amdgcn_logf(t.s) * kLn2;  // natural log-sum-exp
      if (p.conf) p.conf[r] = 1.0f / t.s;                         // exp(max - lz)
      if (p.argmax) p.argmax[r] = t.i;
      if (p.logp) p.logp[r] = xy - lz;
    }
  }
}


// ---------------------------------------------------------------------------------------
// attention masses
// ---------------------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct StatParams {
  const __bf16* q;
  const __bf16* kl;
  const __bf16* kc;
  const int32_t* seed_idx;
  const int32_t* n_seed;
  const float* lse;
  const uint8_t* masked;
  const uint8_t* drafted;
  float* ws;  // [B, Hq, 1 + KG, Lr]: per head, d_in, then the KG partials of d_out
  float* d_in;
  float* d_out;
  int B, Hq, Hkv, L, d, max_seeds, group, r0, Lr, NB;
  int KG, TPG;  // key groups, 32-key tiles per group
  float scale;
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

__device__ __forceinline__ f32x16 mfma16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

constexpr int kStatWaves = 8;

template <int D>
__global__ __launch_bounds__(64 * kStatWaves) void cover_attn_stats_kernel(const StatParams p) {
  constexpr int KS = D / 16;
  __shared__ uint32_t bits[COVER_MAX_L / 32];
  __shared__ float sdin[kStatWaves][COVER_STATS_MAX_LR];  // per-wave d_in partials over its blocks
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5, l32 = lane & 31;
  const int kg = blockIdx.x % p.KG, bh = blockIdx.x / p.KG;
  const int h = bh % p.Hq, b = bh / p.Hq;
  const int kt0 = kg * p.TPG, kt1 = min(p.NB, kt0 + p.TPG);  // this workgroup's key tiles
  float* const wsh = p.ws + ((int64_t)b * p.Hq + h) * (1 + p.KG) * p.Lr;
  const int g = h / p.group;
  const int L = p.L;
  const __bf16* qbh = p.q + b * p.q_sb + h * p.q_sh;
  const int64_t kvo = b * p.kv_sb + g * p.kv_sh;
  const float* lrow = p.lse + ((int64_t)b * p.Hq + h) * L;
  const float scale = p.scale;
  // Everything that does not depend on the seed set is requested before the seed bitmap is
  // built (the kernel is latency bound: a few dependent memory round trips): the seed count
  // with the first 512 seed positions, and for this wave's first query block its Q rows,
  // membership flags and lse, and the drafted flags of the group's first key tile.
  const int ns_raw = p.max_seeds > 0 ? p.n_seed[b] : 0;
  const int j_first = tid < p.max_seeds ? p.seed_idx[(int64_t)b * p.max_seeds + tid] : -1;
  // one query block's operands: Q (query qi, d-chunk 2ks+hl; also the A operand of S = Q K^T),
  // its membership flag byte, the lse of the lane's query and of the queries in S's registers
  bf16x8 qf[KS];
  uint8_t mq_byte = 0;
  float lse_own = 0.0f, lse_r[16];
  auto load_block = [&](int qb) {
    const int rb = qb * 32, qn = min(32, p.Lr - rb);
    const int qi = p.r0 + rb + min(l32, qn - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8*)(qbh + (int64_t)qi * p.q_sl + (2 * ks + hl) * 8);
    mq_byte = p.masked[(int64_t)b * p.Lr + rb + min(l32, qn - 1)];
    lse_own = lrow[qi];
#pragma unroll
    for (int r = 0; r < 16; ++r) lse_r[r] = lrow[p.r0 + rb + min(8 * (r >> 2) + 4 * hl + (r & 3), qn - 1)];
  };
  auto drafted_byte = [&](int kt) -> uint8_t {
    const int kb = kt * 32, kn = min(32, p.Lr - kb);
    return p.drafted[(int64_t)b * p.Lr + kb + min(l32, kn - 1)];
  };
  if (wave < p.NB) load_block(wave);
  const uint8_t dk_first = kt0 < kt1 ? drafted_byte(kt0) : (uint8_t)0;
  // seed bitmap of this sequence; the d_in rows start at zero
  const int nwords = (L + 31) >> 5;
  for (int w = tid; w < nwords; w += 64 * kStatWaves) bits[w] = 0u;
  for (int j = lane; j < p.Lr; j += 64) sdin[wave][j] = 0.0f;
  __syncthreads();
  const int ns = ns_raw < 0 ? 0 : (ns_raw > p.max_seeds ? p.max_seeds : ns_raw);
  if (tid < ns && (unsigned)j_first < (unsigned)L) atomicOr(&bits[j_first >> 5], 1u << (j_first & 31));
  for (int t = tid + 64 * kStatWaves; t < ns; t += 64 * kStatWaves) {  // long seed lists
    const int j = p.seed_idx[(int64_t)b * p.max_seeds + t];
    if ((unsigned)j < (unsigned)L) atomicOr(&bits[j >> 5], 1u << (j & 31));
  }
  __syncthreads();
  auto is_seed = [&](int j) -> bool { return (bits[j >> 5] >> (j & 31)) & 1u; };

  // the K rows of key tile kt (this lane's row, d-chunks 2ks+hl; seeds from the cache)
  auto load_k = [&](bf16x8* kf, int kt) {
    const int kb = kt * 32;
    const int kn = min(32, p.Lr - kb);
    const int kj = p.r0 + kb + min(l32, kn - 1);
    const __bf16* ksrc = (is_seed(kj) ? p.kc : p.kl) + kvo + (int64_t)kj * p.kv_sl;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = *(const bf16x8*)(ksrc + (2 * ks + hl) * 8);
  };
  for (int qb = wave; qb < p.NB; qb += kStatWaves) {
    if (qb != wave) load_block(qb);  // (the first block's operands were requested above)
    const int rb = qb * 32;                       // region offset of this query block
    const int qn = min(32, p.Lr - rb);            // queries of the block inside the region
    const int qi = p.r0 + rb + min(l32, qn - 1);  // this lane's query (clamped)
    // the first key tile's rows go out before the live diagonal row below, so that the two
    // round trips overlap
    bf16x8 kf[KS], kn_f[KS];
    if (kt0 < kt1) load_k(kf, kt0);
    // live diagonal score of this lane's position, for seed rows
    float s_live = 0.0f;
    const bool own_seed = l32 < qn && is_seed(qi);
    if (__builtin_amdgcn_ballot_w64(own_seed) != 0) {
      const __bf16* kr = p.kl + kvo + (int64_t)qi * p.kv_sl;
      float acc = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kv = *(const bf16x8*)(kr + (2 * ks + hl) * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = __builtin_fmaf((float)qf[ks][e], (float)kv[e], acc);
      }
      s_live = acc + __shfl_xor(acc, 32);
    }
    // membership bits of the block's queries
    const uint64_t mq = __builtin_amdgcn_ballot_w64(l32 < qn && mq_byte != 0) & 0xffffffffull;
    float dout = 0.0f;  // this lane's query: sum over drafted keys (its 16 of each tile)
    for (int kt = kt0; kt < kt1; ++kt) {
      if (kt + 1 < kt1) load_k(kn_f, kt + 1);  // the next tile's rows are requested first
      const int kb = kt * 32;
      const int kn = min(32, p.Lr - kb);
      f32x16 st = {}, sq = {};  // S^T (lane = query, registers = keys), S (lane = key)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        st = mfma16(kf[ks], qf[ks], st);
        sq = mfma16(qf[ks], kf[ks], sq);
      }
      const uint8_t dkb = kt == kt0 ? dk_first : drafted_byte(kt);
      const uint64_t dk = __builtin_amdgcn_ballot_w64(l32 < kn && dkb != 0) & 0xffffffffull;
      const bool diag_tile = kt == qb;
      float din = 0.0f;  // this lane's key: sum over masked queries (its 16 of the block)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 8 * (r >> 2) + 4 * hl + (r & 3);  // key (in st) / query (in sq) of register r
        // seed rows see their own live key on the diagonal
        float a = st[r], c = sq[r];
        if (diag_tile && row == l32 && own_seed) { a = s_live; c = s_live; }
        const float wt = __expf(a * scale - lse_own);
        const float wq = __expf(c * scale - lse_r[r]);
        dout += ((dk >> row) & 1) ? wt : 0.0f;
        din += ((mq >> row) & 1) ? wq : 0.0f;
      }
      din += __shfl_xor(din, 32);
      if (hl == 0 && l32 < kn) sdin[wave][kb + l32] += din;  // this wave's row only
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[ks] = kn_f[ks];
    }
    dout += __shfl_xor(dout, 32);
    if (hl == 0 && l32 < qn) wsh[(int64_t)(1 + kg) * p.Lr + rb + l32] = dout;
  }
  __syncthreads();
  // d_in of this head at the group's keys: the waves' rows added in a fixed order
  const int j1 = min(p.Lr, kt1 * 32);
  for (int j = kt0 * 32 + tid; j < j1; j += 64 * kStatWaves) {
    float s = 0.0f;
#pragma unroll
    for (int w = 0; w < kStatWaves; ++w) s += sdin[w][j];
    wsh[j] = s;
  }
}

// d_in(j) = (1/Hq) sum_h ws[h][0][j], d_out(j) = (1/Hq) sum_h sum_g ws[h][1+g][j].  A block
// of 32 keys x 8 head lanes: lane y adds heads y, y+8, ... (groups in order inside each
// head), then the 8 lane sums are added in order: a fixed order, so deterministic.
__global__ __launch_bounds__(256) void cover_attn_stats_reduce_kernel(const StatParams p) {
  __shared__ float sin_[8][32], sout[8][32];
  const int b = blockIdx.y, jx = threadIdx.x & 31, hy = threadIdx.x >> 5;
  const int j = blockIdx.x * 32 + jx;
  const int rec = 1 + p.KG;
  float din = 0.0f, dout = 0.0f;
  if (j < p.Lr) {
    const float* w = p.ws + (int64_t)b * p.Hq * rec * p.Lr + j;
    for (int h = hy; h < p.Hq; h += 8) {
      const float* wh = w + (int64_t)(rec * h) * p.Lr;
      din += wh[0];
      float part = 0.0f;
#pragma unroll 8
      for (int g = 0; g < p.KG; ++g) part += wh[(int64_t)(1 + g) * p.Lr];
      dout += part;
    }
  }
  sin_[hy][jx] = din;
  sout[hy][jx] = dout;
  __syncthreads();
  if (hy == 0 && j < p.Lr) {
    float a = 0.0f, c = 0.0f;
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      a += sin_[y][jx];
      c += sout[y][jx];
    }
    const float inv = 1.0f / (float)p.Hq;
    p.d_in[(int64_t)b * p.Lr + j] = a * inv;
    p.d_out[(int64_t)b * p.Lr + j] = c * inv;
  }
}

}  // namespace

hipError_t launch_token_stats(const TokenArgs& a, hipStream_t stream) {
  TokParams p;
  p.logits = (const char*)a.logits;
  p.tokens = a.tokens;
  p.logp = a.logp;
  p.conf = a.conf;
  p.argmax = a.argmax;
  p.row_stride_bytes = a.row_stride * (a.bf16 ? 2 : 4);
  p.V = a.V;
  if (a.bf16)
    hipLaunchKernelGGL(cover_token_stats_kernel<true>, dim3((unsigned)a.R), dim3(kTokThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(cover_token_stats_kernel<false>, dim3((unsigned)a.R), dim3(kTokThreads), 0, stream, p);
  return hipGetLastError();
}

// The workspace of cover_attn_stats_noalloc: one array per GPU, held until the process ends.
// Host code never passes `scratch` itself to a kernel (in host code the name stands for a
// host-side shadow, not a device address); it passes the address hipGetSymbolAddress gives
// for the current device.
static __device__ __align__(256) float scratch[COVER_STATS_SCRATCH_FLOATS];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t stats_scratch(float** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = (float*)p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

void stats_key_groups(int B, int Hq, int Lr, int* tpg, int* kg_out) {
  // key groups: about 256 workgroups in all (at most one group per 32-key tile, none empty)
  const int nb = (Lr + 31) / 32;
  const int64_t heads = (int64_t)B * Hq;
  int64_t kg = heads > 0 ? (256 + heads - 1) / heads : 1;
  kg = kg < 1 ? 1 : (kg > nb ? nb : kg);
  const int t = kg > 0 ? (int)((nb + kg - 1) / kg) : 1;
  *tpg = t;
  *kg_out = t > 0 ? (nb + t - 1) / t : 0;
}

int64_t stats_workspace_floats(int B, int Hq, int Lr) {
  int tpg, kg;
  stats_key_groups(B, Hq, Lr, &tpg, &kg);
  return (int64_t)B * Hq * (1 + kg) * Lr;
}

hipError_t launch_attn_stats(const StatsArgs& a, hipStream_t stream) {
  StatParams p;
  p.q = (const __bf16*)a.q;
  p.kl = (const __bf16*)a.k_live;
  p.kc = (const __bf16*)a.k_cache;
  p.seed_idx = a.seed_idx;
  p.n_seed = a.n_seed;
  p.lse = a.lse;
  p.masked = a.masked;
  p.drafted = a.drafted;
  p.ws = a.workspace;
  p.d_in = a.d_in;
  p.d_out = a.d_out;
  p.B = a.B; p.Hq = a.Hq; p.Hkv = a.Hkv; p.L = a.L; p.d = a.d; p.max_seeds = a.max_seeds;
  p.group = a.Hq / a.Hkv;
  p.r0 = a.r0; p.Lr = a.Lr;
  p.NB = (a.Lr + 31) / 32;
  stats_key_groups(a.B, a.Hq, a.Lr, &p.TPG, &p.KG);
  p.scale = a.scale;
  p.q_sb = a.q_sb; p.q_sh = a.q_sh; p.q_sl = a.q_sl;
  p.kv_sb = a.kv_sb; p.kv_sh = a.kv_sh; p.kv_sl = a.kv_sl;
  const int64_t nwg = (int64_t)a.B * a.Hq * p.KG;
  if (nwg > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (a.d == 128)
    hipLaunchKernelGGL(cover_attn_stats_kernel<128>, dim3((unsigned)nwg), dim3(64 * kStatWaves), 0, stream, p);
  else
    hipLaunchKernelGGL(cover_attn_stats_kernel<64>, dim3((unsigned)nwg), dim3(64 * kStatWaves), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cover_attn_stats_reduce_kernel, dim3((unsigned)((a.Lr + 31) / 32), (unsigned)a.B),
                     dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cover
