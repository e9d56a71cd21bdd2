/*
 * cover.h -- C ABI of the COVER hot path on MI355X (gfx950).
 *
 * COVER (arXiv 2602.06161) verifies previously unmasked "seed" positions inside the same
 * forward pass that drafts new tokens.  This library provides the two per-step device
 * operations of that pass:
 *
 *   cover_attn_fwd      bidirectional attention over the KV-cache-overridden memory with the
 *                       diagonal correction for seed rows (Sec. 5.1; App. B).
 *   cover_select_seeds  stability-aware seed scoring, adaptive budget and top-k
 *                       (Sec. 5.3).
 * and the producers of the selection's inputs:
 *   cover_token_stats   log p of the current token, confidence and argmax per position
 *                       (Sec. 5.3 u(j); Sec. 3 confidence and draft token).
 *   cover_attn_stats    in/out attention masses d_in, d_out over the response region
 *                       (Sec. 5.3 signals).
 *
 * Conventions shared by every entry point
 *   - Every data pointer is device memory owned by the caller (hipMalloc, or a framework
 *     allocator).  The library allocates nothing, frees nothing and never synchronises;
 *     work is enqueued on `stream` (0 = the null stream) and runs asynchronously.
 *   - Descriptor and pointer errors are detected on the host before anything is enqueued:
 *     the call then returns COVER_ERR_INVALID or COVER_ERR_UNSUPPORTED and writes nothing.
 *   - COVER_ERR_HIP means the HIP runtime rejected the launch.
 *   - Device-resident arguments (seed lists, seed counts, selection inputs) are not
 *     validated by default; their contract is stated per function.  Violations give
 *     unspecified results but never out-of-bounds memory accesses.  With the environment
 *     variable COVER_DEBUG=1 at the time of a call, the contract is checked on the device
 *     first and violations are recorded (see cover_debug_status).
 *   - Outputs must not alias inputs.
 */
#ifndef COVER_H
#define COVER_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COVER_OK = 0,
  COVER_ERR_INVALID = -1,     /* bad pointer, size, stride or alignment            */
  COVER_ERR_UNSUPPORTED = -2, /* valid request outside what the kernels implement  */
  COVER_ERR_HIP = -3          /* the HIP runtime reported an error at launch       */
} cover_status;

typedef enum { COVER_F32 = 0, COVER_BF16 = 1 } cover_dtype;

/* Largest sequence length the attention kernels accept (the seed bitmap of a sequence is
 * staged in on-chip memory). */
#define COVER_MAX_L 65536
/* Largest selection region per batch row. */
#define COVER_MAX_LR 16384

/*
 * Attention problem description.
 *   B        batch rows (>= 0; 0 is a no-op)
 *   Hq, Hkv  query heads and key/value heads; Hq % Hkv == 0; query head h reads key/value
 *            head h / (Hq / Hkv) (grouped-query attention; Hq == Hkv is plain multi-head)
 *   L        sequence length, prompt plus response (0 is a no-op; <= COVER_MAX_L)
 *   d        head dimension: 64 or 128
 *   max_seeds  row stride of seed_idx (>= 0)
 *   dtype    element type of q, k_live, v_live, k_cache, v_cache and out
 *   scale    score scale; 0 selects 1/sqrt(d) (Sec. 5.1)
 *   q_sb, q_sh, q_sl     element strides of q and out over (batch, head, position)
 *   kv_sb, kv_sh, kv_sl  element strides shared by k_live, v_live, k_cache, v_cache
 * The head dimension is contiguous (stride 1).  Base pointers must be 16-byte aligned and
 * every stride a multiple of 16 bytes' worth of elements.
 */
typedef struct {
  int32_t B, Hq, Hkv, L, d;
  int32_t max_seeds;
  cover_dtype dtype;
  float scale;
  int64_t q_sb, q_sh, q_sl;
  int64_t kv_sb, kv_sh, kv_sl;
} cover_attn_desc;

/*
 * cover_attn_fwd -- COVER attention of one layer (Sec. 5.1 "KV cache override" and
 * "diagonal correction"; App. B.1-B.4).
 *
 * For batch row b with seed set S_b = { seed_idx[b, t] : 0 <= t < n_seed[b] }, query head h
 * and key/value head g:
 *   override memory   K'_j = k_cache[b,g,j] if j in S_b, else k_live[b,g,j]; V' likewise
 *   row view          K^(i) = K', except K^(i)_i = k_live[b,g,i] when i in S_b (the key of
 *                     the masked input); V^(i) likewise
 *   out[b,h,i,:]      = sum_j softmax_j(scale * <q_i, K^(i)_j>) V^(i)_j
 *   lse[b,h,i]        = log sum_j exp(scale * <q_i, K^(i)_j>)   (natural log)
 * Non-seed rows therefore attend to the overridden memory unchanged, and each seed row sees
 * cached states everywhere except its own diagonal, which is the leave-one-out view the
 * paper's closed-form correction (App. B.4) produces.  All scores are kept in fp32 and the
 * softmax is taken over all L positions (non-causal).
 *
 * Arguments
 *   q        [B,Hq,L,d]   queries of the verification input (seeds masked)
 *   k_live, v_live   [B,Hkv,L,d]  keys/values of the verification input
 *   k_cache, v_cache [B,Hkv,L,d]  keys/values cached from the previous step, indexed by
 *                     absolute position; only rows at seed positions are read
 *   seed_idx [B,max_seeds] int32  seed positions; may be NULL when max_seeds == 0
 *   n_seed   [B] int32            seeds per batch row; may be NULL when max_seeds == 0
 *   out      [B,Hq,L,d]   output, same dtype and strides as q
 *   lse      [B,Hq,L] fp32, contiguous; may be NULL
 *   desc     problem description (host memory)
 * Device-data contract: 0 <= n_seed[b] <= max_seeds; seed_idx[b,0..n_seed[b]) distinct and in
 * [0, L) (any order).  n_seed outside [0, max_seeds] is clamped into it and entries outside
 * [0, L) are ignored.
 * Returns COVER_ERR_UNSUPPORTED for d not in {64, 128} or L > COVER_MAX_L.
 */
cover_status cover_attn_fwd(const void* q, const void* k_live, const void* v_live,
                            const void* k_cache, const void* v_cache,
                            const int32_t* seed_idx, const int32_t* n_seed,
                            void* out, float* lse,
                            const cover_attn_desc* desc, hipStream_t stream);

/*
 * Selection description.
 *   B           batch rows (>= 0)
 *   Lr          candidate region length per row (>= 0, <= COVER_MAX_LR)
 *   max_seeds   row stride / capacity of seed_idx (>= 0)
 *   pos_offset  added to every emitted position (the region's start in the sequence)
 */
typedef struct {
  int32_t B, Lr;
  int32_t max_seeds;
  int32_t pos_offset;
} cover_select_desc;

/*
 * cover_select_seeds -- stability-aware seed selection with an adaptive revision rate
 * (Sec. 5.3 "Stability aware seed scoring", "Adaptive revision rate").
 *
 * Per batch row, over region positions j in [0, Lr):
 *   flags bit 0 = j is unmasked (j in U_t); bit 1 = j is excluded (a seed of the previous
 *   step, or its ReMask budget is used up); other bits are ignored.
 *   score s_j   = ((-(double)logp_j) * (1 + (double)d_in_j)) / (1 + (double)d_out_j), for j
 *                 in U_t, in IEEE fp64 with round-to-nearest and this exact association
 *   mean        = (sum of s_j over U_t) / |U_t|, the sum taken as a stride-halving tree over
 *                 the region zero-padded to the next power of two
 *   budget      = least k >= 0 with k*k >= c, c = #{ j in U_t : s_j > mean } (= n_t pi_t)
 *   selection   = the min(budget, #eligible, max_seeds) eligible positions (in U_t, not
 *                 excluded) ranked first by score descending then position ascending
 * Outputs
 *   seed_idx [B,max_seeds] int32: selected positions + pos_offset in ascending order,
 *            then -1; n_seed [B] int32: how many; score [B,Lr] fp64 (may be NULL): s_j on
 *            U_t, 0 elsewhere.  The results are bit-exact functions of the inputs.
 * Inputs: logp, d_in, d_out fp32 [B,Lr] row-major (logp = log p_j(y_j) <= 0, the model's
 * log-probability of the token currently at j; d_in, d_out >= 0 are the in/out attention
 * masses); flags uint8 [B,Lr].  Values at positions outside U_t are ignored (they may be
 * anything, including non-finite).  Device-data contract: values on U_t finite, d_in and
 * d_out >= 0.
 * The output layout matches cover_attn_fwd's seed_idx / n_seed, so the next step's
 * attention can consume it without a host round-trip.
 */
cover_status cover_select_seeds(const float* logp, const float* d_in, const float* d_out,
                                const uint8_t* flags,
                                int32_t* seed_idx, int32_t* n_seed, double* score,
                                const cover_select_desc* desc, hipStream_t stream);

/*
 * Token statistics description.
 *   R           rows (positions; >= 0, 0 is a no-op)
 *   V           vocabulary size (>= 1)
 *   dtype       element type of logits (COVER_BF16 or COVER_F32)
 *   row_stride  elements between consecutive rows of logits (>= V); the base pointer and
 *               row_stride * element size must be multiples of 16 bytes
 */
typedef struct {
  int32_t R, V;
  cover_dtype dtype;
  int64_t row_stride;
} cover_token_desc;

/*
 * cover_token_stats -- per-position statistics of the model's output distribution
 * (Sec. 5.3: u(j) = -log p_j(y_j); Sec. 3: confidence = max_v p_j(v), draft token = argmax).
 *
 * For row r with logits x_r[0..V) and lz_r = log sum_v exp(x_r[v]) (natural log):
 *   logp[r]   = x_r[tokens[r]] - lz_r
 *   conf[r]   = exp(max_v x_r[v] - lz_r)
 *   argmax[r] = the smallest v attaining max_v x_r[v]
 * Arithmetic in fp32 (exp/log of the exp2/log2 units); one pass over the logits.
 * Arguments: logits [R, row_stride] (device); tokens int32 [R] (device; may be NULL when
 * logp is NULL); logp, conf fp32 [R] and argmax int32 [R] (device outputs, each may be
 * NULL).  Device-data contract: tokens in [0, V) (a token outside gives logp = NaN, never
 * an out-of-bounds read); logits finite.
 */
cover_status cover_token_stats(const void* logits, const int32_t* tokens,
                               float* logp, float* conf, int32_t* argmax,
                               const cover_token_desc* desc, hipStream_t stream);

/*
 * cover_token_sample -- temperature sampling of the draft tokens (the stochastic decoding of
 * the paper's appendix on robustness): per row r of logits (same description and layout
 * rules as cover_token_stats),
 *   token[r] = argmax_v (x_v / T + g_v), g_v = -ln(-ln u_v) (Gumbel-max: a draw from
 *              softmax(x / T); the smallest v on ties)
 *   prob[r]  = softmax(x / T) at token[r] (the confidence compared with the drafting
 *              threshold; may be NULL)
 * u_v = ((w >> 9) + 1/2) 2^-23 with w word v % 4 of Philox4x32-10 (Salmon et al., SC 2011)
 * at counter (v / 4, r, step, 0) and key (seed mod 2^32, seed >> 32): a fixed function of
 * (seed, step, row, token), reproducible across launches and devices.  Arithmetic in fp32.
 * temperature: > 0 and finite.  token int32 [R], prob fp32 [R]: device outputs.
 */
cover_status cover_token_sample(const void* logits, float temperature, uint64_t seed, uint32_t step,
                                int32_t* token, float* prob, const cover_token_desc* desc,
                                hipStream_t stream);

/*
 * Attention-mass description: the attention problem of cover_attn_fwd (same fields and
 * stride rules; bf16 only) plus the response region [r0, r0 + Lr).
 *   r0, Lr      0 <= r0, 1 <= Lr, r0 + Lr <= L (Lr == 0 is a no-op)
 */
typedef struct {
  cover_attn_desc attn;
  int32_t r0, Lr;
} cover_stats_desc;

/* Largest response region cover_attn_stats accepts. */
#define COVER_STATS_MAX_LR 2048
/* An upper bound of the workspace of cover_attn_stats in floats, valid for every launch:
 * B * Hq * (1 + ceil(Lr / 32)) * Lr.  cover_attn_stats_workspace gives the exact need. */
#define COVER_ATTN_STATS_WORKSPACE(B, Hq, Lr) \
  ((int64_t)(B) * (Hq) * (1 + ((int64_t)(Lr) + 31) / 32) * (Lr))

/*
 * cover_attn_stats -- the in/out attention masses of Sec. 5.3 from the last layer's
 * corrected attention weights, averaged over query heads, restricted to the response region.
 *
 * With w^(h)_{i,j} = exp(scale <q_i, K^(i)_j> - lse[b,h,i]) the weights of cover_attn_fwd
 * (override memory, leave-one-out view for seed rows, normalised over all L positions by
 * the lse that call returned) and A_{i->j} = (1/Hq) sum_h w^(h)_{i,j}, for region positions
 * j = r0 + t, t in [0, Lr):
 *   d_in[b,t]  = sum over region rows i with masked[b, i-r0]  of A_{i->j}
 *   d_out[b,t] = sum over region columns i with drafted[b, i-r0] of A_{j->i}
 * Arguments: q, k_live, k_cache, seed_idx, n_seed as for cover_attn_fwd (v is not needed);
 * lse fp32 [B,Hq,L] contiguous, as returned by cover_attn_fwd for the same inputs;
 * masked, drafted uint8 [B,Lr] (nonzero = member; device); d_in, d_out fp32 [B,Lr]
 * (device outputs); workspace: device fp32 buffer of at least
 * cover_attn_stats_workspace(B, Hq, Lr) floats (COVER_ATTN_STATS_WORKSPACE(B, Hq, Lr) always
 * suffices) owned by the caller (its contents on entry are ignored, on exit unspecified).
 * Two kernel launches on `stream`; partial sums are added in a fixed order, so the results
 * are deterministic.  Weights are formed in fp32 from the fp32 lse.
 * Returns COVER_ERR_UNSUPPORTED for a dtype other than bf16, d not in {64, 128},
 * L > COVER_MAX_L or Lr > COVER_STATS_MAX_LR.
 */
cover_status cover_attn_stats(const void* q, const void* k_live, const void* k_cache,
                              const int32_t* seed_idx, const int32_t* n_seed, const float* lse,
                              const uint8_t* masked, const uint8_t* drafted,
                              float* d_in, float* d_out, float* workspace,
                              const cover_stats_desc* desc, hipStream_t stream);

/*
 * cover_attn_stats_workspace -- floats of workspace a cover_attn_stats call with these B, Hq
 * and Lr uses: B * Hq * (1 + G) * Lr, with G the number of key groups the launch splits the
 * region's 32-key tiles into (about 256 workgroups in all; G <= ceil(Lr / 32)).  A host
 * function: no GPU work.  Returns -1 for negative arguments.
 */
int64_t cover_attn_stats_workspace(int32_t B, int32_t Hq, int32_t Lr);

/* Floats of the library's own per-GPU workspace behind cover_attn_stats_noalloc (4 MiB). */
#define COVER_STATS_SCRATCH_FLOATS (1 << 20)

/*
 * cover_attn_stats_noalloc -- cover_attn_stats without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation).  Same arguments, results and checks as cover_attn_stats, except
 * that the partial sums go to a fixed array inside the library: COVER_STATS_SCRATCH_FLOATS
 * floats on each GPU the library runs on, held until the process ends (its device address is
 * looked up on the first call on each GPU; nothing is allocated, by this call or any other).
 * Every call on one GPU shares that array and the work it enqueues reads back only what the
 * same call wrote, so calls that run one after another (on one stream, or ordered by events)
 * are independent; calls that can overlap on one GPU (different streams with no ordering)
 * race on the array and give unspecified results.
 * Returns COVER_ERR_UNSUPPORTED when cover_attn_stats_workspace(B, Hq, Lr) exceeds
 * COVER_STATS_SCRATCH_FLOATS (for instance B * Hq > 256 at Lr = 2048, or B * Hq > 1024 at
 * Lr = 512), before anything is enqueued; COVER_ERR_HIP if the array's address cannot be
 * obtained.
 */
cover_status cover_attn_stats_noalloc(const void* q, const void* k_live, const void* k_cache,
                                      const int32_t* seed_idx, const int32_t* n_seed,
                                      const float* lse, const uint8_t* masked,
                                      const uint8_t* drafted, float* d_in, float* d_out,
                                      const cover_stats_desc* desc, hipStream_t stream);

/*
 * Block-query attention description: the attention problem of cover_attn_fwd (same fields
 * and stride rules, with attn.L the number of keys; q and out hold Lq rows at the q strides)
 * plus the query block [q_off, q_off + Lq) and the number of key splits.
 *   q_off, Lq   0 <= q_off, 0 <= Lq, q_off + Lq <= attn.L (Lq == 0 is a no-op)
 *   n_split     1 <= n_split <= 256.  1: one launch, one workgroup per 32 query rows whose
 *               waves split the keys among themselves (no workspace).  > 1: the keys are cut
 *               into n_split ranges processed by separate workgroups and merged by a second
 *               launch (more workgroups per query row; the partial results go through the
 *               workspace)
 */
typedef struct {
  cover_attn_desc attn;
  int32_t q_off, Lq;
  int32_t n_split;
} cover_rect_desc;

/* 4-byte words per (row, split) record of the cover_attn_rect workspace. */
#define COVER_RECT_RECORD 68
/* Workspace of cover_attn_rect in floats (none for n_split == 1). */
#define COVER_ATTN_RECT_WORKSPACE(B, Hq, Lq, n_split) \
  ((n_split) > 1 ? (int64_t)(B) * (Hq) * (n_split) * (Lq) * COVER_RECT_RECORD : (int64_t)0)

/*
 * cover_attn_rect -- COVER attention for one block of query rows against all L keys (the
 * prefix-cache decoding COVER is combined with in Sec. 6.6: the block's rows are recomputed,
 * the other positions' keys and values are reused).
 *
 * Row r of out/lse is row q_off + r of what cover_attn_fwd computes for a length-L sequence
 * with the same k_live, v_live, k_cache, v_cache and seeds (Sec. 5.1 override memory and
 * the leave-one-out diagonal of a seed row, App. B): q holds only the block's Lq rows.
 * Seeds may lie anywhere in [0, L), inside the block or not.
 * Arguments as for cover_attn_fwd; out [B,Hq,Lq,d] at the q strides; lse fp32 [B,Hq,Lq]
 * contiguous (may be NULL); workspace: for n_split > 1 a device fp32 buffer of
 * COVER_ATTN_RECT_WORKSPACE(B, Hq, Lq, n_split) floats owned by the caller (contents on
 * entry ignored, on exit unspecified); for n_split == 1 not used (may be NULL).  One kernel
 * launch on `stream` for n_split == 1, two otherwise (partial results per key split, then
 * a merge); every sum runs in a fixed order, so results are deterministic.
 * Returns COVER_ERR_UNSUPPORTED for a dtype other than bf16, d != 128, L > COVER_MAX_L, or
 * n_split == 1 with kv_sl >= 2^26.
 */
cover_status cover_attn_rect(const void* q, const void* k_live, const void* v_live,
                             const void* k_cache, const void* v_cache,
                             const int32_t* seed_idx, const int32_t* n_seed,
                             void* out, float* lse, float* workspace,
                             const cover_rect_desc* desc, hipStream_t stream);

/*
 * Decoding-state update description.
 *   B              batch rows (>= 0; 0 is a no-op)
 *   Lr             region length per row (>= 0, <= COVER_MAX_LR)
 *   max_seeds      row stride / capacity of seed_idx (>= 0)
 *   pos_offset     absolute position of region index 0 (seed_idx holds absolute positions)
 *   mask_id        the [MASK] token id
 *   draft_cap      most positions drafted per row and step (>= 0)
 *   remask_budget  ReMasks after which a position is no longer selectable as a seed
 *   tau            confidence threshold (not NaN), used for drafting and for Replace
 *   min_draft      0 <= min_draft <= draft_cap; 0 is the paper's rule.  Otherwise, when fewer
 *                  than min_draft masked positions pass tau, the min_draft most confident
 *                  masked positions (same order; NaN confidences never drafted) are drafted
 *                  instead, so a decoding loop always progresses (not in the paper)
 */
typedef struct {
  int32_t B, Lr;
  int32_t max_seeds;
  int32_t pos_offset;
  int32_t mask_id;
  int32_t draft_cap;
  int32_t remask_budget;
  float tau;
  int32_t min_draft;
} cover_update_desc;

/*
 * cover_decode_update -- one step's update of the decoding state (Sec. 5.2 drafting and
 * revision outcomes, Sec. 3 state update, Sec. 5.3 ReMask budget and exclusion), per row:
 *   drafting   D = the masked positions (tokens == mask_id) with conf > tau, compared in
 *              fp32; if more than draft_cap qualify, the draft_cap largest by (conf
 *              descending, position ascending).  Each takes its argmax token.
 *   revision   each previous seed i (seed_idx[b, :n_seed[b]] - pos_offset; entries outside
 *              [0, Lr) or at masked positions are ignored, repeats count once):
 *              Keep if argmax_i == tokens_i; else Replace (tokens_i = argmax_i) if
 *              conf_i > tau; else ReMask (tokens_i = mask_id, remask_count_i += 1).
 *   flags      bit 0 = unmasked after the update; bit 1 = i was a seed, or
 *              remask_count_i >= remask_budget -- the flags cover_select_seeds takes next.
 * Arguments (all device memory, row-major [B,Lr] unless stated):
 *   tokens int32 (in/out; the state U/M of the region), argmax int32 and conf fp32 (the
 *   step's argmax token and its probability, e.g. from cover_token_stats), seed_idx int32
 *   [B,max_seeds] and n_seed int32 [B] (the seeds of the step, as cover_select_seeds
 *   emits them; may be NULL when max_seeds == 0), remask_count int32 (in/out),
 *   flags uint8 (out, may be NULL), drafted uint8 (out, 1 = drafted this step, may be NULL),
 *   counts int32 [B,5] (out, may be NULL): |D|, kept, replaced, remasked, masked after;
 *   last_unmask int32 (in/out, may be NULL): the token of each position's most recent
 *   [MASK] -> token transition (-1 = none yet); every drafted position records its new
 *   token (Replace is not an unmasking and leaves it alone);
 *   flipflops int32 [B] (out, may be NULL; needs last_unmask): flip-flop events of the
 *   step (Sec. 4 definition): drafted positions whose new token equals their last_unmask
 *   entry on entry.
 * One kernel launch on `stream`; every result is an exact function of the inputs.  n_seed
 * values outside [0, max_seeds] are clamped.
 */
cover_status cover_decode_update(int32_t* tokens, const int32_t* argmax, const float* conf,
                                 const int32_t* seed_idx, const int32_t* n_seed,
                                 int32_t* remask_count, uint8_t* flags, uint8_t* drafted,
                                 int32_t* counts, int32_t* last_unmask, int32_t* flipflops,
                                 const cover_update_desc* desc, hipStream_t stream);

/*
 * cover_debug_status -- the contract checks enabled by COVER_DEBUG=1 (a debugging aid for
 * integrations; not for production paths).
 *
 * While the environment variable COVER_DEBUG is "1", every cover_attn_fwd, cover_attn_rect
 * and cover_attn_stats call first checks its seed lists, and every cover_select_seeds call its
 * inputs on U_t, with a small kernel on the same stream; a violation sets bits of a status
 * word kept on the current GPU:
 */
#define COVER_DEBUG_SEED_COUNT 1        /* some n_seed[b] outside [0, max_seeds]            */
#define COVER_DEBUG_SEED_RANGE 2        /* a listed seed position outside [0, L)             */
#define COVER_DEBUG_SEED_DUPLICATE 4    /* a seed position listed twice in one batch row     */
#define COVER_DEBUG_SELECT_NONFINITE 8  /* logp, d_in or d_out not finite at a j in U_t      */
#define COVER_DEBUG_SELECT_NEGATIVE 16  /* d_in or d_out negative at a j in U_t              */
/*
 * cover_debug_status copies that word of the current GPU to *status (host memory) after
 * the work already enqueued on `stream` and, if clear != 0, resets it to 0.  Unlike every
 * other entry point it waits for `stream` to finish before returning.  Bits accumulate
 * across calls until cleared; the word starts at 0.  Returns COVER_ERR_INVALID for a NULL
 * status, COVER_ERR_HIP if the copy fails.
 */
cover_status cover_debug_status(int32_t* status, int32_t clear, hipStream_t stream);

/* Static string naming a status code. */
const char* cover_status_str(cover_status s);

/* Library version as major*10000 + minor*100 + patch. */
int32_t cover_version(void);

#ifdef __cplusplus
}
#endif

#endif /* COVER_H */
