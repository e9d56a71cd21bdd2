// C ABI of the COVER library: host-side validation, then one kernel launch per call.
// Every check here runs before anything is enqueued, so a rejected call writes nothing.
#include <math.h>
#include <stdint.h>

#include "cover.h"
#include "cover_internal.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

cover_status hip_status(hipError_t e) { return e == hipSuccess ? COVER_OK : COVER_ERR_HIP; }

}  // namespace

extern "C" {

const char* cover_status_str(cover_status s) {
  switch (s) {
    case COVER_OK: return "COVER_OK";
    case COVER_ERR_INVALID: return "COVER_ERR_INVALID";
    case COVER_ERR_UNSUPPORTED: return "COVER_ERR_UNSUPPORTED";
    case COVER_ERR_HIP: return "COVER_ERR_HIP";
  }
  return "COVER_ERR_UNKNOWN";
}

int32_t cover_version(void) { return 100; }  // 0.1.0

cover_status cover_debug_status(int32_t* status, int32_t clear, hipStream_t stream) {
  if (!status) return COVER_ERR_INVALID;
  return hip_status(cover::debug_status(status, clear != 0, stream));
}

cover_status cover_attn_fwd(const void* q, const void* k_live, const void* v_live,
                            const void* k_cache, const void* v_cache,
                            const int32_t* seed_idx, const int32_t* n_seed,
                            void* out, float* lse,
                            const cover_attn_desc* desc, hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_attn_desc& D = *desc;
  if (D.B < 0 || D.L < 0 || D.Hq < 1 || D.Hkv < 1 || D.d < 1 || D.max_seeds < 0)
    return COVER_ERR_INVALID;
  if (D.Hq % D.Hkv != 0) return COVER_ERR_INVALID;
  if (D.dtype != COVER_F32 && D.dtype != COVER_BF16) return COVER_ERR_INVALID;
  if (!(D.scale >= 0.0f) || isinf(D.scale)) return COVER_ERR_INVALID;  // rejects NaN too
  if (D.d != 64 && D.d != 128) return COVER_ERR_UNSUPPORTED;
  if (D.L > COVER_MAX_L) return COVER_ERR_UNSUPPORTED;
  if (D.B == 0 || D.L == 0) return COVER_OK;

  const int64_t esz = D.dtype == COVER_BF16 ? 2 : 4;
  const int64_t vec = 16 / esz;  // elements per 16-byte chunk
  const void* tensors[6] = {q, k_live, v_live, k_cache, v_cache, out};
  for (const void* t : tensors)
    if (!t || !aligned(t, 16)) return COVER_ERR_INVALID;
  const int64_t strides[6] = {D.q_sb, D.q_sh, D.q_sl, D.kv_sb, D.kv_sh, D.kv_sl};
  for (int64_t s : strides)
    if (s < 0 || s % vec != 0) return COVER_ERR_INVALID;
  if (D.L > 1 && (D.q_sl < D.d || D.kv_sl < D.d)) return COVER_ERR_INVALID;
  if (D.max_seeds > 0) {
    if (!seed_idx || !n_seed || !aligned(seed_idx, 4) || !aligned(n_seed, 4))
      return COVER_ERR_INVALID;
  }
  if (lse && !aligned(lse, 4)) return COVER_ERR_INVALID;
  const int64_t qtile = D.dtype == COVER_BF16 ? 128 : 64;
  if ((int64_t)D.B * D.Hq * ((D.L + qtile - 1) / qtile) > 0x7fffffffLL) return COVER_ERR_UNSUPPORTED;

  cover::AttnArgs a;
  a.q = q; a.k_live = k_live; a.v_live = v_live; a.k_cache = k_cache; a.v_cache = v_cache;
  a.seed_idx = D.max_seeds > 0 ? seed_idx : nullptr;
  a.n_seed = D.max_seeds > 0 ? n_seed : nullptr;
  a.out = out; a.lse = lse;
  a.B = D.B; a.Hq = D.Hq; a.Hkv = D.Hkv; a.L = D.L; a.d = D.d; a.max_seeds = D.max_seeds;
  a.scale = D.scale > 0.0f ? D.scale : 1.0f / sqrtf((float)D.d);
  a.q_sb = D.q_sb; a.q_sh = D.q_sh; a.q_sl = D.q_sl;
  a.kv_sb = D.kv_sb; a.kv_sh = D.kv_sh; a.kv_sl = D.kv_sl;
  if (cover::debug_enabled()) {
    const hipError_t e = cover::launch_check_seeds(a.seed_idx, a.n_seed, D.B, D.max_seeds, D.L, stream);
    if (e != hipSuccess) return COVER_ERR_HIP;
  }
  if (D.dtype != COVER_BF16) return hip_status(cover::launch_attn_f32(a, stream));
  if (D.d == 128) return hip_status(cover::launch_attn_bf16_w4(a, stream));
  return hip_status(cover::launch_attn_bf16(a, stream));  // d = 64
}

cover_status cover_select_seeds(const float* logp, const float* d_in, const float* d_out,
                                const uint8_t* flags,
                                int32_t* seed_idx, int32_t* n_seed, double* score,
                                const cover_select_desc* desc, hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_select_desc& D = *desc;
  if (D.B < 0 || D.Lr < 0 || D.max_seeds < 0) return COVER_ERR_INVALID;
  if (D.Lr > COVER_MAX_LR) return COVER_ERR_UNSUPPORTED;
  if (D.B == 0) return COVER_OK;
  if (!n_seed || !aligned(n_seed, 4)) return COVER_ERR_INVALID;
  if (D.max_seeds > 0 && (!seed_idx || !aligned(seed_idx, 4))) return COVER_ERR_INVALID;
  if (D.Lr > 0) {
    if (!logp || !d_in || !d_out || !flags) return COVER_ERR_INVALID;
    if (!aligned(logp, 4) || !aligned(d_in, 4) || !aligned(d_out, 4)) return COVER_ERR_INVALID;
  }
  if (score && !aligned(score, 8)) return COVER_ERR_INVALID;
  // emitted positions must stay representable
  if ((int64_t)D.pos_offset + D.Lr > 0x7fffffffLL || (int64_t)D.pos_offset < -0x7fffffffLL)
    return COVER_ERR_INVALID;

  cover::SelectArgs a;
  a.logp = logp; a.d_in = d_in; a.d_out = d_out; a.flags = flags;
  a.seed_idx = seed_idx; a.n_seed = n_seed; a.score = score;
  a.B = D.B; a.Lr = D.Lr; a.max_seeds = D.max_seeds; a.pos_offset = D.pos_offset;
  if (cover::debug_enabled()) {
    const hipError_t e = cover::launch_check_select(logp, d_in, d_out, flags, (int64_t)D.B * D.Lr, stream);
    if (e != hipSuccess) return COVER_ERR_HIP;
  }
  return hip_status(cover::launch_select(a, stream));
}

cover_status cover_token_stats(const void* logits, const int32_t* tokens,
                               float* logp, float* conf, int32_t* argmax,
                               const cover_token_desc* desc, hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_token_desc& D = *desc;
  if (D.R < 0 || D.V < 1 || D.row_stride < D.V) return COVER_ERR_INVALID;
  if (D.dtype != COVER_F32 && D.dtype != COVER_BF16) return COVER_ERR_INVALID;
  const int64_t esz = D.dtype == COVER_BF16 ? 2 : 4;
  if ((D.row_stride * esz) % 16 != 0) return COVER_ERR_INVALID;
  if (D.R == 0) return COVER_OK;
  if (!logits || !aligned(logits, 16)) return COVER_ERR_INVALID;
  if (logp && (!tokens || !aligned(tokens, 4) || !aligned(logp, 4))) return COVER_ERR_INVALID;
  if ((conf && !aligned(conf, 4)) || (argmax && !aligned(argmax, 4))) return COVER_ERR_INVALID;
  cover::TokenArgs a;
  a.logits = logits; a.tokens = tokens; a.logp = logp; a.conf = conf; a.argmax = argmax;
  a.R = D.R; a.V = D.V; a.bf16 = D.dtype == COVER_BF16; a.row_stride = D.row_stride;
  return hip_status(cover::launch_token_stats(a, stream));
}

cover_status cover_token_sample(const void* logits, float temperature, uint64_t seed, uint32_t step,
                                int32_t* token, float* prob, const cover_token_desc* desc,
                                hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_token_desc& D = *desc;
  if (D.R < 0 || D.V < 1 || D.row_stride < D.V) return COVER_ERR_INVALID;
  if (D.dtype != COVER_F32 && D.dtype != COVER_BF16) return COVER_ERR_INVALID;
  const int64_t esz = D.dtype == COVER_BF16 ? 2 : 4;
  if ((D.row_stride * esz) % 16 != 0) return COVER_ERR_INVALID;
  if (!(temperature > 0.0f) || isinf(temperature)) return COVER_ERR_INVALID;
  if (D.R == 0) return COVER_OK;
  if (!logits || !aligned(logits, 16) || !token || !aligned(token, 4)) return COVER_ERR_INVALID;
  if (prob && !aligned(prob, 4)) return COVER_ERR_INVALID;
  cover::SampleArgs a;
  a.logits = logits; a.token = token; a.prob = prob;
  a.R = D.R; a.V = D.V; a.bf16 = D.dtype == COVER_BF16; a.row_stride = D.row_stride;
  a.temperature = temperature; a.seed = seed; a.step = step;
  return hip_status(cover::launch_token_sample(a, stream));
}

int64_t cover_attn_stats_workspace(int32_t B, int32_t Hq, int32_t Lr) {
  if (B < 0 || Hq < 0 || Lr < 0) return -1;
  if (B == 0 || Hq == 0 || Lr == 0) return 0;
  return cover::stats_workspace_floats(B, Hq, Lr);
}

}  // extern "C"

namespace {

// Host-side checks shared by cover_attn_stats and cover_attn_stats_noalloc: fills `a` (all
// but the workspace) and returns COVER_OK, or the error to return before anything is enqueued.
// *empty is set for a valid call with nothing to do.
cover_status prepare_stats(const void* q, const void* k_live, const void* k_cache,
                           const int32_t* seed_idx, const int32_t* n_seed, const float* lse,
                           const uint8_t* masked, const uint8_t* drafted, float* d_in,
                           float* d_out, const cover_stats_desc* desc, cover::StatsArgs& a,
                           bool* empty) {
  *empty = false;
  if (!desc) return COVER_ERR_INVALID;
  const cover_attn_desc& D = desc->attn;
  const int32_t r0 = desc->r0, Lr = desc->Lr;
  if (D.B < 0 || D.L < 0 || D.Hq < 1 || D.Hkv < 1 || D.d < 1 || D.max_seeds < 0)
    return COVER_ERR_INVALID;
  if (D.Hq % D.Hkv != 0) return COVER_ERR_INVALID;
  if (D.dtype != COVER_F32 && D.dtype != COVER_BF16) return COVER_ERR_INVALID;
  if (!(D.scale >= 0.0f) || isinf(D.scale)) return COVER_ERR_INVALID;
  if (r0 < 0 || Lr < 0 || (int64_t)r0 + Lr > D.L) return COVER_ERR_INVALID;
  if (D.dtype != COVER_BF16) return COVER_ERR_UNSUPPORTED;
  if (D.d != 64 && D.d != 128) return COVER_ERR_UNSUPPORTED;
  if (D.L > COVER_MAX_L || Lr > COVER_STATS_MAX_LR) return COVER_ERR_UNSUPPORTED;
  if (D.B == 0 || Lr == 0) {
    *empty = true;
    return COVER_OK;
  }
  const void* tensors[3] = {q, k_live, k_cache};
  for (const void* t : tensors)
    if (!t || !aligned(t, 16)) return COVER_ERR_INVALID;
  const int64_t strides[6] = {D.q_sb, D.q_sh, D.q_sl, D.kv_sb, D.kv_sh, D.kv_sl};
  for (int64_t s : strides)
    if (s < 0 || s % 8 != 0) return COVER_ERR_INVALID;
  if (D.L > 1 && (D.q_sl < D.d || D.kv_sl < D.d)) return COVER_ERR_INVALID;
  if (D.max_seeds > 0 && (!seed_idx || !n_seed || !aligned(seed_idx, 4) || !aligned(n_seed, 4)))
    return COVER_ERR_INVALID;
  if (!lse || !aligned(lse, 4) || !masked || !drafted) return COVER_ERR_INVALID;
  if (!d_in || !d_out || !aligned(d_in, 4) || !aligned(d_out, 4)) return COVER_ERR_INVALID;
  a.q = q; a.k_live = k_live; a.k_cache = k_cache;
  a.seed_idx = D.max_seeds > 0 ? seed_idx : nullptr;
  a.n_seed = D.max_seeds > 0 ? n_seed : nullptr;
  a.lse = lse; a.masked = masked; a.drafted = drafted;
  a.d_in = d_in; a.d_out = d_out; a.workspace = nullptr;
  a.B = D.B; a.Hq = D.Hq; a.Hkv = D.Hkv; a.L = D.L; a.d = D.d; a.max_seeds = D.max_seeds;
  a.r0 = r0; a.Lr = Lr;
  a.scale = D.scale > 0.0f ? D.scale : 1.0f / sqrtf((float)D.d);
  a.q_sb = D.q_sb; a.q_sh = D.q_sh; a.q_sl = D.q_sl;
  a.kv_sb = D.kv_sb; a.kv_sh = D.kv_sh; a.kv_sl = D.kv_sl;
  return COVER_OK;
}

cover_status run_stats(const cover::StatsArgs& a, const cover_stats_desc* desc, hipStream_t stream) {
  if (cover::debug_enabled()) {
    const hipError_t e = cover::launch_check_seeds(a.seed_idx, a.n_seed, a.B, a.max_seeds,
                                                   desc->attn.L, stream);
    if (e != hipSuccess) return COVER_ERR_HIP;
  }
  return hip_status(cover::launch_attn_stats(a, stream));
}

}  // namespace

extern "C" {

cover_status cover_attn_stats(const void* q, const void* k_live, const void* k_cache,
                              const int32_t* seed_idx, const int32_t* n_seed, const float* lse,
                              const uint8_t* masked, const uint8_t* drafted,
                              float* d_in, float* d_out, float* workspace,
                              const cover_stats_desc* desc, hipStream_t stream) {
  cover::StatsArgs a;
  bool empty;
  const cover_status st = prepare_stats(q, k_live, k_cache, seed_idx, n_seed, lse, masked,
                                        drafted, d_in, d_out, desc, a, &empty);
  if (st != COVER_OK || empty) return st;
  if (!workspace || !aligned(workspace, 4)) return COVER_ERR_INVALID;
  a.workspace = workspace;
  return run_stats(a, desc, stream);
}

cover_status cover_attn_stats_noalloc(const void* q, const void* k_live, const void* k_cache,
                                      const int32_t* seed_idx, const int32_t* n_seed,
                                      const float* lse, const uint8_t* masked,
                                      const uint8_t* drafted, float* d_in, float* d_out,
                                      const cover_stats_desc* desc, hipStream_t stream) {
  cover::StatsArgs a;
  bool empty;
  const cover_status st = prepare_stats(q, k_live, k_cache, seed_idx, n_seed, lse, masked,
                                        drafted, d_in, d_out, desc, a, &empty);
  if (st != COVER_OK || empty) return st;
  if (cover::stats_workspace_floats(a.B, a.Hq, a.Lr) > COVER_STATS_SCRATCH_FLOATS)
    return COVER_ERR_UNSUPPORTED;
  // the library's own per-GPU array (looked up once per device; nothing is allocated)
  float* scratch = nullptr;
  if (cover::stats_scratch(&scratch) != hipSuccess || !scratch) return COVER_ERR_HIP;
  a.workspace = scratch;
  return run_stats(a, desc, stream);
}

cover_status cover_attn_rect(const void* q, const void* k_live, const void* v_live,
                             const void* k_cache, const void* v_cache,
                             const int32_t* seed_idx, const int32_t* n_seed,
                             void* out, float* lse, float* workspace,
                             const cover_rect_desc* desc, hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_attn_desc& D = desc->attn;
  const int32_t q_off = desc->q_off, Lq = desc->Lq, n_split = desc->n_split;
  if (D.B < 0 || D.L < 0 || D.Hq < 1 || D.Hkv < 1 || D.d < 1 || D.max_seeds < 0)
    return COVER_ERR_INVALID;
  if (D.Hq % D.Hkv != 0) return COVER_ERR_INVALID;
  if (D.dtype != COVER_F32 && D.dtype != COVER_BF16) return COVER_ERR_INVALID;
  if (!(D.scale >= 0.0f) || isinf(D.scale)) return COVER_ERR_INVALID;
  if (q_off < 0 || Lq < 0 || (int64_t)q_off + Lq > D.L) return COVER_ERR_INVALID;
  if (n_split < 1 || n_split > 256) return COVER_ERR_INVALID;
  if (D.dtype != COVER_BF16 || D.d != 128) return COVER_ERR_UNSUPPORTED;
  if (D.L > COVER_MAX_L) return COVER_ERR_UNSUPPORTED;
  if (D.B == 0 || Lq == 0) return COVER_OK;
  const void* tensors[6] = {q, k_live, v_live, k_cache, v_cache, out};
  for (const void* t : tensors)
    if (!t || !aligned(t, 16)) return COVER_ERR_INVALID;
  const int64_t strides[6] = {D.q_sb, D.q_sh, D.q_sl, D.kv_sb, D.kv_sh, D.kv_sl};
  for (int64_t s : strides)
    if (s < 0 || s % 8 != 0) return COVER_ERR_INVALID;
  if ((Lq > 1 && D.q_sl < D.d) || (D.L > 1 && D.kv_sl < D.d)) return COVER_ERR_INVALID;
  if (D.max_seeds > 0 && (!seed_idx || !n_seed || !aligned(seed_idx, 4) || !aligned(n_seed, 4)))
    return COVER_ERR_INVALID;
  if (lse && !aligned(lse, 4)) return COVER_ERR_INVALID;
  if (n_split > 1 && (!workspace || !aligned(workspace, 16))) return COVER_ERR_INVALID;
  if (n_split == 1 && D.kv_sl >= (int64_t(1) << 26)) return COVER_ERR_UNSUPPORTED;
  // grids: at most 2^32 work-items per launch (512 per workgroup for n_split == 1; 256 for the
  // split kernel, and one 64-lane wave per row for the merge)
  if (n_split == 1 && (int64_t)D.B * D.Hq * ((Lq + 31) / 32) > (int64_t(1) << 23) - 8)
    return COVER_ERR_UNSUPPORTED;
  if (n_split > 1 && ((int64_t)D.B * D.Hq * ((Lq + 127) / 128) * n_split > (int64_t(1) << 24) - 1 ||
                      (int64_t)D.B * D.Hq * Lq > (int64_t(1) << 26) - 4))
    return COVER_ERR_UNSUPPORTED;
  cover::RectArgs a;
  a.q = q; a.k_live = k_live; a.v_live = v_live; a.k_cache = k_cache; a.v_cache = v_cache;
  a.seed_idx = D.max_seeds > 0 ? seed_idx : nullptr;
  a.n_seed = D.max_seeds > 0 ? n_seed : nullptr;
  a.out = out; a.lse = lse; a.workspace = n_split > 1 ? workspace : nullptr;
  a.B = D.B; a.Hq = D.Hq; a.Hkv = D.Hkv; a.L = D.L; a.max_seeds = D.max_seeds;
  a.q_off = q_off; a.Lq = Lq; a.n_split = n_split;
  a.scale = D.scale > 0.0f ? D.scale : 1.0f / sqrtf((float)D.d);
  a.q_sb = D.q_sb; a.q_sh = D.q_sh; a.q_sl = D.q_sl;
  a.kv_sb = D.kv_sb; a.kv_sh = D.kv_sh; a.kv_sl = D.kv_sl;
  if (cover::debug_enabled()) {
    const hipError_t e = cover::launch_check_seeds(a.seed_idx, a.n_seed, D.B, D.max_seeds, D.L, stream);
    if (e != hipSuccess) return COVER_ERR_HIP;
  }
  return hip_status(cover::launch_attn_rect(a, stream));
}

cover_status cover_decode_update(int32_t* tokens, const int32_t* argmax, const float* conf,
                                 const int32_t* seed_idx, const int32_t* n_seed,
                                 int32_t* remask_count, uint8_t* flags, uint8_t* drafted,
                                 int32_t* counts, int32_t* last_unmask, int32_t* flipflops,
                                 const cover_update_desc* desc, hipStream_t stream) {
  if (!desc) return COVER_ERR_INVALID;
  const cover_update_desc& D = *desc;
  if (D.B < 0 || D.Lr < 0 || D.max_seeds < 0 || D.draft_cap < 0) return COVER_ERR_INVALID;
  if (D.min_draft < 0 || D.min_draft > D.draft_cap) return COVER_ERR_INVALID;
  if (!(D.tau == D.tau)) return COVER_ERR_INVALID;  // NaN
  if (D.Lr > COVER_MAX_LR) return COVER_ERR_UNSUPPORTED;
  if (D.B == 0) return COVER_OK;
  if (D.Lr > 0) {
    if (!tokens || !argmax || !conf || !remask_count) return COVER_ERR_INVALID;
    if (!aligned(tokens, 4) || !aligned(argmax, 4) || !aligned(conf, 4) || !aligned(remask_count, 4))
      return COVER_ERR_INVALID;
  }
  if (D.max_seeds > 0 && (!seed_idx || !n_seed || !aligned(seed_idx, 4) || !aligned(n_seed, 4)))
    return COVER_ERR_INVALID;
  if (counts && !aligned(counts, 4)) return COVER_ERR_INVALID;
  if (flipflops && ((!last_unmask && D.Lr > 0) || !aligned(flipflops, 4))) return COVER_ERR_INVALID;
  if (last_unmask && D.Lr > 0 && !aligned(last_unmask, 4)) return COVER_ERR_INVALID;
  cover::UpdateArgs a;
  a.tokens = tokens; a.argmax = argmax; a.conf = conf;
  a.seed_idx = D.max_seeds > 0 ? seed_idx : nullptr;
  a.n_seed = D.max_seeds > 0 ? n_seed : nullptr;
  a.remask_count = remask_count; a.flags = flags; a.drafted = drafted; a.counts = counts;
  a.last_unmask = D.Lr > 0 ? last_unmask : nullptr;
  a.flipflops = flipflops;
  a.B = D.B; a.Lr = D.Lr; a.max_seeds = D.max_seeds; a.pos_offset = D.pos_offset;
  a.mask_id = D.mask_id; a.draft_cap = D.draft_cap; a.remask_budget = D.remask_budget;
  a.tau = D.tau; a.min_draft = D.min_draft;
  return hip_status(cover::launch_decode_update(a, stream));
}

}  // extern "C"
