// Internal launch interface between the C ABI (api.cpp) and the HIP kernels.
// Host-validated arguments only: every entry here assumes the descriptor checks passed.
#pragma once
#include <stdint.h>
#include <hip/hip_runtime_api.h>

namespace cover {

struct AttnArgs {
  const void* q;
  const void* k_live;
  const void* v_live;
  const void* k_cache;
  const void* v_cache;
  const int32_t* seed_idx;  // may be null when max_seeds == 0
  const int32_t* n_seed;    // may be null when max_seeds == 0
  void* out;
  float* lse;               // may be null
  int32_t B, Hq, Hkv, L, d, max_seeds;
  float scale;              // > 0
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

struct SelectArgs {
  const float* logp;
  const float* d_in;
  const float* d_out;
  const uint8_t* flags;
  int32_t* seed_idx;
  int32_t* n_seed;
  double* score;  // may be null
  int32_t B, Lr, max_seeds, pos_offset;
};

struct TokenArgs {
  const void* logits;
  const int32_t* tokens;  // may be null when logp is null
  float* logp;            // may be null
  float* conf;            // may be null
  int32_t* argmax;        // may be null
  int32_t R, V;
  int bf16;               // element type of logits: bf16 (1) or fp32 (0)
  int64_t row_stride;     // elements
};

struct SampleArgs {
  const void* logits;
  int32_t* token;
  float* prob;  // may be null
  int32_t R, V;
  int bf16;
  int64_t row_stride;  // elements
  float temperature;   // > 0
  uint64_t seed;
  uint32_t step;
};

struct StatsArgs {
  const void* q;
  const void* k_live;
  const void* k_cache;
  const int32_t* seed_idx;  // may be null when max_seeds == 0
  const int32_t* n_seed;    // may be null when max_seeds == 0
  const float* lse;
  const uint8_t* masked;
  const uint8_t* drafted;
  float* d_in;
  float* d_out;
  float* workspace;
  int32_t B, Hq, Hkv, L, d, max_seeds, r0, Lr;
  float scale;  // > 0
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

struct RectArgs {
  const void* q;
  const void* k_live;
  const void* v_live;
  const void* k_cache;
  const void* v_cache;
  const int32_t* seed_idx;  // may be null when max_seeds == 0
  const int32_t* n_seed;    // may be null when max_seeds == 0
  void* out;
  float* lse;  // may be null
  float* workspace;
  int32_t B, Hq, Hkv, L, max_seeds, q_off, Lq, n_split;
  float scale;  // > 0
  int64_t q_sb, q_sh, q_sl, kv_sb, kv_sh, kv_sl;
};

struct UpdateArgs {
  int32_t* tokens;
  const int32_t* argmax;
  const float* conf;
  const int32_t* seed_idx;  // may be null when max_seeds == 0
  const int32_t* n_seed;    // may be null when max_seeds == 0
  int32_t* remask_count;
  uint8_t* flags;    // may be null
  uint8_t* drafted;  // may be null
  int32_t* counts;   // may be null
  int32_t* last_unmask;  // may be null
  int32_t* flipflops;    // may be null (always null when last_unmask is)
  int32_t B, Lr, max_seeds, pos_offset, mask_id, draft_cap, remask_budget;
  float tau;
  int32_t min_draft;
};

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t stream);     // bf16, d = 64
hipError_t launch_attn_bf16_w4(const AttnArgs& a, hipStream_t stream);  // bf16, d = 128
hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t stream);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);
hipError_t launch_token_stats(const TokenArgs& a, hipStream_t stream);
hipError_t launch_token_sample(const SampleArgs& a, hipStream_t stream);
hipError_t launch_attn_stats(const StatsArgs& a, hipStream_t stream);
// key groups of the attention-mass launch (32-key tiles per group, groups) and the workspace
// floats that launch uses
void stats_key_groups(int B, int Hq, int Lr, int* tpg, int* kg);
int64_t stats_workspace_floats(int B, int Hq, int Lr);
// device address of the attention-mass kernels' own static scratch array on the current GPU
// (COVER_STATS_SCRATCH_FLOATS floats), looked up once per device
hipError_t stats_scratch(float** ptr);
hipError_t launch_decode_update(const UpdateArgs& a, hipStream_t stream);
hipError_t launch_attn_rect(const RectArgs& a, hipStream_t stream);  // bf16, d = 128

// contract checks (COVER_DEBUG=1)
bool debug_enabled();
hipError_t launch_check_seeds(const int32_t* seed_idx, const int32_t* n_seed, int B, int max_seeds,
                              int L, hipStream_t stream);
hipError_t launch_check_select(const float* logp, const float* d_in, const float* d_out,
                               const uint8_t* flags, int64_t n, hipStream_t stream);
hipError_t debug_status(int32_t* status, bool clear, hipStream_t stream);

}  // namespace cover
