// Host-side interface between the C ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ippd {

constexpr int kMaxQuestionsPerPrompt = 1024;   // LDS list of a prompt's active questions

struct LoadContextParams {
  const void* k_raw; const void* v_raw;     // [pool][Hkv][D]
  void* ctx_k; void* ctx_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; int32_t* err_flag;
  int64_t pool; int B, Hkv, D, max_ctx_len;
  double base;
};

struct LoadSegmentsParams {
  const void* k_raw; const void* v_raw;     // [Nt][seg_cap][Hkv][D]
  const int32_t* init_len;
  void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start; int32_t* seg_len; int32_t* err_flag;
  int B, Nt, Hkv, D, seg_cap;
  double base;
};

struct AppendParams {
  const void* q_new; const void* k_new; const void* v_new;
  void* q_rot; void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start;
  int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  int B, Nt, Hq, Hkv, D, seg_cap;
  double base;
};

// One decode-attention launch plan (shared by IPPD and the standard baseline).
struct AttnPlan {
  int shared;        // 1: a context unit serves every active question of its prompt
  int rb;            // 16-row MFMA row blocks per wave (1, 2 or 4)
  int nrg;           // row groups of 16*rb rows per (prompt, kv head) in shared mode
  int chunk;         // context tokens per unit (multiple of 32)
  int max_chunks;    // ceil(max_ctx_len / chunk)
  int ctx_per_g;     // context units per kv head
  int units_per_g;   // context + segment units per kv head
  int n_units;       // units_per_g * Hkv
  int grid;          // n_units rounded up to a multiple of 8 (one slice per XCD)
  size_t part_slots;       // (max_chunks + 1) * Nt * Hq
  size_t workspace_bytes;  // part_slots * (D + 2) * 4, 256-byte rounded pieces
};

struct AttnParams {
  const void* ctx_k; const void* ctx_vt; const void* seg_k; const void* seg_vt;
  const void* q;     // q_rot [Nt][Hq][D]
  const int64_t* ctx_off; const int32_t* ctx_len; const int32_t* q_start;
  const int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  float* part_acc;   // [part_slots][D]
  float* part_ml;    // [part_slots][2]  (running max in raw logit units, sum)
  float* out; float* lse;
  int64_t pool;
  int B, Nt, Hq, Hkv, G, D, seg_cap, max_ctx_len, max_questions;
  int shared, nrg, chunk, max_chunks, ctx_per_g, units_per_g, n_units, grid;
  float c;           // scale * log2(e)
  float scale;
};

hipError_t launch_load_context(int dtype, const LoadContextParams& p, hipStream_t s);
hipError_t launch_load_segments(int dtype, const LoadSegmentsParams& p, hipStream_t s);
hipError_t launch_append(int dtype, const AppendParams& p, hipStream_t s);
hipError_t launch_attention(int dtype, int rb, const AttnParams& p, hipStream_t s);

}  // namespace ippd
