// Host-side interface between the C ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ippd {

constexpr int kMaxQuestionsPerPrompt = 1024;   // LDS list of a prompt's active questions
constexpr int kMaxGroup = 16;                  // query heads per kv head (one MFMA row block)
constexpr int kMaxHalfDim = 64;                // D/2 for D <= 128

struct LoadContextParams {
  const void* k_raw; const void* v_raw;     // [pool][Hkv][D]
  void* ctx_k; void* ctx_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; int32_t* err_flag;
  int64_t pool; int B, Hkv, D, max_ctx_len;
  double inv_freq[kMaxHalfDim];
};

struct LoadSegmentsParams {
  const void* k_raw; const void* v_raw;     // [Nt][seg_cap][Hkv][D]
  const int32_t* init_len;
  void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start; int32_t* seg_len; int32_t* err_flag;
  int B, Nt, Hkv, D, seg_cap;
  double inv_freq[kMaxHalfDim];
};

struct AppendParams {
  const void* q_new; const void* k_new; const void* v_new;
  void* q_rot; void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start;
  int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  int B, Nt, Hq, Hkv, D, seg_cap;
  double inv_freq[kMaxHalfDim];
};

// Launch plan of one decode-attention call.  Work is grouped per
// (prompt, kv head) in IPPD mode and per (question, kv head) in the standard
// baseline; a group owns its context units and its segment units, and the
// groups are dealt in contiguous runs to the 8 workgroup slices (XCDs).
struct StepPlan {
  int shared;              // 1: IPPD, context units serve all active questions of a prompt
  int waves;               // waves per workgroup (questions per segment unit in IPPD mode)
  int row_split;           // 1: waves split a context unit's rows (16 each), 0: its tokens
  int rw;                  // query rows per context unit
  int nrg;                 // row groups per group
  int chunk;               // context tokens per context unit (multiple of 32)
  int max_chunks;          // ceil(max_ctx_len / chunk)
  int ctx_units_per_group; // max_chunks * nrg
  int seg_units_per_group; // segment units (one question per wave) per group
  int units_per_group;
  int n_groups;
  int groups_per_slice;
  int per_slice;
  int grid;                // 8 * per_slice workgroups
  size_t part_slots;       // (max_chunks + 1) * Nt * Hq partial softmax states
  size_t counters;         // n_groups * seg_units_per_group + Nt 32-bit counters
  size_t off_acc, off_ml;  // byte offsets of the partial arrays in the workspace
  size_t workspace_bytes;
};

struct StepParams {
  const void* q_new; const void* k_new; const void* v_new;   // fused step: raw token inputs
  const void* q_rot_in;                                        // attention only: rotated queries
  void* q_rot_out;                                             // fused step: rotated queries (or null)
  void* ctx_k; void* ctx_vt; void* seg_k; void* seg_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; const int32_t* q_start;
  int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  float* out; float* lse;
  uint32_t* counters;      // [n_groups * seg_units_per_group] arrivals, then [Nt] per-question
  float* part_acc;         // [part_slots][D]
  float* part_ml;          // [part_slots][2]: running max (raw logit units), sum
  int64_t pool;
  int B, Nt, Hq, Hkv, G, D, seg_cap, max_ctx_len, max_questions;
  int shared, fused, rw, nrg, chunk, max_chunks;
  int ctx_units_per_group, seg_units_per_group, units_per_group, n_groups, groups_per_slice, per_slice;
  float c;                 // scale * log2(e)
  float scale;
  double inv_freq[kMaxHalfDim];
};

hipError_t launch_load_context(int dtype, const LoadContextParams& p, hipStream_t s);
hipError_t launch_load_segments(int dtype, const LoadSegmentsParams& p, hipStream_t s);
hipError_t launch_append(int dtype, const AppendParams& p, hipStream_t s);
hipError_t launch_step(int dtype, int waves, bool row_split, int grid, const StepParams& p, hipStream_t s);

}  // namespace ippd
