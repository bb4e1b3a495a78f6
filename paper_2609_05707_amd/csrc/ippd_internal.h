// Host-side interface between the C ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ippd {

constexpr int kMaxQuestionsPerPrompt = 1024;   // LDS list of a prompt's active questions
constexpr int kMaxGroup = 16;                  // query heads per kv head (one MFMA row block)
constexpr int kMaxHalfDim = 64;                // D/2 for D <= 128
constexpr int kDenseSegTiles = 8;              // dense-mask baseline: 32-token tiles per segment chunk
#ifndef IPPD_MERGE_THREADS
#define IPPD_MERGE_THREADS 256
#endif
constexpr int kMergeThreads = IPPD_MERGE_THREADS;   // merge_kernel workgroup size (256 measured ahead of 512
                                                    // when a call has few questions, equal otherwise)

struct LoadContextParams {
  const void* k_raw; const void* v_raw;     // [pool][Hkv][D]
  void* ctx_k; void* ctx_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; int32_t* err_flag;
  const int32_t* instr_start; const int32_t* instr_len; int S;   // two-level batch: position base (S = 0: none)
  int64_t pool; int B, Hkv, D, max_ctx_len;
  double inv_freq[kMaxHalfDim];
};

struct LoadSegmentsParams {
  const void* k_raw; const void* v_raw;     // [Nt][seg_cap][Hkv][D]
  const int32_t* init_len;
  void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start; int32_t* seg_len; int32_t* err_flag;
  const int32_t* instr_start; const int32_t* instr_len; int S;   // two-level batch: position base (S = 0: none)
  int B, Nt, Hkv, D, seg_cap;
  double inv_freq[kMaxHalfDim];
};

struct AppendParams {
  const void* q_new; const void* k_new; const void* v_new;
  void* q_rot; void* seg_k; void* seg_vt;
  const int32_t* ctx_len; const int32_t* q_start;
  int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  const int32_t* instr_start; const int32_t* instr_len; int S;   // two-level batch: position base (S = 0: none)
  int B, Nt, Hq, Hkv, D, seg_cap;
  double inv_freq[kMaxHalfDim];
};

// Launch plan of one decode call (attend_kernel + merge_kernel).  A group is
// (prompt b, kv head g) for IPPD or (question i, kv head g) for the standard
// baseline; a context unit is (group, chunk, row group) with 16*waves query
// rows; a segment unit serves seg_tpu tasks (question i, kv head g).
struct StepPlan {
  int shared;              // 1: IPPD, context units serve all questions of a prompt
  int waves;               // waves per workgroup; a context unit covers 16 * rb rows per wave
  int rb;                  // 16-row blocks per wave (1, or 2 for bf16 at D = 128)
  int nrg;                 // row groups per group
  int chunk;               // context tokens per context unit (multiple of 32)
  int max_chunks;          // ceil(max_ctx_len / chunk)
  int n_groups;
  int grid;                // attend_kernel workgroups: ctx_blocks + seg_blocks
  int ctx_blocks;          // context units (8 * nrg * ceil(n_groups * max_chunks / 8))
  int seg_blocks;          // segment units: ceil(Nt * Hkv / seg_tpu)
  int seg_tpu;             // segment tasks per unit (power of two dividing waves)
  int deep;                // 1: deep LDS ring (the context units fit the chip in one wave)
  int n_igroups;           // instruction groups: (instruction s, kv head g) or (question i, kv head g)
  int nrg_i;               // row groups per instruction group
  int max_ichunks;         // ceil(max_instr_len / chunk)
  int instr_blocks;        // instruction units, after the context units
  int dense;               // dense-mask baseline: seg_blocks are dense segment units (prompt, kv head, row group)
  size_t part_slots;       // (max_chunks + 1 + max_ichunks) * Nt * Hq partial softmax states
                           // (context chunks, segment, instruction chunks)
  size_t off_acc, off_ml;  // byte offsets of the partial arrays in the workspace
  size_t workspace_bytes;
};

// Launch plan of one prefill call.  A group is (prompt b, kv head g) for
// IPPD or (question i, kv head g) for the standard baseline.  A unit serves
// tb query tokens x G heads (16 * rb * waves rows): question-row units (the
// group's question tokens against its whole context and their own
// questions) come first, then context-row units (causal over the context),
// the longest causal blocks first.  Unit u of either kind runs on XCD u & 7,
// which holds every unit of groups g = 8 j + (u & 7).
struct PrefillPlan {
  int shared, waves, rb, tb;
  int n_groups, gps;       // question-row groups, and groups per XCD slice (ceil(n_groups / 8))
  int n_cgroups, gps_c;    // context-row groups: n_groups, then the instruction groups
  int kq, kc;              // question-row and context-row units per group
  int q_blocks, grid;      // 8 * gps * kq, then + 8 * gps_c * kc
};

struct PrefillParams {
  const void* q_ctx;       // [pool][Hq][D] raw queries of context tokens
  const void* q_seg;       // [Nt][seg_cap][Hq][D] raw queries of question tokens
  const void* ctx_k; const void* ctx_vt; const void* seg_k; const void* seg_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; const int32_t* q_start; const int32_t* seg_len;
  int32_t* err_flag;
  float* out_ctx;          // [pool][Hq][D]
  float* out_seg;          // [Nt][seg_cap][Hq][D]
  int64_t pool;
  int B, Nt, Hq, Hkv, G, D, seg_cap, max_ctx_len;
  int shared, tb, n_groups, gps, kq, kc, q_blocks;
  int n_cgroups, gps_c;
  // two-level batch (S > 0): instruction s at pool rows instr_off[s] .. + instr_len[s]
  const int32_t* instr_start; const int64_t* instr_off; const int32_t* instr_len;
  int S, max_instr_len;
  float c;                 // scale * log2(e)
  double inv_freq[kMaxHalfDim];
};

struct StepParams {
  const void* q_new; const void* k_new; const void* v_new;   // fused step: raw token inputs
  const void* q_rot_in;                                        // attention only: rotated queries
  void* q_rot_out;                                             // fused step: rotated queries (or null)
  void* ctx_k; void* ctx_vt; void* seg_k; void* seg_vt;
  const int64_t* ctx_off; const int32_t* ctx_len; const int32_t* q_start;
  int32_t* seg_len; const uint8_t* active; int32_t* err_flag;
  float* out; float* lse;
  float* part_acc;         // [part_slots][D]
  float* part_ml;          // [part_slots][2]: running max (raw logit units), sum
  int64_t pool;
  int B, Nt, Hq, Hkv, G, D, seg_cap, max_ctx_len, max_questions;
  int shared, fused, nrg, chunk, max_chunks, n_groups, ctx_blocks, seg_tpu;
  // two-level batch: instruction units (blocks ctx_blocks .. ctx_blocks + instr_blocks - 1)
  const int32_t* instr_start; const int64_t* instr_off; const int32_t* instr_len;
  int S, max_instr_len, max_instr_questions, n_igroups, nrg_i, max_ichunks, instr_blocks;
  int dense;               // dense-mask baseline (the merge checks each question's prompt)
  int merge_phases;        // threads per merged item (slots split among them), power of 2
  int merge_parts;         // merge workgroups per question
  float c;                 // scale * log2(e)
  float scale;
  double inv_freq[kMaxHalfDim];
};

hipError_t launch_load_context(int dtype, const LoadContextParams& p, hipStream_t s);
hipError_t launch_load_segments(int dtype, const LoadSegmentsParams& p, hipStream_t s);
hipError_t launch_append(int dtype, const AppendParams& p, hipStream_t s);
hipError_t launch_step(int dtype, int waves, int rb, bool deep, int grid, const StepParams& p, hipStream_t s);
// merge_kernel alone (the dense-mask baseline's second launch)
hipError_t launch_merge(const StepParams& p, hipStream_t s);
// dense-mask baseline: dense_kernel (context-chunk units, then dense segment
// units) followed by merge_kernel
hipError_t launch_dense(int dtype, int waves, int rb, int grid, const StepParams& p, hipStream_t s);
// prefill_kernel for the batch dtype and head dimension, with rb row blocks
// per wave (the waves are fixed per dtype and head dimension: see prefill_variant)
hipError_t launch_prefill(int dtype, int head_dim, int rb, int grid, const PrefillParams& p, hipStream_t s);
// (waves, rb) of the prefill variant for a dtype and head dimension; false if
// none.  bf16 at D = 128 also runs with rb = 1.
bool prefill_variant(int dtype, int head_dim, int* waves, int* rb);

}  // namespace ippd
