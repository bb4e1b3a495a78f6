/*
 * ippd.h -- C ABI of the MI355X (gfx950) library for the decode step of
 * Intra-Prompt Parallel Decoding (IPPD, arXiv 2609.05707).
 *
 * In IPPD the questions that share a context are stacked into one prompt
 * and decoded in parallel (Sec. 4).  At a decode step every still-active
 * question feeds one token; that token's query attends to
 *   - the shared context of its prompt (instruction + context; the mask
 *     clauses M_ctx and M_caus of Sec. 4.1 admit all of it), and
 *   - its own question+answer segment, including the token itself
 *     (M_qtn and M_caus with ">=", Sec. 4.1),
 * and to nothing else.  The token sits at virtual position
 * |p| + |c_j| + |x_jk| + (t-1) (Sec. 4.1), i.e. the context length plus the
 * number of segment tokens already cached.  The result equals independent
 * causal decoding of each question (Sec. 4.2).  Prompts of a batch carry
 * different contexts and question counts; stopped questions take no token
 * and produce no output (Sec. 4.2 end-of-sequence rule, Sec. 4.4 pads).
 *
 * Conventions for every entry point:
 *   - Array arguments are DEVICE pointers unless marked "host".  All work is
 *     enqueued on `stream`; no entry point synchronises, allocates or frees.
 *     The caller owns every buffer.  Calls that share buffers must be
 *     ordered on one stream.
 *   - Host-checkable argument errors return a status before anything is
 *     enqueued.  Problems only visible in device data (see IPPD_FLAG_*) are
 *     reported by OR-ing bits into *err_flag; affected rows are skipped.
 *   - Rotary embedding: rotate-half pairs (j, j + D/2) with
 *     theta_j = rope_base^(-2j/D); the angle pos*theta_j is formed in fp64.
 *   - Softmax scale 1/sqrt(D) unless `scale` > 0 (Sec. 4.2).
 *   - GQA: query head h reads kv head h / (Hq/Hkv).
 */
#ifndef IPPD_H
#define IPPD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  IPPD_DTYPE_F32 = 0,   /* float32 cache and q/k/v */
  IPPD_DTYPE_BF16 = 1   /* bfloat16 cache and q/k/v; fp32 accumulation */
} ippd_dtype_t;

typedef enum {
  IPPD_OK = 0,
  IPPD_ERR_NULL = 1,       /* a required pointer is NULL */
  IPPD_ERR_SHAPE = 2,      /* inconsistent or unsupported sizes */
  IPPD_ERR_DTYPE = 3,      /* unknown dtype */
  IPPD_ERR_ALIGN = 4,      /* a data pointer is not 16-byte aligned */
  IPPD_ERR_WORKSPACE = 5,  /* workspace NULL or smaller than required */
  IPPD_ERR_HIP = 6,        /* a HIP call failed; see ippd_last_hip_error() */
  IPPD_ERR_SCRATCH = 7     /* ippd_decode_step_noalloc: the batch needs more than
                              IPPD_NOALLOC_SCRATCH_BYTES of partial states */
} ippd_status_t;

/* Bits OR-ed into *err_flag by device code. */
#define IPPD_FLAG_SEGMENT_FULL 1  /* append found seg_len[i] == seg_capacity: token dropped */
#define IPPD_FLAG_BAD_LAYOUT   2  /* device arrays break a rule below: rows skipped */

/*
 * Batch description (a host struct; its array fields are device pointers).
 *
 * Prompts b = 0..B-1.  Prompt b's context occupies tokens
 * [ctx_off[b], ctx_off[b] + ctx_len[b]) of the context pool; ctx_off[b] must
 * be a multiple of 8 and the range must lie inside [0, ctx_pool_tokens).
 * Its questions are i = q_start[b] .. q_start[b+1]-1 (q_start[0] = 0,
 * q_start[B] = num_questions, non-decreasing).  Question i owns one segment
 * per kv head holding seg_len[i] <= seg_capacity cached tokens (question +
 * answer tokens so far) at virtual positions ctx_len[b] + 0..seg_len[i]-1.
 * active[i] != 0 marks a question still decoding this step.
 * max_ctx_len >= every ctx_len[b] and max_questions >= every question count
 * are host-side bounds used to size grids and workspaces (violations set
 * IPPD_FLAG_BAD_LAYOUT).
 */
typedef struct ippd_batch {
  int32_t num_prompts;       /* B >= 1 */
  int32_t num_questions;     /* Nt >= 0, total over prompts */
  int32_t num_q_heads;       /* Hq >= 1 */
  int32_t num_kv_heads;      /* Hkv >= 1, Hq % Hkv == 0, Hq/Hkv <= 16 */
  int32_t head_dim;          /* D: 64 or 128 */
  int32_t dtype;             /* ippd_dtype_t */
  int64_t ctx_pool_tokens;   /* context pool capacity, multiple of 8 */
  int32_t seg_capacity;      /* tokens per segment, multiple of 8, >= 8 */
  int32_t max_ctx_len;       /* host bound on ctx_len[b], <= ctx_pool_tokens */
  int32_t max_questions;     /* host bound on questions per prompt, 1..1024 */
  int32_t chunk_tokens;      /* context tokens per work unit: 0 = automatic,
                                else a multiple of 32 (tests use it to vary splits) */
  int32_t tile_rows;         /* query rows per context unit: 0 = automatic, else 16, 32,
                                64, 128 or 256 (256: bf16 at head_dim 128 only); a tuning
                                knob, results do not depend on it.  The bf16 head_dim 128
                                prefill reads 128 and 256 as its unit size and chooses
                                by itself for any other value */
  double  rope_base;         /* > 0, e.g. 10000 */
  float   scale;             /* softmax scale; <= 0 selects 1/sqrt(head_dim) */
  const int64_t *ctx_off;    /* [B]   pool offset of each context */
  const int32_t *ctx_len;    /* [B]   context tokens per prompt (|p| + |c_j|) */
  const int32_t *q_start;    /* [B+1] question CSR offsets */
  int32_t       *seg_len;    /* [Nt]  cached segment tokens; advanced by ippd_append_kv */
  const uint8_t *active;     /* [Nt]  1 = decoding this step */
  int32_t       *err_flag;   /* [1]   IPPD_FLAG_* bits (never cleared by the library) */
  /* Two-level sharing (optional; Sec. 4.4: one stacked prompt holds several
   * contexts behind one instruction p, which is then read once for all of
   * their questions).  num_instr = S instruction blocks; prompts
   * instr_start[s] .. instr_start[s+1]-1 sit behind instruction s
   * (instr_start[0] = 0, instr_start[S] = B, non-decreasing).  Instruction s
   * occupies pool tokens [instr_off[s], instr_off[s] + instr_len[s]) of the
   * context pool (instr_off a multiple of 8) at positions 0..instr_len[s]-1;
   * the contexts behind it and their questions move up by instr_len[s]
   * (Sec. 4.1: p at [0, |p|), c_j from |p|).  A table that breaks these
   * rules (or puts more than max_instr_questions questions behind one
   * instruction) sets IPPD_FLAG_BAD_LAYOUT and the decode calls then serve
   * no question of the batch.  num_instr = 0 disables the level and the
   * fields below are not read. */
  int32_t num_instr;            /* S >= 0 */
  int32_t max_instr_len;        /* host bound on instr_len[s], <= ctx_pool_tokens */
  int32_t max_instr_questions;  /* host bound on the questions behind one instruction, >= 1 */
  const int32_t *instr_start;   /* [S+1] */
  const int64_t *instr_off;     /* [S] */
  const int32_t *instr_len;     /* [S] */
} ippd_batch_t;

/*
 * KV cache (device buffers of the batch dtype).  Keys are stored rotated at
 * their virtual positions, token-major.  Values are stored transposed in
 * 8-token column blocks: for a region of n tokens, token t of dimension d is
 * element (t / 8) * 8 * D + d * 8 + t % 8, so one dimension's 8 tokens are
 * one 16-byte (bf16) fragment of the value-times-probability product and a
 * 32-token tile of all dimensions is one contiguous block.
 *   ctx_k  [Hkv][ctx_pool_tokens][D]      ctx_vt [Hkv][ctx_pool_tokens / 8][D][8]
 *   seg_k  [Nt][Hkv][seg_capacity][D]     seg_vt [Nt][Hkv][seg_capacity / 8][D][8]
 * All four must be 16-byte aligned.
 */
typedef struct ippd_kv_cache {
  void *ctx_k;
  void *ctx_vt;
  void *seg_k;
  void *seg_vt;
} ippd_kv_cache_t;

/*
 * Fill the context part of the cache from raw (pre-rotation) keys and values
 * k_raw/v_raw [ctx_pool_tokens][Hkv][D], laid out like the pool: token t of
 * prompt b is row ctx_off[b] + t and is rotated at position t (Sec. 4.1:
 * context tokens sit at [|p|, |p| + |c_j|), with p folded into the context),
 * or at instr_len[s] + t behind instruction s of a two-level batch.
 * Rows outside every prompt's range are neither read nor written.
 * Stands in for the prefill that would produce this cache.
 */
ippd_status_t ippd_load_context(const ippd_batch_t *batch, const void *k_raw,
                                const void *v_raw, const ippd_kv_cache_t *kv,
                                hipStream_t stream);

/*
 * Fill the instruction blocks of a two-level batch (num_instr > 0) from raw
 * keys/values laid out like the pool, k_raw/v_raw [ctx_pool_tokens][Hkv][D]:
 * token t of instruction s is row instr_off[s] + t and is rotated at
 * position t (Sec. 4.1: p occupies [0, |p|)).  Other rows are neither read
 * nor written, so one raw buffer may hold both the instructions and the
 * contexts (call ippd_load_context for the latter).
 */
ippd_status_t ippd_load_instructions(const ippd_batch_t *batch, const void *k_raw,
                                     const void *v_raw, const ippd_kv_cache_t *kv,
                                     hipStream_t stream);

/*
 * Fill segments from raw keys/values k_raw/v_raw [Nt][seg_capacity][Hkv][D]:
 * slots 0..init_len[i]-1 of question i are rotated at ctx_len[b] + slot
 * (plus instr_len[s] behind instruction s of a two-level batch; Sec. 4.1
 * question/answer positions) and seg_len[i] is set to init_len[i]
 * (device [Nt], each <= seg_capacity; larger values set IPPD_FLAG_BAD_LAYOUT
 * and leave the question untouched).
 */
ippd_status_t ippd_load_segments(const ippd_batch_t *batch, const void *k_raw,
                                 const void *v_raw, const int32_t *init_len,
                                 const ippd_kv_cache_t *kv, hipStream_t stream);

/*
 * Decode-step rotation and append (Sec. 4.1 virtual position of answer
 * tokens; Sec. 4.2: each generated token re-enters the prompt at its virtual
 * position for the next step).
 * For every active question i of prompt b, with s = seg_len[i] and
 * pos = ctx_len[b] + s (plus instr_len of b's instruction in a two-level batch):
 *   q_rot[i][h] = R(pos) q_new[i][h]        for all Hq heads,
 *   seg slot s of (i, g) <- (R(pos) k_new[i][g], v_new[i][g]),
 *   seg_len[i] = s + 1.
 * q_new [Nt][Hq][D], k_new/v_new [Nt][Hkv][D], q_rot [Nt][Hq][D], all of
 * the batch dtype.  Inactive questions are untouched (no append, q_rot rows
 * not written).  s == seg_capacity sets IPPD_FLAG_SEGMENT_FULL and skips i.
 */
ippd_status_t ippd_append_kv(const ippd_batch_t *batch, const void *q_new,
                             const void *k_new, const void *v_new, void *q_rot,
                             const ippd_kv_cache_t *kv, hipStream_t stream);

/*
 * Workspace of the decode calls: device scratch holding the partial softmax
 * states (max, sum, weighted values) of every (context chunk, question, head)
 * and (segment, question, head).  ippd_decode_workspace_bytes serves
 * ippd_decode_attention and ippd_decode_step, standard_decode_workspace_bytes
 * the two standard_* calls (sizes depend only on host-side fields; 0 means an
 * invalid batch).  A workspace must be 256-byte aligned.  It needs no
 * initialisation and carries nothing from one call to the next: every state
 * a call reads was written earlier in the same call.  Calls that run
 * concurrently need separate workspaces.
 */
size_t ippd_decode_workspace_bytes(const ippd_batch_t *batch);
size_t standard_decode_workspace_bytes(const ippd_batch_t *batch);

/*
 * IPPD decode-step attention (Sec. 4.1 mask, Sec. 4.2 attn_IPPD).  For every
 * active question i (prompt b) and query head h (kv head g):
 *   out[i][h] = softmax_k( scale * q_rot[i][h] . K_k ) V_k
 * over the keys of prompt b's context and of segment (i, g) slots
 * 0..seg_len[i]-1 (call after ippd_append_kv, so the step's own token is the
 * last key), and, in a two-level batch, of b's instruction.  Each context
 * tile is read from HBM once for ALL active questions and all heads of its
 * kv group, each instruction tile once for all questions of all prompts
 * behind it; contexts and instructions are split into chunks whose partial
 * softmax states (max, sum, weighted values) are merged exactly.  lse[i][h] = natural-log sum of exp over the same logits
 * (optional, may be NULL).  out [Nt][Hq][D] and lse [Nt][Hq] are float32;
 * rows of inactive questions are not written.
 * workspace: >= ippd_decode_workspace_bytes(batch) bytes (see above).
 * Two kernel launches: the first computes one partial softmax state per
 * (context chunk, row) and per (segment, row); the second merges them.
 */
ippd_status_t ippd_decode_attention(const ippd_batch_t *batch, const void *q_rot,
                                    const ippd_kv_cache_t *kv, float *out, float *lse,
                                    void *workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/*
 * Baseline: the same result computed as standard decoding does it (Sec. 3,
 * batched autoregressive inference; App. A.2.2 PC+PA decode, one query per
 * attention over |p|+|c_j|+|x|+|y_<t| keys): every question attends to its
 * prompt's context separately, so the context is re-read once per active
 * question.  Same arguments and semantics as ippd_decode_attention;
 * workspace >= standard_decode_workspace_bytes(batch).
 */
ippd_status_t standard_decode_attention(const ippd_batch_t *batch, const void *q_rot,
                                        const ippd_kv_cache_t *kv, float *out, float *lse,
                                        void *workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/*
 * Baseline: the dense-mask form of the same attention, the paper's own
 * scheme (Sec. 4.1: the stacked prompt's new tokens attend over ALL its keys
 * under the additive mask M_fin; Sec. 4.2).  The context part is computed as
 * in ippd_decode_attention; the segment part attends every question's rows
 * over the segments of ALL questions of the prompt and masks out the other
 * questions' keys, so it forms and discards the cross-question scores the
 * block-diagonal form never computes.  Same result, arguments and semantics
 * as ippd_decode_attention (call after ippd_append_kv); one-level batches
 * with max_questions <= 64 (else IPPD_ERR_SHAPE); workspace >=
 * dense_decode_workspace_bytes(batch) (0: batch not supported).
 */
size_t dense_decode_workspace_bytes(const ippd_batch_t *batch);
ippd_status_t dense_decode_attention(const ippd_batch_t *batch, const void *q_rot,
                                     const ippd_kv_cache_t *kv, float *out, float *lse,
                                     void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Fused decode step: ippd_append_kv followed by ippd_decode_attention, in
 * the same two kernel launches as ippd_decode_attention.  q_new [Nt][Hq][D], k_new/v_new [Nt][Hkv][D] are the
 * raw (pre-rotation) projections of the token each active question feeds
 * this step.  The launch rotates them at virtual position
 * ctx_len[b] + seg_len[i], appends the key/value to the segment, attends
 * (context + segment including the new token) and advances seg_len[i].
 * q_rot [Nt][Hq][D] receives the rotated queries, or may be NULL.  An active
 * question whose segment is full (seg_len[i] == seg_capacity) sets
 * IPPD_FLAG_SEGMENT_FULL and gets no output row.  workspace as for
 * ippd_decode_attention.
 */
ippd_status_t ippd_decode_step(const ippd_batch_t *batch, const void *q_new, const void *k_new,
                               const void *v_new, void *q_rot, const ippd_kv_cache_t *kv,
                               float *out, float *lse, void *workspace, size_t workspace_bytes,
                               hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the fused
 * IPPD decode step of ippd_decode_step with the same arguments, minus the
 * workspace.  The partial softmax states live instead in a scratch array of
 * IPPD_NOALLOC_SCRATCH_BYTES that the library holds in device memory on
 * every GPU it runs on until the process ends.  A batch fits when
 * ippd_decode_workspace_bytes(batch) <= IPPD_NOALLOC_SCRATCH_BYTES; a larger
 * one returns IPPD_ERR_SCRATCH before anything is enqueued.  The call
 * allocates nothing: on the first call on a device it looks up that device's
 * copy of the array (hipGetSymbolAddress; a failure returns IPPD_ERR_HIP).
 * `stream` must belong to the current device.  Every call on one GPU shares
 * that GPU's array, so calls that may run concurrently on one GPU race and
 * must be ordered (for example on one stream); the array needs no
 * initialisation and nothing carries from one call to the next.
 */
#define IPPD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ippd_status_t ippd_decode_step_noalloc(const ippd_batch_t *batch, const void *q_new, const void *k_new,
                                       const void *v_new, void *q_rot, const ippd_kv_cache_t *kv,
                                       float *out, float *lse, hipStream_t stream);

/* The standard baseline as one fused launch (append + per-question attention);
 * workspace >= standard_decode_workspace_bytes(batch). */
ippd_status_t standard_decode_step(const ippd_batch_t *batch, const void *q_new, const void *k_new,
                                   const void *v_new, void *q_rot, const ippd_kv_cache_t *kv,
                                   float *out, float *lse, void *workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Stacked-prompt prefill attention (Sec. 4.1: the prompt header, every token
 * a query row under the mask M_fin; App. A.2 prefill dimensions).  The cache
 * holds the rotated context keys (ippd_load_context) and each question's
 * tokens as its segment (ippd_load_segments with init_len = the question
 * lengths, so seg_len[i] = |x_i|).  For context token t of prompt b and
 * query head h (kv head g):
 *   out_ctx[ctx_off[b] + t][h] = softmax_k(scale q . K_k) V_k over the
 *                                prompt's context keys 0..t   (causal);
 * for token u < seg_len[i] of question i (prompt b):
 *   out_seg[i][u][h] = the same over ALL context keys of prompt b and the
 *                      question's own keys 0..u   (M_ctx, M_qtn, M_caus),
 * with the queries rotated at t and at ctx_len[b] + u.
 * q_ctx [ctx_pool_tokens][Hq][D] and q_seg [Nt][seg_capacity][Hq][D] are raw
 * (pre-rotation) queries of the batch dtype; out_ctx and out_seg have the
 * same layouts in float32 (16-byte aligned).  Rows outside every prompt's
 * context and slots at or past seg_len[i] are neither read nor written.
 * IPPD serves all question tokens of a prompt from one pass over its
 * context and computes the context rows once.
 * max_prompt_question_tokens: host bound on the sum of seg_len over the
 * questions of any one prompt (it sizes the grid); a prompt above it sets
 * IPPD_FLAG_BAD_LAYOUT and not all of its question rows are written.
 * active[] is ignored (every question is prefilled).  No workspace; one
 * kernel launch.
 * Two-level batch (num_instr > 0, Sec. 4.4): every question's prompt is
 * [p_s; c_b; x_i] with p_s the instruction of prompt b.  Then, for token t
 * of instruction s,
 *   out_ctx[instr_off[s] + t][h] = the same over the instruction keys 0..t
 *                                  (causal), query rotated at t;
 * context rows see all keys of p_s and then their context causally (query
 * at instr_len[s] + t), question rows all keys of p_s and c_b and then
 * their own question causally (query at instr_len[s] + ctx_len[b] + u).
 * q_ctx holds the instruction queries at the instruction rows of the pool
 * (rows instr_off[s] .. instr_off[s] + instr_len[s] - 1); the cache holds
 * the instruction keys (ippd_load_instructions).  IPPD computes the rows of
 * each instruction once.
 */
ippd_status_t ippd_prefill_attention(const ippd_batch_t *batch, int32_t max_prompt_question_tokens,
                                     const void *q_ctx, const void *q_seg, const ippd_kv_cache_t *kv,
                                     float *out_ctx, float *out_seg, hipStream_t stream);

/*
 * Baseline: the same outputs computed as standard prompting does it (Sec. 3:
 * each question is its own prompt [context; question]): every question
 * streams its prompt's context and recomputes the context rows (all copies
 * write the same values to out_ctx).  Same arguments and semantics as
 * ippd_prefill_attention, the bound applying per question, except that the
 * context rows of a prompt without questions are not written (no question's
 * prompt contains them), nor, in a two-level batch, the rows of an
 * instruction none of whose prompts has a question; the instruction rows
 * are recomputed once per question behind the instruction.
 */
ippd_status_t standard_prefill_attention(const ippd_batch_t *batch, int32_t max_prompt_question_tokens,
                                         const void *q_ctx, const void *q_seg, const ippd_kv_cache_t *kv,
                                         float *out_ctx, float *out_seg, hipStream_t stream);

/* Static description of a status code. */
const char *ippd_status_string(ippd_status_t status);

/* hipError_t of the most recent IPPD_ERR_HIP on the calling thread (0 if none). */
int ippd_last_hip_error(void);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int ippd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IPPD_H */
