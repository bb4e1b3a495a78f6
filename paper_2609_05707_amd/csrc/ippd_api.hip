// C ABI of libippd: argument validation, launch planning, kernel launches.
// Nothing here allocates, frees or synchronises; all work is enqueued on the
// caller's stream.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>

#include "ippd.h"
#include "ippd_internal.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kMinChunk = 256;
constexpr int kMaxChunk = 4096;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Host-side checks of the batch sizes and device-array pointers.
ippd_status_t check_batch(const ippd_batch_t* bt) {
  if (bt == nullptr) return IPPD_ERR_NULL;
  if (bt->dtype != IPPD_DTYPE_F32 && bt->dtype != IPPD_DTYPE_BF16) return IPPD_ERR_DTYPE;
  if (bt->num_prompts < 1 || bt->num_questions < 0 || bt->num_q_heads < 1 || bt->num_kv_heads < 1)
    return IPPD_ERR_SHAPE;
  if (bt->num_q_heads % bt->num_kv_heads != 0) return IPPD_ERR_SHAPE;
  if (bt->num_q_heads / bt->num_kv_heads > ippd::kMaxGroup) return IPPD_ERR_SHAPE;
  if (bt->head_dim != 64 && bt->head_dim != 128) return IPPD_ERR_SHAPE;
  if (bt->ctx_pool_tokens < 0 || (bt->ctx_pool_tokens & 7)) return IPPD_ERR_SHAPE;
  if (bt->seg_capacity < 8 || (bt->seg_capacity & 7)) return IPPD_ERR_SHAPE;
  if (bt->max_ctx_len < 0 || bt->max_ctx_len > bt->ctx_pool_tokens) return IPPD_ERR_SHAPE;
  if (bt->max_questions < 1 || bt->max_questions > ippd::kMaxQuestionsPerPrompt) return IPPD_ERR_SHAPE;
  if (bt->chunk_tokens < 0 || (bt->chunk_tokens & 31)) return IPPD_ERR_SHAPE;
  if (bt->tile_rows != 0 && bt->tile_rows != 16 && bt->tile_rows != 32 && bt->tile_rows != 64 &&
      bt->tile_rows != 128 && bt->tile_rows != 256)
    return IPPD_ERR_SHAPE;
  if (bt->tile_rows == 256 && !(bt->dtype == IPPD_DTYPE_BF16 && bt->head_dim == 128)) return IPPD_ERR_SHAPE;
  if (!(bt->rope_base > 0.0) || !isfinite(bt->rope_base)) return IPPD_ERR_SHAPE;
  if (!isfinite(bt->scale)) return IPPD_ERR_SHAPE;
  if (!bt->ctx_off || !bt->ctx_len || !bt->q_start || !bt->seg_len || !bt->active || !bt->err_flag)
    return IPPD_ERR_NULL;
  if (bt->num_instr < 0) return IPPD_ERR_SHAPE;
  if (bt->num_instr > 0) {
    if (bt->num_instr > bt->num_prompts || bt->max_instr_len < 0 || bt->max_instr_len > bt->ctx_pool_tokens ||
        bt->max_instr_questions < 1)
      return IPPD_ERR_SHAPE;
    if (!bt->instr_start || !bt->instr_off || !bt->instr_len) return IPPD_ERR_NULL;
  }
  return IPPD_OK;
}

// Two-level fields of the kernel parameter blocks (S = 0 leaves positions unshifted).
template <typename P>
void set_instr_positions(const ippd_batch_t* bt, P* p) {
  p->S = bt->num_instr;
  p->instr_start = bt->num_instr > 0 ? bt->instr_start : nullptr;
  p->instr_len = bt->num_instr > 0 ? bt->instr_len : nullptr;
}

float softmax_scale(const ippd_batch_t* bt) {
  return bt->scale > 0.f ? bt->scale : 1.0f / sqrtf(static_cast<float>(bt->head_dim));
}

size_t round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Compute units the planner sizes grids for: the 256 of MI355X (gfx950).  A
// constant, not a device query, so that the plan (and with it the workspace
// size) depends on the batch fields only, the library holds no state, and a
// workspace query on one thread or device agrees with the launch on another.
// On a part with fewer compute units the plan is still correct, only sized
// for more of them.
constexpr int kPlanComputeUnits = 256;
int compute_units() { return kPlanComputeUnits; }

// theta_j = base^(-2j/D) in fp64, the rotation frequencies of pair j.
void fill_inv_freq(const ippd_batch_t* bt, double* out) {
  const int half = bt->head_dim / 2;
  for (int j = 0; j < ippd::kMaxHalfDim; ++j)
    out[j] = j < half ? pow(bt->rope_base, -2.0 * j / bt->head_dim) : 0.0;
}

// Launch plan of a decode call.  Depends only on host fields, so the
// workspace query and the launch agree.
bool plan_step(const ippd_batch_t* bt, bool shared, ippd::StepPlan* pl, bool dense = false) {
  if (check_batch(bt) != IPPD_OK) return false;
  // dense-mask baseline: one-level batches, up to 64 questions per prompt
  if (dense && (!shared || bt->num_instr > 0 || bt->max_questions > 64)) return false;
  const int G = bt->num_q_heads / bt->num_kv_heads;
  const int64_t max_rows = shared ? static_cast<int64_t>(bt->max_questions) * G : G;
  // rows per context unit: 16 * rb per wave.  bf16 at D = 128 with more than
  // 64 rows puts two 16-row blocks on each wave (each K/V fragment read from
  // LDS serves both): 128 rows as 4 x 32, 256 as 8 x 32.
  const bool two_blocks_ok = bt->dtype == IPPD_DTYPE_BF16 && bt->head_dim == 128;
  int rows = bt->tile_rows;
  // a two-level batch's instruction rows (all questions behind it) favour at
  // least 64-row units (measured against 32 at 6 contexts per instruction)
  int64_t sized_rows = max_rows;
  if (bt->num_instr > 0 && shared) {
    const int64_t irows = static_cast<int64_t>(bt->max_instr_questions) * G;
    const int64_t want = irows < 64 ? irows : 64;
    if (want > sized_rows) sized_rows = want;
  }
  if (rows == 0) rows = sized_rows <= 16 ? 16 : (sized_rows <= 32 ? 32 : (sized_rows <= 64 ? 64 : (sized_rows <= 128 || !two_blocks_ok ? 128 : 256)));
  // 128-row units at bf16, D = 128 over prompts of (nearly) one length: eight
  // waves of one 16-row block each, one workgroup per compute unit with the
  // deep ring.  Half the units of the four-wave shape (two workgroups per
  // compute unit), so half the partial states, at the same streaming rate;
  // ragged batches keep the four-wave shape, whose second workgroup per
  // compute unit covers the uneven unit lengths.
  const bool near_uniform = bt->ctx_pool_tokens * 10 >= static_cast<int64_t>(bt->num_prompts) * bt->max_ctx_len * 9;
  const bool eight_single = two_blocks_ok && shared && !dense && bt->num_instr == 0 && rows == 128 && near_uniform;
  const int rb = rows > 64 && two_blocks_ok && !eight_single ? 2 : 1;
  int waves = rows / (16 * rb);
  // fp32 at D = 128: the operands of eight waves do not fit their registers
  if (bt->dtype == IPPD_DTYPE_F32 && bt->head_dim == 128 && waves > 4) waves = 4;
  const int unit_rows = 16 * rb * waves;
  const int nrg = static_cast<int>((max_rows + unit_rows - 1) / unit_rows);
  // workgroups resident per compute unit (eight waves of two row blocks use
  // the registers of two, and their ring the LDS of one)
  const int wg_per_cu = (waves == 8 && (rb == 2 || eight_single)) ? 1 : 2;
  const int64_t n_groups = shared ? static_cast<int64_t>(bt->num_prompts) * bt->num_kv_heads
                                  : static_cast<int64_t>(bt->num_questions) * bt->num_kv_heads;
  // two-level batch: instruction groups, (instruction, kv head) or (question, kv head)
  const int S = bt->num_instr;
  const int64_t n_igroups = S == 0 ? 0 : (shared ? static_cast<int64_t>(S) : bt->num_questions) * bt->num_kv_heads;
  const int64_t irows = shared ? static_cast<int64_t>(bt->max_instr_questions) * G : G;
  const int nrg_i = S == 0 ? 1 : static_cast<int>((irows + unit_rows - 1) / unit_rows);
  int chunk = bt->chunk_tokens;
  if (chunk == 0) {
    // context tokens to stream: one-level IPPD reads each prompt once, and the
    // prompts are packed in the pool, so its size bounds their sum (a ragged
    // batch then gets a chunk from its total, not from B times the longest)
    const int64_t ctx_tokens = shared ? std::min<int64_t>(bt->ctx_pool_tokens,
                                                          static_cast<int64_t>(bt->num_prompts) * bt->max_ctx_len)
                                      : static_cast<int64_t>(bt->num_questions) * bt->max_ctx_len;
    const int64_t work = ctx_tokens * bt->num_kv_heads * nrg + n_igroups * nrg_i * (S ? bt->max_instr_len : 0);
    const int64_t target = static_cast<int64_t>(compute_units()) * wg_per_cu;
    int64_t ch = (work + target - 1) / target;
    ch = (ch + 31) / 32 * 32;
    ch = ch < kMinChunk ? kMinChunk : (ch > kMaxChunk ? kMaxChunk : ch);
    chunk = static_cast<int>(ch);
  }
  const int64_t max_chunks = (bt->max_ctx_len + chunk - 1) / chunk;
  const int64_t ctx_blocks = 8 * nrg * ((n_groups * max_chunks + 7) / 8);
  const int64_t max_ichunks = S == 0 ? 0 : (bt->max_instr_len + chunk - 1) / chunk;
  const int64_t instr_blocks = 8 * nrg_i * ((n_igroups * max_ichunks + 7) / 8);
  // segment tasks (question, kv head): as few per unit as keeps the segment
  // units within one round of resident workgroups (they run after the
  // context units), at most `waves` per unit, and all tasks' wave states
  // must fit the smallest LDS ring (32 KB)
  const bool deep = ctx_blocks + instr_blocks <= compute_units() || wg_per_cu == 1;
  const int64_t slots = static_cast<int64_t>(compute_units()) * (deep ? 1 : 2);
  const int64_t seg_tasks = static_cast<int64_t>(bt->num_questions) * bt->num_kv_heads;
  const int64_t state_bytes = static_cast<int64_t>(G) * (bt->head_dim + 4) * 4;
  int tpu = 1;
  while (tpu < waves && (seg_tasks + tpu - 1) / tpu > slots && 2 * tpu * state_bytes <= 32768) tpu *= 2;
  // dense-mask baseline: segment units (prompt, kv head, segment chunk, row
  // group) split the prompt's concatenated segment tiles into chunks of
  // kDenseSegTiles tiles; chunk 0 writes the segment slot, chunks 1.. the
  // slots after it (where a two-level batch keeps its instruction chunks)
  const int64_t seg_tiles = static_cast<int64_t>(bt->max_questions) * ((bt->seg_capacity + 31) / 32);
  const int64_t seg_chunks = dense ? (seg_tiles + ippd::kDenseSegTiles - 1) / ippd::kDenseSegTiles : 0;
  const int64_t seg_blocks = dense ? n_groups * seg_chunks * nrg : (seg_tasks + tpu - 1) / tpu;
  const int64_t dense_grid = n_groups * max_chunks * nrg + seg_blocks;
  const int64_t grid = ctx_blocks + instr_blocks + seg_blocks;
  if (grid > (1ll << 30) || n_groups * max_chunks > (1ll << 30) || n_igroups * max_ichunks > (1ll << 30)) return false;
  pl->shared = shared ? 1 : 0;
  pl->waves = waves;
  pl->rb = rb;
  pl->nrg = nrg;
  pl->chunk = chunk;
  pl->max_chunks = static_cast<int>(max_chunks);
  pl->n_groups = static_cast<int>(n_groups);
  pl->grid = static_cast<int>(dense ? dense_grid : grid);
  pl->ctx_blocks = static_cast<int>(ctx_blocks);
  pl->seg_blocks = static_cast<int>(seg_blocks);
  pl->seg_tpu = tpu;
  pl->deep = deep ? 1 : 0;
  pl->dense = dense ? 1 : 0;
  pl->n_igroups = static_cast<int>(n_igroups);
  pl->nrg_i = nrg_i;
  pl->max_ichunks = static_cast<int>(dense ? seg_chunks - 1 : max_ichunks);
  pl->instr_blocks = static_cast<int>(instr_blocks);
  pl->part_slots = static_cast<size_t>(max_chunks + 1 + pl->max_ichunks) * bt->num_questions * bt->num_q_heads;
  pl->off_acc = 0;
  pl->off_ml = pl->off_acc + round256(pl->part_slots * bt->head_dim * sizeof(float));
  pl->workspace_bytes = pl->off_ml + round256(pl->part_slots * 2 * sizeof(float));
  return true;
}

ippd_status_t hip_status(hipError_t e) {
  if (e == hipSuccess) return IPPD_OK;
  g_last_hip_error = static_cast<int>(e);
  return IPPD_ERR_HIP;
}

// Shared body of the four decode entry points.  fused: q_new/k_new/v_new are
// raw token inputs that this launch rotates and appends (q_rot optional
// output); otherwise q_rot holds rotated queries and the segment already
// contains the step's token.
ippd_status_t decode(const ippd_batch_t* bt, bool shared, bool fused, const void* q_new,
                     const void* k_new, const void* v_new, const void* q_rot_in, void* q_rot_out,
                     const ippd_kv_cache_t* kv, float* out, float* lse, void* workspace,
                     size_t workspace_bytes, hipStream_t stream, bool dense = false) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (!kv || !out || !kv->ctx_k || !kv->ctx_vt || !kv->seg_k || !kv->seg_vt) return IPPD_ERR_NULL;
  if (fused ? (!q_new || !k_new || !v_new) : !q_rot_in) return IPPD_ERR_NULL;
  if (!aligned16(out) || !aligned16(kv->ctx_k) || !aligned16(kv->ctx_vt) || !aligned16(kv->seg_k) ||
      !aligned16(kv->seg_vt) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3)))
    return IPPD_ERR_ALIGN;
  if (fused ? (!aligned16(q_new) || !aligned16(k_new) || !aligned16(v_new) || (q_rot_out && !aligned16(q_rot_out)))
            : !aligned16(q_rot_in))
    return IPPD_ERR_ALIGN;
  ippd::StepPlan pl;
  if (!plan_step(bt, shared, &pl, dense)) return IPPD_ERR_SHAPE;
  if (bt->num_questions == 0) return IPPD_OK;
  if (!workspace || workspace_bytes < pl.workspace_bytes) return IPPD_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) & 255u) return IPPD_ERR_ALIGN;

  ippd::StepParams p;
  p.q_new = q_new; p.k_new = k_new; p.v_new = v_new;
  p.q_rot_in = q_rot_in; p.q_rot_out = q_rot_out;
  p.ctx_k = kv->ctx_k; p.ctx_vt = kv->ctx_vt; p.seg_k = kv->seg_k; p.seg_vt = kv->seg_vt;
  p.ctx_off = bt->ctx_off; p.ctx_len = bt->ctx_len; p.q_start = bt->q_start;
  p.seg_len = bt->seg_len; p.active = bt->active; p.err_flag = bt->err_flag;
  p.out = out; p.lse = lse;
  char* ws = static_cast<char*>(workspace);
  p.part_acc = reinterpret_cast<float*>(ws + pl.off_acc);
  p.part_ml = reinterpret_cast<float*>(ws + pl.off_ml);
  p.pool = bt->ctx_pool_tokens;
  p.B = bt->num_prompts; p.Nt = bt->num_questions; p.Hq = bt->num_q_heads; p.Hkv = bt->num_kv_heads;
  p.G = bt->num_q_heads / bt->num_kv_heads; p.D = bt->head_dim; p.seg_cap = bt->seg_capacity;
  p.max_ctx_len = bt->max_ctx_len; p.max_questions = bt->max_questions;
  p.shared = pl.shared; p.fused = fused ? 1 : 0; p.nrg = pl.nrg; p.chunk = pl.chunk;
  p.max_chunks = pl.max_chunks; p.n_groups = pl.n_groups; p.ctx_blocks = pl.ctx_blocks;
  p.seg_tpu = pl.seg_tpu;
  p.instr_start = bt->num_instr > 0 ? bt->instr_start : nullptr;
  p.instr_off = bt->num_instr > 0 ? bt->instr_off : nullptr;
  p.instr_len = bt->num_instr > 0 ? bt->instr_len : nullptr;
  p.S = bt->num_instr; p.max_instr_len = bt->max_instr_len; p.max_instr_questions = bt->max_instr_questions;
  p.n_igroups = pl.n_igroups; p.nrg_i = pl.nrg_i; p.max_ichunks = pl.max_ichunks; p.instr_blocks = pl.instr_blocks;
  // merge: enough threads per item that each folds at most 8 of the
  // max_chunks + 1 partial states; items split over workgroups of kMergeThreads
  {
    int ph = 1;
    while (ph < 8 && (pl.max_chunks + 1 + pl.max_ichunks + ph - 1) / ph > 8) ph *= 2;
    const int items = bt->num_q_heads * (bt->head_dim / 8);
    const int per = ippd::kMergeThreads / ph;
    p.merge_phases = ph;
    p.merge_parts = (items + per - 1) / per;
  }
  p.scale = softmax_scale(bt);
  p.c = p.scale * 1.4426950408889634f;
  p.dense = pl.dense;
  fill_inv_freq(bt, p.inv_freq);
  if (pl.dense) return hip_status(ippd::launch_dense(bt->dtype, pl.waves, pl.rb, pl.grid, p, stream));
  return hip_status(ippd::launch_step(bt->dtype, pl.waves, pl.rb, pl.deep != 0, pl.grid, p, stream));
}


// Launch plan of a prefill call (host fields only).
bool plan_prefill(const ippd_batch_t* bt, bool shared, int32_t max_q_tokens, ippd::PrefillPlan* pl) {
  if (check_batch(bt) != IPPD_OK || max_q_tokens < 0) return false;
  int waves = 0, rb = 0;
  if (!ippd::prefill_variant(bt->dtype, bt->head_dim, &waves, &rb)) return false;
  const int G = bt->num_q_heads / bt->num_kv_heads;
  // 256-row units that would not fill the chip (an estimate from the host
  // bounds) are halved: twice the units, each K/V fragment serving one row
  // block.  tile_rows 128 or 256 fixes the choice.
  if (rb == 2 && bt->tile_rows == 128) {
    rb = 1;
  } else if (rb == 2 && bt->tile_rows != 256) {
    const int tb2 = 16 * rb * waves / G;
    const int64_t groups = static_cast<int64_t>(shared ? bt->num_prompts : bt->num_questions) * bt->num_kv_heads;
    const int64_t qt = shared ? max_q_tokens : (max_q_tokens < bt->seg_capacity ? max_q_tokens : bt->seg_capacity);
    const int64_t units = groups * ((qt + tb2 - 1) / tb2 + (static_cast<int64_t>(bt->max_ctx_len) + tb2 - 1) / tb2);
    if (units < compute_units()) rb = 1;
  }
  const int tb = 16 * rb * waves / G;
  const int64_t n_groups = static_cast<int64_t>(shared ? bt->num_prompts : bt->num_questions) * bt->num_kv_heads;
  const int64_t gps = (n_groups + 7) / 8;
  // two-level batch: instruction rows once per instruction (IPPD) or per question (baseline)
  const int S = bt->num_instr;
  const int64_t n_igroups = S == 0 ? 0 : static_cast<int64_t>(shared ? S : bt->num_questions) * bt->num_kv_heads;
  const int64_t n_cgroups = n_groups + n_igroups, gps_c = (n_cgroups + 7) / 8;
  const int64_t qtok = shared ? max_q_tokens : (max_q_tokens < bt->seg_capacity ? max_q_tokens : bt->seg_capacity);
  const int64_t rows_c = S > 0 && bt->max_instr_len > bt->max_ctx_len ? bt->max_instr_len : bt->max_ctx_len;
  const int64_t kq = (qtok + tb - 1) / tb, kc = (rows_c + tb - 1) / tb;
  const int64_t q_blocks = 8 * gps * kq, grid = q_blocks + 8 * gps_c * kc;
  if (grid > (1ll << 30)) return false;
  pl->shared = shared ? 1 : 0;
  pl->waves = waves;
  pl->rb = rb;
  pl->tb = tb;
  pl->n_groups = static_cast<int>(n_groups);
  pl->gps = static_cast<int>(gps);
  pl->n_cgroups = static_cast<int>(n_cgroups);
  pl->gps_c = static_cast<int>(gps_c);
  pl->kq = static_cast<int>(kq);
  pl->kc = static_cast<int>(kc);
  pl->q_blocks = static_cast<int>(q_blocks);
  pl->grid = static_cast<int>(grid);
  return true;
}

// Shared body of the two prefill entry points.
ippd_status_t prefill(const ippd_batch_t* bt, bool shared, int32_t max_q_tokens, const void* q_ctx,
                      const void* q_seg, const ippd_kv_cache_t* kv, float* out_ctx, float* out_seg,
                      hipStream_t stream) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (!q_ctx || !q_seg || !kv || !out_ctx || !out_seg || !kv->ctx_k || !kv->ctx_vt || !kv->seg_k || !kv->seg_vt)
    return IPPD_ERR_NULL;
  if (!aligned16(q_ctx) || !aligned16(q_seg) || !aligned16(out_ctx) || !aligned16(out_seg) ||
      !aligned16(kv->ctx_k) || !aligned16(kv->ctx_vt) || !aligned16(kv->seg_k) || !aligned16(kv->seg_vt))
    return IPPD_ERR_ALIGN;
  ippd::PrefillPlan pl;
  if (!plan_prefill(bt, shared, max_q_tokens, &pl)) return IPPD_ERR_SHAPE;
  if (pl.grid == 0) return IPPD_OK;
  ippd::PrefillParams p;
  p.q_ctx = q_ctx; p.q_seg = q_seg;
  p.ctx_k = kv->ctx_k; p.ctx_vt = kv->ctx_vt; p.seg_k = kv->seg_k; p.seg_vt = kv->seg_vt;
  p.ctx_off = bt->ctx_off; p.ctx_len = bt->ctx_len; p.q_start = bt->q_start; p.seg_len = bt->seg_len;
  p.err_flag = bt->err_flag;
  p.out_ctx = out_ctx; p.out_seg = out_seg;
  p.pool = bt->ctx_pool_tokens;
  p.B = bt->num_prompts; p.Nt = bt->num_questions; p.Hq = bt->num_q_heads; p.Hkv = bt->num_kv_heads;
  p.G = bt->num_q_heads / bt->num_kv_heads; p.D = bt->head_dim; p.seg_cap = bt->seg_capacity;
  p.max_ctx_len = bt->max_ctx_len;
  p.shared = pl.shared; p.tb = pl.tb; p.n_groups = pl.n_groups; p.gps = pl.gps;
  p.kq = pl.kq; p.kc = pl.kc; p.q_blocks = pl.q_blocks;
  p.n_cgroups = pl.n_cgroups; p.gps_c = pl.gps_c;
  p.S = bt->num_instr;
  p.max_instr_len = bt->num_instr > 0 ? bt->max_instr_len : 0;
  p.instr_start = bt->num_instr > 0 ? bt->instr_start : nullptr;
  p.instr_off = bt->num_instr > 0 ? bt->instr_off : nullptr;
  p.instr_len = bt->num_instr > 0 ? bt->instr_len : nullptr;
  p.c = softmax_scale(bt) * 1.4426950408889634f;
  fill_inv_freq(bt, p.inv_freq);
  return hip_status(ippd::launch_prefill(bt->dtype, bt->head_dim, pl.rb, pl.grid, p, stream));
}

// Per-device address of the no-allocation scratch array, looked up once per
// device (concurrent first calls look up the same address).
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

}  // namespace

// Partial softmax states of ippd_decode_step_noalloc: each GPU the library
// runs on holds its own copy until the process ends.  In host code this name
// is a stand-in, not a device address: kernels get the address looked up with
// hipGetSymbolAddress on the device concerned.
static __device__ __align__(256) unsigned char scratch[IPPD_NOALLOC_SCRATCH_BYTES];

extern "C" {

ippd_status_t ippd_load_context(const ippd_batch_t* bt, const void* k_raw, const void* v_raw,
                                const ippd_kv_cache_t* kv, hipStream_t stream) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (!k_raw || !v_raw || !kv || !kv->ctx_k || !kv->ctx_vt) return IPPD_ERR_NULL;
  if (!aligned16(k_raw) || !aligned16(v_raw) || !aligned16(kv->ctx_k) || !aligned16(kv->ctx_vt))
    return IPPD_ERR_ALIGN;
  ippd::LoadContextParams p;
  p.k_raw = k_raw; p.v_raw = v_raw; p.ctx_k = kv->ctx_k; p.ctx_vt = kv->ctx_vt;
  p.ctx_off = bt->ctx_off; p.ctx_len = bt->ctx_len; p.err_flag = bt->err_flag;
  p.pool = bt->ctx_pool_tokens; p.B = bt->num_prompts; p.Hkv = bt->num_kv_heads; p.D = bt->head_dim;
  p.max_ctx_len = bt->max_ctx_len;
  set_instr_positions(bt, &p);
  fill_inv_freq(bt, p.inv_freq);
  return hip_status(ippd::launch_load_context(bt->dtype, p, stream));
}

ippd_status_t ippd_load_instructions(const ippd_batch_t* bt, const void* k_raw, const void* v_raw,
                                     const ippd_kv_cache_t* kv, hipStream_t stream) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (bt->num_instr == 0) return IPPD_ERR_SHAPE;
  if (!k_raw || !v_raw || !kv || !kv->ctx_k || !kv->ctx_vt) return IPPD_ERR_NULL;
  if (!aligned16(k_raw) || !aligned16(v_raw) || !aligned16(kv->ctx_k) || !aligned16(kv->ctx_vt))
    return IPPD_ERR_ALIGN;
  // the context loader over the instruction blocks, at positions 0..len-1
  ippd::LoadContextParams p;
  p.k_raw = k_raw; p.v_raw = v_raw; p.ctx_k = kv->ctx_k; p.ctx_vt = kv->ctx_vt;
  p.ctx_off = bt->instr_off; p.ctx_len = bt->instr_len; p.err_flag = bt->err_flag;
  p.pool = bt->ctx_pool_tokens; p.B = bt->num_instr; p.Hkv = bt->num_kv_heads; p.D = bt->head_dim;
  p.max_ctx_len = bt->max_instr_len;
  p.S = 0; p.instr_start = nullptr; p.instr_len = nullptr;
  fill_inv_freq(bt, p.inv_freq);
  return hip_status(ippd::launch_load_context(bt->dtype, p, stream));
}

ippd_status_t ippd_load_segments(const ippd_batch_t* bt, const void* k_raw, const void* v_raw,
                                 const int32_t* init_len, const ippd_kv_cache_t* kv,
                                 hipStream_t stream) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (!k_raw || !v_raw || !init_len || !kv || !kv->seg_k || !kv->seg_vt) return IPPD_ERR_NULL;
  if (!aligned16(k_raw) || !aligned16(v_raw) || !aligned16(kv->seg_k) || !aligned16(kv->seg_vt))
    return IPPD_ERR_ALIGN;
  ippd::LoadSegmentsParams p;
  p.k_raw = k_raw; p.v_raw = v_raw; p.init_len = init_len; p.seg_k = kv->seg_k; p.seg_vt = kv->seg_vt;
  p.ctx_len = bt->ctx_len; p.q_start = bt->q_start; p.seg_len = bt->seg_len; p.err_flag = bt->err_flag;
  p.B = bt->num_prompts; p.Nt = bt->num_questions; p.Hkv = bt->num_kv_heads; p.D = bt->head_dim;
  p.seg_cap = bt->seg_capacity;
  set_instr_positions(bt, &p);
  fill_inv_freq(bt, p.inv_freq);
  return hip_status(ippd::launch_load_segments(bt->dtype, p, stream));
}

ippd_status_t ippd_append_kv(const ippd_batch_t* bt, const void* q_new, const void* k_new,
                             const void* v_new, void* q_rot, const ippd_kv_cache_t* kv,
                             hipStream_t stream) {
  ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  if (!q_new || !k_new || !v_new || !q_rot || !kv || !kv->seg_k || !kv->seg_vt) return IPPD_ERR_NULL;
  if (!aligned16(q_new) || !aligned16(k_new) || !aligned16(v_new) || !aligned16(q_rot) ||
      !aligned16(kv->seg_k) || !aligned16(kv->seg_vt))
    return IPPD_ERR_ALIGN;
  ippd::AppendParams p;
  p.q_new = q_new; p.k_new = k_new; p.v_new = v_new; p.q_rot = q_rot;
  p.seg_k = kv->seg_k; p.seg_vt = kv->seg_vt;
  p.ctx_len = bt->ctx_len; p.q_start = bt->q_start; p.seg_len = bt->seg_len;
  p.active = bt->active; p.err_flag = bt->err_flag;
  p.B = bt->num_prompts; p.Nt = bt->num_questions; p.Hq = bt->num_q_heads; p.Hkv = bt->num_kv_heads;
  p.D = bt->head_dim; p.seg_cap = bt->seg_capacity;
  set_instr_positions(bt, &p);
  fill_inv_freq(bt, p.inv_freq);
  return hip_status(ippd::launch_append(bt->dtype, p, stream));
}

size_t ippd_decode_workspace_bytes(const ippd_batch_t* bt) {
  ippd::StepPlan pl;
  return plan_step(bt, true, &pl) ? pl.workspace_bytes : 0;
}

size_t standard_decode_workspace_bytes(const ippd_batch_t* bt) {
  ippd::StepPlan pl;
  return plan_step(bt, false, &pl) ? pl.workspace_bytes : 0;
}

ippd_status_t ippd_decode_attention(const ippd_batch_t* bt, const void* q_rot,
                                    const ippd_kv_cache_t* kv, float* out, float* lse,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return decode(bt, true, false, nullptr, nullptr, nullptr, q_rot, nullptr, kv, out, lse, workspace,
                workspace_bytes, stream);
}

ippd_status_t standard_decode_attention(const ippd_batch_t* bt, const void* q_rot,
                                        const ippd_kv_cache_t* kv, float* out, float* lse,
                                        void* workspace, size_t workspace_bytes,
                                        hipStream_t stream) {
  return decode(bt, false, false, nullptr, nullptr, nullptr, q_rot, nullptr, kv, out, lse, workspace,
                workspace_bytes, stream);
}

size_t dense_decode_workspace_bytes(const ippd_batch_t* bt) {
  ippd::StepPlan pl;
  return plan_step(bt, true, &pl, true) ? pl.workspace_bytes : 0;
}

ippd_status_t dense_decode_attention(const ippd_batch_t* bt, const void* q_rot, const ippd_kv_cache_t* kv,
                                     float* out, float* lse, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
  return decode(bt, true, false, nullptr, nullptr, nullptr, q_rot, nullptr, kv, out, lse, workspace,
                workspace_bytes, stream, true);
}

ippd_status_t ippd_decode_step(const ippd_batch_t* bt, const void* q_new, const void* k_new,
                               const void* v_new, void* q_rot, const ippd_kv_cache_t* kv, float* out,
                               float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return decode(bt, true, true, q_new, k_new, v_new, nullptr, q_rot, kv, out, lse, workspace,
                workspace_bytes, stream);
}

ippd_status_t ippd_decode_step_noalloc(const ippd_batch_t* bt, const void* q_new, const void* k_new,
                                       const void* v_new, void* q_rot, const ippd_kv_cache_t* kv, float* out,
                                       float* lse, hipStream_t stream) {
  const ippd_status_t st = check_batch(bt);
  if (st != IPPD_OK) return st;
  ippd::StepPlan pl;
  if (!plan_step(bt, true, &pl)) return IPPD_ERR_SHAPE;
  if (pl.workspace_bytes > IPPD_NOALLOC_SCRATCH_BYTES) return IPPD_ERR_SCRATCH;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return hip_status(hipErrorInvalidDevice);
  void* ptr = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e);
    if (ptr == nullptr || (reinterpret_cast<uintptr_t>(ptr) & 255u)) return hip_status(hipErrorInvalidSymbol);
    g_scratch_addr[dev].store(ptr, std::memory_order_release);
  }
  return decode(bt, true, true, q_new, k_new, v_new, nullptr, q_rot, kv, out, lse, ptr, IPPD_NOALLOC_SCRATCH_BYTES,
                stream);
}

ippd_status_t standard_decode_step(const ippd_batch_t* bt, const void* q_new, const void* k_new,
                                   const void* v_new, void* q_rot, const ippd_kv_cache_t* kv,
                                   float* out, float* lse, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  return decode(bt, false, true, q_new, k_new, v_new, nullptr, q_rot, kv, out, lse, workspace,
                workspace_bytes, stream);
}

ippd_status_t ippd_prefill_attention(const ippd_batch_t* bt, int32_t max_prompt_question_tokens,
                                     const void* q_ctx, const void* q_seg, const ippd_kv_cache_t* kv,
                                     float* out_ctx, float* out_seg, hipStream_t stream) {
  return prefill(bt, true, max_prompt_question_tokens, q_ctx, q_seg, kv, out_ctx, out_seg, stream);
}

ippd_status_t standard_prefill_attention(const ippd_batch_t* bt, int32_t max_prompt_question_tokens,
                                         const void* q_ctx, const void* q_seg, const ippd_kv_cache_t* kv,
                                         float* out_ctx, float* out_seg, hipStream_t stream) {
  return prefill(bt, false, max_prompt_question_tokens, q_ctx, q_seg, kv, out_ctx, out_seg, stream);
}

const char* ippd_status_string(ippd_status_t s) {
  // a C caller may pass any int: read it as one (an out-of-range value of the
  // enum type itself would be undefined behaviour here)
  int code;
  static_assert(sizeof(code) == sizeof(s), "status codes are int-sized");
  memcpy(&code, &s, sizeof code);
  switch (code) {
    case IPPD_OK: return "ok";
    case IPPD_ERR_NULL: return "required pointer is NULL";
    case IPPD_ERR_SHAPE: return "inconsistent or unsupported sizes";
    case IPPD_ERR_DTYPE: return "unknown dtype";
    case IPPD_ERR_ALIGN: return "pointer not aligned (16 bytes; workspace 256 bytes)";
    case IPPD_ERR_WORKSPACE: return "workspace missing or too small";
    case IPPD_ERR_HIP: return "HIP call failed";
    case IPPD_ERR_SCRATCH: return "batch needs more partial-state scratch than the no-allocation step holds";
  }
  return "unknown status";
}

int ippd_last_hip_error(void) { return g_last_hip_error; }

int ippd_version(void) { return 700; }

}  // extern "C"
