// IPPD decode-step attention on gfx950: two launches per call.
//
//   attend_kernel  context units (group, chunk, row group): shared-context
//                  attention of 16*NW query rows over one chunk of context
//                  tokens, one unnormalised partial softmax state (running
//                  max, sum, weighted values) per row; then segment units,
//                  seg_tpu tasks (question i, kv head g) each: in the fused
//                  step rotate and append the token fed this step, and
//                  attend the G query heads of group g over the question's
//                  own segment (M_qtn, Sec. 4.1), the segment's tiles split
//                  over the task's waves, whose states are combined in LDS;
//   merge_kernel   combines each question's partial states exactly
//                  (splitting only regroups the sums of attn_IPPD, Sec. 4.2)
//                  and, in the fused step, advances its segment length.
// The launch boundary orders the two, so no unit ever waits for another.
//
// A *group* is (prompt b, kv head g) for IPPD or (question i, kv head g) for
// the standard baseline.  A context unit streams context tokens
// [chunk*C, (chunk+1)*C) of its group against 16*NW query rows, the
// (question, head of group g) pairs of the prompt in order.  IPPD serves all
// questions of the prompt from one pass over the chunk, so K_c and V_c come
// from HBM once for all M_j queries (Sec. 4.3); the baseline serves the G
// rows of one question and reads the context once per question (App. A.2.2,
// PC+PA decode).  The workgroup streams 32-token tiles through an LDS ring
// with LDS-DMA (global_load_lds_dwordx4: HBM -> LDS without passing through
// registers), several tiles ahead of the compute; wave w owns rows
// 16w..16w+15 and reads its MFMA operands from the ring:
//   S^T (keys x rows) = K Q^T       v_mfma_f32_16x16x32_bf16, A = 16 keys x 32 dims
//   P^T = exp2(c * (S^T - m))       online softmax; the row max is reduced over
//                                   the four 16-lane rows with permlane swaps
//   O^T (dims x rows) += V^T P^T    A = V^T (the value cache is transposed),
//                                   B = P^T taken straight from the S^T registers
// Key rows are assigned to MFMA rows so that lane row r of S^T holds 8
// consecutive tokens, exactly the B layout the PV product needs.  Ring rows
// are XOR-swizzled in 16-byte chunks so that the 16 lanes of every ds_read
// hit distinct bank groups of the 64-bank LDS.
//
#include <float.h>
#include <stddef.h>

#include "ippd_device.h"
#include "ippd_internal.h"
#include "tile_attend.h"

namespace ippd {

// Write one 16-row block's partial state to its slots.
template <int D>
__device__ __forceinline__ void publish_rows(const StepParams& p, const RowState<D>& st, int64_t slot, int lg) {
  float* dst = p.part_acc + slot * D + 4 * lg;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) *reinterpret_cast<f32x4_t*>(dst + 16 * db) = st.o[db];
  if (lg == 0) *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(st.m, st.ls[0]);
}

__device__ __forceinline__ bool prompt_layout_ok(const StepParams& p, int b) {
  const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
  const int64_t off = p.ctx_off[b];
  const int len = p.ctx_len[b];
  return q0 >= 0 && q1 >= q0 && q1 <= p.Nt && q1 - q0 <= p.max_questions &&
         off >= 0 && (off & 7) == 0 && len >= 0 && len <= p.max_ctx_len && off + len <= p.pool;
}

// Segment length a question is served with; -1 if the question is skipped.
__device__ __forceinline__ int usable_seg_len(const StepParams& p, int s) {
  if (p.fused) return (s >= 0 && s < p.seg_cap) ? s : -1;
  return (s >= 1 && s <= p.seg_cap) ? s : -1;
}

// Prompt owning question i (q_start non-decreasing): the number of prompts
// whose questions all precede i, with that prompt's layout fields and
// whether they pass prompt_layout_ok and hold i.  Whole wave: up to 64
// prompts come in one round of loads (lane l reads prompt l, and the owner's
// fields are taken from its lane).
struct PromptInfo {
  int b, q0, q1, len;
  int64_t off;
  bool ok;
};

__device__ __forceinline__ PromptInfo find_prompt(const StepParams& p, int i, int lane) {
  PromptInfo r;
  if (p.B <= 64) {
    const int bl = lane < p.B ? lane : p.B - 1;
    const int q0 = p.q_start[bl], q1 = p.q_start[bl + 1], len = p.ctx_len[bl];
    const int64_t off = p.ctx_off[bl];
    r.b = __popcll(__ballot(lane < p.B && q1 <= i));
    const int bs = r.b < p.B ? r.b : p.B - 1;
    r.q0 = __builtin_amdgcn_readlane(q0, bs);
    r.q1 = __builtin_amdgcn_readlane(q1, bs);
    r.len = __builtin_amdgcn_readlane(len, bs);
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(off), bs);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(static_cast<uint64_t>(off) >> 32), bs);
    r.off = static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
  } else {
    int n = 0;
    for (int b0 = 0; b0 < p.B; b0 += 64) {
      const int bb = b0 + lane;
      n += __popcll(__ballot(bb < p.B && p.q_start[bb + 1] <= i));
    }
    r.b = n;
    const int bs = n < p.B ? n : p.B - 1;
    r.q0 = p.q_start[bs];
    r.q1 = p.q_start[bs + 1];
    r.len = p.ctx_len[bs];
    r.off = p.ctx_off[bs];
  }
  r.ok = r.b < p.B && r.q0 >= 0 && r.q1 >= r.q0 && r.q1 <= p.Nt && r.q1 - r.q0 <= p.max_questions &&
         r.off >= 0 && (r.off & 7) == 0 && r.len >= 0 && r.len <= p.max_ctx_len && r.off + r.len <= p.pool &&
         r.q0 <= i && i < r.q1;
  return r;
}

// Two-level batch: whether the instruction table is sound (the prompt ranges
// of the instructions tile [0, B); each instruction lies in the pool and has
// at most max_instr_questions questions behind it) and question i of prompt
// b lies in the question range of its instruction: exactly the questions
// whose instruction slots the instruction units write.  A question for which
// this fails is skipped (its segment slot carries the skip mark), so that no
// output is formed from slots nobody wrote.  Whole wave; lane l checks
// instructions l, l + 64, ...
__device__ __forceinline__ bool instr_serves(const StepParams& p, int b, int i, int lane) {
  bool bad = false;
  for (int s0 = 0; s0 < p.S; s0 += 64) {
    const int s = s0 + lane;
    bool lb = false;
    if (s < p.S) {
      const int pa = p.instr_start[s], pe = p.instr_start[s + 1];
      lb = !(pa >= 0 && pe >= pa && pe <= p.B && (s > 0 || pa == 0) && (s < p.S - 1 || pe == p.B));
      if (!lb) {
        const int qa = p.q_start[pa], qb = p.q_start[pe];
        const int64_t off = p.instr_off[s];
        const int len = p.instr_len[s];
        lb = !(qa >= 0 && qb >= qa && qb <= p.Nt && qb - qa <= p.max_instr_questions && off >= 0 &&
               (off & 7) == 0 && len >= 0 && len <= p.max_instr_len && off + len <= p.pool);
      }
    }
    bad = bad || wave_any(lb);
  }
  if (bad) return false;
  const int s = instr_of_prompt(p.instr_start, p.S, b);
  return p.q_start[p.instr_start[s]] <= i && i < p.q_start[p.instr_start[s + 1]];
}

// ---------------------------------------------------------------------------
// Row loads of a context unit: the lane's active flag, segment length and
// query fragments.  They are issued with inline asm, ahead of the tile DMA,
// so that the compiler's wait counting (which cannot see the DMA) does not
// make their first use wait for the DMA too; wait_row_loads waits for exactly
// them, its asm taking the destination registers as operands so that nothing
// reads them earlier.
// ---------------------------------------------------------------------------
// Position of the k-th set bit (k < popcount(m)) of a 64-bit mask, by
// halving: six rounds of a popcount of the lower half.
__device__ __forceinline__ int nth_set_bit(uint64_t m, int k) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    const int c = __popcll(m & ((1ull << w) - 1));
    if (k >= c) {
      k -= c;
      m >>= w;
      pos += w;
    }
  }
  return pos;
}

// Active-set compaction of the question range [qa, qb): the number of
// active questions, and for each of the lane's row blocks the kq[rb]-th of
// them (-1 if there are fewer).  Questions that have stopped (Sec. 4.2: a
// finished answer takes no further tokens) then hold no rows, so a unit's
// rows are the G heads of its prompt's active questions in order.  Whole
// wave: 64 flags per ballot, four windows per round of loads.
template <int RB>
__device__ __forceinline__ int active_questions(const uint8_t* __restrict__ active, int qa, int qb,
                                                const int (&kq)[RB], int (&qsel)[RB], int lane) {
  int n = 0;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) qsel[rb] = -1;
  for (int w0 = qa; w0 < qb; w0 += 256) {
    // every load unconditional (lanes past qb read flag qb - 1), so that the
    // four go out together
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = active[min(w0 + 64 * u + lane, qb - 1)];
    bool f[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) f[u] = w0 + 64 * u + lane < qb && v[u] != 0u;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint64_t m = __ballot(f[u]);
      const int c = __popcll(m);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int k = kq[rb] - n;
        if (k >= 0 && k < c) qsel[rb] = w0 + 64 * u + nth_set_bit(m, k);
      }
      n += c;
    }
  }
  return n;
}

__device__ __forceinline__ uint32_t gload_u8(const void* p) {
  uint32_t r;
  asm volatile("global_load_ubyte %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}
__device__ __forceinline__ uint32_t gload_b32(const void* p) {
  uint32_t r;
  asm volatile("global_load_dword %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}
__device__ __forceinline__ u32x4_t gload_b128(const void* p) {
  u32x4_t r;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(p) : "memory");
  return r;
}

template <typename T, int D, bool FUSED, int RB>
struct RowLoads {
  static constexpr int QN = D * static_cast<int>(sizeof(T)) / 64;   // 16-byte query pieces per lane and row
  static constexpr int QPF = static_cast<int>(sizeof(T)) / 2;       // pieces per 8-element fragment
  static constexpr int TN = FUSED ? D / 16 : 0;                    // 16-byte pieces of the lane's D/8 frequencies
  uint32_t a[RB], s[RB];
  u32x4_t q[RB][QN];
  u32x4_t th[TN > 0 ? TN : 1];
};

// Lane (lg, lr) of row block rb (question qi[rb], head h[rb]): dims
// 32*ds + 8*lg + u of the query (raw q_new in the fused step, rotated
// q_rot_in otherwise).
template <typename T, int D, bool FUSED, int RB>
__device__ __forceinline__ void issue_row_loads(RowLoads<T, D, FUSED, RB>& r, const StepParams& p, const int (&qi)[RB],
                                                const int (&h)[RB], int lg) {
  using RL = RowLoads<T, D, FUSED, RB>;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    r.a[rb] = gload_u8(p.active + qi[rb]);
    r.s[rb] = gload_b32(p.seg_len + qi[rb]);
    const char* src = static_cast<const char*>(FUSED ? p.q_new : p.q_rot_in) +
                      ((static_cast<int64_t>(qi[rb]) * p.Hq + h[rb]) * D + lg * 8) * static_cast<int64_t>(sizeof(T));
#pragma unroll
    for (int k = 0; k < RL::QN; ++k)
      r.q[rb][k] = gload_b128(src + (k / RL::QPF) * 32 * static_cast<int>(sizeof(T)) + (k % RL::QPF) * 16);
  }
  if constexpr (FUSED) {
    // theta of pairs 32*ds + 8*lg + u, u = 0..7: 64 contiguous bytes per ds,
    // read where the launch placed StepParams (the kernel's only argument)
    const char* th = (const char*)__builtin_amdgcn_kernarg_segment_ptr() +   // address-space conversion
                     offsetof(StepParams, inv_freq) + 8 * lg * sizeof(double);
#pragma unroll
    for (int k = 0; k < RL::TN; ++k) r.th[k] = gload_b128(th + (k / 4) * 32 * 8 + (k % 4) * 16);
  }
}

// The one wait for the row loads: s_waitcnt vmcnt(N), then every destination
// register is tied to an asm statement at that point, so that none is read
// (or copied) before it (volatile asm statements keep their order).
template <int N, typename T, int D, bool FUSED, int RB>
__device__ __forceinline__ void wait_row_loads(RowLoads<T, D, FUSED, RB>& r) {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  using RL = RowLoads<T, D, FUSED, RB>;
  asm volatile("s_waitcnt vmcnt(%2)" : "+v"(r.a[0]), "+v"(r.s[0]) : "n"(N));
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (rb > 0) asm volatile("" : "+v"(r.a[rb]), "+v"(r.s[rb]));
#pragma unroll
    for (int k = 0; k < RL::QN; ++k) asm volatile("" : "+v"(r.q[rb][k]));
  }
#pragma unroll
  for (int k = 0; k < RL::TN; ++k) asm volatile("" : "+v"(r.th[k]));
}

// Theta of pair u (0..7) of fragment ds from the lane's loaded frequency
// pieces (piece 4*ds + u/2, double u % 2).
template <int TN>
__device__ __forceinline__ double lane_theta(const u32x4_t (&th)[TN], int ds, int u) {
  const u32x4_t tp = th[4 * ds + u / 2];
  return __hiloint2double(static_cast<int>(tp[2 * (u & 1) + 1]), static_cast<int>(tp[2 * (u & 1)]));
}

// Value of lane k of this lane's quad (DPP quad_perm broadcast).
template <int K>
__device__ __forceinline__ float quad_bcast(float v) {
  constexpr int ctrl = K | (K << 2) | (K << 4) | (K << 6);
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), ctrl, 0xF, 0xF, false));
}

// Query fragments (B operand) of one row block from its loaded pieces,
// rotated at pos in the fused step.  Pair j < D/2 is (x_j, x_{j+D/2}):
// fragments ds and ds + DS/2.  quad: the four lanes of each lane quad hold
// heads of one question (G a multiple of 4), so they share every angle:
// lane k of the quad evaluates pairs k and k + 4 of each fragment and the
// quad exchanges the rest.
template <typename T, int D, bool FUSED, int QN, int TN>
__device__ __forceinline__ void row_query(typename Mfma<T>::Frag (&qf)[D / 32], const u32x4_t (&q)[QN],
                                          const u32x4_t (&th)[TN], int64_t pos, bool quad, int lane) {
  using M = Mfma<T>;
  constexpr int DS = D / 32;
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) {
    if constexpr (sizeof(T) == 2) {
      qf[ds] = __builtin_bit_cast(typename M::Frag, q[ds]);
    } else {
      const f32x4_t x = __builtin_bit_cast(f32x4_t, q[2 * ds]), y = __builtin_bit_cast(f32x4_t, q[2 * ds + 1]);
      qf[ds] = typename M::Frag{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
    }
  }
  if constexpr (FUSED) {
    float cs[DS / 2][8], sn[DS / 2][8];
    if (quad) {
      const int k = lane & 3;
#pragma unroll
      for (int ds = 0; ds < DS / 2; ++ds) {
        float ca[2], sa[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          // pair k + 4*hf, chosen among the four by value (not by a
          // runtime index into the pieces, which would go through memory)
          const double t0 = lane_theta(th, ds, 4 * hf), t1 = lane_theta(th, ds, 4 * hf + 1);
          const double t2 = lane_theta(th, ds, 4 * hf + 2), t3 = lane_theta(th, ds, 4 * hf + 3);
          const double t = (k & 2) ? ((k & 1) ? t3 : t2) : ((k & 1) ? t1 : t0);
          rope_cos_sin(pos, t, ca[hf], sa[hf]);
        }
        cs[ds][0] = quad_bcast<0>(ca[0]); sn[ds][0] = quad_bcast<0>(sa[0]);
        cs[ds][1] = quad_bcast<1>(ca[0]); sn[ds][1] = quad_bcast<1>(sa[0]);
        cs[ds][2] = quad_bcast<2>(ca[0]); sn[ds][2] = quad_bcast<2>(sa[0]);
        cs[ds][3] = quad_bcast<3>(ca[0]); sn[ds][3] = quad_bcast<3>(sa[0]);
        cs[ds][4] = quad_bcast<0>(ca[1]); sn[ds][4] = quad_bcast<0>(sa[1]);
        cs[ds][5] = quad_bcast<1>(ca[1]); sn[ds][5] = quad_bcast<1>(sa[1]);
        cs[ds][6] = quad_bcast<2>(ca[1]); sn[ds][6] = quad_bcast<2>(sa[1]);
        cs[ds][7] = quad_bcast<3>(ca[1]); sn[ds][7] = quad_bcast<3>(sa[1]);
      }
    } else {
#pragma unroll
      for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
        for (int u = 0; u < 8; ++u) rope_cos_sin(pos, lane_theta(th, ds, u), cs[ds][u], sn[ds][u]);
    }
#pragma unroll
    for (int ds = 0; ds < DS / 2; ++ds) {
      f32x8_t x = M::to_f32v(qf[ds]), y = M::to_f32v(qf[ds + DS / 2]);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float xr, yr;
        rope_rotate(x[u], y[u], cs[ds][u], sn[ds][u], xr, yr);
        x[u] = xr;
        y[u] = yr;
      }
      qf[ds] = M::from_f32(x);
      qf[ds + DS / 2] = M::from_f32(y);
    }
  }
}

// ---------------------------------------------------------------------------
// LDS of one workgroup.  Context units use all of it as the tile ring.
// Segment units (other workgroups) use the same bytes: per task the query
// rows and the rotation table, then the waves' states to be combined, in the
// first SEGMAIN bytes, and the per-task last key and value, per-wave (max,
// sum), per-task last scores and live flags in the small arrays after them.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, int NS>
struct UnitLds {
  static constexpr int RING = NS * Ring<T, D, NS>::STAGE;
  static constexpr int QROW = D * static_cast<int>(sizeof(T)) + 16;   // padded: a read's 16 lanes hit distinct banks
  static constexpr int QAREA = 16 * QROW;                              // one task's query rows
  static constexpr int TASK = QAREA + (D / 2) * 8;                     // + (cos, sin) of its position
  static constexpr int MAIN = RING;
  // the segment units' small arrays, at the end of main
  static constexpr int KV_BYTES = NW * D * static_cast<int>(sizeof(T));
  static constexpr int EXTRA = 2 * KV_BYTES + NW * 16 * 8 + NW * 16 * 4 + NW * 4;
  static constexpr int SEGMAIN = (MAIN - EXTRA) & ~15;
  static_assert(NW * TASK <= SEGMAIN, "segment tasks must fit");
  alignas(16) unsigned char main[MAIN];
  // per task: the segment's last key (the step's token) and its value
  __device__ __forceinline__ T* k(int task) { return reinterpret_cast<T*>(main + SEGMAIN) + task * D; }
  __device__ __forceinline__ T* v(int task) { return reinterpret_cast<T*>(main + SEGMAIN + KV_BYTES) + task * D; }
  // per wave: (max, sum) of its segment rows
  __device__ __forceinline__ float2* ml(int wave) {
    return reinterpret_cast<float2*>(main + SEGMAIN + 2 * KV_BYTES) + wave * 16;
  }
  // per task: score of the last key per row
  __device__ __forceinline__ float* slast(int task) {
    return reinterpret_cast<float*>(main + SEGMAIN + 2 * KV_BYTES + NW * 16 * 8) + task * 16;
  }
  // per task: served this call
  __device__ __forceinline__ int* live() {
    return reinterpret_cast<int*>(main + SEGMAIN + 2 * KV_BYTES + NW * 16 * 8 + NW * 16 * 4);
  }
};

// ---------------------------------------------------------------------------
// Context unit.  blockIdx -> slice (XCD) = blockIdx & 7, local = blockIdx >> 3;
// consecutive locals of a slice are the row groups of one chunk (they share
// its tiles through that XCD's L2) and chunks are dealt to the slices round
// robin.
// ---------------------------------------------------------------------------
//
// INSTR: an instruction unit of a two-level batch: the group is
// (instruction s, kv head g), whose rows are the questions of every prompt
// behind s (or (question i, kv head g) for the baseline), the keys are the
// instruction's chunk, and the states go to the instruction slots
// max_chunks + 1 + chunk.  In the fused step each row's query is rotated at
// its own question's position instr_len[s] + ctx_len[b] + seg_len[i].
template <typename T, int D, int NW, int NS, bool FUSED, int RB, bool INSTR = false>
__device__ __forceinline__ void context_unit(const StepParams& p, unsigned char* ring, int wave, int lane) {
  using RG = Ring<T, D, NS>;
  using M = Mfma<T>;
  using RL = RowLoads<T, D, FUSED, RB>;
  constexpr int RW = 16 * RB * NW, DPT = RG::BLOCKS / NW;
  constexpr int P0 = RG::NS - 1 < 3 ? RG::NS - 1 : 3;      // tiles issued before the queries are rotated
  const int lr = lane & 15, lg = lane >> 4;
  // instruction units follow the context units (blockIdx >= ctx_blocks)
  const unsigned ub = INSTR ? blockIdx.x - static_cast<unsigned>(p.ctx_blocks) : blockIdx.x;
  const int nrg = INSTR ? p.nrg_i : p.nrg;
  const int nch = INSTR ? p.max_ichunks : p.max_chunks;
  const int slice = ub & 7, local = ub >> 3;
  const int cl = local / nrg, rg = local - cl * nrg;
  const int cglob = cl * 8 + slice;
  if (cglob >= (INSTR ? p.n_igroups : p.n_groups) * nch) return;
  const int grp = cglob / nch, chunk = cglob - grp * nch;

  int b = 0, g, qa, qb;
  int ctx_len, slot_k;                             // key-range length; slot index of this chunk's states
  int64_t off;                                     // key-range start in the pool
  int64_t pos_base = 0;                            // position of the first context token (fused step)
  int pa = 0, pe = 0;                              // INSTR: the prompts behind the instruction
  if constexpr (INSTR) {
    int s = 0;
    bool ok;
    if (p.shared) {
      g = grp / p.S;
      s = grp - g * p.S;
      pa = p.instr_start[s];
      pe = p.instr_start[s + 1];
      // the instructions' prompt ranges must tile [0, B) so that every
      // question's instruction slots are written
      ok = pa >= 0 && pe >= pa && pe <= p.B && (s > 0 || pa == 0) && (s < p.S - 1 || pe == p.B);
      qa = ok ? p.q_start[pa] : 0;
      qb = ok ? p.q_start[pe] : 0;
      ok = ok && qa >= 0 && qb >= qa && qb <= p.Nt && qb - qa <= p.max_instr_questions;
    } else {
      g = grp / p.Nt;
      qa = grp - g * p.Nt;
      qb = qa + 1;
      b = find_prompt(p, qa, lane).b;
      ok = b < p.B;
      if (ok) s = instr_of_prompt(p.instr_start, p.S, b);
      pa = b;
      pe = b + 1;
    }
    off = ok ? p.instr_off[s] : 0;
    ctx_len = ok ? p.instr_len[s] : 0;
    if (!ok || off < 0 || (off & 7) != 0 || ctx_len < 0 || ctx_len > p.max_instr_len || off + ctx_len > p.pool) {
      if (threadIdx.x == 0 && chunk == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
    slot_k = p.max_chunks + 1 + chunk;
  } else {
    if (p.shared) {
      g = grp / p.B;
      b = grp - g * p.B;
    } else {
      g = grp / p.Nt;
      qa = grp - g * p.Nt;
      b = find_prompt(p, qa, lane).b;
      if (b >= p.B) {
        if (threadIdx.x == 0 && chunk == 0) raise_flag(p.err_flag, kFlagBadLayout);
        return;
      }
    }
    if (!prompt_layout_ok(p, b)) {
      if (threadIdx.x == 0 && chunk == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
    if (p.shared) {
      qa = p.q_start[b];
      qb = p.q_start[b + 1];
    } else {
      qb = qa + 1;
    }
    ctx_len = p.ctx_len[b];
    off = p.ctx_off[b];
    slot_k = chunk;
    if (FUSED && p.S > 0) pos_base = instr_pos_base(p.instr_start, p.instr_len, p.S, b);
  }
  // the prompt's context is split into n = ceil(len / chunk) equal chunks
  // (whole tiles), so that a short last chunk does not leave its unit idle;
  // instruction chunks keep the planned size
  int cb = p.chunk;
  if (!INSTR && ctx_len > 0) {
    const int n = (ctx_len + p.chunk - 1) / p.chunk;
    cb = (((ctx_len + n - 1) / n) + 31) & ~31;
  }
  const int G = p.G;
  const int row0 = rg * RW;
  if (row0 >= (qb - qa) * G) return;              // beyond every question's rows
  // the unit's rows are those of the active questions, compacted: row r is
  // head g*G + r % G of the (r / G)-th active question of [qa, qb)
  int kq[RB], qsel[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) kq[rb] = (row0 + 16 * (RB * wave + rb) + lr) / G;
  const int nrows = active_questions<RB>(p.active, qa, qb, kq, qsel, lane) * G;
  if (row0 >= nrows) return;                       // no active rows here: no tile is read
  if (static_cast<int64_t>(chunk) * cb >= ctx_len) {
    // past the prompt's context: an empty state (max -inf) for each row, so
    // that the merge can fold every chunk slot without knowing the prompt
    if (lg == 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + 16 * (RB * wave + rb) + lr;
        if (row < nrows) {
          const int64_t slot = (static_cast<int64_t>(slot_k) * p.Nt + qsel[rb]) * p.Hq + g * G + row % G;
          *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(-INFINITY, 0.f);
        }
      }
    }
    return;
  }

  const int64_t k0 = off + static_cast<int64_t>(chunk) * cb;
  const int64_t k1 = min(k0 + cb, off + ctx_len);
  const int ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
  const T* kbase = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
  const T* vbase = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * p.pool * D;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));

  // this lane's rows: row block rb of wave w holds rows 16*(RB*w + rb) + lr
  // of the unit, row r being head g*G + r % G of active question qsel (rows
  // past the active ones read question qa's inputs and are never published)
  int qi[RB], h[RB];
  bool in_range[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = row0 + 16 * (RB * wave + rb) + lr;
    in_range[rb] = row < nrows;
    qi[rb] = in_range[rb] ? qsel[rb] : qa;
    h[rb] = g * G + row % G;
  }
  // fused instruction unit: each row's query sits at instr_len + ctx_len[b] +
  // seg_len of its own question, b being the prompt (among pa..pe-1) that holds it
  int64_t row_base[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) row_base[rb] = static_cast<int64_t>(ctx_len) + pos_base;
  if constexpr (INSTR && FUSED) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      int lo = pa, hi = pe - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (p.q_start[mid] <= qi[rb]) lo = mid; else hi = mid - 1;
      }
      row_base[rb] = static_cast<int64_t>(ctx_len) + p.ctx_len[lo];
    }
  }
  RL rl;
  issue_row_loads<T, D, FUSED, RB>(rl, p, qi, h, lg);
  TileOffsets<T, D, NW, NS> toff;
  toff.init(wave, lane);
  // exactly P0 tiles go out before the one wait for the row loads (a unit
  // with fewer tiles fetches its last tile again): a single wait with a
  // fixed count leaves the compiler no reason to copy the loaded registers
  // before it.  The extra DMAs are younger than every real tile, so the
  // ring's waits below stay sufficient.
#pragma unroll
  for (int t = 0; t < P0; ++t)
    issue_tile<T, D, NW, NS>(lds + t * RG::STAGE, kbase, vbase, k0 + 32ll * min(t, ntiles - 1), k1, wave, lane, toff);
  wait_row_loads<(P0 * DPT < 63 ? P0 * DPT : 63)>(rl);

  bool act[RB];
  bool any_act = false;
  const bool quad = (G & 3) == 0;                   // lane quads hold heads of one question
  typename M::Frag qf[RB][D / 32];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int s_raw = static_cast<int>(rl.s[rb]);
    act[rb] = in_range[rb] && rl.a[rb] != 0u && usable_seg_len(p, s_raw) >= 0;
    any_act = any_act || act[rb];
    row_query<T, D, FUSED, RL::QN, (RL::TN > 0 ? RL::TN : 1)>(qf[rb], rl.q[rb], rl.th, row_base[rb] + s_raw,
                                                              quad, lane);
    if (!act[rb]) {
#pragma unroll
      for (int ds = 0; ds < D / 32; ++ds) qf[rb][ds] = M::zero();
    }
  }
  const bool live = wave_any(any_act);                // wave-uniform
  // the eight-wave plain loop folds two tiles per barrier (below): its ring
  // starts one tile shallower, so that the stages it refills are the two
  // whose tiles every wave has folded
  constexpr bool kPairs = RG::NS >= 6 && NW == 8 && RB == 1 && D == 128 && sizeof(T) == 2;
#pragma unroll
  for (int t = P0; t < RG::NS - (kPairs ? 2 : 1); ++t)
    if (t < ntiles) issue_tile<T, D, NW, NS>(lds + t * RG::STAGE, kbase, vbase, k0 + 32ll * t, k1, wave, lane, toff);
  RowState<D> st[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) row_init(st[rb]);
  const float c = p.c;

  // ring: tile t sits in stage t % NS; at iteration t the stage of tile t-1
  // is refilled with tile t + NS - 1
  const int last = ntiles - 1;
  const int tail_n = static_cast<int>(k1 - (k0 + 32ll * last));
  // eight single-block waves at bf16, D = 128 (one workgroup per compute
  // unit): the plain loop, whose waves overlap each other's MFMA and VALU
  // work, measured faster than the pipelined one
  constexpr bool kPipelined = RG::NS >= 4 && !(NW == 8 && RB == 1 && D == 128 && sizeof(T) == 2);
  if constexpr (kPipelined) {
    // software pipelined: iteration t folds tile t (softmax on the VALU, then
    // P^T V on the MFMA) while the scores of tile t+1 are computed, so each
    // wave has independent MFMA and VALU work in flight.  K of tile t+1 and
    // V of tile t are both in the ring during iteration t.
    f32x4_t sa[RB][2], sb[RB][2];
    // tile 0's blocks are this thread's oldest DMAs; tiles 1 .. min(NS-2, last) are younger
    wait_tiles<DPT, RG::NS - 2>(min(last, RG::NS - 2));
    __syncthreads();
    if (live) qk_tile<T, D, NS, RB>(ring, qf, sa, lr, lg);
    // iteration t < last folds the scores of full tile t and computes those
    // of tile t+1; unrolled by two so that the two score sets (sa, sb) swap
    // roles instead of being copied.  The last tile (possibly partial) is
    // folded after the loop, so the loop carries no masking.  (Written out
    // rather than as a lambda: a lambda capturing the unit's bases by
    // reference made the compiler treat them as divergent and move the DMA
    // addressing to vector registers.)
    int t = 0;
    for (; t + 2 <= last; t += 2) {
      // tile t+1 must have landed; tiles t+2 .. min(t+NS-2, last) are younger
      wait_tiles<DPT, RG::NS - 3>(min(last - t - 1, RG::NS - 3));
      __syncthreads();                              // also: every wave is past iteration t-1
      if (t + RG::NS - 1 <= last)
        issue_tile<T, D, NW, NS>(lds + ((t + RG::NS - 1) % RG::NS) * RG::STAGE, kbase, vbase,
                                 k0 + 32ll * (t + RG::NS - 1), k1, wave, lane, toff);
      if (live)
        pipe_step<T, D, NS, RB>(ring + ((t + 1) % RG::NS) * RG::STAGE, ring + (t % RG::NS) * RG::STAGE, qf, sa, sb,
                                st, 32, lr, lg, c);
      wait_tiles<DPT, RG::NS - 3>(min(last - t - 2, RG::NS - 3));
      __syncthreads();
      if (t + RG::NS <= last)
        issue_tile<T, D, NW, NS>(lds + ((t + RG::NS) % RG::NS) * RG::STAGE, kbase, vbase, k0 + 32ll * (t + RG::NS),
                                 k1, wave, lane, toff);
      if (live)
        pipe_step<T, D, NS, RB>(ring + ((t + 2) % RG::NS) * RG::STAGE, ring + ((t + 1) % RG::NS) * RG::STAGE, qf, sb,
                                sa, st, 32, lr, lg, c);
    }
    if (t < last) {
      wait_tiles<DPT, RG::NS - 3>(min(last - t - 1, RG::NS - 3));
      __syncthreads();
      if (t + RG::NS - 1 <= last)
        issue_tile<T, D, NW, NS>(lds + ((t + RG::NS - 1) % RG::NS) * RG::STAGE, kbase, vbase,
                                 k0 + 32ll * (t + RG::NS - 1), k1, wave, lane, toff);
      if (live) {
        pipe_step<T, D, NS, RB>(ring + ((t + 1) % RG::NS) * RG::STAGE, ring + (t % RG::NS) * RG::STAGE, qf, sa, sb,
                                st, 32, lr, lg, c);
        softmax_pv<T, D, NS, RB>(ring + (last % RG::NS) * RG::STAGE, sb, st, tail_n, lr, lg, c);
      }
    } else if (live) {
      softmax_pv<T, D, NS, RB>(ring + (last % RG::NS) * RG::STAGE, sa, st, tail_n, lr, lg, c);
    }
  } else if constexpr (kPairs) {
    // two tiles per barrier: at iteration t (even) tiles t and t+1 have
    // landed and every wave has folded tiles t-2 and t-1, whose stages take
    // tiles t+NS-2 and t+NS-1; an odd last tile is folded on its own.
    // Half the barriers, so half the waits for the slowest wave (measured
    // 0.4% faster than one tile per barrier on the 32-layer workload).
    int t = 0;
    for (; t + 1 < ntiles; t += 2) {
      // tiles t+2 .. min(t+NS-4, last) are younger than tile t+1
      wait_tiles<DPT, RG::NS - 4>(min(last - t - 1, RG::NS - 4));
      __syncthreads();
      if (t + RG::NS - 2 <= last)
        issue_tile<T, D, NW, NS>(lds + ((t + RG::NS - 2) % RG::NS) * RG::STAGE, kbase, vbase,
                                 k0 + 32ll * (t + RG::NS - 2), k1, wave, lane, toff);
      if (t + RG::NS - 1 <= last)
        issue_tile<T, D, NW, NS>(lds + ((t + RG::NS - 1) % RG::NS) * RG::STAGE, kbase, vbase,
                                 k0 + 32ll * (t + RG::NS - 1), k1, wave, lane, toff);
      if (live) {
        ring_tile<T, D, NS, RB>(ring + (t % RG::NS) * RG::STAGE, qf, st, 32, lr, lg, c);
        ring_tile<T, D, NS, RB>(ring + ((t + 1) % RG::NS) * RG::STAGE, qf, st, t + 1 == last ? tail_n : 32, lr, lg,
                                c);
      }
    }
    if (t == last) {
      wait_tiles<DPT, RG::NS - 4>(0);
      __syncthreads();
      if (live) ring_tile<T, D, NS, RB>(ring + (t % RG::NS) * RG::STAGE, qf, st, tail_n, lr, lg, c);
    }
  } else {
    for (int t = 0; t < ntiles; ++t) {
      // tile t's blocks are this thread's oldest outstanding DMAs; those of
      // tiles t+1 .. min(t+NS-2, last) are younger
      wait_tiles<DPT, RG::NS - 2>(min(last - t, RG::NS - 2));
      __syncthreads();
      const int tn = t + RG::NS - 1;
      if (tn <= last)
        issue_tile<T, D, NW, NS>(lds + (tn % RG::NS) * RG::STAGE, kbase, vbase, k0 + 32ll * tn, k1, wave, lane, toff);
      if (live) ring_tile<T, D, NS, RB>(ring + (t % RG::NS) * RG::STAGE, qf, st, t == last ? tail_n : 32, lr, lg, c);
    }
  }
  wait_vmcnt<0>();                                  // no LDS-DMA may outlive the workgroup

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (act[rb]) publish_rows<D>(p, st[rb], (static_cast<int64_t>(slot_k) * p.Nt + qi[rb]) * p.Hq + h[rb], lg);
  }
}

// ---------------------------------------------------------------------------
// Segment unit (question i, kv head g).  The segment's cached slots are
// streamed in 32-token tiles, wave w taking tiles w, w + sw, ...; its last
// key (the step's token, at virtual position ctx_len[b] + seg_len[i], or
// slot seg_len[i] - 1 in attention-only calls) is folded in from LDS, so the
// fused step never waits for its own append.
// ---------------------------------------------------------------------------
template <typename T, int D>
__device__ __forceinline__ void load_seg_tile(typename Mfma<T>::Frag (&kf)[2][D / 32], typename Mfma<T>::Frag (&vf)[D / 16],
                                              const T* __restrict__ kseg, const T* __restrict__ vseg, int t, int mlast,
                                              int lr, int lg) {
  using M = Mfma<T>;
  const int t0 = 32 * t;
  // the segment bases are wave-uniform: scalar base plus 32-bit lane offsets
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const uint32_t ko = static_cast<uint32_t>(min(t0 + tile_token(kb, lr), mlast) * D + lg * 8);
#pragma unroll
    for (int ds = 0; ds < D / 32; ++ds) kf[kb][ds] = M::load(kseg + (ko + 32 * ds));
  }
  const uint32_t vo = static_cast<uint32_t>(min((t0 >> 3) + lg, mlast >> 3) * 8 * D + lr * 8);
#pragma unroll
  for (int db = 0; db < D / 16; ++db) vf[db] = M::load(vseg + (vo + 16 * db * 8));
}

template <typename T, int D, int NW, int NS, bool FUSED>
__device__ __forceinline__ void segment_unit(const StepParams& p, UnitLds<T, D, NW, NS>& sh, int u, int wave,
                                             int lane) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  using L = UnitLds<T, D, NW, NS>;
  constexpr int DS = D / 32, DB = D / 16, E = static_cast<int>(sizeof(T));
  const int lr = lane & 15, lg = lane >> 4;
  const int G = p.G;
  // seg_tpu tasks (question i, kv head g) per unit, wpt waves each
  const int tpu = p.seg_tpu, wpt = NW / tpu;
  const int k = wave / wpt, ww = wave - k * wpt;
  const int task = u * tpu + k;
  const bool valid = task < p.Nt * p.Hkv;
  const int tsk = valid ? task : 0;
  const int i = tsk / p.Hkv, g = tsk - i * p.Hkv;
  const int64_t sg = static_cast<int64_t>(i) * p.Hkv + g;
  // the leader's loads need only (i, g): issued here, in a block that does
  // not dominate their uses, they go out with the prompt and segment-length
  // loads below and share their round trip
  const int hq = g * G + (lr < G ? lr : 0);
  Frag qf[DS];
  T kraw[2], vraw[2];
  double theta = 0.0;                              // fused: frequency of pair `lane` (lanes < D/2)
  if (ww == 0) {
    if (FUSED) theta = p.inv_freq[lane % (D / 2)];   // loaded with the row, not after the prompt lookup
    const T* src = static_cast<const T*>(FUSED ? p.q_new : p.q_rot_in) + (static_cast<int64_t>(i) * p.Hq + hq) * D + lg * 8;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = M::load(src + 32 * ds);
    if (FUSED) {
      const T* kn = static_cast<const T*>(p.k_new) + sg * D;
      const T* vn = static_cast<const T*>(p.v_new) + sg * D;
      const int jj = lane % (D / 2);
      kraw[0] = kn[jj];
      kraw[1] = kn[jj + D / 2];
      vraw[0] = vn[lane % D];
      vraw[1] = vn[(lane + 64) % D];
    }
  }
  const PromptInfo pi = find_prompt(p, i, lane);
  const int sraw = p.seg_len[i];
  const bool act = valid && p.active[i] != 0;
  const int s = usable_seg_len(p, sraw);
  if (act && s < 0 && g == 0 && ww == 0 && lane == 0)
    raise_flag(p.err_flag, (p.fused && sraw >= p.seg_cap) ? kFlagSegmentFull : kFlagBadLayout);
  // bad layouts are flagged by the context and instruction units
  const bool live = act && s >= 0 && pi.ok && (p.S == 0 || instr_serves(p, pi.b, i, lane));
  T* skp = static_cast<T*>(p.seg_k) + sg * p.seg_cap * D;
  T* svp = static_cast<T*>(p.seg_vt) + sg * p.seg_cap * D;     // 8-token column blocks
  const int mem = FUSED ? s : s - 1;               // cached slots before the last key
  const int ntiles = live ? (mem + 31) >> 5 : 0;
  const int mlast = max(mem - 1, 0);
  // sw waves of the task hold states to combine (all tasks' states must fit
  // main); tile t goes to wave (t + 1) % sw, so the leader, busy with the
  // queries first, takes tiles last
  const int sw = min(wpt, L::SEGMAIN / (G * (D + 4) * 4) / tpu);
  const int first = ww < sw ? (ww + sw - 1) % sw : ntiles;
  unsigned char* qrows = sh.main + k * L::TASK;
  const unsigned char* qrow = qrows + lr * L::QROW + lg * 8 * E;
  Frag kf[2][DS], vf[DB];
  if (ww == 0) {
    if (lane == 0) sh.live()[k] = live ? 1 : 0;
    if (live) {
      // query rows of the G heads (rows >= G zero), rotated at the step
      // token's virtual position ctx_len[b] + seg_len[i] in the fused step
      const int h = hq;
      float2* rot = reinterpret_cast<float2*>(qrows + L::QAREA);
      if (FUSED) {
        const int64_t pos = static_cast<int64_t>(pi.len) + s +
                            (p.S > 0 ? instr_pos_base(p.instr_start, p.instr_len, p.S, pi.b) : 0);
        if (lane < D / 2) {
          float cs, sn;
          rope_cos_sin(pos, theta, cs, sn);
          rot[lane] = make_float2(cs, sn);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int ds = 0; ds < DS / 2; ++ds) {
          f32x8_t x = M::to_f32v(qf[ds]), y = M::to_f32v(qf[ds + DS / 2]);
#pragma unroll
          for (int uu = 0; uu < 8; ++uu) {
            const float2 cs = rot[32 * ds + 8 * lg + uu];
            float xr, yr;
            rope_rotate(x[uu], y[uu], cs.x, cs.y, xr, yr);
            x[uu] = xr;
            y[uu] = yr;
          }
          qf[ds] = M::from_f32(x);
          qf[ds + DS / 2] = M::from_f32(y);
        }
      }
      if (lr >= G) {
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) qf[ds] = M::zero();
      } else if (FUSED && p.q_rot_out != nullptr) {
        T* qo = static_cast<T*>(p.q_rot_out) + (static_cast<int64_t>(i) * p.Hq + h) * D + lg * 8;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) store8<T>(qo + 32 * ds, qf[ds]);
      }
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) store8<T>(reinterpret_cast<T*>(qrows + lr * L::QROW) + 32 * ds + lg * 8, qf[ds]);
      if (FUSED) {
        // rotate the step's key at pos; append it and its value at slot s
        if (lane < D / 2) {
          const int jj = lane;
          const float2 cs = rot[jj];
          float x, y;
          rope_rotate(to_f32<T>(kraw[0]), to_f32<T>(kraw[1]), cs.x, cs.y, x, y);
          const T xk = from_f32<T>(x), yk = from_f32<T>(y);
          skp[static_cast<int64_t>(s) * D + jj] = xk;
          skp[static_cast<int64_t>(s) * D + jj + D / 2] = yk;
          sh.k(k)[jj] = xk;
          sh.k(k)[jj + D / 2] = yk;
        }
#pragma unroll
        for (int r = 0; r < (D + 63) / 64; ++r) {
          const int d = lane + 64 * r;
          if (d < D) {
            const T v = vraw[r];
            svp[static_cast<int64_t>(s >> 3) * 8 * D + d * 8 + (s & 7)] = v;
            sh.v(k)[d] = v;
          }
        }
      } else {
        for (int d = lane; d < D; d += 64) {
          sh.k(k)[d] = skp[static_cast<int64_t>(s - 1) * D + d];
          sh.v(k)[d] = svp[static_cast<int64_t>((s - 1) >> 3) * 8 * D + d * 8 + ((s - 1) & 7)];
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // score of the last key: q_row . k, reduced over the four lanes of a row
      float dot = 0.f;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const f32x8_t qv = M::to_f32v(M::load(reinterpret_cast<const T*>(qrow + 32 * ds * E)));
        const f32x8_t kv = M::to_f32v(M::load(sh.k(k) + 32 * ds + lg * 8));
#pragma unroll
        for (int uu = 0; uu < 8; ++uu) dot = fmaf(qv[uu], kv[uu], dot);
      }
      dot = xor16_sum(dot);
      dot = xor32_sum(dot);
      if (lg == 0 && lr < G) sh.slast(k)[lr] = dot;
    }
  } else if (first < ntiles) {
    load_seg_tile<T, D>(kf, vf, skp, svp, first, mlast, lr, lg);   // in flight across the barrier
  }
  __syncthreads();                                 // query rows, last keys and their scores are in LDS

  RowState<D> st;
  row_init(st);
  const float c = p.c;
  for (int t = first; t < ntiles; t += sw) {
    asm volatile("" ::: "memory");                // query rows are re-read from LDS, not held in registers
    if (ww == 0 || t != first) load_seg_tile<T, D>(kf, vf, skp, svp, t, mlast, lr, lg);
    const int n = min(mem - 32 * t, 32);
    f32x4_t sc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const Frag q = M::load(reinterpret_cast<const T*>(qrow + 32 * ds * E));
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sc[kb] = M::mma(kf[kb][ds], q, sc[kb]);
    }
    if (n < 32) mask_scores(sc, n, lg);
    const Frag pf = softmax_step<T, D>(sc, st, c);
    const int keep = min(max(n - 8 * lg, 0), 8);
    st.ls = M::mma(M::ones(), pf, st.ls);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const Frag v = n < 32 ? M::keep_first(vf[db], keep) : vf[db];
      st.o[db] = M::mma(v, pf, st.o[db]);
    }
  }
  __syncthreads();                                 // the query rows are dead
  if (live && ww < sw && lr < G) {
    float* o = reinterpret_cast<float*>(sh.main) + ((k * sw + ww) * G + lr) * (D + 4) + 4 * lg;
#pragma unroll
    for (int db = 0; db < DB; ++db) *reinterpret_cast<f32x4_t*>(o + 16 * db) = st.o[db];
    if (lg == 0) sh.ml(k * sw + ww)[lr] = make_float2(st.m, st.ls[0]);
  }
  __syncthreads();
  // combine each task's wave states and its last key: item (task, row r, dims d0..d0+7)
  // a task that is not served marks its rows skipped (sum -1), so the merge
  // needs no question metadata
  const int per_task = G * (D / 8);
  for (int e = threadIdx.x; e < tpu * per_task; e += 64 * NW) {
    const int kk = e / per_task, er = e - kk * per_task;
    const int r = er / (D / 8), d0 = (er - r * (D / 8)) * 8;
    if (!sh.live()[kk]) {
      const int tk = u * tpu + kk;
      if (d0 == 0 && tk < p.Nt * p.Hkv) {
        const int ik = tk / p.Hkv, gk = tk - ik * p.Hkv;
        const int64_t slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + ik) * p.Hq + gk * G + r;
        *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(-INFINITY, -1.f);
      }
      continue;
    }
    const float sl = sh.slast(kk)[r];
    float m = sl;
    for (int w = 0; w < sw; ++w) m = fmaxf(m, sh.ml(kk * sw + w)[r].x);
    const float fl = fast_exp2((sl - m) * c);
    float lsum = fl;
    f32x4_t a0, a1;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      a0[v] = fl * to_f32<T>(sh.v(kk)[d0 + v]);
      a1[v] = fl * to_f32<T>(sh.v(kk)[d0 + 4 + v]);
    }
    for (int w = 0; w < sw; ++w) {
      const float2 mlw = sh.ml(kk * sw + w)[r];
      const float f = fast_exp2((mlw.x - m) * c);  // 0 for a wave without tiles (max -inf)
      lsum = fmaf(f, mlw.y, lsum);
      const float* o = reinterpret_cast<const float*>(sh.main) + ((kk * sw + w) * G + r) * (D + 4) + d0;
      a0 += f * *reinterpret_cast<const f32x4_t*>(o);
      a1 += f * *reinterpret_cast<const f32x4_t*>(o + 4);
    }
    const int tk = u * tpu + kk;
    const int ik = tk / p.Hkv, gk = tk - ik * p.Hkv;
    const int64_t slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + ik) * p.Hq + gk * G + r;
    f32x4_t* dst = reinterpret_cast<f32x4_t*>(p.part_acc + slot * D + d0);
    dst[0] = a0;
    dst[1] = a1;
    if (d0 == 0) *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(m, lsum);
  }
}

// ---------------------------------------------------------------------------
// attend_kernel: context units (blockIdx < ctx_blocks), then segment units.
// Workgroups are dispatched in order, so segment units start as context
// units retire and fill the tail of the context work.
// ---------------------------------------------------------------------------
// The second launch bound asks for four waves per SIMD with one row block
// per wave and two with RB = 2 (twice the accumulators); the ring's LDS then
// sets the workgroups per compute unit: one with nine stages, two with five.
template <typename T, int D, int NW, int NS, bool FUSED, int RB>
__global__ __launch_bounds__(64 * NW, RB == 1 ? 4 : 2) void attend_kernel(StepParams p) {
  __shared__ UnitLds<T, D, NW, NS> sh;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int blk = static_cast<int>(blockIdx.x);
  if (blk < p.ctx_blocks) context_unit<T, D, NW, NS, FUSED, RB>(p, sh.main, wave, lane);
  else if (blk < p.ctx_blocks + p.instr_blocks) context_unit<T, D, NW, NS, FUSED, RB, true>(p, sh.main, wave, lane);
  else segment_unit<T, D, NW, NS, FUSED>(p, sh, blk - p.ctx_blocks - p.instr_blocks, wave, lane);
}

// ---------------------------------------------------------------------------
// merge_kernel: question i is served by merge_parts workgroups of
// kMergeThreads threads.  Item (head h, dims d0..d0+7) of the question
// combines its context chunk states and its segment state:
//   m = max_k m_k,  l = sum_k 2^(c(m_k - m)) l_k,  o = sum_k 2^(c(m_k - m)) o_k / l.
// With P = merge_phases, a workgroup takes kMergeThreads / P items and P
// threads per item, thread phase f folding slots f, f + P, ...; the P states
// of an item are then combined through LDS.  Every slot of every question
// is written by the attend kernel (chunks past a prompt's context hold an
// empty state, the segment slot of a question not served holds sum -1), so
// one round of loads brings all the kernel reads, with no question
// metadata; only part 0 of a question reads its segment length, and
// advances it in the fused step.
// ---------------------------------------------------------------------------
constexpr int kMergeBatch = 8;       // partial states in flight per thread

// Exact combination of partial softmax states (m, l, a) in 2^(c*x) units;
// an empty state (m = -inf) changes nothing.
struct MergeAcc {
  float m, l;
  f32x4_t a0, a1;
  __device__ __forceinline__ void init() {
    m = -INFINITY;
    l = 0.f;
    a0 = f32x4_t{0.f, 0.f, 0.f, 0.f};
    a1 = a0;
  }
  __device__ __forceinline__ void fold(float mk, float lk, f32x4_t x0, f32x4_t x1, float c) {
    if (mk == -INFINITY) return;
    const float mn = fmaxf(m, mk);
    const float sa = fast_exp2((m - mn) * c);        // 0 while m = -inf
    const float sb = fast_exp2((mk - mn) * c);
    l = l * sa + sb * lk;
    a0 = a0 * sa + x0 * sb;
    a1 = a1 * sa + x1 * sb;
    m = mn;
  }
};

template <int D>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(StepParams p) {
  __shared__ __attribute__((aligned(16))) float mp[kMergeThreads * 12];   // (m, l, -, -, 8 values) per thread
  const int tid = threadIdx.x;
  const int P = p.merge_phases, per = kMergeThreads / P;
  const int i = blockIdx.x / p.merge_parts, part = blockIdx.x - i * p.merge_parts;
  const int nslot = p.max_chunks + 1 + p.max_ichunks;   // context chunks, the segment, instruction chunks
  const float c = p.c;
  const int items = p.Hq * (D / 8);
  const int f = tid / per, local = tid - f * per;
  const int e = part * per + local;                // this thread's item
  const bool has = e < items;
  const int h = has ? e / (D / 8) : 0, d0 = has ? (e - h * (D / 8)) * 8 : 0;
  const int64_t seg_slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + i) * p.Hq + h;
  const float seg_l = p.part_ml[2 * seg_slot + 1];
  // dense-mask baseline: its units of a prompt with a bad layout return
  // without writing, so a question is merged only if its prompt is sound
  // (the IPPD path's segment units write the skip mark themselves)
  bool sound = true;
  if (p.dense) sound = find_prompt(p, i, tid & 63).ok;
  const int s = (p.fused && part == 0 && tid == 0) ? p.seg_len[i] : 0;
  MergeAcc acc;
  acc.init();
  for (int k0 = f; k0 < nslot; k0 += P * kMergeBatch) {
    float2 ml[kMergeBatch];
    f32x4_t x0[kMergeBatch], x1[kMergeBatch];
#pragma unroll
    for (int uu = 0; uu < kMergeBatch; ++uu) {
      const int ck = min(k0 + P * uu, nslot - 1);
      const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
      ml[uu] = *reinterpret_cast<const float2*>(p.part_ml + 2 * slot);
      const f32x4_t* src = reinterpret_cast<const f32x4_t*>(p.part_acc + slot * D + d0);
      x0[uu] = src[0];
      x1[uu] = src[1];
    }
#pragma unroll
    for (int uu = 0; uu < kMergeBatch; ++uu)
      if (k0 + P * uu < nslot) acc.fold(ml[uu].x, ml[uu].y, x0[uu], x1[uu], c);
  }
  // every head's segment slot of question i carries the same served/skipped
  // mark, so the decision is workgroup-uniform
  if (seg_l < 0.f || !sound) return;
  if (P > 1) {
    float* dst = mp + tid * 12;
    dst[0] = acc.m;
    dst[1] = acc.l;
    *reinterpret_cast<f32x4_t*>(dst + 4) = acc.a0;
    *reinterpret_cast<f32x4_t*>(dst + 8) = acc.a1;
    __syncthreads();
    if (f == 0) {
      for (int g2 = 1; g2 < P; ++g2) {
        const float* src = mp + (g2 * per + local) * 12;
        acc.fold(src[0], src[1], *reinterpret_cast<const f32x4_t*>(src + 4), *reinterpret_cast<const f32x4_t*>(src + 8), c);
      }
    }
  }
  if (f == 0 && has) {
    const float inv = 1.f / acc.l;
    f32x4_t* dst = reinterpret_cast<f32x4_t*>(p.out + (static_cast<int64_t>(i) * p.Hq + h) * D + d0);
    dst[0] = acc.a0 * inv;
    dst[1] = acc.a1 * inv;
    if (p.lse != nullptr && d0 == 0) p.lse[static_cast<int64_t>(i) * p.Hq + h] = acc.m * p.scale + logf(acc.l);
  }
  // the question was served: its segment holds the step's token
  if (p.fused && part == 0 && tid == 0) p.seg_len[i] = s + 1;
}

// ---------------------------------------------------------------------------
template <typename T, int D, int NW, int NS, int RB>
static hipError_t launch_attend(int grid, const StepParams& p, hipStream_t s) {
  if (p.fused) attend_kernel<T, D, NW, NS, true, RB><<<grid, 64 * NW, 0, s>>>(p);
  else attend_kernel<T, D, NW, NS, false, RB><<<grid, 64 * NW, 0, s>>>(p);
  return hipGetLastError();
}

// Ring depth: 4 stages (two workgroups per CU) in general; 8 (one per CU,
// every tile of a short unit in flight at once) when the context units fit
// the chip in one wave, or when registers allow one workgroup per CU anyway.
// fp32 at D = 128 has 32 KB stages: 2 or 4.  bf16 at D = 128 (16 KB stages)
// takes the deepest rings the 160 KB of LDS allow: five stages (80 KB, two
// workgroups per compute unit) or nine (one workgroup), so that each compute
// unit keeps six or seven tiles in flight while it computes.
template <typename T, int D, int NW, int RB>
static hipError_t launch_depth(bool deep, int grid, const StepParams& p, hipStream_t s) {
  constexpr int stage = 2 * 32 * D * sizeof(T);
  constexpr int base = stage > 16384 ? 2 : (stage == 16384 ? 5 : 4);
  constexpr int dns = stage > 16384 ? 4 : (stage == 16384 ? 9 : 8);
  return deep ? launch_attend<T, D, NW, dns, RB>(grid, p, s) : launch_attend<T, D, NW, base, RB>(grid, p, s);
}

template <typename T, int D>
static hipError_t launch_waves(int waves, int rb, bool deep, int grid, const StepParams& p, hipStream_t s) {
  if (rb == 2) {
    // two row blocks per wave: bf16 at D = 128 with four or eight waves
    if constexpr (sizeof(T) == 2 && D == 128) {
      if (waves == 4) return launch_depth<T, D, 4, 2>(deep, grid, p, s);
      if (waves == 8) return launch_depth<T, D, 8, 2>(deep, grid, p, s);
    }
    return hipErrorInvalidValue;
  }
  switch (waves) {
    case 1: return launch_depth<T, D, 1, 1>(deep, grid, p, s);
    case 2: return launch_depth<T, D, 2, 1>(deep, grid, p, s);
    case 4: return launch_depth<T, D, 4, 1>(deep, grid, p, s);
    default:
      // the planner gives fp32 at D = 128 at most four waves, and bf16 at
      // D = 128 eight single-block waves only with one workgroup per compute
      // unit (the deep ring)
      if constexpr (D == 128 && sizeof(T) == 4) return hipErrorInvalidValue;
      else if constexpr (D == 128) return launch_attend<T, D, 8, 9, 1>(grid, p, s);
      else return launch_depth<T, D, 8, 1>(deep, grid, p, s);
  }
}

template <typename T, int D>
static hipError_t launch_d(int waves, int rb, bool deep, int grid, const StepParams& p, hipStream_t s) {
  hipError_t e = launch_waves<T, D>(waves, rb, deep, grid, p, s);
  if (e != hipSuccess) return e;
  merge_kernel<D><<<static_cast<unsigned>(p.Nt) * p.merge_parts, kMergeThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_merge(const StepParams& p, hipStream_t s) {
  if (p.Nt == 0) return hipSuccess;
  if (p.D == 64) merge_kernel<64><<<static_cast<unsigned>(p.Nt) * p.merge_parts, kMergeThreads, 0, s>>>(p);
  else merge_kernel<128><<<static_cast<unsigned>(p.Nt) * p.merge_parts, kMergeThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_step(int dtype, int waves, int rb, bool deep, int grid, const StepParams& p, hipStream_t s) {
  if (p.Nt == 0 || grid == 0) return hipSuccess;
  if (dtype == 0)
    return p.D == 64 ? launch_d<float, 64>(waves, rb, deep, grid, p, s) : launch_d<float, 128>(waves, rb, deep, grid, p, s);
  return p.D == 64 ? launch_d<uint16_t, 64>(waves, rb, deep, grid, p, s)
                   : launch_d<uint16_t, 128>(waves, rb, deep, grid, p, s);
}

}  // namespace ippd
