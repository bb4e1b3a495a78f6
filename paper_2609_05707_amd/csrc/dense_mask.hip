// Dense-mask baseline of the decode-step attention on gfx950.
//
// The paper's own scheme attends the new-token rows of a stacked prompt over
// ALL of its keys and removes the keys a row may not see with the additive
// mask M_fin (Sec. 4.1; Sec. 4.2 attn_IPPD).  This kernel computes the same
// result that way, so that its cost can be set against the block-diagonal
// kernels of decode_step.hip:
//   context-chunk units  (prompt b, kv head g, chunk, row group): rows = every
//                        question of b x the G heads of g, keys = one context
//                        chunk (every row sees all of them), as the split-K
//                        context units of the IPPD path;
//   dense segment units  (prompt b, kv head g, segment chunk, row group): the
//                        same rows, keys = one chunk of the segments of ALL
//                        questions of b, concatenated in question order (in
//                        32-token tiles, kDenseSegTiles tiles per chunk);
//                        a segment tile is visible only to its own question's
//                        rows, so the unit forms and discards the
//                        cross-question scores that the per-question segment
//                        units never compute.
// Both write the partial states that merge_kernel folds: context chunk slots,
// the segment slot (segment chunk 0, also the skip mark of a question not
// served) and, for segment chunks 1.., the slots after it; so the launch is
// followed by the IPPD merge.  Rows load their
// rotated queries with ordinary loads consumed before the first tile DMA (no
// loads in flight across the ring's counted waits).  A prompt holds at most
// 64 questions: lane l of every wave keeps the length of question l.
#include <float.h>
#include <stddef.h>

#include "ippd.h"
#include "ippd_device.h"
#include "ippd_internal.h"
#include "tile_attend.h"

namespace ippd {

// First question at or after j with keys (lane l of len_v holds question l's length).
__device__ __forceinline__ int dense_next_question(int len_v, int nq, int j) {
  while (j < nq && __builtin_amdgcn_readlane(len_v, j) == 0) ++j;
  return j;
}

// Next tile (j, tt) of the segment sequence: tile tt of question j.
__device__ __forceinline__ void dense_advance(int len_v, int nq, int& j, int& tt) {
  if (++tt >= ((__builtin_amdgcn_readlane(len_v, j) + 31) >> 5)) {
    tt = 0;
    j = dense_next_question(len_v, nq, j + 1);
  }
}

template <typename T, int D, int NW, int NS, int RB>
__global__ __launch_bounds__(64 * NW) void dense_kernel(StepParams p) {
  using RG = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int RW = 16 * RB * NW, DS = D / 32, DPT = RG::BLOCKS / NW;
  static_assert(RG::NS >= 4, "the pipelined loop needs at least four stages");
  __shared__ __attribute__((aligned(16))) unsigned char ring[RG::NS * RG::STAGE];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const int blk = static_cast<int>(blockIdx.x);
  const int nctx = p.n_groups * p.max_chunks * p.nrg;
  const int nseg = p.max_ichunks + 1;             // segment chunks per group
  const bool seg = blk >= nctx;
  int grp, chunk, rg;                             // chunk: context chunk, or segment chunk
  {
    const int u = seg ? blk - nctx : blk;
    const int nch = seg ? nseg : p.max_chunks;
    const int cg = u / p.nrg;
    rg = u - cg * p.nrg;
    grp = cg / nch;
    chunk = cg - grp * nch;
  }
  if (grp >= p.n_groups) return;
  const int g = grp / p.B, b = grp - g * p.B;
  const int qa = p.q_start[b], qb = p.q_start[b + 1];
  const int64_t off = p.ctx_off[b];
  const int ctx_len = p.ctx_len[b];
  if (qa < 0 || qb < qa || qb > p.Nt || qb - qa > 64 || off < 0 || (off & 7) != 0 || ctx_len < 0 ||
      ctx_len > p.max_ctx_len || off + ctx_len > p.pool) {
    if (threadIdx.x == 0 && !seg && chunk == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  const int nq = qb - qa, G = p.G, nrows = nq * G, row0 = rg * RW;
  if (row0 >= nrows) return;
  if (!seg && static_cast<int64_t>(chunk) * p.chunk >= ctx_len) {
    // past the prompt's context: an empty state for every row
    if (lg == 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = row0 + 16 * (RB * wave + rb) + lr;
        if (row < nrows) {
          const int64_t slot = (static_cast<int64_t>(chunk) * p.Nt + qa + row / G) * p.Hq + g * G + row % G;
          *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(-INFINITY, 0.f);
        }
      }
    }
    return;
  }

  // rows: question qa + r / G, head g*G + r % G; lengths of the step (the appended token included)
  int len_v = lane < nq ? p.seg_len[qa + lane] : 0;
  len_v = len_v < 0 ? 0 : (len_v > p.seg_cap ? p.seg_cap : len_v);
  int qi[RB], h[RB];
  bool act[RB];
  typename M::Frag qf[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = row0 + 16 * (RB * wave + rb) + lr;
    const bool in_range = row < nrows;
    const int rr = in_range ? row : nrows - 1;
    qi[rb] = qa + rr / G;
    h[rb] = g * G + rr % G;
    const int s = p.seg_len[qi[rb]];
    act[rb] = in_range && p.active[qi[rb]] != 0 && s >= 1 && s <= p.seg_cap;
    const T* src = static_cast<const T*>(p.q_rot_in) + (static_cast<int64_t>(qi[rb]) * p.Hq + h[rb]) * D + 8 * lg;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = M::load(src + 32 * ds);
    if (seg && chunk == 0 && in_range && !act[rb] && lg == 0) {   // not served: the merge skips the question
      const int64_t slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + qi[rb]) * p.Hq + h[rb];
      *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(-INFINITY, -1.f);
    }
  }
  bool any = false;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) any = any || act[rb];
  if (!__syncthreads_or(any)) return;

  // key tiles: one context chunk, or one chunk of the concatenated segment tiles
  const int64_t k0 = off + static_cast<int64_t>(chunk) * p.chunk;
  const int64_t k1 = min(k0 + p.chunk, off + static_cast<int64_t>(ctx_len));
  int ntiles, j0 = 0, tt0 = 0;
  if (!seg) {
    ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
  } else {
    // tiles per question (lane l: question l), their inclusive prefix over the lanes
    const int nt_v = (len_v + 31) >> 5;
    int incl = nt_v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(incl, d, 64);
      incl += lane >= d ? y : 0;
    }
    const int total = __builtin_amdgcn_readlane(incl, 63);
    const int tpc = kDenseSegTiles;
    const int first = chunk * tpc;
    ntiles = max(0, min(first + tpc, total) - first);
    // the chunk starts in question j0 (the first whose tiles reach past `first`), tile tt0 of it
    j0 = __popcll(__ballot(lane < nq && incl <= first));
    tt0 = j0 < nq ? first - (__builtin_amdgcn_readlane(incl, j0) - __builtin_amdgcn_readlane(nt_v, j0)) : 0;
  }
  ntiles = __builtin_amdgcn_readfirstlane(ntiles);
  const int slot_k = !seg ? chunk : (chunk == 0 ? p.max_chunks : p.max_chunks + chunk);
  if (ntiles == 0) {
    // a segment chunk past the prompt's tiles: an empty state for every served row
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (act[rb] && lg == 0) {
        const int64_t slot = (static_cast<int64_t>(slot_k) * p.Nt + qi[rb]) * p.Hq + h[rb];
        *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(-INFINITY, 0.f);
      }
    }
    return;
  }
  const T* kctx = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
  const T* vctx = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * p.pool * D;
  const T* kseg = static_cast<const T*>(p.seg_k) + (static_cast<int64_t>(qa) * p.Hkv + g) * p.seg_cap * D;
  const T* vseg = static_cast<const T*>(p.seg_vt) + (static_cast<int64_t>(qa) * p.Hkv + g) * p.seg_cap * D;
  const int64_t qstride = static_cast<int64_t>(p.Hkv) * p.seg_cap * D;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));
  TileOffsets<T, D, NW, NS> toff;
  toff.init(wave, lane);

  wait_vmcnt<0>();                                // only tile DMAs are counted from here
  int ti_idx = 0, ji = j0, ti = tt0;              // issue cursor
  const int last = ntiles - 1;
#pragma unroll
  for (int st = 0; st < RG::NS - 1; ++st) {
    if (st <= last) {
      if (!seg) {
        issue_tile<T, D, NW, NS>(lds + st * RG::STAGE, kctx, vctx, k0 + 32ll * ti_idx, k1, wave, lane, toff);
        ++ti_idx;
      } else {
        issue_tile<T, D, NW, NS>(lds + st * RG::STAGE, kseg + ji * qstride, vseg + ji * qstride, 32ll * ti,
                                 __builtin_amdgcn_readlane(len_v, ji), wave, lane, toff);
        dense_advance(len_v, nq, ji, ti);
      }
    }
  }
  RowState<D> rs[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) row_init(rs[rb]);
  const float c = p.c;
  f32x4_t sc[RB][2], sn[RB][2];
  wait_tiles<DPT, RG::NS - 2>(min(last, RG::NS - 2));
  __syncthreads();
  qk_tile<T, D, NS, RB>(ring, qf, sc, lr, lg);
  int jc = j0, tc = tt0;                          // compute cursor (segment units)
  for (int t = 0; t < ntiles; ++t) {
    if (t < last) {
      wait_tiles<DPT, RG::NS - 3>(min(last - t - 1, RG::NS - 3));
      __syncthreads();                            // also: every wave is past iteration t-1
      if (t + RG::NS - 1 <= last) {
        const uint32_t stage = lds + ((t + RG::NS - 1) % RG::NS) * RG::STAGE;
        if (!seg) {
          issue_tile<T, D, NW, NS>(stage, kctx, vctx, k0 + 32ll * ti_idx, k1, wave, lane, toff);
          ++ti_idx;
        } else {
          issue_tile<T, D, NW, NS>(stage, kseg + ji * qstride, vseg + ji * qstride, 32ll * ti,
                                   __builtin_amdgcn_readlane(len_v, ji), wave, lane, toff);
          dense_advance(len_v, nq, ji, ti);
        }
      }
    }
    // tile t: valid tokens, and the rows that may see them
    int n, l[RB];
    if (!seg) {
      n = static_cast<int>(min(static_cast<int64_t>(32), k1 - (k0 + 32ll * t)));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) l[rb] = n - 1;
    } else {
      n = min(32, __builtin_amdgcn_readlane(len_v, jc) - 32 * tc);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) l[rb] = (act[rb] && qi[rb] == qa + jc) ? n - 1 : -1;
    }
    bool need = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) need = need || l[rb] < 31;
    need = wave_any(need);
    // the decode loop's wave priority, as the IPPD and standard steps have it
    pipe_step_masked<T, D, NS, RB, true>(ring + ((t + 1) % RG::NS) * RG::STAGE, ring + (t % RG::NS) * RG::STAGE, qf,
                                         sc, sn, rs, n, lr, lg, c, [&](f32x4_t (&x)[2], int rb) {
                                           if (need) mask_after(x, l[rb], lg);
                                         });
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      sc[rb][0] = sn[rb][0];
      sc[rb][1] = sn[rb][1];
    }
    if (seg) dense_advance(len_v, nq, jc, tc);
  }
  wait_vmcnt<0>();                                // no LDS-DMA may outlive the workgroup

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (!act[rb]) continue;
    const int64_t slot = (static_cast<int64_t>(slot_k) * p.Nt + qi[rb]) * p.Hq + h[rb];
    float* dst = p.part_acc + slot * D + 4 * lg;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) *reinterpret_cast<f32x4_t*>(dst + 16 * db) = rs[rb].o[db];
    if (lg == 0) *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(rs[rb].m, rs[rb].ls[0]);
  }
}

template <typename T, int D>
static hipError_t launch_dense_d(int waves, int rb, int grid, const StepParams& p, hipStream_t s) {
  constexpr int NS = 4;
  if (rb == 2) {
    if constexpr (sizeof(T) == 2 && D == 128) {
      if (waves == 4) dense_kernel<T, D, 4, NS, 2><<<grid, 256, 0, s>>>(p);
      else if (waves == 8) dense_kernel<T, D, 8, NS, 2><<<grid, 512, 0, s>>>(p);
      else return hipErrorInvalidValue;
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  switch (waves) {
    case 1: dense_kernel<T, D, 1, NS, 1><<<grid, 64, 0, s>>>(p); break;
    case 2: dense_kernel<T, D, 2, NS, 1><<<grid, 128, 0, s>>>(p); break;
    case 4: dense_kernel<T, D, 4, NS, 1><<<grid, 256, 0, s>>>(p); break;
    default:
      if constexpr (D == 128) return hipErrorInvalidValue;
      else dense_kernel<T, D, 8, NS, 1><<<grid, 512, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_dense(int dtype, int waves, int rb, int grid, const StepParams& p, hipStream_t s) {
  if (p.Nt == 0 || grid == 0) return hipSuccess;
  hipError_t e;
  if (dtype == IPPD_DTYPE_F32)
    e = p.D == 64 ? launch_dense_d<float, 64>(waves, rb, grid, p, s) : launch_dense_d<float, 128>(waves, rb, grid, p, s);
  else
    e = p.D == 64 ? launch_dense_d<uint16_t, 64>(waves, rb, grid, p, s)
                  : launch_dense_d<uint16_t, 128>(waves, rb, grid, p, s);
  if (e != hipSuccess) return e;
  return launch_merge(p, s);
}

}  // namespace ippd
