// IPPD stacked-prompt prefill attention on gfx950 (one launch per call).
//
// The prefill is the forward pass over the prompt header before any answer
// token exists (Sec. 4.1): every header token is a query row.  With the mask
// M_fin of the stacked prompt, a context token attends causally to its own
// context, and a question token attends to the whole context of its prompt
// and causally to its own question (M_ctx, M_qtn, M_caus with >=); every
// question's tokens start at the same virtual position, right after the
// context.  The IPPD form of this computation serves the rows of all
// questions of a prompt from one pass over the context (the shared keys and
// values come from memory once for the whole question set, Sec. 4.3, and
// App. A.2 for the prefill dimensions), and computes the context rows once.
// The standard baseline prefills every question's own prompt
// [context; question] (Sec. 3), so it streams the context and recomputes the
// context rows once per question.
//
// A group is (prompt b, kv head g) for IPPD or (question i, kv head g) for
// the baseline.  A unit serves tb query tokens x G heads (16 * RB * NW rows,
// row r = token r / G, head g*G + r % G) and streams 32-token key/value
// tiles through the LDS ring of the decode kernels (tile_attend.h), with the
// same MFMA products and online softmax; a per-row limit hides the keys a
// row may not see.  Every unit sees all keys of its rows, so it writes
// normalised outputs directly: no split-K, no workspace.
//   question-row units  tokens k*tb .. of the group's questions (packed in
//                       question order): the whole context unmasked, then the
//                       tiles of each question present, visible to that
//                       question's rows up to their own token (causal);
//   context-row units   context tokens k*tb .. (k+1)*tb - 1: context tiles
//                       up to the block's last token, causal on the diagonal.
//   instruction-row units (two-level batch, Sec. 4.4) instruction tokens
//                       k*tb .., causal over the instruction alone.
// In a two-level batch every prompt behind instruction p is [p; c_b; x_i]:
// question-row and context-row units first stream p's tiles, all visible,
// and the positions of c_b and x_i move up by |p|.  IPPD computes p's rows
// once per instruction; the baseline recomputes them (and the context rows)
// once per question.
// Question-row units come first in the grid (each streams a whole context),
// then context-row and instruction-row units, longest causal block first.  Unit u of either kind
// runs on XCD u & 7, which holds every unit of the groups 8j + (u & 7): the
// units of a group share its tiles through that XCD's L2.  Groups are
// numbered kv head minor, so each XCD gets its share of every prompt.
#include <float.h>
#include <stddef.h>

#include "ippd.h"
#include "ippd_device.h"
#include "ippd_internal.h"
#include "tile_attend.h"

namespace ippd {

template <typename T, int D, int NS>
struct PrefillLds {
  alignas(16) unsigned char ring[NS * Ring<T, D, NS>::STAGE];
  int pre[kMaxQuestionsPerPrompt + 1];   // question-row units: prefix sums of the group's question lengths
};

// Index j with pre[j] <= tau < pre[j + 1] (pre non-decreasing, pre[0] = 0 <= tau < pre[n]).
__device__ __forceinline__ int find_question(const int* pre, int n, int tau) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= tau) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Key tile of a unit: instruction tiles 0..npt-1 (two-level batch), context
// tiles npt..npt+nct-1, then the tiles of questions jlo..jhi (relative to the
// group's first question) in order.
struct TilePos {
  int idx;    // tile index in the unit's sequence
  int j;      // question of a segment tile (relative), or -1 for an instruction or context tile
  int tt;     // tile index within that question's tokens
};

template <typename T, int D, int NW, int NS, int RB>
__device__ __forceinline__ void prefill_unit(const PrefillParams& p, PrefillLds<T, D, NS>& sh, int wave, int lane) {
  using RG = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int DS = D / 32, DPT = RG::BLOCKS / NW;
  static_assert(RG::NS >= 4, "the pipelined loop needs at least four stages");
  const int lr = lane & 15, lg = lane >> 4;
  const int blk = static_cast<int>(blockIdx.x);
  const bool qunit = blk < p.q_blocks;
  const int ub = qunit ? blk : blk - p.q_blocks;
  const int slice = ub & 7, local = ub >> 3;
  const int gps = qunit ? p.gps : p.gps_c;
  const int kk = local / gps, grp = 8 * (local - kk * gps) + slice;
  if (grp >= (qunit ? p.n_groups : p.n_cgroups)) return;
  const int k = qunit ? kk : p.kc - 1 - kk;
  const int G = p.G, TB = p.tb;
  // context-row groups past n_groups hold the rows of an instruction
  const bool irows = grp >= p.n_groups;
  const int gl = irows ? grp - p.n_groups : grp;

  int b, g, qa, nq, s = 0;
  // kv head minor: the XCD slice (group % 8) cycles over kv heads, which
  // carry equal work, rather than over prompts of different lengths
  if (irows && p.shared) {
    s = gl / p.Hkv;
    g = gl - s * p.Hkv;
    b = 0;
    qa = 0;
    nq = 0;
  } else if (p.shared) {
    b = gl / p.Hkv;
    g = gl - b * p.Hkv;
    qa = p.q_start[b];
    nq = p.q_start[b + 1] - qa;
  } else {
    qa = gl / p.Hkv;
    g = gl - qa * p.Hkv;
    nq = 1;
    b = prompt_of(p.q_start, p.B, qa);
  }
  if (b >= p.B || qa < 0 || nq < 0 || nq > kMaxQuestionsPerPrompt || qa + nq > p.Nt || (irows && s >= p.S)) {
    if (threadIdx.x == 0 && k == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  if (p.S > 0 && !(irows && p.shared)) s = instr_of_prompt(p.instr_start, p.S, b);
  // this unit's rows: tokens coff .. coff+lc-1, after lp visible prefix tokens at poff
  int64_t coff, poff = 0;
  int lc, lp = 0;
  if (p.S > 0) {
    poff = p.instr_off[s];
    lp = p.instr_len[s];
    if (lp < 0 || lp > p.max_instr_len || (poff & 7) != 0 || poff < 0 || poff + lp > p.pool) {
      if (threadIdx.x == 0 && k == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
  }
  if (irows) {
    coff = poff;
    lc = lp;
    poff = 0;
    lp = 0;
  } else {
    coff = p.ctx_off[b];
    lc = p.ctx_len[b];
    if (lc < 0 || lc > p.max_ctx_len || (coff & 7) != 0 || coff < 0 || coff + lc > p.pool) {
      if (threadIdx.x == 0 && k == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
  }

  // question-row units: prefix sums of the group's question lengths
  int S = 0;                                      // question tokens of the group
  if (qunit) {
    for (int e = threadIdx.x; e < nq; e += 64 * NW) {
      int s = p.seg_len[qa + e];
      if (s < 0 || s > p.seg_cap) {
        raise_flag(p.err_flag, kFlagBadLayout);
        s = s < 0 ? 0 : p.seg_cap;
      }
      sh.pre[e + 1] = s;
    }
    if (threadIdx.x == 0) sh.pre[0] = 0;
    __syncthreads();
    if (wave == 0) {
      // lane l sums entries l*per+1 .. (l+1)*per, then an exclusive scan of the lane sums
      const int per = (nq + 63) / 64;
      int run = 0;
      for (int e = 0; e < per; ++e) {
        const int x = lane * per + e;
        run += x < nq ? sh.pre[x + 1] : 0;
      }
      int incl = run;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(incl, d, 64);
        incl += lane >= d ? y : 0;
      }
      int acc = incl - run;
      for (int e = 0; e < per; ++e) {
        const int x = lane * per + e;
        if (x < nq) {
          acc += sh.pre[x + 1];
          sh.pre[x + 1] = acc;
        }
      }
    }
    __syncthreads();
    S = sh.pre[nq];
    if (k == 0 && threadIdx.x == 0 && S > p.kq * TB) raise_flag(p.err_flag, kFlagBadLayout);
    if (k * TB >= S) return;                      // uniform: every thread read the same total
  } else if (k * TB >= lc) {
    return;
  }

  // this lane's rows: row block rb of wave w holds rows 16*(RB*w + rb) + lr
  const T* qsrc[RB];
  float* dst[RB];
  bool valid[RB];
  int lim[RB];                                    // ctx unit: causal limit (context token); q unit: own token
  int rj[RB];                                     // q unit: question of the row (relative)
  int64_t pos[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = 16 * (RB * wave + rb) + lr;
    const int tr = row / G, h = g * G + row % G;
    if (qunit) {
      const int tau = k * TB + tr;
      valid[rb] = row < TB * G && tau < S;
      const int tc = valid[rb] ? tau : k * TB;
      const int j = nq == 1 ? 0 : find_question(sh.pre, nq, tc);
      const int u = tc - sh.pre[j];
      rj[rb] = j;
      lim[rb] = u;
      pos[rb] = static_cast<int64_t>(lp) + lc + u;
      const int64_t r = (static_cast<int64_t>(qa + j) * p.seg_cap + u) * p.Hq + h;
      qsrc[rb] = static_cast<const T*>(p.q_seg) + r * D;
      dst[rb] = p.out_seg + r * D;
    } else {
      const int t = k * TB + tr;
      valid[rb] = row < TB * G && t < lc;
      const int tc = valid[rb] ? t : k * TB;
      rj[rb] = -1;
      lim[rb] = tc;
      pos[rb] = static_cast<int64_t>(lp) + tc;
      const int64_t r = (coff + tc) * p.Hq + h;
      qsrc[rb] = static_cast<const T*>(p.q_ctx) + r * D;
      dst[rb] = p.out_ctx + r * D;
    }
  }

  // queries, rotated at their (virtual) positions
  typename M::Frag qf[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = M::load(qsrc[rb] + 32 * ds + 8 * lg);
#pragma unroll
    for (int ds = 0; ds < DS / 2; ++ds) {
      f32x8_t x = M::to_f32v(qf[rb][ds]), y = M::to_f32v(qf[rb][ds + DS / 2]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float cs, sn, xr, yr;
        rope_cos_sin(pos[rb], p.inv_freq[32 * ds + 8 * lg + e], cs, sn);
        rope_rotate(x[e], y[e], cs, sn, xr, yr);
        x[e] = xr;
        y[e] = yr;
      }
      qf[rb][ds] = M::from_f32(x);
      qf[rb][ds + DS / 2] = M::from_f32(y);
    }
  }

  // key range: instruction tiles, context tiles, then (question-row units) the questions present
  const int kv_end = qunit ? lc : min(k * TB + TB, lc);
  const int npt = (lp + 31) >> 5, nct = (kv_end + 31) >> 5, npc = npt + nct;
  int jlo = 0, jhi = -1, nst = 0;
  if (qunit) {
    jlo = nq == 1 ? 0 : find_question(sh.pre, nq, k * TB);
    jhi = nq == 1 ? 0 : find_question(sh.pre, nq, min(k * TB + TB, S) - 1);
    for (int j = jlo; j <= jhi; ++j) nst += (sh.pre[j + 1] - sh.pre[j] + 31) >> 5;
  }
  const int ntiles = __builtin_amdgcn_readfirstlane(npc + nst);
  const int64_t kvoff = static_cast<int64_t>(g) * p.pool * D;
  const T* kctx = static_cast<const T*>(p.ctx_k) + kvoff;
  const T* vctx = static_cast<const T*>(p.ctx_vt) + kvoff;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sh.ring));
  TileOffsets<T, D, NW, NS> toff;
  toff.init(wave, lane);

  auto seg_len_of = [&](int j) { return __builtin_amdgcn_readfirstlane(sh.pre[j + 1] - sh.pre[j]); };
  auto next = [&](TilePos tp) {
    ++tp.idx;
    if (tp.j < 0) {
      if (tp.idx < npc) return tp;
      tp.j = jlo - 1;
      tp.tt = 0;
    } else if (++tp.tt < ((seg_len_of(tp.j) + 31) >> 5)) {
      return tp;
    }
    // first tile of the next question that has tokens
    do {
      ++tp.j;
      tp.tt = 0;
    } while (tp.j < jhi && seg_len_of(tp.j) == 0);
    return tp;
  };
  auto issue = [&](const TilePos& tp, uint32_t stage) {
    if (tp.j < 0 && tp.idx < npt) {
      issue_tile<T, D, NW, NS>(stage, kctx, vctx, poff + 32ll * tp.idx, poff + lp, wave, lane, toff);
    } else if (tp.j < 0) {
      issue_tile<T, D, NW, NS>(stage, kctx, vctx, coff + 32ll * (tp.idx - npt), coff + kv_end, wave, lane, toff);
    } else {
      const int64_t so = (static_cast<int64_t>(qa + tp.j) * p.Hkv + g) * p.seg_cap * D;
      issue_tile<T, D, NW, NS>(stage, static_cast<const T*>(p.seg_k) + so, static_cast<const T*>(p.seg_vt) + so,
                               32ll * tp.tt, seg_len_of(tp.j), wave, lane, toff);
    }
  };

  // without instruction or context tiles the sequence starts at question jlo, which has tokens
  const TilePos first{0, npc > 0 ? -1 : jlo, 0};
  // every compiler-issued load has been consumed; from here the only vector
  // memory operations in flight are this wave's tile DMAs, which the waits count
  wait_vmcnt<0>();
  TilePos ti = first;
  const int last = ntiles - 1;
#pragma unroll
  for (int s = 0; s < RG::NS - 1; ++s) {
    if (s <= last) {
      issue(ti, lds + s * RG::STAGE);
      ti = next(ti);
    }
  }

  RowState<D> st[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) row_init(st[rb]);
  const float c = p.c;
  f32x4_t sc[RB][2], sn[RB][2];
  wait_tiles<DPT, RG::NS - 2>(min(last, RG::NS - 2));
  __syncthreads();
  qk_tile<T, D, NS, RB>(sh.ring, qf, sc, lr, lg);
  TilePos tc = first;
  for (int t = 0; t < ntiles; ++t) {
    if (t < last) {
      wait_tiles<DPT, RG::NS - 3>(min(last - t - 1, RG::NS - 3));
      __syncthreads();                            // also: every wave is past iteration t-1
      if (t + RG::NS - 1 <= last) {
        issue(ti, lds + ((t + RG::NS - 1) % RG::NS) * RG::STAGE);
        ti = next(ti);
      }
    }
    // tile t: valid tokens and each row's visible limit (relative to the tile start)
    int n, l[RB];
    if (tc.j < 0 && tc.idx < npt) {
      n = min(32, lp - 32 * tc.idx);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) l[rb] = n - 1;
    } else if (tc.j < 0) {
      const int ci = tc.idx - npt;
      n = min(32, kv_end - 32 * ci);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) l[rb] = qunit ? n - 1 : min(lim[rb] - 32 * ci, n - 1);
    } else {
      n = min(32, seg_len_of(tc.j) - 32 * tc.tt);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) l[rb] = rj[rb] == tc.j ? min(lim[rb] - 32 * tc.tt, n - 1) : -1;
    }
    bool need = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) need = need || l[rb] < 31;
    need = wave_any(need);
    pipe_step_masked<T, D, NS, RB>(sh.ring + ((t + 1) % RG::NS) * RG::STAGE, sh.ring + (t % RG::NS) * RG::STAGE,
                                   qf, sc, sn, st, n, lr, lg, c, [&](f32x4_t (&s)[2], int rb) {
                                     if (need) mask_after(s, l[rb], lg);
                                   });
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      sc[rb][0] = sn[rb][0];
      sc[rb][1] = sn[rb][1];
    }
    tc = next(tc);
  }
  wait_vmcnt<0>();                                // no LDS-DMA may outlive the workgroup

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (!valid[rb]) continue;
    const float inv = 1.f / st[rb].ls[0];
    float* o = dst[rb] + 4 * lg;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) *reinterpret_cast<f32x4_t*>(o + 16 * db) = st[rb].o[db] * inv;
  }
}

template <typename T, int D, int NW, int NS, int RB>
__global__ __launch_bounds__(64 * NW, NW >= 8 ? 2 : 1) void prefill_kernel(PrefillParams p) {
  __shared__ PrefillLds<T, D, NS> sh;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  prefill_unit<T, D, NW, NS, RB>(p, sh, wave, lane);
}

// Variants: bf16 at D = 128 puts two 16-row blocks on each of eight waves
// (256 rows, every K/V fragment read from LDS serves both), or one (128
// rows) when the planner finds too few 256-row units to fill the chip; the
// others use one block per wave.  fp32 at D = 128 has 32 KB stages: four of
// them.
bool prefill_variant(int dtype, int head_dim, int* waves, int* rb) {
  const bool bf = dtype == IPPD_DTYPE_BF16;
  if (head_dim != 64 && head_dim != 128) return false;
  *waves = (!bf && head_dim == 128) ? 4 : 8;
  *rb = (bf && head_dim == 128) ? 2 : 1;
  return true;
}

hipError_t launch_prefill(int dtype, int head_dim, int rb, int grid, const PrefillParams& p, hipStream_t s) {
  const bool bf = dtype == IPPD_DTYPE_BF16;
  if (bf && head_dim == 128 && rb == 2) prefill_kernel<uint16_t, 128, 8, 8, 2><<<grid, 512, 0, s>>>(p);
  else if (bf && head_dim == 128) prefill_kernel<uint16_t, 128, 8, 8, 1><<<grid, 512, 0, s>>>(p);
  else if (bf && head_dim == 64) prefill_kernel<uint16_t, 64, 8, 8, 1><<<grid, 512, 0, s>>>(p);
  else if (!bf && head_dim == 128) prefill_kernel<float, 128, 4, 4, 1><<<grid, 256, 0, s>>>(p);
  else if (!bf && head_dim == 64) prefill_kernel<float, 64, 8, 8, 1><<<grid, 512, 0, s>>>(p);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace ippd
