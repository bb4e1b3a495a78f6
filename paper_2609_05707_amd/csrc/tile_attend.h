// Building blocks of the attention tile loop shared by the decode-step and
// prefill kernels on gfx950: MFMA operand traits, the LDS tile ring filled by
// LDS-DMA, the online-softmax row state and the per-tile products
//   S^T (keys x rows) = K Q^T       v_mfma_f32_16x16x32_bf16, A = 16 keys x 32 dims
//   P^T = exp2(c * (S^T - m))       online softmax in exp2 units
//   O^T (dims x rows) += V^T P^T    A = V^T (the value cache is transposed),
//                                   B = P^T taken straight from the S^T registers
// Key rows are assigned to MFMA rows so that lane row r of S^T holds 8
// consecutive tokens, exactly the B layout the PV product needs.
#pragma once

#include <float.h>
#include <stddef.h>

#include "ippd_device.h"

namespace ippd {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kRescaleLog2 = 8.f;   // lazy-rescale threshold of the online softmax

// ---------------------------------------------------------------------------
// MFMA operand traits: 8 contraction elements per lane per 32-wide step.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<uint16_t> {   // bf16: one v_mfma_f32_16x16x32_bf16 per step
  typedef bf16x8_t Frag;
  static __device__ __forceinline__ Frag load(const uint16_t* p) {
    return __builtin_bit_cast(Frag, *reinterpret_cast<const u32x4_t*>(p));
  }
  static __device__ __forceinline__ Frag lds2(const unsigned char* a, const unsigned char*) {
    return __builtin_bit_cast(Frag, *reinterpret_cast<const u32x4_t*>(a));
  }
  static __device__ __forceinline__ Frag zero() { return __builtin_bit_cast(Frag, u32x4_t{0u, 0u, 0u, 0u}); }
  static __device__ __forceinline__ Frag ones() {   // bf16 1.0 = 0x3f80
    return __builtin_bit_cast(Frag, u32x4_t{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
  }
  static __device__ __forceinline__ Frag keep_first(Frag f, int n) {
    u16x8_t u = __builtin_bit_cast(u16x8_t, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = e < n ? u[e] : 0;
    return __builtin_bit_cast(Frag, u);
  }
  static __device__ __forceinline__ Frag put(Frag f, int e, uint16_t x) {
    u16x8_t u = __builtin_bit_cast(u16x8_t, f);
#pragma unroll
    for (int k = 0; k < 8; ++k) u[k] = k == e ? x : u[k];
    return __builtin_bit_cast(Frag, u);
  }
  static __device__ __forceinline__ f32x4_t mma(Frag a, Frag b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Frag from_f32(f32x8_t x) { return __builtin_convertvector(x, bf16x8_t); }
  static __device__ __forceinline__ f32x8_t to_f32v(Frag f) { return __builtin_convertvector(f, f32x8_t); }
};

template <> struct Mfma<float> {      // fp32: eight v_mfma_f32_16x16x4_f32 per step
  typedef f32x8_t Frag;
  static __device__ __forceinline__ Frag load(const float* p) {
    const f32x4_t a = reinterpret_cast<const f32x4_t*>(p)[0];
    const f32x4_t b = reinterpret_cast<const f32x4_t*>(p)[1];
    return Frag{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
  static __device__ __forceinline__ Frag lds2(const unsigned char* a, const unsigned char* b) {
    const f32x4_t x = *reinterpret_cast<const f32x4_t*>(a);
    const f32x4_t y = *reinterpret_cast<const f32x4_t*>(b);
    return Frag{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
  }
  static __device__ __forceinline__ Frag zero() { return Frag{0, 0, 0, 0, 0, 0, 0, 0}; }
  static __device__ __forceinline__ Frag ones() { return Frag{1, 1, 1, 1, 1, 1, 1, 1}; }
  static __device__ __forceinline__ Frag keep_first(Frag f, int n) {
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = e < n ? f[e] : 0.f;
    return f;
  }
  static __device__ __forceinline__ Frag put(Frag f, int e, float x) {
#pragma unroll
    for (int k = 0; k < 8; ++k) f[k] = k == e ? x : f[k];
    return f;
  }
  static __device__ __forceinline__ f32x4_t mma(Frag a, Frag b, f32x4_t c) {
#pragma unroll
    for (int u = 0; u < 8; ++u) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], b[u], c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ Frag from_f32(f32x8_t x) { return x; }
  static __device__ __forceinline__ f32x8_t to_f32v(Frag f) { return f; }
};

template <typename T> __device__ __forceinline__ void store8(T* p, typename Mfma<T>::Frag f);
template <> __device__ __forceinline__ void store8<uint16_t>(uint16_t* p, bf16x8_t f) {
  *reinterpret_cast<u32x4_t*>(p) = __builtin_bit_cast(u32x4_t, f);
}
template <> __device__ __forceinline__ void store8<float>(float* p, f32x8_t f) {
  reinterpret_cast<f32x4_t*>(p)[0] = f32x4_t{f[0], f[1], f[2], f[3]};
  reinterpret_cast<f32x4_t*>(p)[1] = f32x4_t{f[4], f[5], f[6], f[7]};
}

// Key row of 32-token tile held by MFMA row lr of key block kb (see header).
__device__ __forceinline__ int tile_token(int kb, int lr) { return 8 * (lr >> 2) + 4 * kb + (lr & 3); }

// ---------------------------------------------------------------------------
// LDS ring of the context units.  A stage is one 32-token tile: K rows in
// MFMA order (row r = 16*kb + lr), stored in 16-byte chunks with chunk c of
// row r at position c ^ swizzle(r), then the tile's values exactly as cached
// (four 8-token column blocks, contiguous).  A stage is filled by 1 KB DMA
// blocks: lane l of a block writes bytes 16l..16l+15, so each lane fetches
// the global chunk that lands at its position.
// ---------------------------------------------------------------------------
template <typename T, int D, int NSTAGES>
struct Ring {
  static constexpr int E = sizeof(T);
  static constexpr int KBYTES = 32 * D * E;
  static constexpr int STAGE = 2 * KBYTES;
  static constexpr int NS = NSTAGES;                     // stages (tiles in flight + 1)
  static constexpr int BLOCKS = STAGE / 1024;
  static constexpr int KBLOCKS = KBYTES / 1024;
  static constexpr int CPR = D * E / 16;                 // chunks per key row
  static constexpr int KSH = CPR >= 16 ? 0 : 1;          // swizzle: bank groups distinct over
  static constexpr int KMASK = (CPR >= 16 ? 16 : CPR) - 1;   //   the 16 lanes of one read
  static constexpr int VBLK = 8 * D * E;                 // bytes of one 8-token value block
  static_assert(64 % CPR == 0 || CPR == 64, "key rows must tile a 1 KB block");
};

// One 16-byte LDS-DMA: this lane's 16 bytes at gptr land at lds_block + 16*lane.
// M0 carries the (wave-uniform) LDS address; the compiler loads it.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_block) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(gptr), "{m0}"(__builtin_amdgcn_readfirstlane(lds_block)) : "memory");
}

// s_waitcnt vmcnt(n) (expcnt, lgkmcnt left free).
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until at most k * DPT vector memory operations are outstanding, for
// a wave-uniform k in [0, K] (counts above 63 wait for 63: longer, never
// shorter, than needed).
template <int DPT, int K>
__device__ __forceinline__ void wait_tiles(int k) {
  if constexpr (K == 0) {
    wait_vmcnt<0>();
  } else {
    if (k >= K) wait_vmcnt<(K * DPT < 63 ? K * DPT : 63)>();
    else wait_tiles<DPT, K - 1>(k);
  }
}

// One 16-byte LDS-DMA from a wave-uniform base plus this lane's 32-bit
// offset (the SGPR-base form: no per-lane 64-bit address arithmetic).  The
// compiler cannot see the SGPR read inside the asm, so the asm itself waits
// out the hazard of a vector instruction having written those SGPRs just
// before (five wait states: s_nop 4).
__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, uint32_t lds_block) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "{m0}"(__builtin_amdgcn_readfirstlane(lds_block)) : "memory");
}

// This lane's byte offsets, from the tile's first token, of the 16 bytes it
// fetches for each of its DMA blocks (blocks wave, wave + NW, ...) of a full
// 32-token tile: K rows in MFMA order with swizzled 16-byte chunks, then the
// values' four 8-token column blocks.  Keys and values of a tile both start
// at element t0 * D of their arrays (t0 is a multiple of 8).
template <typename T, int D, int NW, int NS>
struct TileOffsets {
  using R = Ring<T, D, NS>;
  static constexpr int DPT = R::BLOCKS / NW;
  uint32_t off[DPT];
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int d = 0; d < DPT; ++d) {
      const int q = wave + NW * d;
      if (q < R::KBLOCKS) {
        const int r = q * (64 / R::CPR) + lane / R::CPR;
        const int c = (lane % R::CPR) ^ ((r >> R::KSH) & R::KMASK);
        off[d] = static_cast<uint32_t>(tile_token(r >> 4, r & 15) * D * R::E + c * 16);
      } else {
        off[d] = static_cast<uint32_t>((q - R::KBLOCKS) * 1024 + lane * 16);
      }
    }
  }
};

// Issue the DMA blocks of one tile (tokens [t0, t0+32) of [.., k1)) owned by
// this wave: blocks wave, wave + NW, ...  A full tile uses the precomputed
// offsets; in a partial one, tokens past k1 are clamped to the last valid
// one (the compute masks them).
template <typename T, int D, int NW, int NS>
__device__ __forceinline__ void issue_tile(uint32_t stage, const T* __restrict__ kbase,
                                           const T* __restrict__ vbase, int64_t t0, int64_t k1, int wave,
                                           int lane, const TileOffsets<T, D, NW, NS>& to) {
  using R = Ring<T, D, NS>;
  constexpr int DPT = R::BLOCKS / NW;
  if (t0 + 32 <= k1) {
    const T* kt = kbase + t0 * D;
    const T* vt = vbase + t0 * D;
#pragma unroll
    for (int d = 0; d < DPT; ++d) {
      const int q = wave + NW * d;          // wave-uniform
      dma16s(q < R::KBLOCKS ? kt : vt, to.off[d], stage + static_cast<uint32_t>(q) * 1024u);
    }
    return;
  }
  const int64_t vblk_last = (k1 - 1) >> 3;
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    const int q = wave + NW * d;          // wave-uniform
    const void* src;
    if (q < R::KBLOCKS) {
      const int r = q * (64 / R::CPR) + lane / R::CPR;
      const int c = (lane % R::CPR) ^ ((r >> R::KSH) & R::KMASK);
      int64_t tok = t0 + tile_token(r >> 4, r & 15);
      tok = tok < k1 ? tok : k1 - 1;
      src = reinterpret_cast<const char*>(kbase + tok * D) + c * 16;
    } else {
      const int o = (q - R::KBLOCKS) * 1024 + lane * 16;     // byte offset in the tile's values
      const int jb = o / R::VBLK;
      int64_t blk = (t0 >> 3) + jb;
      blk = blk < vblk_last ? blk : vblk_last;
      src = reinterpret_cast<const char*>(vbase + blk * 8 * D) + (o - jb * R::VBLK);
    }
    dma16(src, stage + static_cast<uint32_t>(q) * 1024u);
  }
}

// ---------------------------------------------------------------------------
// Online softmax state of one 16-row block (O^T registers: lane (lg, lr)
// holds row lr, dims 16*db + 4*lg + v).  The row sums come from the MFMA
// unit: ls += ONES * P^T, an all-ones 16 x 32 V^T block, so every element of
// ls is row lr's sum of the (rounded) weights, the same weights the values
// are multiplied by.
// ---------------------------------------------------------------------------
template <int D>
struct RowState {
  f32x4_t o[D / 16];
  f32x4_t ls;
  float m;
};

template <int D>
__device__ __forceinline__ void row_init(RowState<D>& st) {
#pragma unroll
  for (int db = 0; db < D / 16; ++db) st.o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  st.ls = f32x4_t{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
}

// Fold one tile's scores (lane (lg, lr): tokens 8*lg + 4*kb + v of row lr)
// into the state; returns P^T as the B operand of the PV product.  The
// running max m used as the exponent offset is raised only when some lane's
// tile max exceeds it by more than kRescaleLog2 (in log2 units): below that
// the weights exp2(c*(s - m)) stay under 2^kRescaleLog2, harmless in fp32,
// and the rescale of the sums and values is skipped.  Only that rare path
// reduces the max across the four lanes of a row, so that the row's lanes
// keep one common offset.  Any offset at or below the true max gives the
// same normalised result.
template <typename T, int D>
__device__ __forceinline__ typename Mfma<T>::Frag softmax_step(const f32x4_t (&sc)[2], RowState<D>& st, float c) {
  const float lmx = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                          fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
  if (wave_any((lmx - st.m) * c > kRescaleLog2)) {
    float mx = xor16_max(lmx);
    mx = xor32_max(mx);
    const float mn = fmaxf(st.m, mx);
    const float alpha = fast_exp2((st.m - (mn == -INFINITY ? 0.f : mn)) * c);
    st.ls *= alpha;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) st.o[db] *= alpha;
    st.m = mn;
  }
  const float cm = (st.m == -INFINITY ? 0.f : st.m) * c;
  f32x8_t pv;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 4; ++v) pv[4 * kb + v] = fast_exp2(fmaf(sc[kb][v], c, -cm));
  return Mfma<T>::from_f32(pv);
}

// Scores of tokens >= n (relative to the tile start) are -inf.
__device__ __forceinline__ void mask_scores(f32x4_t (&sc)[2], int n, int lg) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 4; ++v) sc[kb][v] = 8 * lg + 4 * kb + v >= n ? -INFINITY : sc[kb][v];
}

// One ring tile for RB 16-row blocks of one wave: every K and V fragment is
// read from LDS once and used by all RB blocks.  n = valid tokens of the tile
// (32 except for the chunk's last tile).
template <typename T, int D, int NS, int RB>
__device__ __forceinline__ void ring_tile(const unsigned char* stage, const typename Mfma<T>::Frag (&qf)[RB][D / 32],
                                          RowState<D> (&st)[RB], int n, int lr, int lg, float c) {
  using R = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  f32x4_t sc[RB][2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = 16 * kb + lr;
    const int sw = (r >> R::KSH) & R::KMASK;
    const unsigned char* row = stage + r * (R::CPR * 16);
    f32x4_t acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const int c0 = (8 * lg + 32 * ds) * R::E / 16;        // logical chunk of this fragment
      const typename M::Frag kf = M::lds2(row + ((c0 ^ sw) * 16), row + (((c0 + 1) ^ sw) * 16));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[rb] = M::mma(kf, qf[rb][ds], acc[rb]);
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sc[rb][kb] = acc[rb];
  }
  typename M::Frag pf[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (n < 32) mask_scores(sc[rb], n, lg);
    pf[rb] = softmax_step<T, D>(sc[rb], st[rb], c);
  }
  const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) st[rb].ls = M::mma(M::ones(), pf[rb], st[rb].ls);
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    // block lg holds this lane's 8 tokens; dimension 16*db + lr of it
    const unsigned char* vp = stage + R::KBYTES + lg * R::VBLK + (16 * db + lr) * 8 * R::E;
    typename M::Frag vf = M::lds2(vp, vp + 16);
    if (n < 32) vf = M::keep_first(vf, keep);                // never NaN * 0 past the end
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) st[rb].o[db] = M::mma(vf, pf[rb], st[rb].o[db]);
  }
}

// The two halves of ring_tile, for the software-pipelined loop: qk_tile
// computes the raw scores of a stage, softmax_pv folds them (n valid
// tokens) into the row states and adds P^T times the stage's values.
template <typename T, int D, int NS, int RB>
__device__ __forceinline__ void qk_tile(const unsigned char* stage, const typename Mfma<T>::Frag (&qf)[RB][D / 32],
                                        f32x4_t (&sc)[RB][2], int lr, int lg) {
  using R = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int DS = D / 32;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = 16 * kb + lr;
    const int sw = (r >> R::KSH) & R::KMASK;
    const unsigned char* row = stage + r * (R::CPR * 16);
    f32x4_t acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const int c0 = (8 * lg + 32 * ds) * R::E / 16;
      const typename M::Frag kf = M::lds2(row + ((c0 ^ sw) * 16), row + (((c0 + 1) ^ sw) * 16));
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[rb] = M::mma(kf, qf[rb][ds], acc[rb]);
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sc[rb][kb] = acc[rb];
  }
}

template <typename T, int D, int NS, int RB>
__device__ __forceinline__ void softmax_pv(const unsigned char* stage, f32x4_t (&sc)[RB][2], RowState<D> (&st)[RB],
                                           int n, int lr, int lg, float c) {
  using R = Ring<T, D, NS>;
  using M = Mfma<T>;
  typename M::Frag pf[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (n < 32) mask_scores(sc[rb], n, lg);
    pf[rb] = softmax_step<T, D>(sc[rb], st[rb], c);
  }
  const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) st[rb].ls = M::mma(M::ones(), pf[rb], st[rb].ls);
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const unsigned char* vp = stage + R::KBYTES + lg * R::VBLK + (16 * db + lr) * 8 * R::E;
    typename M::Frag vf = M::lds2(vp, vp + 16);
    if (n < 32) vf = M::keep_first(vf, keep);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) st[rb].o[db] = M::mma(vf, pf[rb], st[rb].o[db]);
  }
}

// One iteration of the software-pipelined loop: fold tile t (scores sc,
// values at stv) and compute the scores of the next tile (keys at stk) into
// sn.  The key reads go out first and are covered by the softmax VALU work;
// the value reads go out behind the score MFMAs, which cover them; key and
// value fragments are never live together.  On the last iteration stk is
// any ring stage and sn is not used.  mask(sc[rb], rb) sets the scores of
// keys a row may not see to -inf; n = valid tokens of tile t (values past
// them are zeroed, never NaN * 0).  With PRIO the wave raises its priority
// from its first score product to its last P.V product, so its products
// issue back to back while the other waves of the SIMD run their softmax or
// wait for tiles.
template <typename T, int D, int NS, int RB, bool PRIO = false, typename MaskFn>
__device__ __forceinline__ void pipe_step_masked(const unsigned char* stk, const unsigned char* stv,
                                                 const typename Mfma<T>::Frag (&qf)[RB][D / 32], f32x4_t (&sc)[RB][2],
                                                 f32x4_t (&sn)[RB][2], RowState<D> (&st)[RB], int n, int lr, int lg,
                                                 float c, MaskFn mask) {
  using R = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int DS = D / 32, DB = D / 16;
  typename M::Frag kf[2][DS], vf[DB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = 16 * kb + lr;
    const int sw = (r >> R::KSH) & R::KMASK;
    const unsigned char* row = stk + r * (R::CPR * 16);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const int c0 = (8 * lg + 32 * ds) * R::E / 16;
      kf[kb][ds] = M::lds2(row + ((c0 ^ sw) * 16), row + (((c0 + 1) ^ sw) * 16));
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) mask(sc[rb], rb);
  typename M::Frag pf[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) pf[rb] = softmax_step<T, D>(sc[rb], st[rb], c);
  if (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    f32x4_t acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[rb] = M::mma(kf[kb][ds], qf[rb][ds], acc[rb]);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sn[rb][kb] = acc[rb];
  }
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const unsigned char* vp = stv + R::KBYTES + lg * R::VBLK + (16 * db + lr) * 8 * R::E;
    vf[db] = M::lds2(vp, vp + 16);
  }
  if (n < 32) {
    const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[db] = M::keep_first(vf[db], keep);   // never NaN * 0 past the end
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) st[rb].ls = M::mma(M::ones(), pf[rb], st[rb].ls);
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) st[rb].o[db] = M::mma(vf[db], pf[rb], st[rb].o[db]);
  if (PRIO) __builtin_amdgcn_s_setprio(0);
}

// The decode form: only the tile's tail (tokens >= n) is masked, and the
// wave's priority is raised over its products (measured faster on decode
// steps with 64 rows per kv head; the 256-row prefill units gained nothing).
template <typename T, int D, int NS, int RB>
__device__ __forceinline__ void pipe_step(const unsigned char* stk, const unsigned char* stv,
                                          const typename Mfma<T>::Frag (&qf)[RB][D / 32], f32x4_t (&sc)[RB][2],
                                          f32x4_t (&sn)[RB][2], RowState<D> (&st)[RB], int n, int lr, int lg,
                                          float c) {
  pipe_step_masked<T, D, NS, RB, true>(stk, stv, qf, sc, sn, st, n, lr, lg, c, [n, lg](f32x4_t (&s)[2], int) {
    if (n < 32) mask_scores(s, n, lg);
  });
}

// Scores of tokens > lim (relative to the tile start) are -inf: a row's
// causal limit, or -1 to hide the whole tile from it.
__device__ __forceinline__ void mask_after(f32x4_t (&sc)[2], int lim, int lg) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 4; ++v) sc[kb][v] = 8 * lg + 4 * kb + v > lim ? -INFINITY : sc[kb][v];
}

}  // namespace ippd
