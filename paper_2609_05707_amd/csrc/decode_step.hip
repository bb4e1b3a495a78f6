// IPPD decode-step attention on gfx950: two launches per call.
//
//   attend_kernel       context units: shared-context attention, one
//                       unnormalised partial softmax state (running max,
//                       sum, weighted values) per query row and chunk;
//   segment_merge_kernel  one workgroup per (question, kv head): in the fused
//                       step it rotates and appends the token fed this step,
//                       attends over the question's own segment, and merges
//                       that state exactly with the context chunks' (splitting
//                       only regroups the sums of attn_IPPD, Sec. 4.2).
// The launch boundary orders the two, so no unit ever waits for another.
//
// A *group* is (prompt b, kv head g) for IPPD or (question i, kv head g) for
// the standard baseline.  Context unit (group, chunk, row group): context
// tokens [chunk*C, (chunk+1)*C) of prompt b against 16*NW query rows, the
// (question, head of group g) pairs of the prompt in order.  IPPD serves all
// questions of the prompt from one pass over the chunk, so K_c and V_c come
// from HBM once for all M_j queries (Sec. 4.3); the baseline serves the G
// rows of one question and reads the context once per question (App. A.2.2,
// PC+PA decode).  The workgroup streams 32-token tiles through an LDS ring
// with LDS-DMA (global_load_lds_dwordx4: HBM -> LDS without passing through
// registers), three tiles ahead of the compute; wave w owns rows 16w..16w+15
// and reads its MFMA operands from the ring:
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
// Segment (M_qtn, Sec. 4.1): four waves split the tiles of the question's
// cached slots; its last key (the step's token, at virtual position
// ctx_len[b] + seg_len[i]) is folded in from LDS, so the fused step never
// waits for its own append.
#include <float.h>

#include "ippd_device.h"
#include "ippd_internal.h"

namespace ippd {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

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

// Issue the DMA blocks of one tile (tokens [t0, t0+32) of [.., k1)) owned by
// this wave: blocks wave, wave + NW, ...  Tokens past k1 are clamped to the
// last valid one; the compute masks them.
template <typename T, int D, int NW, int NS>
__device__ __forceinline__ void issue_tile(uint32_t stage, const T* __restrict__ kbase,
                                           const T* __restrict__ vbase, int64_t t0, int64_t k1, int wave,
                                           int lane) {
  using R = Ring<T, D, NS>;
  constexpr int DPT = R::BLOCKS / NW;
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
// holds row lr, dims 16*db + 4*lg + v).
// ---------------------------------------------------------------------------
template <int D>
struct RowState {
  f32x4_t o[D / 16];
  float m, l;
};

template <int D>
__device__ __forceinline__ void row_init(RowState<D>& st) {
#pragma unroll
  for (int db = 0; db < D / 16; ++db) st.o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
}

// Fold one tile's scores (lane (lg, lr): tokens 8*lg + 4*kb + v of row lr)
// into the state; returns P^T as the B operand of the PV product.  The
// rescale by exp2(c*(m_old - m_new)) is skipped when no row's max moved,
// where it would multiply by exactly 1.
template <typename T, int D>
__device__ __forceinline__ typename Mfma<T>::Frag softmax_step(const f32x4_t (&sc)[2], RowState<D>& st, float c) {
  float mx = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                   fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
  mx = xor16_max(mx);
  mx = xor32_max(mx);
  if (__any(mx > st.m)) {
    const float mn = fmaxf(st.m, mx);
    const float alpha = fast_exp2((st.m - (mn == -INFINITY ? 0.f : mn)) * c);
    st.l *= alpha;
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
  st.l += ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
  return Mfma<T>::from_f32(pv);
}

// Scores of tokens >= n (relative to the tile start) are -inf.
__device__ __forceinline__ void mask_scores(f32x4_t (&sc)[2], int n, int lg) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 4; ++v) sc[kb][v] = 8 * lg + 4 * kb + v >= n ? -INFINITY : sc[kb][v];
}

// One ring tile for one 16-row block.  n = valid tokens of the tile (32 except
// for the chunk's last tile).
template <typename T, int D, int NS>
__device__ __forceinline__ void ring_tile(const unsigned char* stage, const typename Mfma<T>::Frag (&qf)[D / 32],
                                          RowState<D>& st, int n, int lr, int lg, float c) {
  using R = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  f32x4_t sc[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = 16 * kb + lr;
    const int sw = (r >> R::KSH) & R::KMASK;
    const unsigned char* row = stage + r * (R::CPR * 16);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const int c0 = (8 * lg + 32 * ds) * R::E / 16;        // logical chunk of this fragment
      const typename M::Frag kf = M::lds2(row + ((c0 ^ sw) * 16), row + (((c0 + 1) ^ sw) * 16));
      acc = M::mma(kf, qf[ds], acc);
    }
    sc[kb] = acc;
  }
  if (n < 32) mask_scores(sc, n, lg);
  const typename M::Frag pf = softmax_step<T, D>(sc, st, c);
  const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    // block lg holds this lane's 8 tokens; dimension 16*db + lr of it
    const unsigned char* vp = stage + R::KBYTES + lg * R::VBLK + (16 * db + lr) * 8 * R::E;
    typename M::Frag vf = M::lds2(vp, vp + 16);
    if (n < 32) vf = M::keep_first(vf, keep);                // never NaN * 0 past the end
    st.o[db] = M::mma(vf, pf, st.o[db]);
  }
}

// Write one 16-row block's partial state to its slots.
template <int D>
__device__ __forceinline__ void publish_rows(const StepParams& p, const RowState<D>& st, int64_t slot, int lg) {
  float* dst = p.part_acc + slot * D + 4 * lg;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) *reinterpret_cast<f32x4_t*>(dst + 16 * db) = st.o[db];
  if (lg == 0) *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(st.m, st.l);
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

// Query fragments (B operand) of one row (question qi, head h), in two
// steps so that all loads can be issued, and waited for, before the tile DMA
// starts: fetch_q loads q_new (fused step; plus the rotation frequencies of
// the lane's pairs) or the given rotated queries; rotate_q rotates q_new at
// pos.  Lane (lg, lr) holds dims 32*ds + 8*lg + u; pair j (j < D/2) is
// (x_j, x_{j+D/2}), i.e. fragment ds and ds + DS/2.
template <typename T, int D, bool FUSED>
struct QFetch {
  typename Mfma<T>::Frag f[D / 32];
  double th[FUSED ? D / 8 : 1];
};

template <typename T, int D, bool FUSED>
__device__ __forceinline__ void fetch_q(QFetch<T, D, FUSED>& q, const StepParams& p, int qi, int h, int lg) {
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  const T* src = static_cast<const T*>(FUSED ? p.q_new : p.q_rot_in) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) q.f[ds] = M::load(src + 32 * ds);
  if (FUSED) {
#pragma unroll
    for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
      for (int u = 0; u < 8; ++u) q.th[8 * ds + u] = p.inv_freq[lg * 8 + 32 * ds + u];
  }
}

template <typename T, int D, bool FUSED>
__device__ __forceinline__ void rotate_q(typename Mfma<T>::Frag (&qf)[D / 32], const QFetch<T, D, FUSED>& q,
                                         int64_t pos) {
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  if (!FUSED) {
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = q.f[ds];
    return;
  }
  f32x8_t x[DS];
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) x[ds] = M::to_f32v(q.f[ds]);
#pragma unroll
  for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float cs, sn, xr, yr;
      rope_cos_sin(pos, q.th[FUSED ? 8 * ds + u : 0], cs, sn);
      rope_rotate(x[ds][u], x[ds + DS / 2][u], cs, sn, xr, yr);
      x[ds][u] = xr;
      x[ds + DS / 2][u] = yr;
    }
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) qf[ds] = M::from_f32(x[ds]);
}

// ---------------------------------------------------------------------------
// Segment task (question i of prompt b, kv head g; one wave), run by the
// context units once their chunk is done.  Fused step: rotate the step's
// key at virtual position ctx_len + seg_len[i] and append it with its value;
// the task's own attention folds that key in from LDS after streaming the
// cached slots, so it never waits for the store.  Attention-only calls fold
// slot seg_len[i] - 1 the same way, so both give identical sums.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct SegScratch {
  static constexpr int QROW = D * sizeof(T) + 16;   // padded: the 16 lanes of a read hit distinct banks
  alignas(16) unsigned char q[16 * QROW];           // rotated queries of the G heads (rows >= G zero)
  alignas(16) T k[D];                               // the last key and value
  alignas(16) T v[D];
};

template <typename T, int D, bool FUSED>
__device__ void segment_task(const StepParams& p, SegScratch<T, D>& ws, int i, int ctx_len, int g, int lane) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  using SS = SegScratch<T, D>;
  constexpr int DS = D / 32, DB = D / 16;
  const int lr = lane & 15, lg = lane >> 4;
  const int G = p.G;
  const int sraw = p.seg_len[i];
  const int s = usable_seg_len(p, sraw);
  if (s < 0) {
    if (lane == 0 && g == 0) raise_flag(p.err_flag, (p.fused && sraw >= p.seg_cap) ? kFlagSegmentFull : kFlagBadLayout);
    return;
  }
  const int64_t sg = static_cast<int64_t>(i) * p.Hkv + g;
  T* skp = static_cast<T*>(p.seg_k) + sg * p.seg_cap * D;
  T* svp = static_cast<T*>(p.seg_vt) + sg * p.seg_cap * D;     // 8-token column blocks
  const int64_t pos = static_cast<int64_t>(ctx_len) + s;
  {
    // query rows: lane (lg, lr) holds head g*G + lr, dims 32*ds + 8*lg + u
    const int h = g * G + (lr < G ? lr : 0);
    const T* src = static_cast<const T*>(FUSED ? p.q_new : p.q_rot_in) + (static_cast<int64_t>(i) * p.Hq + h) * D + lg * 8;
    Frag qf[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = M::load(src + 32 * ds);
    if (FUSED) {
      // rotate pairs (j, j + D/2), j = 32*ds + 8*lg + u, at pos
#pragma unroll
      for (int ds = 0; ds < DS / 2; ++ds) {
        f32x8_t x = M::to_f32v(qf[ds]), y = M::to_f32v(qf[ds + DS / 2]);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          float cs, sn, xr, yr;
          rope_cos_sin(pos, p.inv_freq[lg * 8 + 32 * ds + u], cs, sn);
          rope_rotate(x[u], y[u], cs, sn, xr, yr);
          x[u] = xr;
          y[u] = yr;
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
    for (int ds = 0; ds < DS; ++ds) store8<T>(reinterpret_cast<T*>(ws.q + lr * SS::QROW) + 32 * ds + lg * 8, qf[ds]);
  }
  if (FUSED) {
    const T* kn = static_cast<const T*>(p.k_new) + sg * D;
    const T* vn = static_cast<const T*>(p.v_new) + sg * D;
    for (int jj = lane; jj < D / 2; jj += 64) {
      float cs, sn, x, y;
      rope_cos_sin(pos, p.inv_freq[jj], cs, sn);
      rope_rotate(to_f32<T>(kn[jj]), to_f32<T>(kn[jj + D / 2]), cs, sn, x, y);
      const T xk = from_f32<T>(x), yk = from_f32<T>(y);
      skp[static_cast<int64_t>(s) * D + jj] = xk;
      skp[static_cast<int64_t>(s) * D + jj + D / 2] = yk;
      ws.k[jj] = xk;
      ws.k[jj + D / 2] = yk;
    }
    for (int d = lane; d < D; d += 64) {
      const T v = vn[d];
      svp[static_cast<int64_t>(s >> 3) * 8 * D + d * 8 + (s & 7)] = v;
      ws.v[d] = v;
    }
  } else {
    for (int d = lane; d < D; d += 64) {
      ws.k[d] = skp[static_cast<int64_t>(s - 1) * D + d];
      ws.v[d] = svp[static_cast<int64_t>((s - 1) >> 3) * 8 * D + d * 8 + ((s - 1) & 7)];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");

  RowState<D> st;
  row_init(st);
  const float c = p.c;
  const unsigned char* qrow = ws.q + lr * SS::QROW + lg * 8 * sizeof(T);
  const int mem = FUSED ? s : s - 1;            // cached slots before the last key
  const int ntiles = (mem + 31) >> 5;
  const int mlast = max(mem - 1, 0);
  // the segment bases are wave-uniform: loads take them as scalar bases plus
  // 32-bit lane offsets (a segment holds < 2^31 elements)
  const T* __restrict__ kseg = skp;
  const T* __restrict__ vseg = svp;
  for (int t = 0; t < ntiles; ++t) {
    const int t0 = 32 * t;
    Frag kf[2][DS], vf[DB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint32_t ko = static_cast<uint32_t>(min(t0 + tile_token(kb, lr), mlast) * D + lg * 8);
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = M::load(kseg + (ko + 32 * ds));
    }
    const uint32_t vo = static_cast<uint32_t>(min((t0 >> 3) + lg, mlast >> 3) * 8 * D + lr * 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[db] = M::load(vseg + (vo + 16 * db * 8));
    const int n = min(mem - t0, 32);
    f32x4_t sc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const Frag qf = M::load(reinterpret_cast<const T*>(qrow + 32 * ds * sizeof(T)));
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) sc[kb] = M::mma(kf[kb][ds], qf, sc[kb]);
    }
    if (n < 32) mask_scores(sc, n, lg);
    const Frag pf = softmax_step<T, D>(sc, st, c);
    const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const Frag v = n < 32 ? M::keep_first(vf[db], keep) : vf[db];
      st.o[db] = M::mma(v, pf, st.o[db]);
    }
  }
  {
    // the last key: score = q_row . k, folded in as one more token
    float dot = 0.f;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const f32x8_t qv = M::to_f32v(M::load(reinterpret_cast<const T*>(qrow + 32 * ds * sizeof(T))));
      const f32x8_t kv = M::to_f32v(M::load(ws.k + 32 * ds + lg * 8));
#pragma unroll
      for (int u = 0; u < 8; ++u) dot = fmaf(qv[u], kv[u], dot);
    }
    dot = xor16_sum(dot);
    dot = xor32_sum(dot);
    if (__any(dot > st.m)) {
      const float mn = fmaxf(st.m, dot);
      const float alpha = fast_exp2((st.m - mn) * c);
      st.l *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) st.o[db] *= alpha;
      st.m = mn;
    }
    const float pn = fast_exp2((dot - st.m) * c);
    if (lg == 0) st.l += pn;                 // one lane per row: the sum is reduced over lg below
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int v = 0; v < 4; ++v) st.o[db][v] = fmaf(pn, to_f32<T>(ws.v[16 * db + 4 * lg + v]), st.o[db][v]);
  }
  float l = xor16_sum(st.l);
  st.l = xor32_sum(l);
  if (lr < G) publish_rows<D>(p, st, (static_cast<int64_t>(p.max_chunks) * p.Nt + i) * p.Hq + g * G + lr, lg);
}

// ---------------------------------------------------------------------------
// attend_kernel.  The first ctx_blocks workgroups are context units:
// blockIdx -> slice (XCD) = blockIdx & 7, local = blockIdx >> 3;
// consecutive locals of a slice are the row groups of one chunk (they share
// its tiles through that XCD's L2) and chunks are dealt to the slices round
// robin.  The remaining workgroups are segment units, NW segment tasks each
// (task (b, j, g): question slot j of prompt b, kv head g).  Workgroups are
// dispatched in order, so segment units start as context units retire and
// fill the tail of the context work.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, int NS>
union AttendShared {
  alignas(16) unsigned char ring[NS * 2 * 32 * D * sizeof(T)];
  SegScratch<T, D> seg[NW];
};

template <typename T, int D, int NW, int NS, bool FUSED>
__global__ __launch_bounds__(64 * NW, 4) void attend_kernel(StepParams p) {
  using RG = Ring<T, D, NS>;
  using M = Mfma<T>;
  constexpr int RW = 16 * NW, DPT = RG::BLOCKS / NW;
  __shared__ AttendShared<T, D, NW, NS> sh;
  unsigned char* ring = sh.ring;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  if (static_cast<int>(blockIdx.x) >= p.ctx_blocks) {
    // segment unit: task (b, j, g) per wave
    const int task = (static_cast<int>(blockIdx.x) - p.ctx_blocks) * NW + wave;
    const int g = task % p.Hkv, bj = task / p.Hkv;
    const int b = bj / p.max_questions, j = bj - b * p.max_questions;
    if (b >= p.B || !prompt_layout_ok(p, b)) return;
    const int i = p.q_start[b] + j;
    if (i >= p.q_start[b + 1] || !p.active[i]) return;
    segment_task<T, D, FUSED>(p, sh.seg[wave], i, p.ctx_len[b], g, lane);
    return;
  }
  const int slice = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int cl = local / p.nrg, rg = local - cl * p.nrg;
  const int cglob = cl * 8 + slice;
  if (cglob >= p.n_groups * p.max_chunks) return;
  const int grp = cglob / p.max_chunks, chunk = cglob - grp * p.max_chunks;

  int b, g, qa, qb;
  if (p.shared) {
    g = grp / p.B;
    b = grp - g * p.B;
  } else {
    g = grp / p.Nt;
    qa = grp - g * p.Nt;
    b = prompt_of(p.q_start, p.B, qa);
  }
  if (!prompt_layout_ok(p, b)) {
    if (threadIdx.x == 0 && chunk == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  if (p.shared) { qa = p.q_start[b]; qb = p.q_start[b + 1]; } else { qb = qa + 1; }
  const int G = p.G;
  const int nq = qb - qa;
  const int nrows = nq * G;
  const int row0 = rg * RW;
  const int ctx_len = p.ctx_len[b];
  if (static_cast<int64_t>(chunk) * p.chunk >= ctx_len || row0 >= nrows) return;
  {
    const int64_t off = p.ctx_off[b];
    const int64_t k0 = off + static_cast<int64_t>(chunk) * p.chunk;
    const int64_t k1 = min(k0 + p.chunk, off + ctx_len);
    const int ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
    const T* kbase = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
    const T* vbase = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * p.pool * D;
    const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));

    // this lane's row: question qa + row / G, head g*G + row % G.  Its loads
    // all go out, and land, before the tile DMA: queued behind the DMA of
    // every workgroup they would wait for all of it.
    const int row = row0 + 16 * wave + lr;
    const bool in_range = row < nrows;
    const int rr = in_range ? row : nrows - 1;
    const int qi = qa + rr / G, h = g * G + rr % G;
    const bool a_raw = p.active[qi] != 0;
    const int s_raw = FUSED ? p.seg_len[qi] : 0;
    QFetch<T, D, FUSED> qraw;
    fetch_q<T, D, FUSED>(qraw, p, qi, h, lg);
    wait_vmcnt<0>();

    // the first NS-1 tiles; the rotation below overlaps with them
#pragma unroll
    for (int t = 0; t < RG::NS - 1; ++t)
      issue_tile<T, D, NW, NS>(lds + t * RG::STAGE, kbase, vbase, k0 + 32ll * min(t, ntiles - 1), k1, wave, lane);

    const bool act = in_range && a_raw;
    const bool live = __any(act);                   // wave-uniform
    typename M::Frag qf[D / 32];
    rotate_q<T, D, FUSED>(qf, qraw, static_cast<int64_t>(ctx_len) + s_raw);
    if (!act) {
#pragma unroll
      for (int ds = 0; ds < D / 32; ++ds) qf[ds] = M::zero();
    }
    RowState<D> st;
    row_init(st);
    const float c = p.c;

    // ring: tile t sits in stage t % NS; at iteration t the stage of tile t-1
    // is refilled with tile t + NS - 1
    const int last = ntiles - 1;
    const int tail_n = static_cast<int>(k1 - (k0 + 32ll * last));
    for (int t = 0; t < ntiles; ++t) {
      // tile t's blocks are this thread's oldest DMAs (at most 63 can be
      // tracked: beyond that the wait is merely longer than needed)
      wait_vmcnt<((RG::NS - 2) * DPT < 63 ? (RG::NS - 2) * DPT : 63)>();
      __syncthreads();
      const int tn = t + RG::NS - 1;
      issue_tile<T, D, NW, NS>(lds + (tn % RG::NS) * RG::STAGE, kbase, vbase, k0 + 32ll * min(tn, last), k1,
                               wave, lane);
      if (live) ring_tile<T, D, NS>(ring + (t % RG::NS) * RG::STAGE, qf, st, t == last ? tail_n : 32, lr, lg, c);
    }
    wait_vmcnt<0>();                                // no LDS-DMA may outlive the workgroup

    float l = xor16_sum(st.l);
    st.l = xor32_sum(l);
    if (act) publish_rows<D>(p, st, (static_cast<int64_t>(chunk) * p.Nt + qi) * p.Hq + h, lg);
  }

}

// ---------------------------------------------------------------------------
// merge_kernel: question i = q_start[b] + j is served by merge_parts
// workgroups of kMergeThreads threads.  Item (head h, dims d0..d0+7) of the
// question combines its context chunks and its segment state:
//   m = max_k m_k,  l = sum_k 2^(c(m_k - m)) l_k,  o = sum_k 2^(c(m_k - m)) o_k / l.
// With P = merge_phases, a workgroup takes kMergeThreads / P items and P
// threads per item, thread phase f folding slots f, f + P, ...; the P states
// of an item are then combined through LDS.  The partial states are requested
// together with the question's active flag and segment length.
// ---------------------------------------------------------------------------
constexpr int kMergeThreads = 512;
constexpr int kMergeBatch = 8;       // partial states in flight per thread

// Exact combination of partial softmax states (m, l, a) in 2^(c*x) units.
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
    const float mn = fmaxf(m, mk);
    const float ms = mn == -INFINITY ? 0.f : mn;
    const float sa = fast_exp2((m - ms) * c);        // 0 while m = -inf
    const float sb = fast_exp2((mk - ms) * c);
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
  const int part = blockIdx.x % p.merge_parts, bj = blockIdx.x / p.merge_parts;
  const int b = bj / p.max_questions, j = bj - b * p.max_questions;
  if (!prompt_layout_ok(p, b)) return;             // flagged by the context units
  const int i = p.q_start[b] + j;
  if (i >= p.q_start[b + 1]) return;
  const int nc = min((p.ctx_len[b] + p.chunk - 1) / p.chunk, p.max_chunks);
  const int nslot = nc + 1;                        // chunks, then the segment
  const float c = p.c;
  const int items = p.Hq * (D / 8);
  const bool act = p.active[i] != 0;
  const int s = usable_seg_len(p, p.seg_len[i]);
  const int f = tid / per, local = tid - f * per;
  const int e = part * per + local;                // this thread's item
  const bool has = e < items;
  const int h = has ? e / (D / 8) : 0, d0 = has ? (e - h * (D / 8)) * 8 : 0;
  MergeAcc acc;
  acc.init();
  for (int k0 = f; k0 < nslot; k0 += P * kMergeBatch) {
    float2 ml[kMergeBatch];
    f32x4_t x0[kMergeBatch], x1[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
      const int k = min(k0 + P * u, nslot - 1);
      const int ck = k < nc ? k : p.max_chunks;
      const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
      ml[u] = *reinterpret_cast<const float2*>(p.part_ml + 2 * slot);
      const f32x4_t* src = reinterpret_cast<const f32x4_t*>(p.part_acc + slot * D + d0);
      x0[u] = src[0];
      x1[u] = src[1];
    }
    if (!act || s < 0) break;                      // inactive or skipped: nothing to write
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u)
      if (k0 + P * u < nslot) acc.fold(ml[u].x, ml[u].y, x0[u], x1[u], c);
  }
  if (!act || s < 0) return;                       // workgroup-uniform
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
  if (p.fused) {
    // every thread of the workgroup has read seg_len[i] above; with several
    // workgroups per question the last one to arrive advances it
    __syncthreads();
    if (tid == 0) {
      if (p.merge_parts == 1 || atomicAdd(p.counters + i, 1u) == static_cast<uint32_t>(p.merge_parts - 1)) {
        if (p.merge_parts > 1) p.counters[i] = 0;
        p.seg_len[i] = s + 1;
      }
    }
  }
}

// ---------------------------------------------------------------------------
template <typename T, int D, int NW, int NS>
static hipError_t launch_attend(int grid, const StepParams& p, hipStream_t s) {
  if (p.fused) attend_kernel<T, D, NW, NS, true><<<grid, 64 * NW, 0, s>>>(p);
  else attend_kernel<T, D, NW, NS, false><<<grid, 64 * NW, 0, s>>>(p);
  return hipGetLastError();
}

// Ring depth: 4 stages (two workgroups per CU) in general; 8 (one per CU,
// every tile of a short unit in flight at once) when the grid fits the chip
// in one wave.  fp32 at D = 128 has 32 KB stages: 2 or 4.
template <typename T, int D, int NW>
static hipError_t launch_depth(bool deep, int grid, const StepParams& p, hipStream_t s) {
  constexpr int base = (2 * 32 * D * sizeof(T)) > 16384 ? 2 : 4;
  return deep ? launch_attend<T, D, NW, 2 * base>(grid, p, s) : launch_attend<T, D, NW, base>(grid, p, s);
}

template <typename T, int D>
static hipError_t launch_d(int waves, bool deep, int grid, const StepParams& p, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (grid > 0) {
    switch (waves) {
      case 1: e = launch_depth<T, D, 1>(deep, grid, p, s); break;
      case 2: e = launch_depth<T, D, 2>(deep, grid, p, s); break;
      case 4: e = launch_depth<T, D, 4>(deep, grid, p, s); break;
      default: e = launch_depth<T, D, 8>(deep, grid, p, s); break;
    }
    if (e != hipSuccess) return e;
  }
  const unsigned nblk = static_cast<unsigned>(p.B) * p.max_questions * p.merge_parts;
  merge_kernel<D><<<nblk, kMergeThreads, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_step(int dtype, int waves, bool deep, int grid, const StepParams& p, hipStream_t s) {
  if (p.Nt == 0) return hipSuccess;
  if (dtype == 0)
    return p.D == 64 ? launch_d<float, 64>(waves, deep, grid, p, s) : launch_d<float, 128>(waves, deep, grid, p, s);
  return p.D == 64 ? launch_d<uint16_t, 64>(waves, deep, grid, p, s)
                   : launch_d<uint16_t, 128>(waves, deep, grid, p, s);
}

}  // namespace ippd
