// IPPD decode-step attention on gfx950: two launches per call.
//
//   attend_kernel  context units and segment tasks.  Each leaves, for every
//                  query row it serves, an unnormalised partial softmax state
//                  (running max, sum, weighted values) in the workspace.
//   merge_kernel   one workgroup per question combines that question's
//                  partial states exactly (splitting only regroups the sums
//                  of attn_IPPD, Sec. 4.2), writes out/lse and, in the fused
//                  step, advances the segment length.
// The launch boundary orders the two, so no unit ever waits for another.
//
// A *group* is (prompt b, kv head g) for IPPD or (question i, kv head g) for
// the standard baseline.
//
// Context unit (group, chunk, row group): context tokens
// [chunk*C, (chunk+1)*C) of prompt b against up to 16*NW query rows, the
// (active question, head of group g) pairs.  IPPD serves all active
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
// Segment task (question i, kv head g; one wave): the question's own
// question+answer segment (M_qtn, Sec. 4.1).  In the fused step the wave
// first rotates the step's key at virtual position ctx_len[b] + seg_len[i]
// (Sec. 4.1) and appends key and value to the cache; its own attention takes
// that token from registers, so it never waits for the store.
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
// MFMA order (row r = 16*kb + lr), then the V^T rows (D rows of 32 tokens).
// Both are stored in 16-byte chunks with chunk c of row r at position
// c ^ swizzle(r).  A stage is filled by 1 KB DMA blocks: lane l of a block
// writes bytes 16l..16l+15, so each lane fetches the global chunk that lands
// at its position.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct Ring {
  static constexpr int E = sizeof(T);
  static constexpr int KBYTES = 32 * D * E;
  static constexpr int STAGE = 2 * KBYTES;
  static constexpr int NS = STAGE <= 16384 ? 4 : 2;     // stages (tiles in flight + 1)
  static constexpr int BLOCKS = STAGE / 1024;
  static constexpr int KBLOCKS = KBYTES / 1024;
  static constexpr int CPR = D * E / 16;                 // chunks per key row
  static constexpr int KSH = CPR >= 16 ? 0 : 1;          // swizzle: bank groups distinct over
  static constexpr int KMASK = (CPR >= 16 ? 16 : CPR) - 1;   //   the 16 lanes of one read
  static constexpr int VCPR = 2 * E;                     // chunks per V^T row (32 tokens)
  static constexpr int VSH = VCPR == 4 ? 2 : 1;
  static constexpr int VMASK = VCPR - 1;
  static constexpr int TPC = 16 / E;                     // tokens per V^T chunk
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
template <typename T, int D, int NW>
__device__ __forceinline__ void issue_tile(uint32_t stage, const T* __restrict__ kbase,
                                           const T* __restrict__ vbase, int64_t pool, int64_t t0,
                                           int64_t k1, int wave, int lane) {
  using R = Ring<T, D>;
  constexpr int DPT = R::BLOCKS / NW;
  const int64_t vlast = (k1 - 1) & ~static_cast<int64_t>(R::TPC - 1);
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
      const int dr = (q - R::KBLOCKS) * (64 / R::VCPR) + lane / R::VCPR;
      const int c = (lane % R::VCPR) ^ ((dr >> R::VSH) & R::VMASK);
      int64_t tok = t0 + c * R::TPC;
      tok = tok < vlast ? tok : vlast;
      src = vbase + static_cast<int64_t>(dr) * pool + tok;
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
template <typename T, int D>
__device__ __forceinline__ void ring_tile(const unsigned char* stage, const typename Mfma<T>::Frag (&qf)[D / 32],
                                          RowState<D>& st, int n, int lr, int lg, float c) {
  using R = Ring<T, D>;
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
    const int d = 16 * db + lr;
    const int sw = (d >> R::VSH) & R::VMASK;
    const unsigned char* row = stage + R::KBYTES + d * (R::VCPR * 16);
    const int c0 = 2 * lg * R::E / 4;                       // bf16: lg, fp32: 2*lg
    typename M::Frag vf = M::lds2(row + ((c0 ^ sw) * 16), row + (((c0 + 1) ^ sw) * 16));
    if (n < 32) vf = M::keep_first(vf, keep);                // never NaN * 0 past the end
    st.o[db] = M::mma(vf, pf, st.o[db]);
  }
}

// Write one 16-row block's partial state to its slots (rows with valid).
template <int D>
__device__ __forceinline__ void publish_rows(const StepParams& p, const RowState<D>& st, int64_t slot,
                                             bool valid, int lg) {
  if (!valid) return;
  float* dst = p.part_acc + slot * D + 4 * lg;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) *reinterpret_cast<f32x4_t*>(dst + 16 * db) = st.o[db];
  if (lg == 0) *reinterpret_cast<float2*>(p.part_ml + 2 * slot) = make_float2(st.m, st.l);
}

// ---------------------------------------------------------------------------
// Shared memory of attend_kernel.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW>
struct AttendSmem {
  alignas(16) unsigned char ring[Ring<T, D>::NS * Ring<T, D>::STAGE];   // context units
  alignas(16) T seg_k[NW][D];                 // segment tasks: the step's rotated key
  alignas(16) T seg_v[NW][D];                 //   and value, per wave
  int q[kMaxQuestionsPerPrompt];              // compacted active questions
  int s[kMaxQuestionsPerPrompt];              // their segment lengths
  int cnt[NW];
};

__device__ __forceinline__ bool prompt_layout_ok(const StepParams& p, int b) {
  const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
  const int64_t off = p.ctx_off[b];
  const int len = p.ctx_len[b];
  return q0 >= 0 && q1 >= q0 && q1 <= p.Nt && q1 - q0 <= p.max_questions &&
         off >= 0 && (off & 7) == 0 && len >= 0 && len <= p.max_ctx_len && off + len <= p.pool;
}

// Segment length a question's units work from; -1 if the question is skipped.
__device__ __forceinline__ int usable_seg_len(const StepParams& p, int s) {
  if (p.fused) return (s >= 0 && s < p.seg_cap) ? s : -1;
  return (s >= 1 && s <= p.seg_cap) ? s : -1;
}

// Query fragments (B operand) of row `row` (question qi, head h): raw q_new
// rotated at pos (fused step) or the given rotated queries.
template <typename T, int D, bool FUSED>
__device__ __forceinline__ void load_q(typename Mfma<T>::Frag (&qf)[D / 32], const StepParams& p, int qi, int h,
                                       int64_t pos, int lg) {
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  if (FUSED) {
    const T* qp = static_cast<const T*>(p.q_new) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
    f32x8_t x[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) x[ds] = M::to_f32v(M::load(qp + 32 * ds));
#pragma unroll
    for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float cs, sn, xr, yr;
        rope_cos_sin(pos, p.inv_freq[lg * 8 + 32 * ds + u], cs, sn);
        rope_rotate(x[ds][u], x[ds + DS / 2][u], cs, sn, xr, yr);
        x[ds][u] = xr;
        x[ds + DS / 2][u] = yr;
      }
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = M::from_f32(x[ds]);
  } else {
    const T* qp = static_cast<const T*>(p.q_rot_in) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[ds] = M::load(qp + 32 * ds);
  }
}

// ---------------------------------------------------------------------------
// Context unit.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, bool FUSED>
__device__ void context_unit(const StepParams& p, AttendSmem<T, D, NW>& sm, int grp, int chunk, int rg,
                             int wave, int lane) {
  using RG = Ring<T, D>;
  using M = Mfma<T>;
  constexpr int NT = 64 * NW, RW = 16 * NW, DPT = RG::BLOCKS / NW;
  const int tid = threadIdx.x, lr = lane & 15, lg = lane >> 4;
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
    if (tid == 0 && chunk == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  if (p.shared) { qa = p.q_start[b]; qb = p.q_start[b + 1]; } else { qb = qa + 1; }
  const int ctx_len = p.ctx_len[b];
  const int64_t off = p.ctx_off[b];
  if (static_cast<int64_t>(chunk) * p.chunk >= ctx_len || qb == qa) return;
  const int64_t k0 = off + static_cast<int64_t>(chunk) * p.chunk;
  const int64_t k1 = min(k0 + p.chunk, off + ctx_len);
  const int ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
  const T* kbase = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
  const T* vbase = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * D * p.pool;
  const uint32_t ring = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sm.ring));

  // the first NS-1 tiles go out before anything else
#pragma unroll
  for (int t = 0; t < RG::NS - 1; ++t)
    issue_tile<T, D, NW>(ring + t * RG::STAGE, kbase, vbase, p.pool, k0 + 32ll * min(t, ntiles - 1), k1, wave, lane);

  // rows: active questions of the group, compacted (with their segment lengths)
  const int nq = qb - qa;
  int n_act = 0;
  for (int t0 = 0; t0 < nq; t0 += NT) {
    const int t = t0 + tid;
    const bool a = t < nq && p.active[qa + t];
    const int s = t < nq ? p.seg_len[qa + t] : 0;
    const unsigned long long ball = __ballot(a);
    const int before = __popcll(ball & ((1ull << lane) - 1ull));
    if (lane == 0) sm.cnt[wave] = __popcll(ball);
    __syncthreads();
    int wbase = n_act;
    for (int w = 0; w < wave; ++w) wbase += sm.cnt[w];
    if (a) { sm.q[wbase + before] = qa + t; sm.s[wbase + before] = s; }
    for (int w = 0; w < NW; ++w) n_act += sm.cnt[w];
    __syncthreads();
  }
  const int G = p.G;
  const int nrows = n_act * G;
  const int row0 = rg * RW;
  if (row0 >= nrows) {
    wait_vmcnt<0>();      // no LDS-DMA may outlive the workgroup
    return;
  }
  const int rb0 = row0 + 16 * wave;
  const bool live = rb0 < nrows;
  const int row = rb0 + lr;
  typename M::Frag qf[D / 32];
  if (row < nrows) {
    const int lq = row / G;
    load_q<T, D, FUSED>(qf, p, sm.q[lq], g * G + row % G, static_cast<int64_t>(ctx_len) + sm.s[lq], lg);
  } else {
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
    wait_vmcnt<(RG::NS - 2) * DPT>();
    __syncthreads();
    const int tn = t + RG::NS - 1;
    issue_tile<T, D, NW>(ring + (tn % RG::NS) * RG::STAGE, kbase, vbase, p.pool, k0 + 32ll * min(tn, last), k1,
                         wave, lane);
    if (live)
      ring_tile<T, D>(sm.ring + (t % RG::NS) * RG::STAGE, qf, st, t == last ? tail_n : 32, lr, lg, c);
  }
  wait_vmcnt<0>();

  float l = xor16_sum(st.l);
  st.l = xor32_sum(l);
  if (live && row < nrows) {
    const int lq = row / G;
    const int64_t slot = (static_cast<int64_t>(chunk) * p.Nt + sm.q[lq]) * p.Hq + g * G + row % G;
    publish_rows<D>(p, st, slot, true, lg);
  }
}

// ---------------------------------------------------------------------------
// Segment task: question i (prompt b), kv head g, one wave.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct SegTile {
  typename Mfma<T>::Frag k[2][D / 32];
  typename Mfma<T>::Frag v[D / 16];
};

template <typename T, int D, int NW, bool FUSED>
__device__ void segment_task(const StepParams& p, AttendSmem<T, D, NW>& sm, int i, int b, int g, int wave,
                             int lane) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  constexpr int DS = D / 32, DB = D / 16;
  const int lr = lane & 15, lg = lane >> 4;
  const int G = p.G;
  const int sraw = p.seg_len[i];
  const int s = usable_seg_len(p, sraw);
  if (s < 0) {
    if (lane == 0) {
      raise_flag(p.err_flag, (p.fused && sraw >= p.seg_cap) ? kFlagSegmentFull : kFlagBadLayout);
      if (g == 0) p.qmeta[i] = 0;
    }
    return;
  }
  const int ctx_len = p.ctx_len[b];
  if (g == 0 && lane == 0) p.qmeta[i] = (ctx_len + p.chunk - 1) / p.chunk + 1;
  const int64_t sg = static_cast<int64_t>(i) * p.Hkv + g;
  T* skp = static_cast<T*>(p.seg_k) + sg * p.seg_cap * D;
  T* svp = static_cast<T*>(p.seg_vt) + sg * D * p.seg_cap;
  Frag qf[DS];
  int n_tok;                                   // keys attended: memory slots [0, s) (+ slot s)
  if (FUSED) {
    // rotate and append this step's key/value at slot s, virtual position ctx_len + s
    const int64_t pos = static_cast<int64_t>(ctx_len) + s;
    const T* kn = static_cast<const T*>(p.k_new) + sg * D;
    const T* vn = static_cast<const T*>(p.v_new) + sg * D;
    for (int jj = lane; jj < D / 2; jj += 64) {
      float cs, sn, x, y;
      rope_cos_sin(pos, p.inv_freq[jj], cs, sn);
      rope_rotate(to_f32<T>(kn[jj]), to_f32<T>(kn[jj + D / 2]), cs, sn, x, y);
      const T xk = from_f32<T>(x), yk = from_f32<T>(y);
      skp[static_cast<int64_t>(s) * D + jj] = xk;
      skp[static_cast<int64_t>(s) * D + jj + D / 2] = yk;
      sm.seg_k[wave][jj] = xk;
      sm.seg_k[wave][jj + D / 2] = yk;
    }
    for (int d = lane; d < D; d += 64) {
      const T v = vn[d];
      svp[static_cast<int64_t>(d) * p.seg_cap + s] = v;
      sm.seg_v[wave][d] = v;
    }
    // rotated queries of the G heads of group g (written out if asked)
    if (lr < G) {
      load_q<T, D, true>(qf, p, i, g * G + lr, pos, lg);
      if (p.q_rot_out != nullptr) {
        T* qo = static_cast<T*>(p.q_rot_out) + (static_cast<int64_t>(i) * p.Hq + g * G + lr) * D + lg * 8;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) store8<T>(qo + 32 * ds, qf[ds]);
      }
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[ds] = M::zero();
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    n_tok = s + 1;
  } else {
    if (lr < G) {
      load_q<T, D, false>(qf, p, i, g * G + lr, 0, lg);
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[ds] = M::zero();
    }
    n_tok = s;
  }
  RowState<D> st;
  row_init(st);
  const float c = p.c;
  const int mem = FUSED ? s : n_tok;            // tokens read from the cache
  const int ntiles = (n_tok + 31) >> 5;
  const int mlast = max(mem - 1, 0);
  const int vlast = mlast & ~7;
  for (int t = 0; t < ntiles; ++t) {
    const int t0 = 32 * t;
    SegTile<T, D> tl;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int tok = min(t0 + tile_token(kb, lr), mlast);
      const T* kp = skp + static_cast<int64_t>(tok) * D + lg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) tl.k[kb][ds] = M::load(kp + 32 * ds);
    }
    {
      const int tv = min(t0 + 8 * lg, vlast);
      const T* vp = svp + static_cast<int64_t>(lr) * p.seg_cap + tv;
#pragma unroll
      for (int db = 0; db < DB; ++db) tl.v[db] = M::load(vp + static_cast<int64_t>(16 * db) * p.seg_cap);
    }
    const int n = min(n_tok - t0, 32);
    if (FUSED && t == ntiles - 1) {
      // slot s (the step's token) comes from the wave's own copy
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        if (t0 + tile_token(kb, lr) == s) {
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) tl.k[kb][ds] = M::load(&sm.seg_k[wave][32 * ds + lg * 8]);
        }
      const int e = s - t0 - 8 * lg;
      if (e >= 0 && e < 8) {
#pragma unroll
        for (int db = 0; db < DB; ++db) tl.v[db] = M::put(tl.v[db], e, sm.seg_v[wave][16 * db + lr]);
      }
    }
    f32x4_t sc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) acc = M::mma(tl.k[kb][ds], qf[ds], acc);
      sc[kb] = acc;
    }
    if (n < 32) mask_scores(sc, n, lg);
    const Frag pf = softmax_step<T, D>(sc, st, c);
    const int keep = min(max(n - 8 * lg, 0), 8);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const Frag vf = n < 32 ? M::keep_first(tl.v[db], keep) : tl.v[db];
      st.o[db] = M::mma(vf, pf, st.o[db]);
    }
  }
  float l = xor16_sum(st.l);
  st.l = xor32_sum(l);
  const int64_t slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + i) * p.Hq + g * G + lr;
  publish_rows<D>(p, st, slot, lr < G, lg);
}

// ---------------------------------------------------------------------------
// attend_kernel: blockIdx -> slice (XCD) = blockIdx & 7, local = blockIdx >> 3.
// The first seg_locals locals of every slice are segment units, then come
// context units: consecutive locals of a slice are the row groups of one
// chunk (they share its tiles through that XCD's L2), chunks are dealt to
// the slices round robin.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, bool FUSED>
__global__ __launch_bounds__(64 * NW, 4) void attend_kernel(StepParams p) {
  __shared__ AttendSmem<T, D, NW> sm;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int slice = blockIdx.x & 7, local = blockIdx.x >> 3;
  if (local < p.seg_locals) {
    const int u = local * 8 + slice;
    if (u >= p.seg_units) return;
    int i, b, g;
    if (p.shared) {
      const int grp = u / p.seg_per_group, j = u - grp * p.seg_per_group;
      g = grp / p.B;
      b = grp - g * p.B;
      if (!prompt_layout_ok(p, b)) return;     // flagged by the group's context units
      i = p.q_start[b] + NW * j + wave;
      if (i >= p.q_start[b + 1]) return;
    } else {
      const int grp = u * NW + wave;
      if (grp >= p.n_groups) return;
      g = grp / p.Nt;
      i = grp - g * p.Nt;
      b = prompt_of(p.q_start, p.B, i);
      if (!prompt_layout_ok(p, b)) return;
    }
    if (!p.active[i]) return;
    segment_task<T, D, NW, FUSED>(p, sm, i, b, g, wave, lane);
    return;
  }
  const int z = local - p.seg_locals;
  const int cl = z / p.nrg, rg = z - cl * p.nrg;
  const int cglob = cl * 8 + slice;
  if (cglob >= p.n_groups * p.max_chunks) return;
  const int grp = cglob / p.max_chunks, chunk = cglob - grp * p.max_chunks;
  context_unit<T, D, NW, FUSED>(p, sm, grp, chunk, rg, wave, lane);
}

// ---------------------------------------------------------------------------
// merge_kernel: workgroup per question; thread (head h, 8 dims) combines the
// question's context chunks and its segment state:
//   m = max_k m_k,  l = sum_k 2^(c(m_k - m)) l_k,  o = sum_k 2^(c(m_k - m)) o_k / l.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void merge_kernel(StepParams p) {
  __shared__ int s_meta;
  const int i = blockIdx.x;
  if (threadIdx.x == 0) {
    // qmeta[i] = 1 + context chunks when this call's segment task of (i, head 0)
    // ran; reset here so that a question no task reaches next call is skipped
    const int meta = p.qmeta[i];
    p.qmeta[i] = 0;
    s_meta = p.active[i] ? meta : 0;
  }
  __syncthreads();
  const int meta = s_meta;
  if (meta <= 0) return;
  const int nc = min(meta - 1, p.max_chunks);   // context chunks of the question's prompt
  const int D = p.D;
  const float c = p.c;
  constexpr int kBatch = 8;
  for (int e = threadIdx.x; e < p.Hq * D / 8; e += blockDim.x) {
    const int h = (e * 8) / D, d0 = e * 8 - h * D;
    float mx = -INFINITY, l = 0.f;
    f32x4_t a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 <= nc; k0 += kBatch) {
      float2 ml[kBatch];
      f32x4_t x0[kBatch], x1[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int k = min(k0 + u, nc);
        const int ck = k < nc ? k : p.max_chunks;
        const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
        ml[u] = *reinterpret_cast<const float2*>(p.part_ml + 2 * slot);
        const f32x4_t* src = reinterpret_cast<const f32x4_t*>(p.part_acc + slot * D + d0);
        x0[u] = src[0];
        x1[u] = src[1];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const bool live = k0 + u <= nc;
        const float mn = live ? fmaxf(mx, ml[u].x) : mx;
        const float ms = mn == -INFINITY ? 0.f : mn;
        const float sa = fast_exp2((mx - ms) * c);                        // 0 while mx = -inf
        const float sb = live ? fast_exp2((ml[u].x - ms) * c) : 0.f;
        l = l * sa + sb * ml[u].y;
        a0 = a0 * sa + x0[u] * sb;
        a1 = a1 * sa + x1[u] * sb;
        mx = mn;
      }
    }
    const float inv = 1.f / l;
    f32x4_t* dst = reinterpret_cast<f32x4_t*>(p.out + (static_cast<int64_t>(i) * p.Hq + h) * D + d0);
    dst[0] = a0 * inv;
    dst[1] = a1 * inv;
    if (p.lse != nullptr && d0 == 0) p.lse[static_cast<int64_t>(i) * p.Hq + h] = mx * p.scale + logf(l);
  }
  if (p.fused && threadIdx.x == 0) p.seg_len[i] = p.seg_len[i] + 1;
}

// ---------------------------------------------------------------------------
template <typename T, int D, int NW>
static hipError_t launch_attend(int grid, const StepParams& p, hipStream_t s) {
  if (p.fused) attend_kernel<T, D, NW, true><<<grid, 64 * NW, 0, s>>>(p);
  else attend_kernel<T, D, NW, false><<<grid, 64 * NW, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_d(int waves, int grid, const StepParams& p, hipStream_t s) {
  switch (waves) {
    case 1: return launch_attend<T, D, 1>(grid, p, s);
    case 2: return launch_attend<T, D, 2>(grid, p, s);
    case 4: return launch_attend<T, D, 4>(grid, p, s);
    default: return launch_attend<T, D, 8>(grid, p, s);
  }
}

hipError_t launch_step(int dtype, int waves, int grid, const StepParams& p, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipError_t e;
  if (dtype == 0)
    e = p.D == 64 ? launch_d<float, 64>(waves, grid, p, s) : launch_d<float, 128>(waves, grid, p, s);
  else
    e = p.D == 64 ? launch_d<uint16_t, 64>(waves, grid, p, s) : launch_d<uint16_t, 128>(waves, grid, p, s);
  if (e != hipSuccess) return e;
  merge_kernel<<<p.Nt, 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace ippd
