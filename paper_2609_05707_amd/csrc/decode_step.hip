// Single-launch IPPD decode step on gfx950: rotation + append (optional),
// shared-context attention, own-segment attention and the exact merge.
//
// Work decomposition.  A *group* is (prompt b, kv head g) for IPPD, or
// (question i, kv head g) for the standard baseline.  A group owns
//   - context units (chunk c, row group rg): context tokens
//     [c*chunk, (c+1)*chunk) of prompt b applied to a block of query rows =
//     (active question, head of group g) pairs.  IPPD serves all active
//     questions of the prompt from one pass over the chunk, so K_c, V_c are
//     read from HBM once for all M_j queries (Sec. 4.3); the baseline serves
//     the G rows of one question, reading the context once per question
//     (App. A.2.2, PC+PA decode);
//   - segment units (one question per wave): the question's own
//     question+answer segment (M_qtn, Sec. 4.1), including the token fed this
//     step, whose key/value the fused step first appends at virtual position
//     ctx_len[b] + seg_len[i] (Sec. 4.1).
// Every unit leaves an unnormalised partial softmax state (max, sum,
// weighted values) per row.  Each segment group has an arrival counter that
// every context unit of the group and the segment unit bump after publishing
// their partials; whoever arrives last merges the group's rows exactly
// (splitting only regroups the sums of attn_IPPD, Sec. 4.2) and resets the
// counter.  No unit waits for another and no L2 writeback or invalidate is
// issued (see publish4).
//
// Context units come in two shapes:
//   row split (IPPD, > 16 rows): NW waves each own a 16-row block.  All
//     threads load each 32-token K/V tile with coalesced 16-byte loads into a
//     small register stage and write it to a double-buffered LDS tile; every
//     wave then reads its MFMA operands from LDS, so the tile is fetched from
//     HBM once for all rows.  Loads run two tiles ahead of the compute.
//   token split (<= 16 rows: baseline, small prompts): four waves stream
//     interleaved tiles straight into registers and meet once in LDS.
// Per tile and 16-row block:
//   S^T (keys x rows) = K Q^T           v_mfma_f32_16x16x32_bf16, A = 16 keys x 32 dims
//   P^T = exp2(c * (S^T - m))           online softmax; row max across the four
//                                       16-lane rows through permlane swaps
//   O^T (dims x rows) += V^T P^T        A = V^T rows, token-contiguous in the
//                                       transposed value cache; B = P^T taken
//                                       straight from the S^T registers
// Key rows are assigned to MFMA rows so that lane row r of S^T holds 8
// consecutive tokens, exactly the B layout PV needs: K and V^T fragments are
// single 16-byte reads and P never leaves registers.
#include <float.h>

#include "ippd_device.h"
#include "ippd_internal.h"

namespace ippd {

constexpr int kWaves = 4;             // waves of a token-split context unit

// ---------------------------------------------------------------------------
// MFMA operand traits: 8 contraction elements per lane per 32-wide step.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<uint16_t> {   // bf16: one v_mfma_f32_16x16x32_bf16 per step
  typedef bf16x8_t Frag;
  static __device__ __forceinline__ Frag load(const uint16_t* p) {
    return __builtin_bit_cast(Frag, *reinterpret_cast<const uint4*>(p));
  }
  static __device__ __forceinline__ Frag zero() { return __builtin_bit_cast(Frag, make_uint4(0, 0, 0, 0)); }
  static __device__ __forceinline__ Frag keep_first(Frag f, int n) {
    u16x8_t u = __builtin_bit_cast(u16x8_t, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) u[e] = e < n ? u[e] : 0;
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
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    Frag f = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    return f;
  }
  static __device__ __forceinline__ Frag zero() { Frag f = {0, 0, 0, 0, 0, 0, 0, 0}; return f; }
  static __device__ __forceinline__ Frag keep_first(Frag f, int n) {
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = e < n ? f[e] : 0.f;
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
  *reinterpret_cast<uint4*>(p) = __builtin_bit_cast(uint4, f);
}
template <> __device__ __forceinline__ void store8<float>(float* p, f32x8_t f) {
  reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
}

// ---------------------------------------------------------------------------
// Publishing partial states between units.  A merger may run on another XCD,
// whose L2 is not coherent with the writer's.  Partials are therefore written
// with device-scope stores (write-through past L2) and read with device-scope
// loads (miss in L2); before bumping an arrival counter every wave waits for
// its stores to be acknowledged.  The counters themselves are device-scope
// atomics.  No L2 writeback or invalidate is ever needed.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void publish4(float* p, float a, float b, float c, float d) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const uint64_t lo = (static_cast<uint64_t>(__float_as_uint(b)) << 32) | __float_as_uint(a);
  const uint64_t hi = (static_cast<uint64_t>(__float_as_uint(d)) << 32) | __float_as_uint(c);
  __hip_atomic_store(q, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void publish2(float* p, float a, float b) {
  const uint64_t v = (static_cast<uint64_t>(__float_as_uint(b)) << 32) | __float_as_uint(a);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 fetch2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float(static_cast<uint32_t>(v)), __uint_as_float(static_cast<uint32_t>(v >> 32)));
}
// s_waitcnt vmcnt(0): every vector memory operation of this wave has completed.
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ uint32_t arrive(uint32_t* c) {
  return __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void clear(uint32_t* c) {
  __hip_atomic_store(c, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// ---------------------------------------------------------------------------
// One 32-token tile of one wave: K fragments (2 key blocks x D/32 steps) and
// V^T fragments (D/16 dim blocks).
// ---------------------------------------------------------------------------
template <typename T, int D>
struct Tile {
  typename Mfma<T>::Frag k[2][D / 32];
  typename Mfma<T>::Frag v[D / 16];
};

// Register-streamed tile (token-split units and segments).  Loads are
// unconditional, with addresses clamped into [k0, k1) and tail data masked
// where it is used: a branch around a load would make the compiler's
// wait-count tracking wait for every load in flight, including the
// prefetched next tile.
template <typename T, int D>
__device__ __forceinline__ void load_tile(Tile<T, D>& tl, const T* __restrict__ kbase,
                                          const T* __restrict__ vbase, int64_t vstride,
                                          int64_t t0, int64_t k1, int lr, int lg) {
  using M = Mfma<T>;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    int64_t tk = t0 + 8 * (lr >> 2) + 4 * kb + (lr & 3);
    tk = tk < k1 ? tk : k1 - 1;
    const T* kp = kbase + tk * D + lg * 8;
#pragma unroll
    for (int ds = 0; ds < D / 32; ++ds) tl.k[kb][ds] = M::load(kp + 32 * ds);
  }
  int64_t tv = t0 + 8 * lg;
  const int64_t tv_last = (k1 - 1) & ~static_cast<int64_t>(7);   // last 8-token group in range
  tv = tv < tv_last ? tv : tv_last;
  const T* vp = vbase + static_cast<int64_t>(lr) * vstride + tv;
#pragma unroll
  for (int db = 0; db < D / 16; ++db) tl.v[db] = M::load(vp + static_cast<int64_t>(16 * db) * vstride);
}

// Online-softmax update of one wave with one tile; nrb row blocks are live.
template <typename T, int D, int RB>
__device__ __forceinline__ void process_tile(const Tile<T, D>& tl, const typename Mfma<T>::Frag (&qf)[RB][D / 32],
                                             f32x4_t (&o)[D / 16][RB], float (&m_run)[RB], float (&l_run)[RB],
                                             int64_t t0, int64_t k1, int lg, float c, int nrb) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  constexpr int DS = D / 32, DB = D / 16;
  f32x4_t sc[2][RB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
      if (rb < nrb) {
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) acc = M::mma(tl.k[kb][ds], qf[rb][ds], acc);
      }
      sc[kb][rb] = acc;
    }
  // lane (lg, lr) holds, for row lr of each block, tokens t0 + 8*lg + 4*kb + v
  if (t0 + 32 > k1) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const bool dead = t0 + 8 * lg + 4 * kb + v >= k1;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) sc[kb][rb][v] = dead ? -INFINITY : sc[kb][rb][v];
      }
  }
  Frag pf[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (rb >= nrb) { pf[rb] = M::zero(); continue; }
    float mx = fmaxf(fmaxf(fmaxf(sc[0][rb][0], sc[0][rb][1]), fmaxf(sc[0][rb][2], sc[0][rb][3])),
                     fmaxf(fmaxf(sc[1][rb][0], sc[1][rb][1]), fmaxf(sc[1][rb][2], sc[1][rb][3])));
    mx = xor16_max(mx);
    mx = xor32_max(mx);
    const float m_new = fmaxf(m_run[rb], mx);
    const float m_safe = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2((m_run[rb] - m_safe) * c);
    const float cm = m_safe * c;
    f32x8_t pv;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 4; ++v) pv[4 * kb + v] = fast_exp2(fmaf(sc[kb][rb][v], c, -cm));
    const float ps = ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
    l_run[rb] = l_run[rb] * alpha + ps;
    m_run[rb] = m_new;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][rb] *= alpha;
    pf[rb] = M::from_f32(pv);
  }
  // tail tile: zero values of tokens past the end (never NaN * 0)
  const bool tail = t0 + 32 > k1;
  int keep = static_cast<int>(min(max(k1 - (t0 + 8 * lg), static_cast<int64_t>(0)), static_cast<int64_t>(8)));
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const Frag v = tail ? M::keep_first(tl.v[db], keep) : tl.v[db];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      if (rb < nrb) o[db][rb] = M::mma(v, pf[rb], o[db][rb]);
  }
}

// Stream this wave's tiles first, first+stride, ... of [k0, k1) through
// registers, one tile ahead.  A counted loop over tile pairs (tail peeled)
// keeps the load pattern identical on every path into the loop, which lets
// the compiler wait for exactly one tile.
template <typename T, int D>
__device__ __forceinline__ void stream_tiles(const T* __restrict__ kbase, const T* __restrict__ vbase,
                                             int64_t vstride, int64_t k0, int64_t k1, int first, int stride,
                                             const typename Mfma<T>::Frag (&qf)[1][D / 32],
                                             f32x4_t (&o)[D / 16][1], float (&m_run)[1], float (&l_run)[1],
                                             int lr, int lg, float c) {
  const int ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
  if (first >= ntiles) return;
  const int mine = (ntiles - first + stride - 1) / stride;      // tiles of this wave
  auto start = [&](int n) { return k0 + 32ll * (first + min(n, mine - 1) * stride); };
  Tile<T, D> a, b;
  load_tile<T, D>(a, kbase, vbase, vstride, start(0), k1, lr, lg);
  load_tile<T, D>(b, kbase, vbase, vstride, start(1), k1, lr, lg);
  const int pairs = mine >> 1;
  for (int n = 0; n < pairs; ++n) {
    process_tile<T, D, 1>(a, qf, o, m_run, l_run, start(2 * n), k1, lg, c, 1);
    load_tile<T, D>(a, kbase, vbase, vstride, start(2 * n + 2), k1, lr, lg);
    process_tile<T, D, 1>(b, qf, o, m_run, l_run, start(2 * n + 1), k1, lg, c, 1);
    load_tile<T, D>(b, kbase, vbase, vstride, start(2 * n + 3), k1, lr, lg);
  }
  if (mine & 1) process_tile<T, D, 1>(a, qf, o, m_run, l_run, start(mine - 1), k1, lg, c, 1);
}

// ---------------------------------------------------------------------------
// Row-split staging: geometry of one 32-token tile in LDS and its
// cooperative load (16-byte chunks, CPT per thread).
// ---------------------------------------------------------------------------
template <typename T, int D, int NW>
struct RowGeom {
  static constexpr int E = sizeof(T);
  static constexpr int KROW = D * E + 16;        // padded key row (bytes): rows shift 4 banks
  static constexpr int KBYTES = 32 * KROW;
  static constexpr int VROW = 32 * E;            // one V^T dim row of the tile (bytes)
  static constexpr int VBYTES = D * VROW;
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int NK = 2 * D * E;           // key chunks per tile
  static constexpr int NCH = 2 * NK;             // key + value chunks
  static constexpr int THREADS = 64 * NW;
  static constexpr int CPT = NCH / THREADS;
  static constexpr int KCPR = D * E / 16;        // key chunks per token
  static constexpr int VCPR = 2 * E;             // value chunks per dim row
  static constexpr int TPC = 16 / E;             // tokens per value chunk
  static_assert(NCH % THREADS == 0, "tile chunks must split evenly over the threads");
};

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <typename T, int D, int NW>
struct Stage {                       // native vectors, so the array stays in registers
  u32x4_t x[RowGeom<T, D, NW>::CPT];
};

template <typename T, int D, int NW>
__device__ __forceinline__ void stage_load(Stage<T, D, NW>& st, const T* __restrict__ kbase,
                                           const T* __restrict__ vbase, int64_t vstride, int64_t t0,
                                           int64_t k1, int tid) {
  using G = RowGeom<T, D, NW>;
  const int64_t tv_last = (k1 - 1) & ~static_cast<int64_t>(G::TPC - 1);
#pragma unroll
  for (int u = 0; u < G::CPT; ++u) {
    const int q = tid + G::THREADS * u;
    const int rk = q / G::KCPR, ck = q - rk * G::KCPR;
    int64_t tk = t0 + rk;
    tk = tk < k1 ? tk : k1 - 1;
    const int qv = q >= G::NK ? q - G::NK : 0;
    const int dv = qv / G::VCPR, cv = qv - dv * G::VCPR;
    int64_t tv = t0 + cv * G::TPC;
    tv = tv < tv_last ? tv : tv_last;
    const char* ka = reinterpret_cast<const char*>(kbase + tk * D) + ck * 16;
    const char* va = reinterpret_cast<const char*>(vbase + static_cast<int64_t>(dv) * vstride + tv);
    st.x[u] = *reinterpret_cast<const u32x4_t*>(q < G::NK ? ka : va);
  }
}

template <typename T, int D, int NW>
__device__ __forceinline__ void stage_store(const Stage<T, D, NW>& st, unsigned char* ring, int tid) {
  using G = RowGeom<T, D, NW>;
#pragma unroll
  for (int u = 0; u < G::CPT; ++u) {
    const int q = tid + G::THREADS * u;
    const int rk = q / G::KCPR, ck = q - rk * G::KCPR;
    const int qv = q >= G::NK ? q - G::NK : 0;
    const int dv = qv / G::VCPR, cv = qv - dv * G::VCPR;
    const int off = q < G::NK ? rk * G::KROW + ck * 16 : G::KBYTES + dv * G::VROW + cv * 16;
    *reinterpret_cast<u32x4_t*>(ring + off) = st.x[u];
  }
}

// One wave's online-softmax update from an LDS tile: key fragments are read
// for the score MFMAs, value fragments one dim block at a time for PV, so
// only one operand set is live at once.
template <typename T, int D, int NW>
__device__ __forceinline__ void process_lds_tile(const unsigned char* ring, const typename Mfma<T>::Frag (&qf)[1][D / 32],
                                                 f32x4_t (&o)[D / 16][1], float (&m_run)[1], float (&l_run)[1],
                                                 int64_t t0, int64_t k1, int lr, int lg, float c) {
  using G = RowGeom<T, D, NW>;
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  constexpr int DS = D / 32, DB = D / 16;
  f32x4_t sc[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int tk = 8 * (lr >> 2) + 4 * kb + (lr & 3);
    const T* kp = reinterpret_cast<const T*>(ring + tk * G::KROW) + lg * 8;
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) acc = M::mma(M::load(kp + 32 * ds), qf[0][ds], acc);
    sc[kb] = acc;
  }
  if (t0 + 32 > k1) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 4; ++v) sc[kb][v] = t0 + 8 * lg + 4 * kb + v >= k1 ? -INFINITY : sc[kb][v];
  }
  float mx = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                   fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
  mx = xor16_max(mx);
  mx = xor32_max(mx);
  const float m_new = fmaxf(m_run[0], mx);
  const float m_safe = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = fast_exp2((m_run[0] - m_safe) * c);
  const float cm = m_safe * c;
  f32x8_t pv;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 4; ++v) pv[4 * kb + v] = fast_exp2(fmaf(sc[kb][v], c, -cm));
  l_run[0] = l_run[0] * alpha + (((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7])));
  m_run[0] = m_new;
  const Frag pf = M::from_f32(pv);
  const bool tail = t0 + 32 > k1;
  const int keep = static_cast<int>(min(max(k1 - (t0 + 8 * lg), static_cast<int64_t>(0)), static_cast<int64_t>(8)));
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    Frag v = M::load(reinterpret_cast<const T*>(ring + G::KBYTES + (16 * db + lr) * G::VROW) + lg * 8);
    if (tail) v = M::keep_first(v, keep);
    o[db][0] = M::mma(v, pf, o[db][0] * alpha);
  }
}

// ---------------------------------------------------------------------------
// Shared memory: the phases of a unit never overlap, so they share storage.
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, bool RS>
struct StepSmem {
  static constexpr int RW = RS ? 16 * NW : 16;     // rows of a context unit
  union {
    unsigned char ring[RS ? 2 * RowGeom<T, D, NW>::STAGE : 16];   // row split: tile double buffer
    float o[RS ? 1 : kWaves][16][D + 4];                          // token split: cross-wave merge
    float2 cs[RW + 1][D / 2];                                      // cos/sin per question of a unit
    float2 seg_cs[NW][D / 2];                                      // segment unit: per wave
  } u;
  float m[kWaves][16];
  float l[kWaves][16];
  int q[kMaxQuestionsPerPrompt];                   // compacted active questions of the prompt
  int merge_list[kMaxQuestionsPerPrompt];
  int cnt[NW];
  int n_merge;
};

__device__ __forceinline__ bool prompt_layout_ok(const StepParams& p, int b) {
  const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
  const int64_t off = p.ctx_off[b];
  const int len = p.ctx_len[b];
  return q0 >= 0 && q1 >= q0 && q1 <= p.Nt && q1 - q0 <= p.max_questions &&
         off >= 0 && (off & 7) == 0 && len >= 0 && len <= p.max_ctx_len && off + len <= p.pool;
}

// Segment length a question's units work from; -1 if the question is skipped.
__device__ __forceinline__ int usable_seg_len(const StepParams& p, int i) {
  const int s = p.seg_len[i];
  if (p.fused) return (s >= 0 && s < p.seg_cap) ? s : -1;
  return (s >= 1 && s <= p.seg_cap) ? s : -1;
}

// Rotated query fragments (B operand) of one 16-row block: row r of the
// block is the (question, head) pair in LDS list q at index row0b + r.
template <typename T, int D, bool FUSED>
__device__ __forceinline__ void load_q(typename Mfma<T>::Frag (&qf)[1][D / 32], const StepParams& p,
                                       const int* qlist, const float2 (*cs)[D / 2], int row_block0, int R,
                                       int q_first, int g, int lr, int lg) {
  using M = Mfma<T>;
  constexpr int DS = D / 32;
  const int G = p.G;
  const int row = row_block0 + lr;
  if (row >= R) {
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::zero();
    return;
  }
  const int qi = qlist[row / G];
  const int h = g * G + row % G;
  if (FUSED) {
    const T* qp = static_cast<const T*>(p.q_new) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
    f32x8_t x[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) x[ds] = M::to_f32v(M::load(qp + 32 * ds));
    const int lq = row / G - q_first;
#pragma unroll
    for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float2 csv = cs[lq][lg * 8 + 32 * ds + u];
        float xr, yr;
        rope_rotate(x[ds][u], x[ds + DS / 2][u], csv.x, csv.y, xr, yr);
        x[ds][u] = xr;
        x[ds + DS / 2][u] = yr;
      }
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::from_f32(x[ds]);
  } else {
    const T* qp = static_cast<const T*>(p.q_rot_in) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::load(qp + 32 * ds);
  }
}

// ---------------------------------------------------------------------------
// Exact merge of segment group j: wave w merges question qa + NW*j + w (IPPD)
// or the group's single question (baseline, wave 0).  Online over the slots,
// eight slots' loads in flight at a time.
// ---------------------------------------------------------------------------
template <int D, int NW>
__device__ void merge_segment_group(const StepParams& p, int b, int g, int qa, int qb, int j, int wave) {
  const int lane = threadIdx.x & 63;
  const int i = p.shared ? qa + NW * j + wave : qa;
  if (!p.shared && wave != 0) return;
  if (i >= qb || !p.active[i]) return;
  const int s = usable_seg_len(p, i);
  if (s < 0) return;
  const int nc = (p.ctx_len[b] + p.chunk - 1) / p.chunk;
  const int G = p.G;
  const float c = p.c;
  constexpr int kBatch = 8;
  for (int e0 = lane * 8; e0 < G * D; e0 += 64 * 8) {
    const int row = e0 / D, d0 = e0 - row * D;
    const int h = g * G + row;
    float mx = -INFINITY, l = 0.f;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int k0 = 0; k0 <= nc; k0 += kBatch) {
      float2 ml[kBatch], x[kBatch][4];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int k = min(k0 + u, nc);
        const int ck = k < nc ? k : p.max_chunks;
        const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
        ml[u] = fetch2(p.part_ml + 2 * slot);
        const float* src = p.part_acc + slot * D + d0;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) x[u][qq] = fetch2(src + 2 * qq);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const bool live = k0 + u <= nc;
        const float mn = live ? fmaxf(mx, ml[u].x) : mx;
        const float sa = fast_exp2((mx - mn) * c);                     // 0 while mx = -inf
        const float sb = live ? fast_exp2((ml[u].x - mn) * c) : 0.f;
        l = l * sa + sb * ml[u].y;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          acc[2 * qq] = acc[2 * qq] * sa + sb * x[u][qq].x;
          acc[2 * qq + 1] = acc[2 * qq + 1] * sa + sb * x[u][qq].y;
        }
        mx = mn;
      }
    }
    const float inv = 1.f / l;
    float4* dst = reinterpret_cast<float4*>(p.out + (static_cast<int64_t>(i) * p.Hq + h) * D + d0);
    dst[0] = make_float4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    dst[1] = make_float4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
    if (p.lse != nullptr && d0 == 0) p.lse[static_cast<int64_t>(i) * p.Hq + h] = mx * p.scale + logf(l);
  }
  if (p.fused && lane == 0) {
    // The last of the Hkv merges of question i advances its segment: every
    // unit that reads seg_len[i] this step has arrived before any merge of i.
    uint32_t* qc = p.counters + static_cast<size_t>(p.n_groups) * p.seg_units_per_group + i;
    if (arrive(qc) == static_cast<uint32_t>(p.Hkv - 1)) {
      clear(qc);
      __hip_atomic_fetch_add(p.seg_len + i, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Write one 16-row block's partial state (O^T registers; lane (lg, lr) holds
// row lr, dims 16*db + 4*lg + v) to its slots.
template <int D>
__device__ __forceinline__ void publish_rows(const StepParams& p, const f32x4_t (&o)[D / 16][1], float m,
                                             float l, int64_t slot, bool valid, int lg) {
  if (!valid) return;
#pragma unroll
  for (int db = 0; db < D / 16; ++db)
    publish4(p.part_acc + slot * D + 16 * db + 4 * lg, o[db][0][0], o[db][0][1], o[db][0][2], o[db][0][3]);
  if (lg == 0) publish2(p.part_ml + 2 * slot, m, l);
}

// ---------------------------------------------------------------------------
// The kernel.  NW waves per workgroup; RS selects the row-split context
// units (otherwise token split with NW = 4).
// ---------------------------------------------------------------------------
template <typename T, int D, int NW, bool RS, bool FUSED>
__global__ __launch_bounds__(64 * NW, 2) void decode_step_kernel(StepParams p) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  using SM = StepSmem<T, D, NW, RS>;
  constexpr int DS = D / 32, DB = D / 16, NT = 64 * NW, RW = SM::RW;
  static_assert(RS || NW == kWaves, "token-split units use four waves");
  __shared__ SM sm;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar control flow
  const int lr = lane & 15, lg = lane >> 4;

  // ---- unit decode: groups are dealt to the 8 slices (XCDs) in contiguous runs ----
  const int slice = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int gl = local / p.units_per_group;
  const int r = local - gl * p.units_per_group;
  const int grp = slice * p.groups_per_slice + gl;
  if (grp >= p.n_groups) return;
  int b, g, qa, qb;
  if (p.shared) {
    g = grp / p.B;
    b = grp - g * p.B;
    qa = qb = 0;
  } else {
    g = grp / p.Nt;
    qa = grp - g * p.Nt;
    qb = qa + 1;
    b = prompt_of(p.q_start, p.B, qa);
  }
  if (!prompt_layout_ok(p, b)) {
    if (tid == 0 && r == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  if (p.shared) { qa = p.q_start[b]; qb = p.q_start[b + 1]; }
  const int nseg = p.shared ? (qb - qa + NW - 1) / NW : 1;
  if (nseg == 0) return;
  uint32_t* grp_cnt = p.counters + static_cast<size_t>(grp) * p.seg_units_per_group;
  const int G = p.G;
  const float c = p.c;
  const int ctx_len = p.ctx_len[b];

  if (r < p.ctx_units_per_group) {
    // =========================== context unit ===============================
    const int cidx = r / p.nrg, rg = r - cidx * p.nrg;
    const int64_t off = p.ctx_off[b];
    const int64_t k0 = off + static_cast<int64_t>(cidx) * p.chunk;
    const int64_t k1 = min(k0 + p.chunk, off + ctx_len);
    const int row0 = rg * RW;
    const int nq = qb - qa;
    const bool maybe = static_cast<int64_t>(cidx) * p.chunk < ctx_len && row0 < nq * G;
    const T* kbase = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
    const T* vbase = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * D * p.pool;
    const int ntiles = maybe ? static_cast<int>((k1 - k0 + 31) >> 5) : 0;

    // first two tiles of the row-split pipeline go out before any setup
    Stage<T, D, NW> sa, sb;
    if (RS && ntiles > 0) {
      stage_load<T, D, NW>(sa, kbase, vbase, p.pool, k0, k1, tid);
      stage_load<T, D, NW>(sb, kbase, vbase, p.pool, k0 + 32ll * min(1, ntiles - 1), k1, tid);
    }

    // rows: active questions of the group, compacted
    int n_act = 0;
    if (maybe) {
      if (p.shared) {
        int base_cnt = 0;
        for (int t0 = 0; t0 < nq; t0 += NT) {
          const int t = t0 + tid;
          const bool a = t < nq && p.active[qa + t];
          const unsigned long long ball = __ballot(a);
          const int before = __popcll(ball & ((1ull << lane) - 1ull));
          if (lane == 0) sm.cnt[wave] = __popcll(ball);
          __syncthreads();
          int wbase = base_cnt;
          for (int w = 0; w < wave; ++w) wbase += sm.cnt[w];
          if (a) sm.q[wbase + before] = qa + t;
          for (int w = 0; w < NW; ++w) base_cnt += sm.cnt[w];
          __syncthreads();
        }
        n_act = base_cnt;
      } else {
        n_act = p.active[qa] ? 1 : 0;
        if (tid == 0) sm.q[0] = qa;
        __syncthreads();
      }
    }
    const int R = n_act * G;
    if (maybe && row0 < R) {
      // questions touched by rows [row0, row_end); with G not dividing 16 the
      // first and last may straddle a neighbouring unit's window
      const int q_first = row0 / G;
      const int row_end = min(R, row0 + RW);
      if (FUSED) {
        const int nlq = (row_end - 1) / G - q_first + 1;
        for (int e = tid; e < nlq * (D / 2); e += NT) {
          const int lq = e / (D / 2), jj = e - lq * (D / 2);
          const int qi = sm.q[q_first + lq];
          float cs, sn;
          rope_cos_sin(static_cast<int64_t>(ctx_len) + p.seg_len[qi], p.inv_freq[jj], cs, sn);
          sm.u.cs[lq][jj] = make_float2(cs, sn);
        }
        __syncthreads();
      }
      f32x4_t o[DB][1];
      float m_run[1] = {-INFINITY}, l_run[1] = {0.f};
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      Frag qf[1][DS];

      if (RS) {
        // ---- row split: wave w owns rows row0 + 16w .. +15 ----
        const int rb0 = row0 + 16 * wave;
        const bool live = rb0 < R;
        load_q<T, D, FUSED>(qf, p, sm.q, sm.u.cs, rb0, R, q_first, g, lr, lg);
        __syncthreads();   // cos/sin table (aliasing the ring) fully read
        unsigned char* ring0 = sm.u.ring;
        unsigned char* ring1 = sm.u.ring + RowGeom<T, D, NW>::STAGE;
        const int last = ntiles - 1;
        const int pairs = ntiles >> 1;
        for (int n = 0; n < pairs; ++n) {
          const int t = 2 * n;
          stage_store<T, D, NW>(sa, ring0, tid);
          stage_load<T, D, NW>(sa, kbase, vbase, p.pool, k0 + 32ll * min(t + 2, last), k1, tid);
          __syncthreads();
          if (live) process_lds_tile<T, D, NW>(ring0, qf, o, m_run, l_run, k0 + 32ll * t, k1, lr, lg, c);
          stage_store<T, D, NW>(sb, ring1, tid);
          stage_load<T, D, NW>(sb, kbase, vbase, p.pool, k0 + 32ll * min(t + 3, last), k1, tid);
          __syncthreads();
          if (live) process_lds_tile<T, D, NW>(ring1, qf, o, m_run, l_run, k0 + 32ll * (t + 1), k1, lr, lg, c);
        }
        if (ntiles & 1) {
          stage_store<T, D, NW>(sa, ring0, tid);
          __syncthreads();
          if (live) process_lds_tile<T, D, NW>(ring0, qf, o, m_run, l_run, k0 + 32ll * last, k1, lr, lg, c);
        }
        float l = xor16_sum(l_run[0]);
        l = xor32_sum(l);
        const int row = rb0 + lr;
        if (live && row < R) {
          const int qi = sm.q[row / G];
          const int64_t slot = (static_cast<int64_t>(cidx) * p.Nt + qi) * p.Hq + g * G + row % G;
          publish_rows<D>(p, o, m_run[0], l, slot, true, lg);
        }
      } else {
        // ---- token split: four waves take interleaved tiles of the same 16 rows ----
        load_q<T, D, FUSED>(qf, p, sm.q, sm.u.cs, row0, R, q_first, g, lr, lg);
        stream_tiles<T, D>(kbase, vbase, p.pool, k0, k1, wave, kWaves, qf, o, m_run, l_run, lr, lg, c);
        float l = xor16_sum(l_run[0]);
        l = xor32_sum(l);
        if (lg == 0) {
          sm.m[wave][lr] = m_run[0];
          sm.l[wave][lr] = l;
        }
        __syncthreads();   // also retires every read of the cos/sin table before o reuses it
        {
          const float mall = fmaxf(fmaxf(sm.m[0][lr], sm.m[1][lr]), fmaxf(sm.m[2][lr], sm.m[3][lr]));
          const float msafe = mall == -INFINITY ? 0.f : mall;
          const float f = fast_exp2((m_run[0] - msafe) * c);
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const f32x4_t v = o[db][0] * f;
            *reinterpret_cast<float4*>(&sm.u.o[wave][lr][16 * db + 4 * lg]) = make_float4(v[0], v[1], v[2], v[3]);
          }
        }
        __syncthreads();
        const int64_t slot_base = static_cast<int64_t>(cidx) * p.Nt;
        for (int e = tid * 4; e < 16 * D; e += NT * 4) {
          const int rw = e / D, d = e - rw * D;
          const int row = row0 + rw;
          if (row >= R) continue;
          const int qi = sm.q[row / G];
          const int64_t slot = (slot_base + qi) * p.Hq + g * G + row % G;
          const float4 o0 = *reinterpret_cast<const float4*>(&sm.u.o[0][rw][d]);
          const float4 o1 = *reinterpret_cast<const float4*>(&sm.u.o[1][rw][d]);
          const float4 o2 = *reinterpret_cast<const float4*>(&sm.u.o[2][rw][d]);
          const float4 o3 = *reinterpret_cast<const float4*>(&sm.u.o[3][rw][d]);
          publish4(p.part_acc + slot * D + d, (o0.x + o1.x) + (o2.x + o3.x), (o0.y + o1.y) + (o2.y + o3.y),
                   (o0.z + o1.z) + (o2.z + o3.z), (o0.w + o1.w) + (o2.w + o3.w));
        }
        if (tid < 16) {
          const int row = row0 + tid;
          if (row < R) {
            const int qi = sm.q[row / G];
            const int64_t slot = (slot_base + qi) * p.Hq + g * G + row % G;
            const float mall = fmaxf(fmaxf(sm.m[0][tid], sm.m[1][tid]), fmaxf(sm.m[2][tid], sm.m[3][tid]));
            const float msafe = mall == -INFINITY ? 0.f : mall;
            float l2 = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) l2 += sm.l[w][tid] * fast_exp2((sm.m[w][tid] - msafe) * c);
            publish2(p.part_ml + 2 * slot, mall, l2);
          }
        }
      }
    }

    // ---- arrive at every segment group of the prompt; merge where last ----
    wait_vm();
    if (tid == 0) sm.n_merge = 0;
    __syncthreads();
    for (int j = tid; j < nseg; j += NT) {
      if (arrive(grp_cnt + j) == static_cast<uint32_t>(p.ctx_units_per_group))
        sm.merge_list[atomicAdd(&sm.n_merge, 1)] = j;
    }
    __syncthreads();
    const int nm = sm.n_merge;
    for (int k = 0; k < nm; ++k) {
      const int j = sm.merge_list[k];
      merge_segment_group<D, NW>(p, b, g, qa, qb, j, wave);
      if (tid == 0) clear(grp_cnt + j);
    }
    return;
  }

  // ============================= segment unit ================================
  const int j = r - p.ctx_units_per_group;
  if (j >= nseg) return;
  {
    const int i = p.shared ? qa + NW * j + wave : qa;
    const bool mine = (p.shared || wave == 0) && i < qb && p.active[i];
    const int s = mine ? usable_seg_len(p, i) : -1;
    if (mine && s < 0 && lane == 0)
      raise_flag(p.err_flag, (p.fused && p.seg_len[i] >= p.seg_cap) ? kFlagSegmentFull : kFlagBadLayout);
    if (s >= 0) {
      const int64_t sg = static_cast<int64_t>(i) * p.Hkv + g;
      T* skp = static_cast<T*>(p.seg_k) + sg * p.seg_cap * D;
      T* svp = static_cast<T*>(p.seg_vt) + sg * D * p.seg_cap;
      Frag qf[1][DS];
      int64_t k1;
      if (FUSED) {
        // append this step's key/value at slot s, rotated at ctx_len + s
        const int64_t pos = static_cast<int64_t>(ctx_len) + s;
        for (int jj = lane; jj < D / 2; jj += 64) {
          float cs, sn;
          rope_cos_sin(pos, p.inv_freq[jj], cs, sn);
          sm.u.seg_cs[wave][jj] = make_float2(cs, sn);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        const T* kn = static_cast<const T*>(p.k_new) + sg * D;
        const T* vn = static_cast<const T*>(p.v_new) + sg * D;
        for (int jj = lane; jj < D / 2; jj += 64) {
          const float2 cs = sm.u.seg_cs[wave][jj];
          float x, y;
          rope_rotate(to_f32<T>(kn[jj]), to_f32<T>(kn[jj + D / 2]), cs.x, cs.y, x, y);
          skp[static_cast<int64_t>(s) * D + jj] = from_f32<T>(x);
          skp[static_cast<int64_t>(s) * D + jj + D / 2] = from_f32<T>(y);
        }
        for (int d = lane; d < D; d += 64) svp[static_cast<int64_t>(d) * p.seg_cap + s] = vn[d];
        // rotated queries of the G heads of group g (B operand; written out if asked)
        if (lr < G) {
          const int h = g * G + lr;
          const T* qp = static_cast<const T*>(p.q_new) + (static_cast<int64_t>(i) * p.Hq + h) * D + lg * 8;
          f32x8_t x[DS];
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) x[ds] = M::to_f32v(M::load(qp + 32 * ds));
#pragma unroll
          for (int ds = 0; ds < DS / 2; ++ds)
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const float2 cs = sm.u.seg_cs[wave][lg * 8 + 32 * ds + u];
              float xr, yr;
              rope_rotate(x[ds][u], x[ds + DS / 2][u], cs.x, cs.y, xr, yr);
              x[ds][u] = xr;
              x[ds + DS / 2][u] = yr;
            }
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::from_f32(x[ds]);
          if (p.q_rot_out != nullptr) {
            T* qo = static_cast<T*>(p.q_rot_out) + (static_cast<int64_t>(i) * p.Hq + h) * D + lg * 8;
#pragma unroll
            for (int ds = 0; ds < DS; ++ds) store8<T>(qo + 32 * ds, qf[0][ds]);
          }
        } else {
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::zero();
        }
        // the wave reads back the slot it just wrote: its stores must have landed
        wait_vm();
        __builtin_amdgcn_wave_barrier();
        k1 = s + 1;
      } else {
        if (lr < G) {
          const T* qp = static_cast<const T*>(p.q_rot_in) + (static_cast<int64_t>(i) * p.Hq + g * G + lr) * D + lg * 8;
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::load(qp + 32 * ds);
        } else {
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) qf[0][ds] = M::zero();
        }
        k1 = s;
      }
      f32x4_t o[DB][1];
      float m_run[1] = {-INFINITY}, l_run[1] = {0.f};
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      stream_tiles<T, D>(skp, svp, p.seg_cap, 0, k1, 0, 1, qf, o, m_run, l_run, lr, lg, c);
      float l = xor16_sum(l_run[0]);
      l = xor32_sum(l);
      const int64_t slot = (static_cast<int64_t>(p.max_chunks) * p.Nt + i) * p.Hq + g * G + lr;
      publish_rows<D>(p, o, m_run[0], l, slot, lr < G, lg);
    }
  }
  wait_vm();
  __syncthreads();
  if (tid == 0) sm.n_merge = arrive(grp_cnt + j) == static_cast<uint32_t>(p.ctx_units_per_group) ? 1 : 0;
  __syncthreads();
  if (sm.n_merge) {
    merge_segment_group<D, NW>(p, b, g, qa, qb, j, wave);
    if (tid == 0) clear(grp_cnt + j);
  }
}

// ---------------------------------------------------------------------------
template <typename T, int D, int NW, bool RS>
static hipError_t launch_shape(int grid, const StepParams& p, hipStream_t s) {
  if (p.fused) decode_step_kernel<T, D, NW, RS, true><<<grid, 64 * NW, 0, s>>>(p);
  else decode_step_kernel<T, D, NW, RS, false><<<grid, 64 * NW, 0, s>>>(p);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_d(int waves, bool row_split, int grid, const StepParams& p, hipStream_t s) {
  if (!row_split) return launch_shape<T, D, kWaves, false>(grid, p, s);
  switch (waves) {
    case 2: return launch_shape<T, D, 2, true>(grid, p, s);
    case 4: return launch_shape<T, D, 4, true>(grid, p, s);
    default: return launch_shape<T, D, 8, true>(grid, p, s);
  }
}

hipError_t launch_step(int dtype, int waves, bool row_split, int grid, const StepParams& p, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  if (dtype == 0)
    return p.D == 64 ? launch_d<float, 64>(waves, row_split, grid, p, s)
                     : launch_d<float, 128>(waves, row_split, grid, p, s);
  return p.D == 64 ? launch_d<uint16_t, 64>(waves, row_split, grid, p, s)
                   : launch_d<uint16_t, 128>(waves, row_split, grid, p, s);
}

}  // namespace ippd
