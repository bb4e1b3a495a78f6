// Decode-step attention for IPPD on gfx950.
//
// Work is split into units, each one workgroup of four waves:
//   context unit  (kv head g, prompt b, chunk c, row group rg): the chunk's
//                 keys/values are streamed from HBM once for up to 16*RB query
//                 rows = (active question, head of group g) pairs of the whole
//                 prompt (IPPD, Sec. 4.3: K_c, V_c reused by all M_j queries).
//                 In the standard baseline a context unit serves one question.
//   segment unit  (kv head g, question i): the G rows of question i against its
//                 own question+answer segment (M_qtn, Sec. 4.1).
// Each unit leaves an unnormalised partial softmax state per row (max m, sum
// l, weighted values); the merge kernel combines a row's partials exactly
// (the split only regroups the sums of softmax(qK^T/sqrt(d_k))V, Sec. 4.2).
//
// Inside a unit the four waves take interleaved 32-token tiles.  Per tile:
//   S^T (tokens x rows) = K . Q^T     MFMA, A = 16 keys x 32 dims, B = Q^T
//   P^T = exp2(c*(S^T - m))           online softmax, per-row max across the
//                                     four 16-lane rows via permlane swaps
//   O^T (dims x rows) += V^T . P^T    MFMA, A = V^T rows (token-contiguous
//                                     thanks to the transposed value cache),
//                                     B = P^T straight from the S^T registers
// Key rows are assigned to MFMA rows so that lane row r of the S^T result
// holds 8 consecutive tokens, which is exactly the B layout PV needs; both
// K and V^T fragments are single 16-byte loads, no LDS staging.
#include <float.h>

#include "ippd_device.h"
#include "ippd_internal.h"

namespace ippd {

// ---------------------------------------------------------------------------
// MFMA operand traits: 8 k-elements per lane per 32-wide contraction step.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<uint16_t> {   // bf16: one v_mfma_f32_16x16x32_bf16
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
};

template <> struct Mfma<float> {      // fp32: eight v_mfma_f32_16x16x4_f32
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
};

// Per-prompt layout checks shared by the partials and merge kernels.
__device__ __forceinline__ bool prompt_layout_ok(const AttnParams& p, int b) {
  const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
  const int64_t off = p.ctx_off[b];
  const int len = p.ctx_len[b];
  return q0 >= 0 && q1 >= q0 && q1 <= p.Nt && q1 - q0 <= p.max_questions &&
         off >= 0 && (off & 7) == 0 && len >= 0 && len <= p.max_ctx_len && off + len <= p.pool;
}

// ---------------------------------------------------------------------------
// Partials kernel.
// ---------------------------------------------------------------------------
template <typename T, int D, int RB>
__global__ __launch_bounds__(256) void attn_partials_kernel(AttnParams p) {
  using M = Mfma<T>;
  using Frag = typename M::Frag;
  constexpr int DS = D / 32;      // 32-wide contraction steps over the head dim
  constexpr int DB = D / 16;      // 16-dim blocks of the output
  constexpr int RW = RB * 16;     // query rows per unit
  constexpr int OSTRIDE = D + 4;  // padded LDS row of the cross-wave merge

  __shared__ float s_o[4][RW][OSTRIDE];
  __shared__ float s_m[4][RW];
  __shared__ float s_l[4][RW];
  __shared__ int s_q[kMaxQuestionsPerPrompt];
  __shared__ int s_cnt[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  // ---- unit decode: consecutive units share an XCD (8 round-robin slices) ----
  const int per_xcd = p.grid >> 3;
  const int u = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (u >= p.n_units) return;
  const int g = u / p.units_per_g;
  const int r = u - g * p.units_per_g;
  const int G = p.G;

  const T* kbase;      // row of token 0 of this key source
  const T* vbase;      // V^T: row d=0, token 0
  int64_t vstride;     // tokens per V^T row
  int64_t k0, k1;      // token range of this unit
  int b, rg = 0, n_act, slot_chunk;
  bool is_seg = false;
  int seg_q = -1;

  if (r < p.ctx_per_g) {
    int c;
    if (p.shared) {
      b = r / (p.max_chunks * p.nrg);
      const int rem = r - b * p.max_chunks * p.nrg;
      c = rem / p.nrg;
      rg = rem - c * p.nrg;
    } else {
      seg_q = r / p.max_chunks;          // the single question of this unit
      c = r - seg_q * p.max_chunks;
      if (!p.active[seg_q]) return;
      b = prompt_of(p.q_start, p.B, seg_q);
    }
    if (!prompt_layout_ok(p, b)) {
      if (tid == 0 && c == 0 && rg == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
    const int64_t off = p.ctx_off[b];
    const int len = p.ctx_len[b];
    if (static_cast<int64_t>(c) * p.chunk >= len) return;
    k0 = off + static_cast<int64_t>(c) * p.chunk;
    k1 = min(k0 + p.chunk, off + len);
    kbase = static_cast<const T*>(p.ctx_k) + static_cast<int64_t>(g) * p.pool * D;
    vbase = static_cast<const T*>(p.ctx_vt) + static_cast<int64_t>(g) * D * p.pool;
    vstride = p.pool;
    slot_chunk = c;
  } else {
    seg_q = r - p.ctx_per_g;
    if (!p.active[seg_q]) return;
    b = prompt_of(p.q_start, p.B, seg_q);
    const int s = p.seg_len[seg_q];
    if (s < 1 || s > p.seg_cap) {
      if (tid == 0 && g == 0) raise_flag(p.err_flag, kFlagBadLayout);
      return;
    }
    is_seg = true;
    k0 = 0;
    k1 = s;
    const int64_t sg = static_cast<int64_t>(seg_q) * p.Hkv + g;
    kbase = static_cast<const T*>(p.seg_k) + sg * p.seg_cap * D;
    vbase = static_cast<const T*>(p.seg_vt) + sg * D * p.seg_cap;
    vstride = p.seg_cap;
    slot_chunk = p.max_chunks;
  }

  // ---- rows: (active question, head of group g), compacted ----
  if (p.shared && !is_seg) {
    const int q0 = p.q_start[b], nq = p.q_start[b + 1] - q0;
    int base_cnt = 0;
    for (int t0 = 0; t0 < nq; t0 += 256) {
      const int t = t0 + tid;
      const bool a = t < nq && p.active[q0 + t];
      const unsigned long long ball = __ballot(a);
      const int before = __popcll(ball & ((1ull << lane) - 1ull));
      if (lane == 0) s_cnt[wave] = __popcll(ball);
      __syncthreads();
      int wbase = base_cnt;
      for (int w = 0; w < wave; ++w) wbase += s_cnt[w];
      if (a) s_q[wbase + before] = q0 + t;
      base_cnt += s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
      __syncthreads();
    }
    n_act = base_cnt;
  } else {
    if (tid == 0) s_q[0] = seg_q;
    __syncthreads();
    n_act = 1;
  }
  const int R = n_act * G;
  const int row0 = rg * RW;
  if (row0 >= R) return;

  // ---- Q^T fragments of this unit's rows (B operand) ----
  Frag qf[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = row0 + rb * 16 + lr;
    if (row < R) {
      const int qi = s_q[row / G];
      const int h = g * G + row % G;
      const T* qp = static_cast<const T*>(p.q) + (static_cast<int64_t>(qi) * p.Hq + h) * D + lg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = M::load(qp + 32 * ds);
    } else {
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) qf[rb][ds] = M::zero();
    }
  }

  const float c = p.c;
  f32x4_t o[DB][RB];
  float m_run[RB], l_run[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  const int ntiles = static_cast<int>((k1 - k0 + 31) >> 5);
  for (int tile = wave; tile < ntiles; tile += 4) {
    const int64_t t0 = k0 + static_cast<int64_t>(tile) * 32;
    // K fragments: MFMA row lr of key block kb <- token t0 + 8*(lr/4) + 4*kb + lr%4
    Frag kf[2][DS];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      int64_t tk = t0 + 8 * (lr >> 2) + 4 * kb + (lr & 3);
      tk = tk < k1 ? tk : k1 - 1;
      const T* kp = kbase + tk * D + lg * 8;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[kb][ds] = M::load(kp + 32 * ds);
    }
    // V^T fragments: dim 16*db + lr, tokens t0 + 8*lg .. +7
    Frag vf[DB];
    const int64_t tv = t0 + 8 * lg;
    if (tv < k1) {
      const T* vp = vbase + static_cast<int64_t>(lr) * vstride + tv;
#pragma unroll
      for (int db = 0; db < DB; ++db) vf[db] = M::load(vp + static_cast<int64_t>(16 * db) * vstride);
      if (tv + 8 > k1) {
        const int keep = static_cast<int>(k1 - tv);
#pragma unroll
        for (int db = 0; db < DB; ++db) vf[db] = M::keep_first(vf[db], keep);
      }
    } else {
#pragma unroll
      for (int db = 0; db < DB; ++db) vf[db] = M::zero();
    }

    // S^T = K Q^T
    f32x4_t sc[2][RB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) acc = M::mma(kf[kb][ds], qf[rb][ds], acc);
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

    // online softmax per row, P^T fragments
    Frag pf[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
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
      float ps = ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
      l_run[rb] = l_run[rb] * alpha + ps;
      m_run[rb] = m_new;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][rb] *= alpha;
      pf[rb] = M::from_f32(pv);
    }
    // O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) o[db][rb] = M::mma(vf[db], pf[rb], o[db][rb]);
  }

  // ---- combine the four waves (rows lr of each block; sums over the lane rows) ----
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    float l = xor16_sum(l_run[rb]);
    l = xor32_sum(l);
    if (lg == 0) {
      s_m[wave][rb * 16 + lr] = m_run[rb];
      s_l[wave][rb * 16 + lr] = l;
    }
  }
  __syncthreads();
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int rw = rb * 16 + lr;
    const float mall = fmaxf(fmaxf(s_m[0][rw], s_m[1][rw]), fmaxf(s_m[2][rw], s_m[3][rw]));
    const float msafe = mall == -INFINITY ? 0.f : mall;
    const float f = fast_exp2((m_run[rb] - msafe) * c);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const f32x4_t v = o[db][rb] * f;
      *reinterpret_cast<float4*>(&s_o[wave][rw][16 * db + 4 * lg]) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
  __syncthreads();

  // ---- write the unit's partial state ----
  const int64_t slot_base = static_cast<int64_t>(slot_chunk) * p.Nt;
  for (int e = tid; e < RW * D; e += 256) {
    const int rw = e / D, d = e - rw * D;
    const int row = row0 + rw;
    if (row >= R) continue;
    const int qi = s_q[row / G];
    const int h = g * G + row % G;
    const int64_t slot = (slot_base + qi) * p.Hq + h;
    p.part_acc[slot * D + d] = (s_o[0][rw][d] + s_o[1][rw][d]) + (s_o[2][rw][d] + s_o[3][rw][d]);
  }
  if (tid < RW) {
    const int rw = tid, row = row0 + rw;
    if (row < R) {
      const int qi = s_q[row / G];
      const int h = g * G + row % G;
      const int64_t slot = (slot_base + qi) * p.Hq + h;
      const float mall = fmaxf(fmaxf(s_m[0][rw], s_m[1][rw]), fmaxf(s_m[2][rw], s_m[3][rw]));
      const float msafe = mall == -INFINITY ? 0.f : mall;
      float l = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) l += s_l[w][rw] * fast_exp2((s_m[w][rw] - msafe) * c);
      p.part_ml[2 * slot] = mall;
      p.part_ml[2 * slot + 1] = l;
    }
  }
}

// ---------------------------------------------------------------------------
// Merge kernel: one wave per (question, head) row.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void attn_merge_kernel(AttnParams p) {
  constexpr int PER = D / 64;
  const int row = blockIdx.x;
  const int i = row / p.Hq, h = row - i * p.Hq;
  if (!p.active[i]) return;
  const int b = prompt_of(p.q_start, p.B, i);
  if (!prompt_layout_ok(p, b)) return;
  const int s = p.seg_len[i];
  if (s < 1 || s > p.seg_cap) return;
  const int len = p.ctx_len[b];
  const int nc = (len + p.chunk - 1) / p.chunk;
  if (nc > p.max_chunks) {
    if (threadIdx.x == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  const float c = p.c;
  const int lane = threadIdx.x;
  float mx = -INFINITY;
  for (int k = 0; k <= nc; ++k) {
    const int ck = k < nc ? k : p.max_chunks;
    const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
    mx = fmaxf(mx, p.part_ml[2 * slot]);
  }
  const float ms = mx == -INFINITY ? 0.f : mx;
  float l = 0.f;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int k = 0; k <= nc; ++k) {
    const int ck = k < nc ? k : p.max_chunks;
    const int64_t slot = (static_cast<int64_t>(ck) * p.Nt + i) * p.Hq + h;
    const float w = fast_exp2((p.part_ml[2 * slot] - ms) * c);
    l += w * p.part_ml[2 * slot + 1];
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += w * p.part_acc[slot * D + lane + 64 * e];
  }
  const float inv = 1.f / l;
  float* op = p.out + static_cast<int64_t>(row) * D;
#pragma unroll
  for (int e = 0; e < PER; ++e) op[lane + 64 * e] = acc[e] * inv;
  if (p.lse != nullptr && lane == 0) p.lse[row] = ms * p.scale + logf(l);
}

// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t launch_typed(int rb, const AttnParams& p, hipStream_t s) {
  if (p.grid > 0) {
    switch (rb) {
      case 1: attn_partials_kernel<T, D, 1><<<p.grid, 256, 0, s>>>(p); break;
      case 2: attn_partials_kernel<T, D, 2><<<p.grid, 256, 0, s>>>(p); break;
      default: attn_partials_kernel<T, D, 4><<<p.grid, 256, 0, s>>>(p); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t rows = static_cast<int64_t>(p.Nt) * p.Hq;
  if (rows > 0) attn_merge_kernel<D><<<static_cast<unsigned>(rows), 64, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, int rb, const AttnParams& p, hipStream_t s) {
  if (dtype == 0) return p.D == 64 ? launch_typed<float, 64>(rb, p, s) : launch_typed<float, 128>(rb, p, s);
  return p.D == 64 ? launch_typed<uint16_t, 64>(rb, p, s) : launch_typed<uint16_t, 128>(rb, p, s);
}

}  // namespace ippd
