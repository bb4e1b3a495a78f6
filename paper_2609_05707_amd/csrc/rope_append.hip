// Rotary embedding at virtual positions: decode-step append and cache loaders.
//
// Positions follow the virtual-position rule of Sec. 4.1: a context token t
// sits at t (instruction folded into the context), segment slot t of a
// question of prompt b at ctx_len[b] + t, and the token fed at a decode step
// at ctx_len[b] + seg_len[i]; behind an instruction of a two-level batch all
// of them move up by its length.  theta_j = base^(-2j/D) comes from the host in
// fp64; cos/sin use the fp64-reduced angle (rope_cos_sin).
#include "ippd_device.h"
#include "ippd_internal.h"

namespace ippd {

// Rotate 8 consecutive pairs (x[j], x[j + D/2]) for j = j0..j0+7.
template <typename T>
__device__ __forceinline__ void rotate8(const T* __restrict__ src, T* __restrict__ dst, int j0, int half,
                                        const float2* cs) {
  float a[8], bb[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) { a[u] = to_f32<T>(src[j0 + u]); bb[u] = to_f32<T>(src[j0 + half + u]); }
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float2 c = cs[j0 + u];
    float x, y;
    rope_rotate(a[u], bb[u], c.x, c.y, x, y);
    dst[j0 + u] = from_f32<T>(x);
    dst[j0 + half + u] = from_f32<T>(y);
  }
}

// ---------------------------------------------------------------------------
// Decode-step append: one workgroup per question, one 16-byte vector per
// thread and item.  Item e of question i is
//   e < Hq*QP                 pairs [v*VE, v*VE + VE) of query head e / QP,
//                             rotated into q_rot (QP = D/2 / VE pair vectors),
//   e < (Hq + Hkv)*QP         the same pairs of key head (e - Hq*QP) / QP,
//                             rotated into segment slot s of (i, head),
//   e < (Hq + Hkv)*QP + Hkv*VG  dims [v*VE, v*VE + VE) of value head (e - ..) / VG,
//                             written into slot s of the transposed value cache
// (VE = 16 bytes / element size, VG = D / VE).  Every load is issued before
// the question's state is known; the prompt is found with one ballot over
// the prompts (lane l reads prompt l), so a question costs one round trip of
// loads and then its stores.  The D/2 (cos, sin) pairs of the question's
// position are evaluated once, into LDS; rotations use the same cos/sin and
// rounding as the fused decode step, so both give identical bits.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(1024) void append_kernel(AppendParams p) {
  constexpr int VE = 16 / static_cast<int>(sizeof(T));
  typedef T vec_t __attribute__((ext_vector_type(VE)));
  const int i = blockIdx.x;
  const int D = p.D, half = D / 2;
  const int QP = half / VE, VG = D / VE;
  const int nq = p.Hq * QP, nk = p.Hkv * QP, nitems = nq + nk + p.Hkv * VG;
  const int lane = threadIdx.x & 63;
  // the thread's items (a block covers a question in one pass when it can)
  constexpr int kMaxPass = 2;
  vec_t lo[kMaxPass], hi[kMaxPass];
  // every head of the question turns by the same D/2 angles: thread j < D/2
  // evaluates pair j's once into LDS (its frequency read first, with the
  // other loads, so that it shares their round trip)
  __shared__ float2 rot[kMaxHalfDim];
  const double theta = threadIdx.x < static_cast<unsigned>(half) ? p.inv_freq[threadIdx.x] : 0.0;
  // the question's state, and the first 64 prompts' question ends and
  // context lengths for the prompt lookup below, all loaded before any wait
  const bool act = p.active[i] != 0;
  const int s = p.seg_len[i];
  const int bl0 = lane < p.B ? lane : p.B - 1;
  const int q10 = p.q_start[bl0 + 1], cl0 = p.ctx_len[bl0];
  const T* __restrict__ qn = static_cast<const T*>(p.q_new);
  const T* __restrict__ kn = static_cast<const T*>(p.k_new);
  const T* __restrict__ vn = static_cast<const T*>(p.v_new);
  // one load site per pass (a value item reads its vector twice): loads
  // issued from separate branches into the same registers would each wait
  // for the one before
#pragma unroll
  for (int r = 0; r < kMaxPass; ++r) {
    const int e = threadIdx.x + r * blockDim.x;
    const T* src;
    int hoff;
    if (e < nq + nk) {
      const bool isq = e < nq;
      const int ee = isq ? e : e - nq;
      src = (isq ? qn + (static_cast<int64_t>(i) * p.Hq + ee / QP) * D
                 : kn + (static_cast<int64_t>(i) * p.Hkv + ee / QP) * D) + (ee % QP) * VE;
      hoff = half;
    } else {
      const int ev = e - nq - nk;
      src = vn + (static_cast<int64_t>(i) * p.Hkv + ev / VG) * D + (ev % VG) * VE;
      hoff = 0;
    }
    if (e < nitems) {
      lo[r] = *reinterpret_cast<const vec_t*>(src);
      hi[r] = *reinterpret_cast<const vec_t*>(src + hoff);
    }
  }
  // the question's prompt: the number of prompts whose questions all precede
  // i (windows of 64 prompts; the first was loaded above)
  int n = __popcll(__ballot(lane < p.B && q10 <= i));
  int b = n, len = __shfl(cl0, n < 64 ? n : 63, 64);
  for (int b0 = 64; n == 64 && b0 < p.B; b0 += 64) {
    const int bb = b0 + lane;
    const int bl = bb < p.B ? bb : p.B - 1;
    const int q1 = p.q_start[bl + 1], cl = p.ctx_len[bl];
    n = __popcll(__ballot(bb < p.B && q1 <= i));
    b = b0 + n;
    len = __shfl(cl, n < 64 ? n : 63, 64);
  }
  if (b >= p.B) {                                  // i past the last prompt's questions
    b = p.B - 1;
    len = p.ctx_len[b];
  }
  if (!act) return;
  if (s < 0 || s >= p.seg_cap) {
    if (threadIdx.x == 0) raise_flag(p.err_flag, s >= p.seg_cap ? kFlagSegmentFull : kFlagBadLayout);
    return;
  }
  const int64_t pos = instr_pos_base(p.instr_start, p.instr_len, p.S, b) + len + s;
  if (threadIdx.x < static_cast<unsigned>(half)) {
    float c, sn;
    rope_cos_sin(pos, theta, c, sn);
    rot[threadIdx.x] = make_float2(c, sn);
  }
  __syncthreads();                                 // act and s are the question's: every thread is here
  T* __restrict__ qr = static_cast<T*>(p.q_rot);
  T* __restrict__ sk = static_cast<T*>(p.seg_k);
  T* __restrict__ svt = static_cast<T*>(p.seg_vt);
#pragma unroll
  for (int r = 0; r < kMaxPass; ++r) {
    const int e = threadIdx.x + r * blockDim.x;
    if (e < nq + nk) {
      const bool isq = e < nq;
      const int ee = isq ? e : e - nq;
      const int j0 = (ee % QP) * VE;
      vec_t x, y;
#pragma unroll
      for (int u = 0; u < VE; ++u) {
        const float2 cs = rot[j0 + u];
        float xr, yr;
        rope_rotate(to_f32<T>(lo[r][u]), to_f32<T>(hi[r][u]), cs.x, cs.y, xr, yr);
        x[u] = from_f32<T>(xr);
        y[u] = from_f32<T>(yr);
      }
      T* dst = isq ? qr + (static_cast<int64_t>(i) * p.Hq + ee / QP) * D + j0
                   : sk + ((static_cast<int64_t>(i) * p.Hkv + ee / QP) * p.seg_cap + s) * D + j0;
      *reinterpret_cast<vec_t*>(dst) = x;
      *reinterpret_cast<vec_t*>(dst + half) = y;
    } else if (e < nitems) {
      const int ev = e - nq - nk;
      const int g = ev / VG, d0 = (ev % VG) * VE;
#pragma unroll
      for (int u = 0; u < VE; ++u)
        svt[vt_index(static_cast<int64_t>(i) * p.Hkv + g, p.seg_cap, D, s, d0 + u)] = lo[r][u];
    }
  }
  __syncthreads();   // every thread has read seg_len[i] before it moves
  if (threadIdx.x == 0) p.seg_len[i] = s + 1;
}

// ---------------------------------------------------------------------------
// Context loader: workgroup per (prompt b, 64-token tile, kv head g).
// ---------------------------------------------------------------------------
constexpr int kLoadTile = 64;

template <typename T>
__global__ __launch_bounds__(256) void load_context_kernel(LoadContextParams p, int tiles_per_prompt) {
  __shared__ T s_v[kLoadTile][128 + 1];
  const int g = blockIdx.y;
  const int b = blockIdx.x / tiles_per_prompt;
  const int tile = blockIdx.x - b * tiles_per_prompt;
  const int64_t off = p.ctx_off[b];
  const int len = p.ctx_len[b];
  if (off < 0 || (off & 7) || len < 0 || len > p.max_ctx_len || off + len > p.pool) {
    if (threadIdx.x == 0 && tile == 0 && g == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  const int t0 = tile * kLoadTile;
  if (t0 >= len) return;
  const int nt = min(kLoadTile, len - t0);
  const int D = p.D, half = D / 2;
  const int64_t base_pos = instr_pos_base(p.instr_start, p.instr_len, p.S, b);
  const T* __restrict__ kr = static_cast<const T*>(p.k_raw);
  const T* __restrict__ vr = static_cast<const T*>(p.v_raw);
  T* __restrict__ ck = static_cast<T*>(p.ctx_k);
  T* __restrict__ cvt = static_cast<T*>(p.ctx_vt);
  for (int e = threadIdx.x; e < nt * half; e += blockDim.x) {
    const int tt = e / half, j = e - tt * half;
    const int t = t0 + tt;
    float c, sn;
    rope_cos_sin(base_pos + t, p.inv_freq[j], c, sn);
    const int64_t src = ((off + t) * p.Hkv + g) * D;
    const int64_t dst = (static_cast<int64_t>(g) * p.pool + off + t) * D;
    float x, y;
    rope_rotate(to_f32<T>(kr[src + j]), to_f32<T>(kr[src + j + half]), c, sn, x, y);
    ck[dst + j] = from_f32<T>(x);
    ck[dst + j + half] = from_f32<T>(y);
  }
  // values: transpose a [tokens][D] tile into 8-token column blocks through LDS
  for (int e = threadIdx.x; e < nt * D; e += blockDim.x) {
    const int tt = e / D, d = e - tt * D;
    s_v[tt][d] = vr[((off + t0 + tt) * p.Hkv + g) * D + d];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < nt * D; e += blockDim.x) {
    const int d = e / nt, tt = e - d * nt;
    cvt[vt_index(g, p.pool, D, off + t0 + tt, d)] = s_v[tt][d];
  }
}

// ---------------------------------------------------------------------------
// Segment loader: workgroup per (question i, 64-slot tile, kv head g).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void load_segments_kernel(LoadSegmentsParams p, int tiles) {
  __shared__ T s_v[kLoadTile][128 + 1];
  const int g = blockIdx.y;
  const int i = blockIdx.x / tiles;
  const int tile = blockIdx.x - i * tiles;
  const int n = p.init_len[i];
  if (n < 0 || n > p.seg_cap) {
    if (threadIdx.x == 0 && tile == 0 && g == 0) raise_flag(p.err_flag, kFlagBadLayout);
    return;
  }
  const int b = prompt_of(p.q_start, p.B, i);
  if (threadIdx.x == 0 && tile == 0 && g == 0) p.seg_len[i] = n;
  const int t0 = tile * kLoadTile;
  if (t0 >= n) return;
  const int nt = min(kLoadTile, n - t0);
  const int D = p.D, half = D / 2;
  const int64_t base_pos = instr_pos_base(p.instr_start, p.instr_len, p.S, b) + p.ctx_len[b];
  const T* __restrict__ kr = static_cast<const T*>(p.k_raw);
  const T* __restrict__ vr = static_cast<const T*>(p.v_raw);
  T* __restrict__ sk = static_cast<T*>(p.seg_k);
  T* __restrict__ svt = static_cast<T*>(p.seg_vt);
  for (int e = threadIdx.x; e < nt * half; e += blockDim.x) {
    const int tt = e / half, j = e - tt * half;
    const int t = t0 + tt;
    float c, sn;
    rope_cos_sin(base_pos + t, p.inv_freq[j], c, sn);
    const int64_t src = ((static_cast<int64_t>(i) * p.seg_cap + t) * p.Hkv + g) * D;
    const int64_t dst = ((static_cast<int64_t>(i) * p.Hkv + g) * p.seg_cap + t) * D;
    float x, y;
    rope_rotate(to_f32<T>(kr[src + j]), to_f32<T>(kr[src + j + half]), c, sn, x, y);
    sk[dst + j] = from_f32<T>(x);
    sk[dst + j + half] = from_f32<T>(y);
  }
  for (int e = threadIdx.x; e < nt * D; e += blockDim.x) {
    const int tt = e / D, d = e - tt * D;
    s_v[tt][d] = vr[((static_cast<int64_t>(i) * p.seg_cap + t0 + tt) * p.Hkv + g) * D + d];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < nt * D; e += blockDim.x) {
    const int d = e / nt, tt = e - d * nt;
    svt[vt_index(static_cast<int64_t>(i) * p.Hkv + g, p.seg_cap, D, t0 + tt, d)] = s_v[tt][d];
  }
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
hipError_t launch_load_context(int dtype, const LoadContextParams& p, hipStream_t s) {
  const int tiles = (p.max_ctx_len + kLoadTile - 1) / kLoadTile;
  if (tiles == 0 || p.B == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(p.B) * tiles, p.Hkv);
  if (dtype == 0) load_context_kernel<float><<<grid, 256, 0, s>>>(p, tiles);
  else load_context_kernel<uint16_t><<<grid, 256, 0, s>>>(p, tiles);
  return hipGetLastError();
}

hipError_t launch_load_segments(int dtype, const LoadSegmentsParams& p, hipStream_t s) {
  const int tiles = (p.seg_cap + kLoadTile - 1) / kLoadTile;
  if (p.Nt == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(p.Nt) * tiles, p.Hkv);
  if (dtype == 0) load_segments_kernel<float><<<grid, 256, 0, s>>>(p, tiles);
  else load_segments_kernel<uint16_t><<<grid, 256, 0, s>>>(p, tiles);
  return hipGetLastError();
}

// One workgroup per question, as many threads (whole waves, at most 1024) as
// the question has items, or half of them when that exceeds 1024 (each
// thread then takes two: the kernel covers at most two passes).
hipError_t launch_append(int dtype, const AppendParams& p, hipStream_t s) {
  if (p.Nt == 0) return hipSuccess;
  const int ve = dtype == 0 ? 4 : 8;
  const int items = (p.Hq + p.Hkv) * (p.D / 2 / ve) + p.Hkv * (p.D / ve);
  int threads = (items + 63) / 64 * 64;
  if (threads > 1024) threads = ((items + 1) / 2 + 63) / 64 * 64;
  if (threads > 1024) return hipErrorInvalidValue;
  if (dtype == 0) append_kernel<float><<<p.Nt, threads, 0, s>>>(p);
  else append_kernel<uint16_t><<<p.Nt, threads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace ippd
