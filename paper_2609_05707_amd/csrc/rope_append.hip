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
// Decode-step append: one workgroup per question.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void append_kernel(AppendParams p) {
  __shared__ float2 s_cs[kMaxHalfDim];
  const int i = blockIdx.x;
  if (i >= p.Nt || !p.active[i]) return;
  const int b = prompt_of(p.q_start, p.B, i);
  const int s = p.seg_len[i];
  if (s < 0 || s >= p.seg_cap) {
    if (threadIdx.x == 0) raise_flag(p.err_flag, s >= p.seg_cap ? kFlagSegmentFull : kFlagBadLayout);
    return;
  }
  const int D = p.D, half = D / 2;
  const int64_t pos = instr_pos_base(p.instr_start, p.instr_len, p.S, b) + p.ctx_len[b] + s;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    float c, sn;
    rope_cos_sin(pos, p.inv_freq[j], c, sn);
    s_cs[j] = make_float2(c, sn);
  }
  __syncthreads();

  const T* __restrict__ qn = static_cast<const T*>(p.q_new);
  const T* __restrict__ kn = static_cast<const T*>(p.k_new);
  const T* __restrict__ vn = static_cast<const T*>(p.v_new);
  T* __restrict__ qr = static_cast<T*>(p.q_rot);
  T* __restrict__ sk = static_cast<T*>(p.seg_k);
  T* __restrict__ svt = static_cast<T*>(p.seg_vt);
  const int oct = half / 8;                    // groups of 8 pairs per head
  const int heads = p.Hq + p.Hkv;
  for (int e = threadIdx.x; e < heads * oct; e += blockDim.x) {
    const int hh = e / oct, j0 = (e - hh * oct) * 8;
    if (hh < p.Hq) {
      const int64_t off = (static_cast<int64_t>(i) * p.Hq + hh) * D;
      rotate8<T>(qn + off, qr + off, j0, half, s_cs);
    } else {
      const int g = hh - p.Hq;
      const int64_t src = (static_cast<int64_t>(i) * p.Hkv + g) * D;
      const int64_t dst = ((static_cast<int64_t>(i) * p.Hkv + g) * p.seg_cap + s) * D;
      rotate8<T>(kn + src, sk + dst, j0, half, s_cs);
    }
  }
  for (int e = threadIdx.x; e < p.Hkv * D; e += blockDim.x) {
    const int g = e / D, d = e - g * D;
    const int64_t src = (static_cast<int64_t>(i) * p.Hkv + g) * D + d;
    svt[vt_index(static_cast<int64_t>(i) * p.Hkv + g, p.seg_cap, D, s, d)] = vn[src];
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

hipError_t launch_append(int dtype, const AppendParams& p, hipStream_t s) {
  if (p.Nt == 0) return hipSuccess;
  if (dtype == 0) append_kernel<float><<<p.Nt, 256, 0, s>>>(p);
  else append_kernel<uint16_t><<<p.Nt, 256, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace ippd
