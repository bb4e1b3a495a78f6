// Device-side helpers shared by the IPPD kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ippd {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8_t __attribute__((ext_vector_type(8)));

constexpr int kFlagSegmentFull = 1;
constexpr int kFlagBadLayout = 2;

// bf16 storage is handled as raw 16-bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even float -> bf16 (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_to_f32(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f32_to_bf16(x); }

// cos/sin of pos * theta.  The angle is formed in fp64 and reduced to
// r in [-pi/4, pi/4] about the nearest multiple k*pi/2 (pi/2 split hi + lo),
// so the reduction is exact to ~1e-16 for any position; sin r and cos r then
// come from their Taylor series in fp32 (terms to r^9 and r^10: truncation
// below 2e-9 on that interval) and k mod 4 picks and signs them.  Accurate to
// about 1e-7 everywhere, where an fp32 angle would be off by ~pos * 6e-8 rad.
__device__ __forceinline__ void rope_cos_sin(int64_t pos, double theta, float& c, float& s) {
  const double ang = static_cast<double>(pos) * theta;
  const double k = rint(ang * 0.63661977236758134);                          // 2/pi
  const double r = fma(-k, 1.5707963267948966, ang) - k * 6.123233995736766e-17;
  const float x = static_cast<float>(r), x2 = x * x;
  float sp = fmaf(x2, 2.75573192e-6f, -1.98412698e-4f);     //  1/9!, -1/7!
  sp = fmaf(x2, sp, 8.33333333e-3f);                        //  1/5!
  sp = fmaf(x2, sp, -1.66666667e-1f);                       // -1/3!
  const float sn = fmaf(x * x2, sp, x);
  float cp = fmaf(x2, -2.75573192e-7f, 2.48015873e-5f);     // -1/10!, 1/8!
  cp = fmaf(x2, cp, -1.38888889e-3f);                       // -1/6!
  cp = fmaf(x2, cp, 4.16666667e-2f);                        //  1/4!
  cp = fmaf(x2, cp, -0.5f);                                 // -1/2!
  const float cs = fmaf(x2, cp, 1.0f);
  const int q = static_cast<int>(static_cast<int64_t>(k) & 3);   // angle = r + q*pi/2
  const float c0 = (q & 1) ? sn : cs, s0 = (q & 1) ? cs : sn;
  c = ((q + 1) & 2) ? -c0 : c0;                             // q = 1, 2: cos < 0 side
  s = (q & 2) ? -s0 : s0;                                   // q = 2, 3: sin < 0 side
}

// Rotate one pair (a, b) = (x_j, x_{j+D/2}) by (c, s) = (cos, sin); written with
// explicit fmaf so every call site rounds identically.
__device__ __forceinline__ void rope_rotate(float a, float b, float c, float s, float& x, float& y) {
  x = fmaf(a, c, -(b * s));
  y = fmaf(b, c, a * s);
}

// Butterfly partners across the four 16-lane rows of a wave64, via the gfx950
// permlane swaps.  After swapping a value with itself, the two results hold
// {own value, partner value} in every lane, so an associative op over them is
// the pairwise reduction.
__device__ __forceinline__ float xor16_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Whether the predicate holds in any active lane.  Built on the ballot
// intrinsic, whose result the compiler knows to be wave-uniform, so that a
// branch on it stays a scalar branch and the values computed under it stay
// in scalar registers.
__device__ __forceinline__ bool wave_any(bool pred) { return __builtin_amdgcn_ballot_w64(pred) != 0; }

// Values are cached transposed in 8-token column blocks: for a region of n
// tokens (n a multiple of 8), token t of dimension d sits at
//   region * n * D + (t / 8) * 8 * D + d * 8 + t % 8,
// so the 8 tokens of one dimension are 16 (bf16) or 32 (fp32) contiguous
// bytes and a 32-token tile of all D dimensions is one contiguous block.
__device__ __forceinline__ int64_t vt_index(int64_t region, int64_t n, int D, int64_t t, int d) {
  return region * n * D + (t >> 3) * 8 * D + d * 8 + (t & 7);
}

// Prompt owning question i: the largest b with q_start[b] <= i (q_start has B+1 entries).
__device__ __forceinline__ int prompt_of(const int32_t* q_start, int B, int i) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (q_start[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Instruction of prompt b in a two-level batch: the largest s in [0, S) with
// instr_start[s] <= b.
__device__ __forceinline__ int instr_of_prompt(const int32_t* instr_start, int S, int b) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (instr_start[mid] <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Virtual position of prompt b's first context token: the length of the
// instruction it sits behind in a two-level batch, 0 without an instruction level.
__device__ __forceinline__ int64_t instr_pos_base(const int32_t* instr_start, const int32_t* instr_len, int S, int b) {
  return S > 0 ? instr_len[instr_of_prompt(instr_start, S, b)] : 0;
}

__device__ __forceinline__ void raise_flag(int32_t* err_flag, int bits) {
  atomicOr(reinterpret_cast<int*>(err_flag), bits);
}

}  // namespace ippd
