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

// cos/sin of pos * theta.  The angle is formed and reduced to [-pi, pi] in
// fp64 (2*pi split hi + lo), then evaluated with fp32 sincos: the result is
// accurate to a few 1e-7 for any position, where an fp32 angle would be off
// by ~pos * 6e-8 rad.
__device__ __forceinline__ void rope_cos_sin(int64_t pos, double theta, float& c, float& s) {
  const double ang = static_cast<double>(pos) * theta;
  const double k = rint(ang * 0.15915494309189535);
  const double r = fma(-k, 6.283185307179586, ang) - k * 2.4492935982947064e-16;
  sincosf(static_cast<float>(r), &s, &c);
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

// Prompt owning question i: the largest b with q_start[b] <= i (q_start has B+1 entries).
__device__ __forceinline__ int prompt_of(const int32_t* q_start, int B, int i) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (q_start[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ void raise_flag(int32_t* err_flag, int bits) {
  atomicOr(reinterpret_cast<int*>(err_flag), bits);
}

}  // namespace ippd
