// Streaming ceiling of the decode kernels' context path on one MI355X.
//
// A standalone measurement program (not part of libippd.so).  It streams the
// context K/V cache of the 32-layer workload's shape (8 prompts x 8 kv heads
// x 8192 tokens, bf16, D = 128: 268 MB per layer) the way the context units
// do, with no attention arithmetic, and times it.  The gap between what this
// reaches and the decode kernels' own rate is what the tile products, the
// unit start-up, the segment units and the merge cost; the gap between this
// and 8 TB/s is what the memory system gives this access pattern.
//
//   ring   one unit per compute unit: eight waves, the nine-stage LDS ring of
//          the decode units, 2048-token chunks (64 tiles), the same LDS-DMA
//          issue (issue_tile with the swizzled key rows and 8-token value
//          blocks), the same waits and one barrier per tile
//   loads  the same bytes read by a grid-stride loop of 16-byte register
//          loads (eight in flight per thread), for comparison
//
// Each kernel runs over a rotation of eight layers' caches (2.1 GB), so no
// launch finds its bytes in the 256 MB last-level cache; time per launch from
// HIP events over 24 launches after 4 warm-up launches.
//
// Usage: stream_ceiling            (built next to libippd.so by build.py)
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <vector>

#include "tile_attend.h"

namespace {

using T = uint16_t;
constexpr int D = 128, NW = 8, NS = 9;
constexpr int kPrompts = 8, kKvHeads = 8, kCtx = 8192, kChunk = 2048;
constexpr int64_t kPool = static_cast<int64_t>(kPrompts) * kCtx;            // tokens per kv head
constexpr int64_t kElems = kKvHeads * kPool * D;                            // per cache (K or V^T)
constexpr int kUnits = kPrompts * kKvHeads * (kCtx / kChunk);               // 256
constexpr int kLayers = 8;

// One context unit's stream: group (kv head g, prompt b), chunk c.
__global__ __launch_bounds__(64 * NW) void ring_stream(const T* __restrict__ kc, const T* __restrict__ vc,
                                                       unsigned* __restrict__ sink) {
  using RG = ippd::Ring<T, D, NS>;
  constexpr int DPT = RG::BLOCKS / NW;
  __shared__ __attribute__((aligned(16))) unsigned char ring[NS * RG::STAGE];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int u = blockIdx.x;
  const int per_head = kPrompts * (kCtx / kChunk);
  const int g = u / per_head, r = u - g * per_head;
  const int b = r / (kCtx / kChunk), c = r - b * (kCtx / kChunk);
  const T* kbase = kc + static_cast<int64_t>(g) * kPool * D;
  const T* vbase = vc + static_cast<int64_t>(g) * kPool * D;
  const int64_t k0 = static_cast<int64_t>(b) * kCtx + static_cast<int64_t>(c) * kChunk, k1 = k0 + kChunk;
  const int ntiles = kChunk / 32, last = ntiles - 1;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));
  ippd::TileOffsets<T, D, NW, NS> toff;
  toff.init(wave, lane);
  for (int t = 0; t < NS - 1; ++t)
    ippd::issue_tile<T, D, NW, NS>(lds + t * RG::STAGE, kbase, vbase, k0 + 32ll * t, k1, wave, lane, toff);
  for (int t = 0; t < ntiles; ++t) {
    ippd::wait_tiles<DPT, NS - 2>(min(last - t, NS - 2));
    __syncthreads();
    const int tn = t + NS - 1;
    if (tn <= last)
      ippd::issue_tile<T, D, NW, NS>(lds + (tn % NS) * RG::STAGE, kbase, vbase, k0 + 32ll * tn, k1, wave, lane, toff);
  }
  ippd::wait_vmcnt<0>();
  __syncthreads();
  // one word per thread out of the last stage, so the ring has a reader
  sink[static_cast<int64_t>(u) * blockDim.x + threadIdx.x] =
      reinterpret_cast<const unsigned*>(ring + (last % NS) * RG::STAGE)[threadIdx.x];
}

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void register_loads(const u4* __restrict__ a, const u4* __restrict__ b, int64_t n,
                                                      unsigned* __restrict__ sink) {
  u4 acc = {0u, 0u, 0u, 0u};
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int h = 0; h < 2; ++h) {
    const u4* p = h == 0 ? a : b;
    int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i + 7 * stride < n; i += 8 * stride) {
      u4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = p[i + k * stride];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc ^= v[k];
    }
    for (; i < n; i += stride) acc ^= p[i];
  }
  sink[static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

#define CHECK(x)                                                                          \
  do {                                                                                    \
    const hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) {                                                               \
      std::fprintf(stderr, "%s failed: %s (line %d)\n", #x, hipGetErrorString(e_), __LINE__); \
      return 1;                                                                           \
    }                                                                                     \
  } while (0)

template <typename F>
int time_kernel(const char* name, F launch, double bytes) {
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  constexpr int kWarm = 4, kReps = 24;
  for (int r = 0; r < kWarm; ++r) launch(r % kLayers);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  CHECK(hipEventRecord(e0));
  for (int r = 0; r < kReps; ++r) launch(r % kLayers);
  CHECK(hipEventRecord(e1));
  CHECK(hipEventSynchronize(e1));
  CHECK(hipGetLastError());
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  const double us = 1e3 * ms / kReps;
  std::printf("%-16s %10.0f %10.2f %10.1f %8.3f\n", name, bytes, us, bytes / us / 1e3, bytes / us / 1e3 / 8000.0);
  std::fflush(stdout);
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return 0;
}

}  // namespace

int main() {
  const size_t cache_bytes = static_cast<size_t>(kElems) * sizeof(T);
  std::vector<T*> kc(kLayers), vc(kLayers);
  for (int l = 0; l < kLayers; ++l) {
    CHECK(hipMalloc(&kc[l], cache_bytes));
    CHECK(hipMalloc(&vc[l], cache_bytes));
    CHECK(hipMemset(kc[l], 0x3c, cache_bytes));
    CHECK(hipMemset(vc[l], 0x3c, cache_bytes));
  }
  unsigned* sink = nullptr;
  const int loads_grid = 2048;
  CHECK(hipMalloc(&sink, sizeof(unsigned) * static_cast<size_t>(kUnits > loads_grid ? kUnits : loads_grid) * 512));
  const double bytes = 2.0 * static_cast<double>(cache_bytes);
  std::printf("# K + V^T bytes per launch %.0f (%d units x %d tokens x 2 x %d B)\n", bytes, kUnits, kChunk,
              static_cast<int>(D * sizeof(T)));
  std::printf("%-16s %10s %10s %10s %8s\n", "kernel", "bytes", "us", "GB/s", "of8TB/s");
  if (time_kernel("ring", [&](int l) {
        ring_stream<<<kUnits, 64 * NW, 0, 0>>>(kc[l], vc[l], sink);
      }, bytes))
    return 1;
  const int64_t n16 = static_cast<int64_t>(cache_bytes / 16);
  if (time_kernel("loads", [&](int l) {
        register_loads<<<loads_grid, 256, 0, 0>>>(reinterpret_cast<const u4*>(kc[l]), reinterpret_cast<const u4*>(vc[l]),
                                                  n16, sink);
      }, bytes))
    return 1;
  for (int l = 0; l < kLayers; ++l) {
    CHECK(hipFree(kc[l]));
    CHECK(hipFree(vc[l]));
  }
  CHECK(hipFree(sink));
  return 0;
}
