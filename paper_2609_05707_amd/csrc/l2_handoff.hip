// Whether data one kernel writes stays in the writer's L2 for the next
// kernel on the same stream, on one MI355X.
//
// A standalone measurement program (not part of libippd.so), for the decode
// step's split-K partial states: the attend kernel writes them and the merge
// kernel, the next launch, reads them back.  If the reader found them in the
// L2 of the XCD that wrote them, placing each group's units and its merge
// workgroups on one XCD would take those reads off HBM.
//
// The writer's workgroups with blockIdx % 8 == 0 (one XCD: workgroups are
// dealt to the eight XCDs round robin) write 2 MiB, 32 KiB each; the reader,
// launched next, reads the same bytes from the workgroups with
// blockIdx % 8 == x, for x = 0 (the writer's XCD) and x = 1 (another).
// Per-launch time from HIP events; the rocprofv3 FETCH_SIZE of each reader
// launch (L2 fills from the fabric) answers the question.
//
// Usage: l2_handoff            (built next to libippd.so by build.py)
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
constexpr int kRegions = 64;                  // writer workgroups on XCD 0
constexpr int kRegionBytes = 32768;           // 2 MiB in all
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void writer(u4* __restrict__ buf, unsigned v) {
  if (blockIdx.x % 8 != 0) return;
  u4* p = buf + static_cast<size_t>(blockIdx.x / 8) * (kRegionBytes / 16);
  for (int i = threadIdx.x; i < kRegionBytes / 16; i += kThreads) p[i] = u4{v, v + 1u, v + 2u, static_cast<unsigned>(i)};
}

__global__ __launch_bounds__(kThreads) void reader(const u4* __restrict__ buf, unsigned* __restrict__ sink, int xcd) {
  if (static_cast<int>(blockIdx.x % 8) != xcd) return;
  const u4* p = buf + static_cast<size_t>(blockIdx.x / 8) * (kRegionBytes / 16);
  u4 acc = {0u, 0u, 0u, 0u};
  for (int i = threadIdx.x; i < kRegionBytes / 16; i += kThreads) acc ^= p[i];
  sink[blockIdx.x * kThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

#define CHECK(x)                                                                          \
  do {                                                                                    \
    const hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) {                                                               \
      std::fprintf(stderr, "%s failed: %s (line %d)\n", #x, hipGetErrorString(e_), __LINE__); \
      return 1;                                                                           \
    }                                                                                     \
  } while (0)

}  // namespace

int main() {
  u4* buf = nullptr;
  unsigned* sink = nullptr;
  CHECK(hipMalloc(&buf, static_cast<size_t>(kRegions) * kRegionBytes));
  CHECK(hipMalloc(&sink, sizeof(unsigned) * 8 * kRegions * kThreads));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  constexpr int kWarm = 10, kReps = 40;
  for (int xcd : {0, 1, 0, 1}) {
    float total = 0.f;
    for (int rep = 0; rep < kWarm + kReps; ++rep) {
      writer<<<8 * kRegions, kThreads>>>(buf, static_cast<unsigned>(rep));
      CHECK(hipEventRecord(e0));
      reader<<<8 * kRegions, kThreads>>>(buf, sink, xcd);
      CHECK(hipEventRecord(e1));
      CHECK(hipEventSynchronize(e1));
      float ms = 0.f;
      CHECK(hipEventElapsedTime(&ms, e0, e1));
      if (rep >= kWarm) total += ms;
    }
    std::printf("reader on XCD %d, writer on XCD 0: %.2f us per 2 MiB read (%d launches)\n", xcd, 1e3 * total / kReps,
                kReps);
    std::fflush(stdout);
  }
  CHECK(hipGetLastError());
  CHECK(hipFree(buf));
  CHECK(hipFree(sink));
  return 0;
}
