// read_probe.hip -- measured HBM read ceiling for the segmented diff.
//
// Streams two buffers the way the diff kernel reads a candidate and a
// reference state (16-byte non-temporal loads, 64 lanes x U chunks per tile,
// each wave walking a contiguous range of tiles) and folds them with XOR, so
// the only work is the read.  It runs the read at 1, 2 and 4 workgroups of 4
// waves per CU and prints one JSON line: the best shape's median and best
// GB/s over several launches, and every shape's median.  Built by the
// package build step; bench.py runs it and reports the result beside the
// diff kernel's bandwidth.
//
// usage: read_probe [GiB per side (default 32)] [reps (default 7)] [offset]
//
// With an offset (bytes, a multiple of 4096, at most 1 GiB) the two buffers
// are one allocation, the second starting `offset` bytes after the end of
// the first, so that their placement relative to each other is fixed; an
// offset of -1 reads one buffer of twice the size as a single stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                                      \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::printf("{\"error\": \"%s at line %d\"}\n", hipGetErrorString(e_), __LINE__); \
      std::exit(1);                                                                   \
    }                                                                                 \
  } while (0)

constexpr int kU = 4;          // chunks per lane per tile, as in the diff kernel
constexpr int kWavesPerBlock = 4;

__global__ __launch_bounds__(kWavesPerBlock * 64) void read_one(const uint8_t* a, uint64_t n_tiles,
                                                               uint32_t* out) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t wave = (uint64_t)blockIdx.x * kWavesPerBlock +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const uint64_t nw = (uint64_t)gridDim.x * kWavesPerBlock;
  const uint64_t lo = n_tiles * wave / nw, hi = n_tiles * (wave + 1) / nw;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (uint64_t t = lo; t < hi; ++t) {
    const uint8_t* pa = a + (t * kU * 64 + lane) * 16;
    u32x4 va[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) va[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(pa + j * 1024));
#pragma unroll
    for (int j = 0; j < kU; ++j) acc ^= va[j];
  }
  out[(uint64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc.x | acc.y | acc.z | acc.w;
}

__global__ __launch_bounds__(kWavesPerBlock * 64) void read_two(const uint8_t* a, const uint8_t* b,
                                                               uint64_t n_tiles, uint32_t* out) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t wave = (uint64_t)blockIdx.x * kWavesPerBlock +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const uint64_t nw = (uint64_t)gridDim.x * kWavesPerBlock;
  const uint64_t lo = n_tiles * wave / nw, hi = n_tiles * (wave + 1) / nw;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (uint64_t t = lo; t < hi; ++t) {
    const uint8_t* pa = a + (t * kU * 64 + lane) * 16;
    const uint8_t* pb = b + (t * kU * 64 + lane) * 16;
    u32x4 va[kU], vb[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      va[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(pa + j * 1024));
      vb[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(pb + j * 1024));
    }
#pragma unroll
    for (int j = 0; j < kU; ++j) acc ^= va[j] ^ vb[j];
  }
  out[(uint64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc.x | acc.y | acc.z | acc.w;
}

int main(int argc, char** argv) {
  const uint64_t per_side = (argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 32ull) << 30;
  const int reps = argc > 2 ? std::atoi(argv[2]) : 7;
  const bool placed = argc > 3;
  const long long offset = placed ? std::atoll(argv[3]) : 0;
  if (reps < 1 || (placed && (offset < -1 || offset > (1ll << 30) || (offset > 0 && offset % 4096 != 0)))) {
    std::printf("{\"error\": \"reps must be >= 1; offset -1 or a multiple of 4096 in [0, 2^30]\"}\n");
    return 2;
  }
  int cus = 0;
  CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
  const int max_blocks = cus * 4;
  const uint64_t tile_bytes = (uint64_t)kU * 64 * 16;
  const uint64_t n_tiles = per_side / tile_bytes;         // every tile lies inside both buffers
  uint8_t *a = nullptr, *b = nullptr, *base = nullptr;
  uint32_t* out = nullptr;
  if (placed) {
    const uint64_t total = 2 * per_side + (offset > 0 ? (uint64_t)offset : 0);
    CHECK(hipMalloc(&base, total));
    CHECK(hipMemset(base, 0x5A, total));
    a = base;
    b = offset >= 0 ? base + per_side + offset : nullptr;
  } else {
    CHECK(hipMalloc(&a, per_side));
    CHECK(hipMalloc(&b, per_side));
    CHECK(hipMemset(a, 0x5A, per_side));
    CHECK(hipMemset(b, 0x5A, per_side));
  }
  CHECK(hipMalloc(&out, (size_t)max_blocks * kWavesPerBlock * 64 * sizeof(uint32_t)));
  CHECK(hipDeviceSynchronize());
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  const double bytes = 2.0 * (double)n_tiles * (double)tile_bytes;
  double best_med = 1e30, best_min = 1e30;
  int best_per_cu = 0;
  char shapes[256] = {0};
  size_t used = 0;
  for (int per_cu : {1, 2, 4}) {
    const int blocks = cus * per_cu;
    std::vector<float> ms;
    for (int r = 0; r < reps + 1; ++r) {
      CHECK(hipEventRecord(e0));
      if (b)
        hipLaunchKernelGGL(read_two, dim3(blocks), dim3(kWavesPerBlock * 64), 0, 0, a, b, n_tiles, out);
      else
        hipLaunchKernelGGL(read_one, dim3(blocks), dim3(kWavesPerBlock * 64), 0, 0, a, 2 * n_tiles, out);
      CHECK(hipGetLastError());
      CHECK(hipEventRecord(e1));
      CHECK(hipEventSynchronize(e1));
      float t = 0.f;
      CHECK(hipEventElapsedTime(&t, e0, e1));
      if (r > 0) ms.push_back(t);                           // first launch is a warmup
    }
    std::sort(ms.begin(), ms.end());
    const double med = ms[ms.size() / 2];
    used += std::snprintf(shapes + used, sizeof(shapes) - used, "%s\"%d\": %.1f", used ? ", " : "", per_cu,
                          bytes / (med * 1e-3) / 1e9);
    if (med < best_med) {
      best_med = med;
      best_min = ms[0];
      best_per_cu = per_cu;
    }
  }
  char where[96];
  if (!placed)
    std::snprintf(where, sizeof(where), "two allocations");
  else if (b)
    std::snprintf(where, sizeof(where), "one allocation, second buffer %lld bytes after the first", offset);
  else
    std::snprintf(where, sizeof(where), "one stream over both");
  std::printf("{\"GBps\": %.1f, \"best_GBps\": %.1f, \"median_ms\": %.4f, \"bytes\": %.0f, "
              "\"GBps_by_workgroups_per_cu\": {%s}, "
              "\"config\": \"2 x %llu GiB (%s), nt dwordx4, U=%d, best of 1/2/4 workgroups x %d waves per CU: %d\"}\n",
              bytes / (best_med * 1e-3) / 1e9, bytes / (best_min * 1e-3) / 1e9, best_med, bytes, shapes,
              (unsigned long long)(per_side >> 30), where, kU, kWavesPerBlock, best_per_cu);
  if (placed) {
    CHECK(hipFree(base));
  } else {
    CHECK(hipFree(a));
    CHECK(hipFree(b));
  }
  CHECK(hipFree(out));
  return 0;
}
