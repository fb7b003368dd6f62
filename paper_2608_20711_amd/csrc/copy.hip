// copy.hip -- segmented multi-region copy: snapshot and restore of a captured
// pre-dispatch state (AsmEvo section 3.4, Tier 2: candidates replay the
// captured dispatch with identical launch parameters and memory contents,
// restored in place so that absolute pointers inside the state stay valid).
//
// All regions share one flat tile space of 4 KiB tiles; the four waves of a
// workgroup share a contiguous range of tiles and take them in turn.  A
// region whose source and destination have the same address phase modulo 16
// is copied with 16-byte non-temporal loads and stores after a byte-wise
// head; other regions are copied byte by byte.
#include "device_math.h"
#include "kernels.h"
#include "layout.h"

namespace asmevo {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyBlock = 256;

#ifndef ASMEVO_COPY_WAVE_STEP                        // waves of a workgroup sharing one tile range
#define ASMEVO_COPY_WAVE_STEP 4
#endif
#ifndef ASMEVO_COPY_NT_LOAD
#define ASMEVO_COPY_NT_LOAD 1
#endif
#ifndef ASMEVO_COPY_NT_STORE
#define ASMEVO_COPY_NT_STORE 1
#endif

__device__ __forceinline__ void copy_bytes(uint64_t dst, uint64_t src, uint64_t n, uint64_t first,
                                           uint64_t step) {
  for (uint64_t k = first; k < n; k += step) *gptr_mut<uint8_t>(dst + k) = *gptr_mut<uint8_t>(src + k);
}

__global__ __launch_bounds__(kCopyBlock) void copy_kernel(const CopyRegion* __restrict__ regs, int n,
                                                          uint64_t total_tiles) {
  // kStep consecutive waves of a workgroup share one contiguous tile range
  // and take its tiles in turn (kStep = 1: every wave has a range of its own).
  constexpr uint32_t kStep = ASMEVO_COPY_WAVE_STEP;
  static_assert(kStep >= 1 && (kCopyBlock / kWave) % kStep == 0, "a tile range stays inside a workgroup");
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = (uint64_t)blockIdx.x * (kCopyBlock / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t ngroups = (uint64_t)gridDim.x * (kCopyBlock / kWave) / kStep;
  const uint64_t group = wave / kStep;
  const uint64_t lo = total_tiles * group / ngroups;
  const uint64_t hi = total_tiles * (group + 1) / ngroups;
  const uint64_t first = lo + wave % kStep;
  if (first >= hi) return;
  int s_lo = 0, s_hi = n - 1;            // last region with tile_begin <= first
  while (s_lo < s_hi) {
    const int mid = (s_lo + s_hi + 1) >> 1;
    if (regs[mid].tile_begin <= first) s_lo = mid;
    else s_hi = mid - 1;
  }
  int s = s_lo;
  for (uint64_t t = first; t < hi; t += kStep) {
    while (s + 1 < n && regs[s + 1].tile_begin <= t) ++s;
    const CopyRegion R = regs[s];
    const uint64_t tile = t - R.tile_begin;
    if (R.vec) {
      // body = bytes [head, head + body_bytes) move in 16-byte chunks; the head
      // and the tail are copied by the first and last tiles
      const uint64_t c0 = tile * kTileChunks;
      if (tile == 0 && R.head) copy_bytes(R.dst, R.src, R.head, lane, kWave);
      const uint64_t body_chunks = R.body_bytes / kChunk;
      if (c0 + kTileChunks <= body_chunks) {
        u32x4 v[kDiffUnroll];
#pragma unroll
        for (int j = 0; j < kDiffUnroll; ++j) {
          const auto* p = gptr_mut<u32x4>(R.src + R.head + (c0 + j * kWave + lane) * kChunk);
          v[j] = ASMEVO_COPY_NT_LOAD ? __builtin_nontemporal_load(p) : *p;
        }
#pragma unroll
        for (int j = 0; j < kDiffUnroll; ++j) {
          auto* p = gptr_mut<u32x4>(R.dst + R.head + (c0 + j * kWave + lane) * kChunk);
          if (ASMEVO_COPY_NT_STORE) __builtin_nontemporal_store(v[j], p);
          else *p = v[j];
        }
      } else {
        for (int j = 0; j < kDiffUnroll; ++j) {
          const uint64_t c = c0 + j * kWave + lane;
          if (c < body_chunks)
            *gptr_mut<u32x4>(R.dst + R.head + c * kChunk) = *gptr_mut<u32x4>(R.src + R.head + c * kChunk);
        }
      }
      if (tile + 1 == R.tile_count) {
        const uint64_t done = R.head + body_chunks * kChunk;
        if (done < R.bytes) copy_bytes(R.dst + done, R.src + done, R.bytes - done, lane, kWave);
      }
    } else {
      const uint64_t b0 = tile * (uint64_t)kTileChunks * kChunk;
      const uint64_t len = R.bytes - b0 < (uint64_t)kTileChunks * kChunk ? R.bytes - b0
                                                                        : (uint64_t)kTileChunks * kChunk;
      copy_bytes(R.dst + b0, R.src + b0, len, lane, kWave);
    }
  }
}

}  // namespace

hipError_t launch_copy(const CopyRegion* regs, int n, uint64_t total_tiles, int workgroups,
                       hipStream_t stream) {
  if (n == 0 || total_tiles == 0) return hipSuccess;
  const uint64_t max_wg = (total_tiles + (kCopyBlock / kWave) - 1) / (kCopyBlock / kWave);
  const int wg = (uint64_t)workgroups > max_wg ? (int)max_wg : workgroups;
  hipLaunchKernelGGL(copy_kernel, dim3(wg), dim3(kCopyBlock), 0, stream, regs, n, total_tiles);
  return hipGetLastError();
}

}  // namespace asmevo
