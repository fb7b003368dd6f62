// guard.hip -- canary integrity check of guard regions (AsmEvo section 3.2:
// the predicate iota requires intact out-of-bounds guards; section 3.4:
// Tier-1 allocations carry canary-initialised guards, and guard regions are
// checked byte-exactly).  Row padding between the rows of a strided
// allocation is checked the same way, as interior guards.  The expected
// bytes are regenerated from (seed, alloc_id, side) -- the pad bytes from
// the PAD stream at their data offset -- so only the candidate is read.
#include "device_math.h"
#include "kernels.h"
#include "layout.h"

namespace asmevo {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ void guard_init_kernel(asmevo_guard_result* results, int n) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  asmevo_guard_result r;
  r.bad_lo = 0;
  r.bad_hi = 0;
  r.first_bad_lo = -1;
  r.first_bad_hi = -1;
  r.bad_pad = 0;
  r.first_bad_pad = -1;
  results[t] = r;
}

__device__ __forceinline__ void add_bad(asmevo_guard_result* res, uint32_t side, uint64_t cnt, uint64_t first) {
  if (side == 0) {
    atomicAdd(reinterpret_cast<unsigned long long*>(&res->bad_lo), cnt);
    atomicMin(reinterpret_cast<unsigned long long*>(&res->first_bad_lo), first);
  } else if (side == 1) {
    atomicAdd(reinterpret_cast<unsigned long long*>(&res->bad_hi), cnt);
    atomicMin(reinterpret_cast<unsigned long long*>(&res->first_bad_hi), first);
  } else {
    atomicAdd(reinterpret_cast<unsigned long long*>(&res->bad_pad), cnt);
    atomicMin(reinterpret_cast<unsigned long long*>(&res->first_bad_pad), first);
  }
}

// One thread per 16 guard bytes; the chunk's region is found by binary search
// over the regions' chunk prefix.  A wave's corrupted chunks of one region
// (the common case when a write runs over many rows or a whole guard) are
// folded across the wave first, so one lane issues the atomics.
__global__ __launch_bounds__(256) void guard_kernel(const GuardRegion* __restrict__ regs, int n,
                                                    uint64_t total_chunks, uint64_t seed,
                                                    asmevo_guard_result* results) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint32_t lane = threadIdx.x & 63u;
  // the loop bound is uniform per workgroup, so every lane reaches the cross-lane steps
  for (uint64_t base = (uint64_t)blockIdx.x * blockDim.x; base < total_chunks; base += stride) {
    const uint64_t g = base + threadIdx.x;
    uint32_t mask = 0;
    uint64_t first = ~0ull;
    uint32_t key = ~0u;                     // result index * 4 + side
    if (g < total_chunks) {
      int lo = 0, hi = n - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (regs[mid].chunk_begin <= g) lo = mid;
        else hi = mid - 1;
      }
      const GuardRegion R = regs[lo];
      uint64_t p0, q0 = 0;            // byte offset in the guard (pad: in the run), pad data offset
      uint32_t nb;
      U4 C;
      if (R.side < 2) {
        p0 = (g - R.chunk_begin) * kChunk;
        const uint64_t left = R.bytes - p0;
        nb = left < (uint64_t)kChunk ? (uint32_t)left : (uint32_t)kChunk;
        C = stream(seed, R.alloc_id, kCanary, R.side, 0, p0 >> 4);
      } else {
        const uint64_t k = g - R.chunk_begin;
        const uint64_t run = k / R.run_chunks;
        p0 = (k - run * R.run_chunks) * kChunk;
        const uint64_t left = R.bytes - p0;
        nb = left < (uint64_t)kChunk ? (uint32_t)left : (uint32_t)kChunk;
        q0 = run * R.pitch + R.pad_off + p0;
        C = stream(seed, R.alloc_id, kPad, 0, 0, q0 >> 4);
      }
      if (R.side < 2) {
        const uint64_t src = R.addr + p0;
        if (nb == (uint32_t)kChunk && (src & 15u) == 0) {
          const u32x4 v = *gptr_mut<u32x4>(src);
          const uint32_t x[4] = {v.x ^ C.x, v.y ^ C.y, v.z ^ C.z, v.w ^ C.w};
#pragma unroll
          for (int k = 0; k < 16; ++k) mask |= ((x[k >> 2] >> (8 * (k & 3))) & 0xFFu) ? (1u << k) : 0u;
        } else {
          const AS_GLOBAL uint8_t* bytes = gptr_mut<uint8_t>(src);
          for (uint32_t k = 0; k < nb; ++k)
            mask |= (bytes[k] != byte_of(C, k)) ? (1u << k) : 0u;
        }
      } else {
        // pad bytes [q0, q0 + nb) of the data region: PAD blocks q0 / 16 and the next
        const AS_GLOBAL uint8_t* bytes = gptr_mut<uint8_t>(R.addr + q0);
        const uint32_t ph = (uint32_t)(q0 & 15u);
        const U4 C1 = stream(seed, R.alloc_id, kPad, 0, 0, (q0 >> 4) + 1u);
        for (uint32_t k = 0; k < nb; ++k) {
          const uint32_t j = ph + k;
          const uint8_t want = j < 16u ? byte_of(C, j) : byte_of(C1, j - 16u);
          mask |= (bytes[k] != want) ? (1u << k) : 0u;
        }
      }
      if (mask) {
        first = (R.side < 2 ? p0 : q0) + (uint64_t)__builtin_ctz(mask);
        key = (R.result_index << 2) | R.side;
      }
    }
    const uint64_t act = __ballot(mask != 0u);
    if (act == 0ull) continue;                              // uniform across the wave
    const int lead = __builtin_ctzll(act);
    const uint32_t lkey = __shfl(key, lead, 64);
    const bool mine = mask != 0u && key == lkey;
    uint64_t cnt = mine ? (uint64_t)__builtin_popcount(mask) : 0ull;
    uint64_t fst = mine ? first : ~0ull;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      cnt += __shfl_xor(cnt, m, 64);
      const uint64_t o = __shfl_xor(fst, m, 64);
      fst = o < fst ? o : fst;
    }
    if ((int)lane == lead) add_bad(results + (lkey >> 2), lkey & 3u, cnt, fst);
    if (mask != 0u && !mine)                                // another region in the same wave: rare
      add_bad(results + (key >> 2), key & 3u, (uint64_t)__builtin_popcount(mask), first);
  }
}

}  // namespace

hipError_t launch_guard(const GuardRegion* regs, int n_regs, uint64_t total_chunks, uint64_t seed,
                        asmevo_guard_result* results, int n_results, hipStream_t stream) {
  if (n_results == 0) return hipSuccess;
  hipLaunchKernelGGL(guard_init_kernel, dim3((n_results + 255) / 256), dim3(256), 0, stream,
                     results, n_results);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || total_chunks == 0) return e;
  uint64_t blocks = (total_chunks + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(guard_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, regs, n_regs,
                     total_chunks, seed, results);
  return hipGetLastError();
}

}  // namespace asmevo
