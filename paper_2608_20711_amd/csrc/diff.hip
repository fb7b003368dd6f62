// diff.hip -- segmented multi-buffer comparison of a candidate state against
// the reference state (AsmEvo section 3.2, Eq. 1: Delta = K'(x) - O(x) and
// its infinity norm; iota: bit-exact integer buffers; section 3.4: floating
// outputs by tolerance, integer / opaque state byte-exactly).
//
// Streaming, HBM-bound design for gfx950:
//  * every segment is cut into tiles of 512 16-byte chunks (8 KiB per
//    operand); all segments share one flat tile space;
//  * each wave owns a contiguous range of tiles and issues 8 non-temporal
//    dwordx4 loads per operand per lane before looking at any of them;
//  * the common case is a 128-bit XOR that is zero: nothing else runs;
//  * only chunks whose bits differ (or, under the strict NaN policy, hold a
//    NaN) are decoded and tested in fp64;
//  * per-lane partials are reduced across the wave with cross-lane shuffles
//    only when the wave has seen a difference in the segment it leaves, and
//    land in the result with exact 64-bit atomics (sum / min / max of
//    non-negative doubles as bit patterns), so results are identical for any
//    schedule or launch geometry.
#include "device_math.h"
#include "kernels.h"
#include "layout.h"

namespace asmevo {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct Acc {
  uint32_t bw, tol, nf;
  uint64_t first_bw, first_tol;
  uint64_t max_abs, max_rel;   // bit patterns of non-negative doubles
};

__device__ __forceinline__ void acc_reset(Acc& a) {
  a.bw = 0;
  a.tol = 0;
  a.nf = 0;
  a.first_bw = ~0ull;
  a.first_tol = ~0ull;
  a.max_abs = 0;
  a.max_rel = 0;
}

template <int DT> struct Et;
template <> struct Et<ASMEVO_F32> { static constexpr int es = 4; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_BF16> { static constexpr int es = 2; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_F16> { static constexpr int es = 2; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_FP8_E4M3> { static constexpr int es = 1; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_I32> { static constexpr int es = 4; static constexpr bool fp = false; };
template <> struct Et<ASMEVO_I64> { static constexpr int es = 8; static constexpr bool fp = false; };
template <> struct Et<ASMEVO_U8> { static constexpr int es = 1; static constexpr bool fp = false; };

template <int DT>
__device__ __forceinline__ uint64_t elem(const u32x4& v, int e) {
  // e is a compile-time constant at every call of this form
  constexpr int es = Et<DT>::es;
  if constexpr (es == 4) return v[e];
  else if constexpr (es == 2) return (v[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
  else if constexpr (es == 1) return (v[e >> 2] >> (8 * (e & 3))) & 0xFFu;
  else return (uint64_t)v[2 * e] | ((uint64_t)v[2 * e + 1] << 32);
}

// Element e (a run-time value) of a chunk, selected without indexing into
// registers (which would go through scratch memory).
template <int DT>
__device__ __forceinline__ uint64_t elem_dyn(const u32x4& v, uint32_t e) {
  constexpr uint32_t es = Et<DT>::es;
  const uint32_t byte = e * es;
  const uint32_t wi = byte >> 2;
  const uint32_t w = wi == 0 ? v.x : wi == 1 ? v.y : wi == 2 ? v.z : v.w;
  if constexpr (es == 8) {
    const uint32_t w2 = wi == 0 ? v.y : v.w;
    return (uint64_t)w | ((uint64_t)w2 << 32);
  } else if constexpr (es == 4) {
    return w;
  } else {
    return (w >> (8u * (byte & 3u))) & ((1u << (8u * es)) - 1u);
  }
}

template <int DT>
__device__ __forceinline__ bool is_nan_raw(uint64_t r) {
  if constexpr (DT == ASMEVO_F32) return (r & 0x7FFFFFFFu) > 0x7F800000u;
  else if constexpr (DT == ASMEVO_BF16) return (r & 0x7FFFu) > 0x7F80u;
  else if constexpr (DT == ASMEVO_F16) return (r & 0x7FFFu) > 0x7C00u;
  else if constexpr (DT == ASMEVO_FP8_E4M3) return (r & 0x7Fu) == 0x7Fu;
  else return false;
}

// One element pair that needs attention: bits differ, or b is a NaN under the
// strict policy.  Implements the per-pair rule of the tolerance check.
template <int DT>
__device__ __forceinline__ void pair_slow(uint64_t ra, uint64_t rb, uint64_t i, bool tol_mode,
                                       bool strict, double atol, double rtol, Acc& acc) {
  const bool bw = ra != rb;
  if (bw) {
    acc.bw += 1;
    acc.first_bw = i < acc.first_bw ? i : acc.first_bw;
  }
  if constexpr (Et<DT>::fp) {
    if (!tol_mode) return;
    double A = 0.0, B = 0.0;
    const int ca = decode<DT>(ra, A);
    const int cb = decode<DT>(rb, B);
    const bool nonfinite = (ca | cb) != 0;
    bool mism;
    if (!bw) {
      mism = (cb == 3) && strict;
    } else if (ca == 3 || cb == 3) {
      mism = !(ca == 3 && cb == 3 && !strict);
    } else if (nonfinite) {
      mism = true;
    } else {
      const double d = __builtin_fabs(A - B);
      const double scaled = rtol * __builtin_fabs(B);
      const double t = atol + scaled;
      mism = !(d <= t);
      double rel;
      if (B != 0.0) rel = d / __builtin_fabs(B);
      else rel = (d == 0.0) ? 0.0 : __builtin_inf();
      const uint64_t db = (uint64_t)__double_as_longlong(d);
      const uint64_t rb_ = (uint64_t)__double_as_longlong(rel);
      acc.max_abs = db > acc.max_abs ? db : acc.max_abs;
      acc.max_rel = rb_ > acc.max_rel ? rb_ : acc.max_rel;
    }
    if (mism) {
      acc.tol += 1;
      acc.first_tol = i < acc.first_tol ? i : acc.first_tol;
      if (nonfinite) acc.nf += 1;
    }
  }
}

// One 16-byte chunk pair holding `nvalid` elements starting at logical index i0.
template <int DT>
__device__ __forceinline__ void chunk(const u32x4& va, const u32x4& vb, uint64_t i0,
                                      uint32_t nvalid, bool tol_mode, bool strict, double atol,
                                      double rtol, Acc& acc) {
  const u32x4 x = va ^ vb;
  if (((x.x | x.y | x.z | x.w) == 0u) && !strict) return;   // the common case
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  uint32_t mask = 0;
#pragma unroll
  for (int e = 0; e < epc; ++e) {
    const bool need = elem<DT>(x, e) != 0 || (strict && is_nan_raw<DT>(elem<DT>(vb, e)));
    mask |= need ? (1u << e) : 0u;
  }
  mask &= (nvalid >= 32u) ? ~0u : ((1u << nvalid) - 1u);
  while (mask) {
    const uint32_t e = (uint32_t)__builtin_ctz(mask);
    mask &= mask - 1u;
    pair_slow<DT>(elem_dyn<DT>(va, e), elem_dyn<DT>(vb, e), i0 + (uint64_t)e, tol_mode, strict,
                  atol, rtol, acc);
  }
}

// Loads the valid elements of a chunk one by one (misaligned operands or a
// partial chunk at the end of a row); invalid bytes read as zero on both sides.
template <int DT>
__device__ __forceinline__ u32x4 load_elems(const uint8_t* p, uint32_t nv) {
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < epc; ++e) {
    if ((uint32_t)e < nv) {
      if constexpr (es == 1) w[e >> 2] |= (uint32_t)gptr<uint8_t>(p)[e] << (8 * (e & 3));
      else if constexpr (es == 2) w[e >> 1] |= (uint32_t)gptr<uint16_t>(p)[e] << (16 * (e & 1));
      else if constexpr (es == 4) w[e] = gptr<uint32_t>(p)[e];
      else {
        const uint64_t raw = gptr<uint64_t>(p)[e];
        w[2 * e] = (uint32_t)raw;
        w[2 * e + 1] = (uint32_t)(raw >> 32);
      }
    }
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

__device__ __forceinline__ u32x4 ld_nt(const uint8_t* p) {
  return __builtin_nontemporal_load(gptr<u32x4>(p));
}

// Chunk pair of a row whose bytes [c*16, c*16 + nbytes) are valid: a vector
// load when the chunk is whole and aligned, element loads otherwise.
template <int DT>
__device__ __forceinline__ void load_chunk(const uint8_t* pa, const uint8_t* pb, uint32_t nbytes,
                                           bool vec, u32x4& va, u32x4& vb) {
  if (nbytes == (uint32_t)kChunk && vec) {
    va = ld_nt(pa);
    vb = ld_nt(pb);
  } else {
    const uint32_t nv = nbytes / Et<DT>::es;
    va = load_elems<DT>(pa, nv);
    vb = load_elems<DT>(pb, nv);
  }
}

// All tiles [t_begin, t_end) of one segment.
template <int DT>
__device__ __forceinline__ void diff_range(const DiffSeg& S, uint64_t t_begin, uint64_t t_end,
                                           uint32_t lane, Acc& acc) {
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  constexpr int U = kDiffUnroll;
  const bool tol_mode = S.mode == ASMEVO_TOLERANCE;
  const bool strict = (S.flags & kSegStrict) != 0;
  const bool vec = (S.flags & kSegVec) != 0;
  const uint8_t* a0 = reinterpret_cast<const uint8_t*>(S.a);
  const uint8_t* b0 = reinterpret_cast<const uint8_t*>(S.b);

  if (S.flags & kSegNarrow) {
    // Short rows: tiles over the row-major chunk space, each lane finds its row.
    const uint64_t total = S.rows * S.row_chunks;
    for (uint64_t tile = t_begin; tile < t_end; ++tile) {
      const uint64_t k0 = tile * (uint64_t)kTileChunks;
#pragma unroll 1
      for (int j = 0; j < U; ++j) {
        const uint64_t k = k0 + (uint64_t)(j * kWave) + lane;
        u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
        uint32_t nb = 0;
        uint64_t i0 = 0;
        if (k < total) {
          const uint64_t r = k / S.row_chunks;
          const uint64_t c = k - r * S.row_chunks;
          const uint64_t cb = c * kChunk;
          const uint64_t rem = S.row_bytes - cb;
          nb = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
          load_chunk<DT>(a0 + r * S.a_pitch + cb, b0 + r * S.b_pitch + cb, nb, vec, va, vb);
          i0 = r * S.cols + c * epc;
        }
        chunk<DT>(va, vb, i0, nb / es, tol_mode, strict, S.atol, S.rtol, acc);
      }
    }
    return;
  }

  // Row-tiled: every tile lies inside one row.
  const uint64_t tpr = S.tiles_per_row;
  uint64_t tile = t_begin;
#if ASMEVO_DIFF_PIPELINE
  if (S.rows == 1 && vec) {
    // Contiguous segment: its whole tiles run as a software pipeline -- the
    // loads of tile t+1 are in flight while tile t is checked.
    const uint64_t whole = S.full_chunks / kTileChunks;
    const uint64_t t_fast = t_end < whole ? t_end : whole;
    if (tile < t_fast) {
      const uint8_t* qa = a0 + (uint64_t)lane * kChunk;
      const uint8_t* qb = b0 + (uint64_t)lane * kChunk;
      u32x4 va[U], vb[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        va[j] = ld_nt(qa + (tile * kTileChunks + j * kWave) * kChunk);
        vb[j] = ld_nt(qb + (tile * kTileChunks + j * kWave) * kChunk);
      }
      for (; tile < t_fast; ++tile) {
        u32x4 na[U], nb[U];
        if (tile + 1 < t_fast) {
#pragma unroll
          for (int j = 0; j < U; ++j) {
            na[j] = ld_nt(qa + ((tile + 1) * kTileChunks + j * kWave) * kChunk);
            nb[j] = ld_nt(qb + ((tile + 1) * kTileChunks + j * kWave) * kChunk);
          }
        }
        u32x4 x = va[0] ^ vb[0];
#pragma unroll
        for (int j = 1; j < U; ++j) x |= va[j] ^ vb[j];
        if (((x.x | x.y | x.z | x.w) != 0u) || strict) {
          const uint64_t k0 = tile * (uint64_t)kTileChunks;
#pragma unroll
          for (int j = 0; j < U; ++j)
            chunk<DT>(va[j], vb[j], (k0 + (uint64_t)(j * kWave) + lane) * epc, epc, tol_mode, strict,
                      S.atol, S.rtol, acc);
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
          va[j] = na[j];
          vb[j] = nb[j];
        }
      }
    }
  }
#endif
  for (; tile < t_end; ++tile) {
    uint64_t r = 0, kt = tile;
    if (S.rows > 1) {
      r = (uint32_t)tile / (uint32_t)tpr;
      kt = tile - r * tpr;
    }
    const uint8_t* pa = a0 + r * S.a_pitch;
    const uint8_t* pb = b0 + r * S.b_pitch;
    const uint64_t ibase = r * S.cols;
    const uint64_t k0 = kt * (uint64_t)kTileChunks;
    if (vec && k0 + kTileChunks <= S.full_chunks) {
      // Whole tile: issue all loads first, then one combined check.
      const uint8_t* qa = pa + (k0 + lane) * kChunk;
      const uint8_t* qb = pb + (k0 + lane) * kChunk;
      u32x4 va[U], vb[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        va[j] = ld_nt(qa + j * kWave * kChunk);
        vb[j] = ld_nt(qb + j * kWave * kChunk);
      }
      u32x4 x = va[0] ^ vb[0];
#pragma unroll
      for (int j = 1; j < U; ++j) x |= va[j] ^ vb[j];
      if (((x.x | x.y | x.z | x.w) != 0u) || strict) {
#pragma unroll
        for (int j = 0; j < U; ++j)
          chunk<DT>(va[j], vb[j], ibase + (k0 + (uint64_t)(j * kWave) + lane) * epc, epc, tol_mode,
                    strict, S.atol, S.rtol, acc);
      }
      continue;
    }
    // Last tile of a row (or misaligned operands): per-chunk bounds.
#pragma unroll 1
    for (int j = 0; j < U; ++j) {
      const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
      u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
      uint32_t nb = 0;
      if (c < S.row_chunks) {
        const uint64_t cb = c * kChunk;
        const uint64_t rem = S.row_bytes - cb;
        nb = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
        load_chunk<DT>(pa + cb, pb + cb, nb, vec, va, vb);
      }
      chunk<DT>(va, vb, ibase + c * epc, nb / es, tol_mode, strict, S.atol, S.rtol, acc);
    }
  }
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}
__device__ __forceinline__ uint64_t wave_min(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const uint64_t o = __shfl_xor(v, m, kWave);
    v = o < v ? o : v;
  }
  return v;
}
__device__ __forceinline__ uint64_t wave_max(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const uint64_t o = __shfl_xor(v, m, kWave);
    v = o > v ? o : v;
  }
  return v;
}

// Folds the wave's partials for one segment into its result (only if the
// wave saw anything) and resets them.
__device__ __forceinline__ void flush(Acc& acc, const DiffSeg& S, asmevo_segment_result* results, uint32_t lane) {
  if (__ballot((acc.bw | acc.tol) != 0u) == 0ull) return;
  uint64_t bw = wave_sum(acc.bw);
  uint64_t tol = wave_sum(acc.tol);
  const uint64_t nf = wave_sum(acc.nf);
  uint64_t fbw = wave_min(acc.first_bw);
  uint64_t ftol = wave_min(acc.first_tol);
  const uint64_t mab = wave_max(acc.max_abs);
  const uint64_t mre = wave_max(acc.max_rel);
  if (lane == 0) {
    asmevo_segment_result* R = results + S.result_index;
    if (S.mode != ASMEVO_TOLERANCE) {
      tol = bw;
      ftol = fbw;
    }
    if (bw) {
      atomicAdd(reinterpret_cast<unsigned long long*>(&R->bitwise_mismatches), bw);
      atomicMin(reinterpret_cast<unsigned long long*>(&R->first_bitwise), fbw);
    }
    if (tol) {
      atomicAdd(reinterpret_cast<unsigned long long*>(&R->mismatches), tol);
      atomicMin(reinterpret_cast<unsigned long long*>(&R->first_mismatch), ftol);
    }
    if (nf) atomicAdd(reinterpret_cast<unsigned long long*>(&R->nonfinite_mismatches), nf);
    if (mab) atomicMax(reinterpret_cast<unsigned long long*>(&R->max_abs), mab);
    if (mre) atomicMax(reinterpret_cast<unsigned long long*>(&R->max_rel), mre);
  }
  acc_reset(acc);
}

__global__ void diff_init_kernel(asmevo_segment_result* results, int n) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  asmevo_segment_result r;
  r.mismatches = 0;
  r.first_mismatch = -1;
  r.bitwise_mismatches = 0;
  r.first_bitwise = -1;
  r.nonfinite_mismatches = 0;
  r.max_abs = 0.0;
  r.max_rel = 0.0;
  results[t] = r;
}


__global__ __launch_bounds__(kDiffBlock) __attribute__((amdgpu_waves_per_eu(ASMEVO_DIFF_WAVES_PER_EU)))
void diff_kernel(const DiffSeg* __restrict__ segs, int n,
                                                          uint64_t total_tiles,
                                                          asmevo_segment_result* results) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = (uint64_t)blockIdx.x * (kDiffBlock / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t nwaves = (uint64_t)gridDim.x * (kDiffBlock / kWave);
  const uint64_t lo = total_tiles * wave / nwaves;
  const uint64_t hi = total_tiles * (wave + 1) / nwaves;
  if (lo >= hi) return;
  int s_lo = 0, s_hi = n - 1;            // last segment with tile_begin <= lo
  while (s_lo < s_hi) {
    const int mid = (s_lo + s_hi + 1) >> 1;
    if (segs[mid].tile_begin <= lo) s_lo = mid;
    else s_hi = mid - 1;
  }
  int s = s_lo;
  Acc acc;
  acc_reset(acc);
  uint64_t t = lo;
  while (t < hi) {
    while (s + 1 < n && segs[s + 1].tile_begin <= t) ++s;
    const DiffSeg S = segs[s];
    const uint64_t seg_end = S.tile_begin + S.tile_count;
    const uint64_t t_end = seg_end < hi ? seg_end : hi;
    const uint64_t b = t - S.tile_begin, e = t_end - S.tile_begin;
    switch (S.dtype) {
      case ASMEVO_F32: diff_range<ASMEVO_F32>(S, b, e, lane, acc); break;
      case ASMEVO_BF16: diff_range<ASMEVO_BF16>(S, b, e, lane, acc); break;
      case ASMEVO_F16: diff_range<ASMEVO_F16>(S, b, e, lane, acc); break;
      case ASMEVO_FP8_E4M3: diff_range<ASMEVO_FP8_E4M3>(S, b, e, lane, acc); break;
      case ASMEVO_I32: diff_range<ASMEVO_I32>(S, b, e, lane, acc); break;
      case ASMEVO_I64: diff_range<ASMEVO_I64>(S, b, e, lane, acc); break;
      default: diff_range<ASMEVO_U8>(S, b, e, lane, acc); break;
    }
    flush(acc, S, results, lane);
    t = t_end;
  }
}

}  // namespace

int diff_blocks_per_cu() {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, diff_kernel, kDiffBlock, 0) != hipSuccess ||
      blocks <= 0)
    blocks = 4;
  return blocks;
}

hipError_t launch_diff(const DiffSeg* segs, int n, uint64_t total_tiles,
                       asmevo_segment_result* results, int workgroups, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(diff_init_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, results, n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || total_tiles == 0) return e;
  const uint64_t max_wg = (total_tiles + (kDiffBlock / kWave) - 1) / (kDiffBlock / kWave);
  const int wg = (uint64_t)workgroups > max_wg ? (int)max_wg : workgroups;
  hipLaunchKernelGGL(diff_kernel, dim3(wg), dim3(kDiffBlock), 0, stream, segs, n, total_tiles,
                     results);
  return hipGetLastError();
}

}  // namespace asmevo
