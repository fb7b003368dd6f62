// diff.hip -- segmented multi-buffer comparison of a candidate state against
// the reference state (AsmEvo section 3.2, Eq. 1: Delta = K'(x) - O(x) and
// its infinity norm, and the cosine c_x = cos(K'(x), O(x)); iota: bit-exact
// integer buffers; section 3.4: floating outputs by tolerance, integer /
// opaque state byte-exactly).
//
// Streaming, HBM-bound design for gfx950:
//  * every segment is cut into tiles of 256 16-byte chunks (4 KiB per
//    operand), each inside one row; all segments share one flat tile space;
//  * each wave owns a contiguous range of tiles (in the cosine variant the
//    four waves of a workgroup take the tiles of 1 MiB blocks in turn, the
//    blocks dealt to the workgroups round-robin: the cosine's cost per tile
//    depends on the element type) and issues 4 non-temporal dwordx4 loads
//    per operand per lane before looking at any of them;
//  * the common case is a 128-bit XOR that is zero: one combined check per
//    tile, nothing else runs;
//  * only chunks whose bits differ (or, under the strict NaN policy, hold a
//    NaN) are decoded and tested in fp64;
//  * per-lane partials are reduced across the wave with cross-lane shuffles
//    only when the wave has seen a difference in the segment it leaves, and
//    land in the result with exact 64-bit atomics (sum / min / max of
//    non-negative doubles as bit patterns), so results are identical for any
//    schedule or launch geometry;
//  * the cosine variant also accumulates fp64 a*b, a*a, b*b per lane over the
//    same registers, folds each tile (= one 4096-byte block) with the xor
//    butterfly's tree (permlane swaps and DPP) and stores the block sums;
//    cos_level_kernel and cosine_kernel fold the blocks of a segment with the
//    left-complete pairwise tree.
#include "device_math.h"
#include "kernels.h"
#include "layout.h"
#include "pair_rule.h"

namespace asmevo {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Element e (a run-time value) of a chunk, selected without indexing into
// registers (which would go through scratch memory).
template <int DT>
__device__ __forceinline__ uint64_t elem_dyn(const u32x4& v, uint32_t e) {
  constexpr uint32_t es = Et<DT>::es;
  const uint32_t byte = e * es;
  const bool odd = (byte & 4u) != 0, high = (byte & 8u) != 0;   // word = byte / 4
  if constexpr (es == 8) {
    const uint32_t w = high ? v.z : v.x;
    const uint32_t w2 = high ? v.w : v.y;
    return (uint64_t)w | ((uint64_t)w2 << 32);
  }
  const uint32_t w = high ? (odd ? v.w : v.z) : (odd ? v.y : v.x);
  if constexpr (es == 4) {
    return w;
  } else {
    return (w >> (8u * (byte & 3u))) & ((1u << (8u * es)) - 1u);
  }
}

// Bit e set: element e of the chunk pair needs pair_slow (its bits differ,
// or, under the strict policy, b's element is a NaN).  1- and 2-byte
// elements are tested four or two to a word: adding 0x7F.. (0x7FFF..) to the
// low seven (fifteen) bits sets an element's top bit iff they are non-zero,
// and adding the gap between the largest finite magnitude and the top bit
// does the same for a NaN; no sum carries into the next element.
template <int DT>
__device__ __forceinline__ uint32_t need_mask(const u32x4& va, const u32x4& vb, bool strict) {
  constexpr int es = Et<DT>::es;
  constexpr bool fp = Et<DT>::fp;
  uint32_t mask = 0;
  if constexpr (es == 8) {
    mask |= ((va.x ^ vb.x) | (va.y ^ vb.y)) != 0u ? 1u : 0u;
    mask |= ((va.z ^ vb.z) | (va.w ^ vb.w)) != 0u ? 2u : 0u;
  } else if constexpr (es == 4) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      bool need = (va[k] ^ vb[k]) != 0u;
      if constexpr (fp) need = need || (strict && (vb[k] & 0x7FFFFFFFu) > 0x7F800000u);
      mask |= need ? (1u << k) : 0u;
    }
  } else if constexpr (es == 2) {
    constexpr uint32_t kNanGap = DT == ASMEVO_F16 ? 0x03FF03FFu : 0x007F007Fu;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t x = va[k] ^ vb[k];
      uint32_t top = ((x & 0x7FFF7FFFu) + 0x7FFF7FFFu) | x;
      if constexpr (fp) top |= strict ? (vb[k] & 0x7FFF7FFFu) + kNanGap : 0u;
      top &= 0x80008000u;
      mask |= (((top >> 15) & 1u) | (top >> 30)) << (2 * k);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t x = va[k] ^ vb[k];
      uint32_t top = ((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x;
      if constexpr (fp) top |= strict ? (vb[k] & 0x7F7F7F7Fu) + 0x01010101u : 0u;
      top &= 0x80808080u;
      mask |= (((top >> 7) | (top >> 14) | (top >> 21) | (top >> 28)) & 0xFu) << (4 * k);
    }
  }
  return mask;
}

// Logical index of walk position q of a reordered N-D segment.
__device__ __forceinline__ uint64_t nd_logical(const NdExt* X, uint64_t q);

// One 16-byte chunk pair holding `nvalid` elements starting at logical index
// i0 (walk position i0 of a reordered N-D segment when `permuted`).
template <int DT, bool ND = false>
__device__ __forceinline__ void chunk(const u32x4& va, const u32x4& vb, uint64_t i0,
                                      uint32_t nvalid, bool tol_mode, bool strict, double atol,
                                      double rtol, Acc& acc, const NdExt* X = nullptr,
                                      bool permuted = false) {
  const u32x4 x = va ^ vb;
  if (((x.x | x.y | x.z | x.w) == 0u) && !strict) return;   // the common case
  uint32_t mask = need_mask<DT>(va, vb, strict);
  mask &= (nvalid >= 32u) ? ~0u : ((1u << nvalid) - 1u);
  while (mask) {
    const uint32_t e = (uint32_t)__builtin_ctz(mask);
    mask &= mask - 1u;
    uint64_t i = i0 + (uint64_t)e;
    if constexpr (ND) {
      if (permuted) i = nd_logical(X, i);
    }
    pair_slow<DT>(elem_dyn<DT>(va, e), elem_dyn<DT>(vb, e), i, tol_mode, strict, atol, rtol, acc);
  }
}

// ------------------------------------------------------- slow path of a tile
// A tile whose chunk pairs hold differences (or, under the strict NaN
// policy, any tile) runs the per-pair rule for every element its need masks
// mark.  Left to each lane, the rule runs as often as the busiest lane has
// marked elements, with the other lanes idle: with 1 % of the elements
// differing (a GEMM output's last-bit flips) nearly every tile takes ~1.1
// rounds of the ~110-instruction rule per chunk row, four rows a tile.  So
// the marked elements of the whole tile are first gathered into the wave's
// slot of LDS (each lane appends its own, at an offset from a wave-wide
// prefix sum of the counts), and the rule then runs once per 64 of them, one
// element per lane.  A tile with more than kSlowCap marked elements (dense
// differences, where every lane is busy anyway) keeps the per-lane loop.
// BITWISE segments need no rule: counts and first indices come from the
// masks directly.
constexpr uint32_t kSlowCap = 256;
struct SlowEntry {       // 16 bytes
  uint32_t ra, rb;       // raw element bits (at most 4 bytes: the rule runs on float types only)
  uint64_t idx;          // logical index, or walk position of a reordered N-D segment
};

__device__ __forceinline__ uint32_t valid_mask(uint32_t nvalid) {
  return nvalid >= 32u ? ~0u : ((1u << nvalid) - 1u);
}

// The wave's marked elements of U chunk pairs: chunk j holds elements
// i0[j] + e, e < nv[j].  The whole wave must be active (the prefix sum and
// the total are wave-wide); callers branch on wave-uniform conditions only.  (The cosine
// variants keep the per-lane loop: the gathering would exceed their
// register budget.)
template <int DT, bool ND, bool COMPACT, int U>
__device__ __forceinline__ void tile_slow(const u32x4 (&va)[U], const u32x4 (&vb)[U], const uint64_t (&i0)[U],
                                          const uint32_t (&nv)[U], uint32_t lane, bool tol_mode, bool strict,
                                          double atol, double rtol, Acc& acc, const NdExt* X, bool permuted,
                                          SlowEntry* slot) {
  if constexpr (!COMPACT) {
#pragma unroll
    for (int j = 0; j < U; ++j)
      chunk<DT, ND>(va[j], vb[j], i0[j], nv[j], tol_mode, strict, atol, rtol, acc, X, permuted);
    return;
  }
  uint32_t m[U];
  uint32_t cnt = 0;
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const u32x4 x = va[j] ^ vb[j];
    m[j] = (((x.x | x.y | x.z | x.w) == 0u) && !strict) ? 0u : need_mask<DT>(va[j], vb[j], strict);
    m[j] &= valid_mask(nv[j]);
    cnt += (uint32_t)__builtin_popcount(m[j]);
  }
  if (!Et<DT>::fp || !tol_mode) {
    // bits differ: that is the whole verdict (need masks mark exactly the
    // differing elements when the policy is not strict)
    acc.bw += cnt;
#pragma unroll
    for (int j = 0; j < U; ++j) {
      if (m[j] == 0u) continue;
      uint64_t i = i0[j] + (uint64_t)__builtin_ctz(m[j]);
      if constexpr (ND) {
        if (permuted) {                        // the lowest logical index need not be the first in walk order
          uint32_t mm = m[j];
          i = ~0ull;
          while (mm) {
            const uint64_t q = nd_logical(X, i0[j] + (uint64_t)__builtin_ctz(mm));
            mm &= mm - 1u;
            i = q < i ? q : i;
          }
        }
      }
      acc.first_bw = i < acc.first_bw ? i : acc.first_bw;
    }
    return;
  }
  // exclusive prefix sum of the lanes' counts, and the wave's total
  uint32_t inc = cnt;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const uint32_t o = (uint32_t)__shfl_up((int)inc, (unsigned)d, kWave);
    inc += lane >= (uint32_t)d ? o : 0u;
  }
  const uint32_t total = (uint32_t)__shfl((int)inc, kWave - 1, kWave);
  if (total > kSlowCap) {                      // dense: every lane has work of its own
#pragma unroll
    for (int j = 0; j < U; ++j)
      chunk<DT, ND>(va[j], vb[j], i0[j], nv[j], tol_mode, strict, atol, rtol, acc, X, permuted);
    return;
  }
  uint32_t off = inc - cnt;
#pragma unroll
  for (int j = 0; j < U; ++j) {
    uint32_t mm = m[j];
    while (mm) {
      const uint32_t e = (uint32_t)__builtin_ctz(mm);
      mm &= mm - 1u;
      SlowEntry E;
      E.ra = (uint32_t)elem_dyn<DT>(va[j], e);
      E.rb = (uint32_t)elem_dyn<DT>(vb[j], e);
      E.idx = i0[j] + (uint64_t)e;
      slot[off++] = E;
    }
  }
  // the entries of every lane are in LDS before any lane reads them
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (uint32_t k = lane; k < total; k += kWave) {
    const SlowEntry E = slot[k];
    uint64_t i = E.idx;
    if constexpr (ND) {
      if (permuted) i = nd_logical(X, i);
    }
    pair_slow<DT>(E.ra, E.rb, i, true, strict, atol, rtol, acc);
  }
  // every lane has read its entries before the slot is written again
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// A whole tile's slow path is deferred: every lane copies its four chunk
// pairs to the wave's slot of LDS (fixed places, no branches: 8 KiB per
// tile), a ballot per chunk row marks the chunk pairs that need the rule
// (bits differ, or under the strict policy b holds a NaN), and the rule runs
// on the marked ones, one per lane, after the next tile's loads have been
// issued, so that it overlaps their latency instead of adding to it.
constexpr uint32_t kSlotBytes = 8192;   // per wave: a tile's chunk pairs
static_assert(2u * kTileChunks * kChunk <= kSlotBytes, "a tile's chunk pairs fit the slot");
static_assert(kSlowCap * sizeof(SlowEntry) <= kSlotBytes, "element gathering fits the slot");

// Does any element of the chunk hold a NaN?
template <int DT>
__device__ __forceinline__ bool any_nan(const u32x4& v) {
  uint32_t hit = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t w = v[k];
    if constexpr (DT == ASMEVO_F32) hit |= (w & 0x7FFFFFFFu) > 0x7F800000u ? 1u : 0u;
    else if constexpr (DT == ASMEVO_BF16) hit |= ((w & 0x7FFF7FFFu) + 0x007F007Fu) & 0x80008000u;
    else if constexpr (DT == ASMEVO_F16) hit |= ((w & 0x7FFF7FFFu) + 0x03FF03FFu) & 0x80008000u;
    else if constexpr (DT == ASMEVO_FP8_E4M3) hit |= ((w & 0x7F7F7F7Fu) + 0x01010101u) & 0x80808080u;
  }
  return hit != 0u;
}

// The marked chunk pairs of a staged tile: ballot masks per chunk row.
template <int U>
struct Staged {
  uint64_t mask[U];
  uint32_t count;        // marked chunk pairs (wave-uniform)
  uint64_t ibase, k0;    // the tile's first logical index and first chunk
};

// Copies the chunk pairs of a whole tile to the slot (a at [0, 256), b at
// [256, 512) in 16-byte units, chunk j * 64 + lane) and marks those that
// need the rule.  The whole wave must be active.
template <int DT, int U>
__device__ __forceinline__ void stage_tile(const u32x4 (&va)[U], const u32x4 (&vb)[U], uint32_t lane, bool strict,
                                           uint64_t ibase, uint64_t k0, u32x4* slot, Staged<U>& st) {
  st.count = 0;
  st.ibase = ibase;
  st.k0 = k0;
#pragma unroll
  for (int j = 0; j < U; ++j) {
    slot[j * kWave + lane] = va[j];
    slot[kTileChunks + j * kWave + lane] = vb[j];
    const u32x4 x = va[j] ^ vb[j];
    bool need = (x.x | x.y | x.z | x.w) != 0u;
    if (strict) need = need || any_nan<DT>(vb[j]);
    st.mask[j] = __ballot(need);
    st.count += (uint32_t)__builtin_popcountll(st.mask[j]);
  }
}

// Position of the r-th set bit (r counted from 0) of m, which has more than
// r set bits: a binary search over bit counts, without branches.
__device__ __forceinline__ uint32_t nth_set_bit(uint64_t m, uint32_t r) {
  uint32_t pos = 0;
  uint32_t c = (uint32_t)__builtin_popcount((uint32_t)m);
  const bool hi = r >= c;
  r -= hi ? c : 0u;
  uint32_t w = hi ? (uint32_t)(m >> 32) : (uint32_t)m;
  pos += hi ? 32u : 0u;
#pragma unroll
  for (int half = 16; half >= 1; half >>= 1) {
    c = (uint32_t)__builtin_popcount(w & ((1u << half) - 1u));
    const bool up = r >= c;
    r -= up ? c : 0u;
    w = up ? (w >> half) : w;
    pos += up ? (uint32_t)half : 0u;
  }
  return pos;
}

// The rule on the marked chunk pairs of a staged tile, one per lane.
template <int DT, bool ND, int U>
__device__ __forceinline__ void run_staged(const u32x4* slot, const Staged<U>& st, uint32_t lane, bool strict,
                                           double atol, double rtol, Acc& acc, const NdExt* X, bool permuted) {
  constexpr int epc = 16 / Et<DT>::es;
  // the stores of every lane are in LDS before any lane reads them
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (uint32_t k = lane; k < st.count; k += kWave) {
    uint32_t r = k, j = 0;
#pragma unroll
    for (int q = 0; q + 1 < U; ++q) {    // the chunk row holding the k-th marked pair
      const uint32_t c = (uint32_t)__builtin_popcountll(st.mask[q]);
      const bool next = j == (uint32_t)q && r >= c;
      r -= next ? c : 0u;
      j += next ? 1u : 0u;
    }
    uint64_t m = st.mask[0];
#pragma unroll
    for (int q = 1; q < U; ++q) m = j == (uint32_t)q ? st.mask[q] : m;
    const uint32_t pos = j * kWave + nth_set_bit(m, r);
    chunk<DT, ND>(slot[pos], slot[kTileChunks + pos], st.ibase + (st.k0 + pos) * epc, epc, true, strict, atol,
                  rtol, acc, X, permuted);
  }
  // every lane has read before the slot is written again
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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

// Elements of a chunk `step` bytes apart (N-D segments whose innermost
// dimension is not unit-stride); invalid elements read as zero on both sides.
template <int DT>
__device__ __forceinline__ u32x4 load_elems_strided(const uint8_t* p, uint32_t nv, uint64_t step) {
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < epc; ++e) {
    if ((uint32_t)e < nv) {
      const uint8_t* q = p + (uint64_t)e * step;
      if constexpr (es == 1) w[e >> 2] |= (uint32_t)*gptr<uint8_t>(q) << (8 * (e & 3));
      else if constexpr (es == 2) w[e >> 1] |= (uint32_t)*gptr<uint16_t>(q) << (16 * (e & 1));
      else if constexpr (es == 4) w[e] = *gptr<uint32_t>(q);
      else {
        const uint64_t raw = *gptr<uint64_t>(q);
        w[2 * e] = (uint32_t)raw;
        w[2 * e + 1] = (uint32_t)(raw >> 32);
      }
    }
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

// A chunk of elements 2 apart: the 32 bytes at p (16-byte aligned) in two
// vector loads, of which the even elements are kept, packed in order.
template <int DT>
__device__ __forceinline__ u32x4 load_pairs(const uint8_t* p) {
  constexpr int es = Et<DT>::es;
  const u32x4 v0 = ld_nt(p), v1 = ld_nt(p + 16);
  if constexpr (es == 8) {
    return u32x4{v0.x, v0.y, v1.x, v1.y};
  } else if constexpr (es == 4) {
    return u32x4{v0.x, v0.z, v1.x, v1.z};
  } else {
    // v_perm_b32 picks bytes of {hi word, lo word} = bytes 7..4, 3..0
    constexpr uint32_t sel = es == 2 ? 0x05040100u : 0x06040200u;
    return u32x4{__builtin_amdgcn_perm(v0.y, v0.x, sel), __builtin_amdgcn_perm(v0.w, v0.z, sel),
                 __builtin_amdgcn_perm(v1.y, v1.x, sel), __builtin_amdgcn_perm(v1.w, v1.z, sel)};
  }
}

// Chunk c of a row of an N-D segment whose rows start at pa / pb.  A gather
// whose elements are 2 apart in an operand (pair2a / pair2b) loads that
// operand's chunk as 32 contiguous bytes, unless it is the row's last chunk:
// every other chunk is followed by another element of the same row, so the
// 32 bytes end before it and stay inside the view.
template <int DT>
__device__ __forceinline__ void load_nd_chunk(const uint8_t* pa, const uint8_t* pb, uint64_t c,
                                              uint32_t nbytes, bool vec, bool gather, uint64_t in_sa,
                                              uint64_t in_sb, bool pair2a, bool pair2b, bool last,
                                              u32x4& va, u32x4& vb) {
  if (gather) {
    constexpr int epc = 16 / Et<DT>::es;
    const uint32_t nv = nbytes / Et<DT>::es;
    if (pair2a && !last) va = load_pairs<DT>(pa + c * 2 * kChunk);
    else va = load_elems_strided<DT>(pa + c * epc * in_sa, nv, in_sa);
    if (pair2b && !last) vb = load_pairs<DT>(pb + c * 2 * kChunk);
    else vb = load_elems_strided<DT>(pb + c * epc * in_sb, nv, in_sb);
  } else {
    load_chunk<DT>(pa + c * kChunk, pb + c * kChunk, nbytes, vec, va, vb);
  }
}

// A span row (kSegSpan): chunk c of the row's covering bytes keeps the
// elements at row positions that are multiples of s (bits 0-7 of `span`) and
// masks the others to zero, the same on both operands, so they compare equal
// on every path.  `r` is (c * elements per chunk) mod s; bits 8-23 of `span`
// hold the positions k < 16 with k mod s == 0.
template <int DT>
__device__ __forceinline__ void span_mask(uint32_t span, uint32_t r, u32x4& va, u32x4& vb) {
  constexpr uint32_t es = Et<DT>::es, epc = 16 / es;
  const uint32_t s = span & 0xFFu;
  const uint32_t t = r == 0 ? 0u : s - r;                      // first kept position in the chunk
  const uint32_t bits = t < epc ? ((span >> 8) << t) & ((1u << epc) - 1u) : 0u;
  u32x4 m;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint32_t w;
    if constexpr (es == 8) {
      w = (bits >> (k >> 1)) & 1u ? ~0u : 0u;
    } else if constexpr (es == 4) {
      w = (bits >> k) & 1u ? ~0u : 0u;
    } else if constexpr (es == 2) {
      w = ((bits >> (2 * k)) & 1u ? 0x0000FFFFu : 0u) | ((bits >> (2 * k + 1)) & 1u ? 0xFFFF0000u : 0u);
    } else {
      const uint32_t x = (bits >> (4 * k)) & 0xFu;             // four bits to the low bits of four bytes
      w = ((x * 0x00204081u) & 0x01010101u) * 0xFFu;
    }
    m[k] = w;
  }
  va &= m;
  vb &= m;
}

// (c * elements per chunk) mod s for chunk c of a span row.
template <int DT>
__device__ __forceinline__ uint32_t span_residue(uint64_t c, uint32_t span) {
  const uint64_t s = span & 0xFFu;
  const uint64_t p = c * (uint64_t)(16 / Et<DT>::es);
  return (uint32_t)(((p >> 32) == 0) ? (uint32_t)p % (uint32_t)s : p % s);
}

// n / d and n % d, in 32 bits when both fit.
__device__ __forceinline__ void divmod(uint64_t n, uint64_t d, uint64_t& q, uint64_t& r) {
  if (((n | d) >> 32) == 0) {
    const uint32_t q32 = (uint32_t)n / (uint32_t)d;
    q = q32;
    r = n - (uint64_t)q32 * d;
  } else {
    q = n / d;
    r = n - q * d;
  }
}

// Byte offsets of row r of an N-D segment in both operands.
__device__ __forceinline__ void nd_row_offsets(const NdExt* X, uint64_t r, uint64_t& oa, uint64_t& ob) {
  oa = 0;
  ob = 0;
  const int nd = (int)X->nouter;
#pragma unroll 1
  for (int d = nd - 1; d > 0; --d) {
    uint64_t q, idx;
    divmod(r, X->oshape[d], q, idx);
    oa += idx * X->opa[d];
    ob += idx * X->opb[d];
    r = q;
  }
  if (nd > 0) {                     // the outermost index is what remains (r < oshape[0])
    oa += r * X->opa[0];
    ob += r * X->opb[0];
  }
}

// The outer walk of an N-D segment of several short rows (X is then never
// null), read once per range.  The short-row paths find the row of every
// chunk, and reading the extension there cost each wave-load three more
// vector loads: a view of 256-byte rows over 2 x 8 GiB took 3.12 ms against
// 2.64 ms with this in the plain diff, and 5.90 against 4.96 ms with this and
// the DPP group fold in the cosine pass.  With one outer dimension (a matrix,
// or dimensions that merged) a row's offsets are one product each.
struct NdRows {
  const NdExt* X;
  uint32_t nouter;
  uint64_t pa0, pb0;
};
__device__ __forceinline__ NdRows nd_rows(const NdExt* X) {
  return NdRows{X, X->nouter, X->opa[0], X->opb[0]};
}
__device__ __forceinline__ void row_offsets(const NdRows& R, uint64_t r, uint64_t& oa, uint64_t& ob) {
  if (R.nouter == 1) {
    oa = r * R.pa0;
    ob = r * R.pb0;
  } else {
    nd_row_offsets(R.X, r, oa, ob);
  }
}

__device__ __forceinline__ uint64_t nd_logical(const NdExt* X, uint64_t q) {
  uint64_t l = 0;
  const int ni = (int)X->ni;
#pragma unroll 1
  for (int d = ni - 1; d >= 0; --d) {
    uint64_t rest, idx;
    divmod(q, X->ishape[d], rest, idx);
    l += idx * X->lpitch[d];
    q = rest;
  }
  return X->index_base + l;
}

// ------------------------------------------------------------ cosine sums
// Lane sums of one 4096-byte block (a*b, a*a, b*b over pairs with both
// values finite).  Products of two values of any float element type are
// exact in fp64, so fma(A, B, s) rounds exactly like s + A*B.
struct Cos {
  double ab, aa, bb;
};

// Exact fp64 value of finite element e (a compile-time position) of a chunk,
// through the hardware conversions: bf16 by a shift into binary32, fp16 by
// v_cvt_f32_f16 (exact, subnormals kept), fp8 e4m3 by v_cvt_f32_fp8 (the
// OCP E4M3FN decode on gfx950, checked against the oracle for all 256
// patterns), then binary32 -> binary64, which is exact.
template <int DT>
__device__ __forceinline__ double elem_f64(const u32x4& v, int e) {
  if constexpr (DT == ASMEVO_F32) {
    return (double)__uint_as_float(v[e]);
  } else if constexpr (DT == ASMEVO_BF16) {
    const uint32_t w = v[e >> 1];
    return (double)__uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  } else if constexpr (DT == ASMEVO_F16) {
    const uint16_t h = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    return (double)(float)__builtin_bit_cast(_Float16, h);
  } else {
    const int w = (int)v[e >> 2];
    switch (e & 3) {   // the byte selector must be a literal
      case 0: return (double)__builtin_amdgcn_cvt_f32_fp8(w, 0);
      case 1: return (double)__builtin_amdgcn_cvt_f32_fp8(w, 1);
      case 2: return (double)__builtin_amdgcn_cvt_f32_fp8(w, 2);
      default: return (double)__builtin_amdgcn_cvt_f32_fp8(w, 3);
    }
  }
}

// Does any element of the chunk have an all-ones exponent (Inf or NaN)?
template <int DT>
__device__ __forceinline__ bool any_nonfinite(const u32x4& v) {
  uint32_t hit = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t w = v[k];
    if constexpr (DT == ASMEVO_F32) {
      hit |= ((w & 0x7F800000u) == 0x7F800000u) ? 1u : 0u;
    } else if constexpr (DT == ASMEVO_BF16 || DT == ASMEVO_F16) {
      constexpr uint32_t e = DT == ASMEVO_BF16 ? 0x7F80u : 0x7C00u;
      hit |= ((w & e) == e) ? 1u : 0u;
      hit |= (((w >> 16) & e) == e) ? 1u : 0u;
    } else {
      // fp8 e4m3: only S.1111.111 is not finite
      const uint32_t m = w & 0x7F7F7F7Fu;
      const uint32_t t = m ^ 0x7F7F7F7Fu;            // a zero byte where the pattern is 0x7F
      hit |= ((t - 0x01010101u) & ~t & 0x80808080u) ? 1u : 0u;
    }
  }
  return hit != 0;
}

// Lane sums of one chunk with no checks: a NaN or Inf element makes a sum
// non-finite (fp64 cannot overflow here: |a*b| < 2^256 and there are fewer
// than 2^52 terms), which the caller detects to redo the block with checks.
template <int DT>
__device__ __forceinline__ void cos_chunk_fast(const u32x4& va, const u32x4& vb, Cos& c) {
  constexpr int epc = 16 / Et<DT>::es;
  if constexpr (DT == ASMEVO_FP8_E4M3) {
    // v_cvt_pk_f32_fp8: two bytes of a word per instruction
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      // the half selector must be a literal: low bytes first, then high bytes
      const auto fa0 = __builtin_amdgcn_cvt_pk_f32_fp8((int)va[k], false);
      const auto fb0 = __builtin_amdgcn_cvt_pk_f32_fp8((int)vb[k], false);
      const auto fa1 = __builtin_amdgcn_cvt_pk_f32_fp8((int)va[k], true);
      const auto fb1 = __builtin_amdgcn_cvt_pk_f32_fp8((int)vb[k], true);
      const double A[4] = {(double)fa0[0], (double)fa0[1], (double)fa1[0], (double)fa1[1]};
      const double B[4] = {(double)fb0[0], (double)fb0[1], (double)fb1[0], (double)fb1[1]};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c.ab = __builtin_fma(A[q], B[q], c.ab);
        c.aa = __builtin_fma(A[q], A[q], c.aa);
        c.bb = __builtin_fma(B[q], B[q], c.bb);
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < epc; ++e) {
      const double A = elem_f64<DT>(va, e);
      const double B = elem_f64<DT>(vb, e);
      c.ab = __builtin_fma(A, B, c.ab);
      c.aa = __builtin_fma(A, A, c.aa);
      c.bb = __builtin_fma(B, B, c.bb);
    }
  }
}

// Lane sums of the first `nvalid` elements of a chunk, skipping (and
// counting) pairs with a NaN or Inf.
template <int DT>
__device__ __forceinline__ void cos_chunk(const u32x4& va, const u32x4& vb, uint32_t nvalid, Cos& c,
                                          uint32_t& nonfinite) {
#pragma unroll 1
  for (uint32_t e = 0; e < nvalid; ++e) {
    double A = 0.0, B = 0.0;
    if (decode<DT>(elem_dyn<DT>(va, e), A) != 0 || decode<DT>(elem_dyn<DT>(vb, e), B) != 0) {
      nonfinite += 1;
      continue;
    }
    c.ab = __builtin_fma(A, B, c.ab);
    c.aa = __builtin_fma(A, A, c.aa);
    c.bb = __builtin_fma(B, B, c.bb);
  }
}

__device__ __forceinline__ uint32_t lo32(double v) { return (uint32_t)(uint64_t)__double_as_longlong(v); }
__device__ __forceinline__ uint32_t hi32(double v) { return (uint32_t)((uint64_t)__double_as_longlong(v) >> 32); }
__device__ __forceinline__ double f64_of(uint32_t hi, uint32_t lo) {
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// v moved across lanes by one DPP pattern (CTRL: the instruction's dpp_ctrl),
// 32 bits at a time: row_ror:R (0x120 + R) gives lane i of each 16-lane row
// the value of lane (i + 16 - R) mod 16; quad_perm 0x4E and 0xB1 give lane i
// of each group of four the value of lane i ^ 2 and i ^ 1.  Every lane has a
// source under these patterns, so no old value is merged in, and the
// compiler zeroes no register before each move.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Lanes 0-15 and 32-47 receive v of the lane 16 up (v_permlane16_swap);
// the other lanes receive anything.
__device__ __forceinline__ double row_up16(double v) {
  const uint32_t any = __builtin_nondeterministic_value(0u);
  const auto lo = __builtin_amdgcn_permlane16_swap(lo32(v), any, false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap(hi32(v), any, false, false);
  return f64_of(hi[1], lo[1]);
}

// Folds the lane sums of a block and stores its record out[0..3] =
// {Σab, Σaa, Σbb, 0}: the xor butterfly's tree, lanes 32 apart first, then 16,
// 8, 4, 2, 1 (fp64 addition commutes, and the lane sums are finite, so every
// lane that ends with a sum holds the same bits).  The three sums share
// registers as they fold, because each step leaves half the lanes unused:
//  * v_permlane32_swap of Σab (first operand) with Σaa (second) hands lanes
//    0-31 the upper half of Σab and lanes 32-63 the lower half of Σaa, so one
//    addition gives Σab's pair sums in lanes 0-31 and Σaa's in lanes 32-63;
//    Σbb's pair sums go to lanes 0-31 of a second register;
//  * v_permlane16_swap of those two registers, then one addition: Σab's
//    partial sums fill row 0 (lanes 0-15), Σbb's row 1, Σaa's row 2;
//  * the last four steps stay within rows (DPP), all three sums at once.
// Lanes 0-3 write the record with one store.  The whole wave must be active.
__device__ __forceinline__ void cos_store(const Cos& c, double* out, uint32_t lane) {
  const auto l1 = __builtin_amdgcn_permlane32_swap(lo32(c.ab), lo32(c.aa), false, false);
  const auto h1 = __builtin_amdgcn_permlane32_swap(hi32(c.ab), hi32(c.aa), false, false);
  const double p = f64_of(h1[0], l1[0]) + f64_of(h1[1], l1[1]);     // lanes 0-31: Σab, 32-63: Σaa
  const uint32_t any = __builtin_nondeterministic_value(0u);        // its lanes end unused
  const auto l2 = __builtin_amdgcn_permlane32_swap(lo32(c.bb), any, false, false);
  const auto h2 = __builtin_amdgcn_permlane32_swap(hi32(c.bb), any, false, false);
  const double q = f64_of(h2[0], l2[0]) + f64_of(h2[1], l2[1]);     // lanes 0-31: Σbb
  const auto l3 = __builtin_amdgcn_permlane16_swap(lo32(p), lo32(q), false, false);
  const auto h3 = __builtin_amdgcn_permlane16_swap(hi32(p), hi32(q), false, false);
  double t = f64_of(h3[0], l3[0]) + f64_of(h3[1], l3[1]);           // rows 0, 1, 2: Σab, Σbb, Σaa
  t = t + dpp_f64<0x128>(t);      // row_ror:8: lanes 0-7 of a row get i + 8
  t = t + dpp_f64<0x12C>(t);      // row_ror:12: lanes 0-3 get i + 4
  t = t + dpp_f64<0x4E>(t);       // quad_perm [2,3,0,1]
  t = t + dpp_f64<0xB1>(t);       // quad_perm [1,0,3,2]
  const double s_aa = f64_of((uint32_t)__builtin_amdgcn_readlane((int)hi32(t), 32),
                             (uint32_t)__builtin_amdgcn_readlane((int)lo32(t), 32));
  const double s_bb = f64_of((uint32_t)__builtin_amdgcn_readlane((int)hi32(t), 16),
                             (uint32_t)__builtin_amdgcn_readlane((int)lo32(t), 16));
  if (lane < (uint32_t)kCosRec) {
    double v = 0.0;
    v = lane == 2 ? s_bb : v;
    v = lane == 1 ? s_aa : v;
    v = lane == 0 ? t : v;
    out[lane] = v;
  }
}

// All tiles [t_begin, t_end) of one segment.  COS: also the block sums of
// each tile into `partials` (three doubles per global tile index).  ND: rows
// are placed by the segment's N-D extension X (the 2-D code otherwise).
// The cosine variant on rows of at most kNarrowCosChunks chunks, each one
// block (one tile).  Tiling row by row would leave most of a wave idle: a row
// of R chunks fills lanes 0..R-1 only.  Instead, with N the power of two at or
// above R, the block sum is an xor butterfly over the row's first N chunks.
// That is the block sum of the definition: in the 64-lane butterfly of a
// row's block, the steps m >= N add lanes that hold +0.0 to lanes 0..N-1 (a
// lane sum is never -0.0), so lane 0 ends with the butterfly over 0..N-1.
// A row takes P = N / 2 lanes (one lane for a one-chunk row), a wave-load
// G = 64 / P rows, row g in lanes gP..gP+P-1.  Lane t holds chunks t and
// t + P: adding their sums is the butterfly's first step (chunk c with
// c + N / 2) with no data moved, and the other steps go across the P lanes.
constexpr uint32_t kNarrowCosChunks = 32;

// QMAX: chunks a lane at most (2 or 4).
template <int DT, bool ND, uint32_t QMAX = 2>
__device__ __forceinline__ void diff_range_narrow_cos(const DiffSeg& S, const NdExt* X, uint64_t t_begin,
                                                   uint64_t t_end, uint32_t step, uint32_t lane, Acc& acc,
                                                   double* partials, uint32_t& nonfinite, bool tol_mode,
                                                   bool strict, bool vec, bool gather, bool pair2a, bool pair2b,
                                                   uint64_t in_sa, uint64_t in_sb, uint64_t ibase0, bool permuted) {
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  const uint32_t R = (uint32_t)S.row_chunks;
  uint32_t lg = 0;
  while ((1u << lg) < R) ++lg;
  // Q = QMAX chunks a lane, fewer for rows of fewer chunks (in diff_kernel
  // four spilled registers and ran slower than two)
  static_assert(QMAX == 2 || QMAX == 4, "two or four chunks a lane");
  constexpr uint32_t QLOG = QMAX == 4 ? 2u : 1u;
  const uint32_t lq = lg < QLOG ? lg : QLOG;
  const uint32_t P = 1u << (lg - lq), G = (uint32_t)kWave >> (lg - lq);
  const uint32_t Q = 1u << lq;
  const uint32_t g = lane >> (lg - lq), t = lane & (P - 1);
  NdRows walk{};
  if constexpr (ND) walk = nd_rows(X);     // entered for segments of several rows only
  const uint8_t* a0 = reinterpret_cast<const uint8_t*>(S.a);
  const uint8_t* b0 = reinterpret_cast<const uint8_t*>(S.b);
  for (uint64_t tile = t_begin; tile < t_end; tile += (uint64_t)step * G) {
    const uint64_t row = tile + (uint64_t)g * step;
    u32x4 va[QMAX], vb[QMAX];
    uint32_t nb[QMAX];
    uint64_t oa = 0, ob = 0;
    if constexpr (ND) {
      if (row < t_end) row_offsets(walk, row, oa, ob);
    }
#pragma unroll
    for (uint32_t k = 0; k < QMAX; ++k) {
      const uint32_t c = t + k * P;
      va[k] = u32x4{0u, 0u, 0u, 0u};
      vb[k] = u32x4{0u, 0u, 0u, 0u};
      nb[k] = 0;
      if (row < t_end && k < Q && c < R) {
        const uint64_t cb = (uint64_t)c * kChunk;
        const uint64_t rem = S.row_bytes - cb;
        nb[k] = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
        if constexpr (ND) {
          load_nd_chunk<DT>(a0 + oa, b0 + ob, c, nb[k], vec, gather, in_sa, in_sb, pair2a, pair2b, c + 1 == R,
                            va[k], vb[k]);
        } else {
          load_chunk<DT>(a0 + row * S.a_pitch + cb, b0 + row * S.b_pitch + cb, nb[k], vec, va[k], vb[k]);
        }
      }
    }
    Cos s[QMAX];
#pragma unroll
    for (uint32_t k = 0; k < QMAX; ++k) {
      chunk<DT, ND>(va[k], vb[k], ibase0 + row * S.cols + (uint64_t)(t + k * P) * epc, nb[k] / es, tol_mode,
                    strict, S.atol, S.rtol, acc, X, permuted);
      s[k] = Cos{0.0, 0.0, 0.0};
      cos_chunk_fast<DT>(va[k], vb[k], s[k]);
      if (!(__builtin_isfinite(s[k].ab) && __builtin_isfinite(s[k].aa) && __builtin_isfinite(s[k].bb))) {
        s[k] = Cos{0.0, 0.0, 0.0};
        cos_chunk<DT>(va[k], vb[k], nb[k] / es, s[k], nonfinite);
      }
    }
    // the first steps, in the lane (chunk k with k + QMAX / 2, then with k + 1)
#pragma unroll
    for (uint32_t h = QMAX / 2; h >= 1; h /= 2) {
#pragma unroll
      for (uint32_t k = 0; k < h; ++k) {
        s[k].ab = s[k].ab + s[k + h].ab;
        s[k].aa = s[k].aa + s[k + h].aa;
        s[k].bb = s[k].bb + s[k + h].bb;
      }
    }
    Cos cs = s[0];
    // The other steps over each group of P lanes; only the group's first lane
    // (t == 0) keeps its sum, so a step may hand the other lanes anything.
    // Within 16-lane rows the steps are DPP moves (row_ror:8 is xor 8;
    // row_ror:12 gives lanes 0-3 of each 8 the value 4 lanes up), across rows
    // (P = 32, only reached by a build with QMAX = 1) one swap of odd and even
    // rows.
    if (P == 32) {
      cs.ab = cs.ab + row_up16(cs.ab);
      cs.aa = cs.aa + row_up16(cs.aa);
      cs.bb = cs.bb + row_up16(cs.bb);
    }
    if (P >= 16) {
      cs.ab = cs.ab + dpp_f64<0x128>(cs.ab);
      cs.aa = cs.aa + dpp_f64<0x128>(cs.aa);
      cs.bb = cs.bb + dpp_f64<0x128>(cs.bb);
    }
    if (P >= 8) {
      cs.ab = cs.ab + dpp_f64<0x12C>(cs.ab);
      cs.aa = cs.aa + dpp_f64<0x12C>(cs.aa);
      cs.bb = cs.bb + dpp_f64<0x12C>(cs.bb);
    }
    if (P >= 4) {
      cs.ab = cs.ab + dpp_f64<0x4E>(cs.ab);
      cs.aa = cs.aa + dpp_f64<0x4E>(cs.aa);
      cs.bb = cs.bb + dpp_f64<0x4E>(cs.bb);
    }
    if (P >= 2) {
      cs.ab = cs.ab + dpp_f64<0xB1>(cs.ab);
      cs.aa = cs.aa + dpp_f64<0xB1>(cs.aa);
      cs.bb = cs.bb + dpp_f64<0xB1>(cs.bb);
    }
    if (t == 0 && row < t_end) {
      double* rec = partials + kCosRec * (S.tile_begin + row);
      rec[0] = cs.ab;
      rec[1] = cs.aa;
      rec[2] = cs.bb;
      rec[3] = 0.0;
    }
  }
}

// ROWS: only segments of long rows, 16-byte aligned and unit-stride, of a
// float type (the cosine variant for calls made only of such segments): the
// row-tiled whole-tile code alone.  GATHERS: only gathers of long rows (one
// row, or rows of more than kNarrowCosChunks chunks) of a float type whose
// elements are 2 apart in both operands: the chunk-by-chunk code alone, two
// chunks in flight, each a pair of 16-byte loads per operand.
template <int DT, bool COS, bool ND, bool ROWS = false, bool GATHERS = false>
__device__ __forceinline__ void diff_range(const DiffSeg& S, const NdExt* X, uint64_t t_begin,
                                           uint64_t t_end, uint32_t step, uint32_t lane, Acc& acc,
                                           double* partials, uint32_t& nonfinite, uint8_t* slot_bytes) {
  constexpr int es = Et<DT>::es;
  constexpr int epc = 16 / es;
  constexpr int U = kDiffUnroll;
  constexpr bool kCos = COS && Et<DT>::fp;
  // whole tiles defer their slow path in the plain 2-D diff only (the N-D
  // variant would exceed its register budget: 128 for 4 waves per SIMD)
  constexpr bool kDefer = !COS && !ND;
  SlowEntry* slot = reinterpret_cast<SlowEntry*>(slot_bytes);
  u32x4* stage = reinterpret_cast<u32x4*>(slot_bytes);
  const bool tol_mode = S.mode == ASMEVO_TOLERANCE;
  const bool strict = (S.flags & kSegStrict) != 0;
  const bool vec = (S.flags & kSegVec) != 0;
  const uint8_t* a0 = reinterpret_cast<const uint8_t*>(S.a);
  const uint8_t* b0 = reinterpret_cast<const uint8_t*>(S.b);
  uint64_t ibase0 = 0, in_sa = 0, in_sb = 0;
  bool gather = false, permuted = false, pair2a = false, pair2b = false;
  uint32_t span = 0;                      // a span row's stride and pattern (the plain N-D diff)
  if constexpr (ND && !COS) span = (S.flags & kSegSpan) ? S.span : 0u;
  if constexpr (ND) {
    permuted = (S.flags & kSegPermuted) != 0;
    ibase0 = permuted ? 0 : S.nd_index_base;  // reordered: indices are mapped on a mismatch
    gather = (S.flags & kSegGather) != 0;
    pair2a = (S.flags & kSegPair2A) != 0;
    pair2b = (S.flags & kSegPair2B) != 0;
    if (X != nullptr) {
      in_sa = X->in_sa;
      in_sb = X->in_sb;
    }
  }

  if (!kCos && (S.flags & kSegNarrow)) {
    // Short rows: tiles over the row-major chunk space, each lane finds its
    // row; all U chunk pairs of a tile are loaded before any is checked.  A
    // lane divides once per tile (its first chunk) and steps its other chunks,
    // 64 apart, by the quotient and remainder of 64 by the row's chunks.
    const uint64_t total = S.rows * S.row_chunks;
    const uint64_t n_rc = S.row_chunks;
    const uint64_t q64 = (uint64_t)kWave / n_rc, r64 = (uint64_t)kWave - q64 * n_rc;
    // (the cosine kernels compile this path for their integer segments and
    // keep the per-chunk walk: with the new one there, the changed layout of
    // the whole kernel made its sliced-row views 14 % slower)
    NdRows walk{};
    if constexpr (ND && !COS) {
      if (S.rows > 1) walk = nd_rows(X);   // a segment of several rows has an extension
    }
    for (uint64_t tile = t_begin; tile < t_end; tile += step) {
      const uint64_t k0 = tile * (uint64_t)kTileChunks;
      u32x4 va[U], vb[U];
      uint32_t nb[U];
      uint64_t i0[U];
      uint64_t r, c;
      divmod(k0 + lane, n_rc, r, c);
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint64_t k = k0 + (uint64_t)(j * kWave) + lane;
        va[j] = u32x4{0u, 0u, 0u, 0u};
        vb[j] = u32x4{0u, 0u, 0u, 0u};
        nb[j] = 0;
        i0[j] = 0;
        if (j > 0) {                      // (r, c) of chunk k from those of k - 64
          r += q64;
          c += r64;
          if (c >= n_rc) {
            c -= n_rc;
            r += 1;
          }
        }
        if (k < total) {
          const uint64_t cb = c * kChunk;
          const uint64_t rem = S.row_bytes - cb;
          nb[j] = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
          if constexpr (ND) {
            uint64_t oa = 0, ob = 0;
            if (S.rows > 1) {
              if constexpr (COS) nd_row_offsets(X, r, oa, ob);
              else row_offsets(walk, r, oa, ob);
            }
            load_nd_chunk<DT>(a0 + oa, b0 + ob, c, nb[j], vec, gather, in_sa, in_sb, pair2a, pair2b,
                              c + 1 == S.row_chunks, va[j], vb[j]);
            if (span) span_mask<DT>(span, span_residue<DT>(c, span), va[j], vb[j]);
          } else {
            load_chunk<DT>(a0 + r * S.a_pitch + cb, b0 + r * S.b_pitch + cb, nb[j], vec, va[j], vb[j]);
          }
          i0[j] = ibase0 + r * S.cols + c * epc;
        }
      }
      uint32_t nv[U];
#pragma unroll
      for (int j = 0; j < U; ++j) nv[j] = nb[j] / es;
      tile_slow<DT, ND, !COS, U>(va, vb, i0, nv, lane, tol_mode, strict, S.atol, S.rtol, acc, X, permuted, slot);
    }
    return;
  }

  if constexpr (kCos && !ROWS && !GATHERS) {
    if (S.rows > 1 && S.row_chunks <= (uint64_t)kNarrowCosChunks) {
      diff_range_narrow_cos<DT, ND>(S, X, t_begin, t_end, step, lane, acc, partials, nonfinite, tol_mode, strict,
                                    vec, gather, pair2a, pair2b, in_sa, in_sb, ibase0, permuted);
      return;
    }
  }

  // Row-tiled: every tile lies inside one row (and is one cosine block).
  const uint64_t tpr = ND ? (S.row_chunks + kTileChunks - 1) / kTileChunks : (uint64_t)S.tiles_per_row;
  for (uint64_t tile = t_begin; tile < t_end; tile += step) {
    uint64_t r = 0, kt = tile;
    if (S.rows > 1) {
      if constexpr (ND) {
        divmod(tile, tpr, r, kt);
      } else {
        r = (uint32_t)tile / (uint32_t)tpr;
        kt = tile - r * tpr;
      }
    }
    const uint8_t* pa;
    const uint8_t* pb;
    if constexpr (ND) {
      uint64_t oa = 0, ob = 0;
      if (S.rows > 1) nd_row_offsets(X, r, oa, ob);     // one row: no extension, offset 0
      pa = a0 + oa;
      pb = b0 + ob;
    } else {
      pa = a0 + r * S.a_pitch;
      pb = b0 + r * S.b_pitch;
    }
    const uint64_t ibase = ibase0 + r * S.cols;
    const uint64_t k0 = kt * (uint64_t)kTileChunks;
    Cos cs{0.0, 0.0, 0.0};
    const bool whole = vec && k0 + kTileChunks <= S.full_chunks;
    // The cosine variant also takes the last tile of an aligned unit-stride
    // row here, with bounded loads: the bytes past the row's end load as zeros
    // on both sides, and adding a +0.0 product leaves a lane sum unchanged (a
    // lane sum starts at +0.0, so it is never -0.0).
    if (!GATHERS && (ROWS || whole || (kCos && vec && !gather))) {
      // Whole tile: issue all loads first, then one combined check.
      u32x4 va[U], vb[U];
      uint32_t nv[U];                      // valid elements per chunk
      if (kCos && !whole && ND && S.full_chunks > 0) {
        // Every lane loads, with no branch around its loads: a chunk past the
        // row's whole chunks reads the last whole one (which this tile reads
        // too) and is then cleared, and a partial last chunk is read again
        // element by element.  (Loads under a branch, into registers zeroed
        // first, left waits between them in some builds of this kernel.)
        const uint64_t fc = S.full_chunks;
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
          const uint64_t cc = c < fc ? c : fc - 1;
          va[j] = ld_nt(pa + cc * kChunk);
          vb[j] = ld_nt(pb + cc * kChunk);
        }
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
          nv[j] = (uint32_t)epc;
          if (c >= fc) {
            va[j] = u32x4{0u, 0u, 0u, 0u};
            vb[j] = u32x4{0u, 0u, 0u, 0u};
            nv[j] = 0;
            if (c < S.row_chunks) {            // the partial last chunk
              const uint32_t nb = (uint32_t)(S.row_bytes - c * kChunk);
              load_chunk<DT>(pa + c * kChunk, pb + c * kChunk, nb, true, va[j], vb[j]);
              nv[j] = nb / es;
            }
          }
        }
      } else if (kCos && !whole) {
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
          va[j] = u32x4{0u, 0u, 0u, 0u};
          vb[j] = u32x4{0u, 0u, 0u, 0u};
          nv[j] = 0;
          if (c < S.row_chunks) {
            const uint64_t rem = S.row_bytes - c * kChunk;
            const uint32_t nb = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
            load_chunk<DT>(pa + c * kChunk, pb + c * kChunk, nb, true, va[j], vb[j]);
            nv[j] = nb / es;
          }
        }
      } else {
        const uint8_t* qa = pa + (k0 + lane) * kChunk;
        const uint8_t* qb = pb + (k0 + lane) * kChunk;
#pragma unroll
        for (int j = 0; j < U; ++j) {
          va[j] = ld_nt(qa + j * kWave * kChunk);
          vb[j] = ld_nt(qb + j * kWave * kChunk);
          nv[j] = epc;
        }
        if (span) {
          // a lane's chunks are 64 apart: the residue steps by (64 * elements per chunk) mod s
          const uint32_t sp = span & 0xFFu;
          const uint32_t step_r = (uint32_t)(kWave * epc) % sp;
          uint32_t r = span_residue<DT>(k0 + lane, span);
#pragma unroll
          for (int j = 0; j < U; ++j) {
            span_mask<DT>(span, r, va[j], vb[j]);
            r += step_r;
            r = r >= sp ? r - sp : r;
          }
        }
      }
      u32x4 x = va[0] ^ vb[0];
#pragma unroll
      for (int j = 1; j < U; ++j) x |= va[j] ^ vb[j];
      // (unlikely: the slow path is then laid out away from the loop, which
      // runs straight through to the next tile's loads with one taken branch;
      // with the slow path inline and jumped over, the sweep measured 1-2 %
      // slower)
      // (the gathering slow path needs the whole wave: the branch is taken by
      // every lane when any lane's chunks differ)
      if (__builtin_expect(__ballot((x.x | x.y | x.z | x.w) != 0u) != 0ull || strict, 0)) {
        if constexpr (COS) {
#pragma unroll
          for (int j = 0; j < U; ++j)
            chunk<DT, ND>(va[j], vb[j], ibase + (k0 + (uint64_t)(j * kWave) + lane) * epc, nv[j], tol_mode,
                          strict, S.atol, S.rtol, acc, X, permuted);
        } else if constexpr (!kDefer) {
          uint64_t i0[U];
#pragma unroll
          for (int j = 0; j < U; ++j) i0[j] = ibase + (k0 + (uint64_t)(j * kWave) + lane) * epc;
          tile_slow<DT, ND, true, U>(va, vb, i0, nv, lane, tol_mode, strict, S.atol, S.rtol, acc, X, permuted,
                                     slot);
        } else {
          // Slow mode: this tile and the whole tiles after it that need the
          // rule too, each tile's rule run from LDS while the next tile's
          // loads are in flight; back to the loop above after the first tile
          // that needs nothing, or before a tile that is not whole.  (The
          // loop above is left as it was: checking for staged work there
          // cost the difference-free sweep 0.6 %.)
          uint64_t i0[U];
          uint64_t cur = tile;
          uint64_t ib = ibase, kc = k0;
          uint64_t rc = r, ktc = kt;     // row and tile-in-row of `cur`
          Staged<U> st;
          bool pending = false;
          for (;;) {
            if (Et<DT>::fp && tol_mode) {
              stage_tile<DT, U>(va, vb, lane, strict, ib, kc, stage, st);
              pending = st.count != 0;
            } else {                     // bitwise verdicts: cheap, now
#pragma unroll
              for (int j = 0; j < U; ++j) i0[j] = ib + (kc + (uint64_t)(j * kWave) + lane) * epc;
              tile_slow<DT, ND, true, U>(va, vb, i0, nv, lane, tol_mode, strict, S.atol, S.rtol, acc, X,
                                         permuted, slot);
            }
            const uint64_t nxt = cur + step;
            if (nxt >= t_end) break;
            uint64_t r2 = 0, kt2 = nxt;
            if (S.rows > 1) {
              if (step == 1) {           // the next tile of the row, or the first of the next row
                const bool wrap = ktc + 1 == tpr;
                r2 = wrap ? rc + 1 : rc;
                kt2 = wrap ? 0 : ktc + 1;
              } else {
                r2 = (uint32_t)nxt / (uint32_t)tpr;
                kt2 = nxt - r2 * tpr;
              }
            }
            const uint64_t k2 = kt2 * (uint64_t)kTileChunks;
            if (k2 + kTileChunks > S.full_chunks) break;      // not whole: the loop above takes it
            const uint8_t* qa = a0 + r2 * S.a_pitch + (k2 + lane) * kChunk;
            const uint8_t* qb = b0 + r2 * S.b_pitch + (k2 + lane) * kChunk;
#pragma unroll
            for (int j = 0; j < U; ++j) {
              va[j] = ld_nt(qa + j * kWave * kChunk);
              vb[j] = ld_nt(qb + j * kWave * kChunk);
            }
            if (pending) {               // overlaps the loads just issued
              run_staged<DT, ND, U>(stage, st, lane, strict, S.atol, S.rtol, acc, X, permuted);
              pending = false;
            }
            cur = nxt;
            ib = ibase0 + r2 * S.cols;
            kc = k2;
            rc = r2;
            ktc = kt2;
            u32x4 y = va[0] ^ vb[0];
#pragma unroll
            for (int j = 1; j < U; ++j) y |= va[j] ^ vb[j];
            if (!(__ballot((y.x | y.y | y.z | y.w) != 0u) != 0ull || strict)) break;   // a clean tile: done
          }
          if (pending) run_staged<DT, ND, U>(stage, st, lane, strict, S.atol, S.rtol, acc, X, permuted);
          tile = cur;                    // the loop's step moves past it
        }
      }
      if constexpr (kCos) {
#pragma unroll
        for (int j = 0; j < U; ++j) cos_chunk_fast<DT>(va[j], vb[j], cs);
        if (!(__builtin_isfinite(cs.ab) && __builtin_isfinite(cs.aa) && __builtin_isfinite(cs.bb))) {
          cs = Cos{0.0, 0.0, 0.0};                 // this lane met a NaN or Inf: redo with checks
          // (unrolled: a run-time index would move va and vb out of registers)
#pragma unroll
          for (int j = 0; j < U; ++j) cos_chunk<DT>(va[j], vb[j], nv[j], cs, nonfinite);
        }
        cos_store(cs, partials + kCosRec * (S.tile_begin + tile), lane);
      }
      continue;
    }
    // Last tile of a row, misaligned operands or a gather: per-chunk bounds.
    // The plain and N-D diffs issue all the tile's loads before checking any
    // chunk (the latency is then paid once per tile); the cosine variant,
    // short of registers, goes chunk by chunk.
    // (gathers of 1- and 2-byte elements load each element on its own, up
    // to 16 loads per chunk and operand: those keep one chunk in flight)
    if (!COS && (!gather || Et<DT>::es >= 4 || (pair2a && pair2b))) {
      u32x4 va[U], vb[U];
      uint32_t nb[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
        va[j] = u32x4{0u, 0u, 0u, 0u};
        vb[j] = u32x4{0u, 0u, 0u, 0u};
        nb[j] = 0;
        if (c < S.row_chunks) {
          const uint64_t cb = c * kChunk;
          const uint64_t rem = S.row_bytes - cb;
          nb[j] = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
          if constexpr (ND) {
            load_nd_chunk<DT>(pa, pb, c, nb[j], vec, gather, in_sa, in_sb, pair2a, pair2b,
                              c + 1 == S.row_chunks, va[j], vb[j]);
            if (span) span_mask<DT>(span, span_residue<DT>(c, span), va[j], vb[j]);
          } else {
            load_chunk<DT>(pa + cb, pb + cb, nb[j], vec, va[j], vb[j]);
          }
        }
      }
      uint64_t i0[U];
      uint32_t nv[U];
#pragma unroll
      for (int j = 0; j < U; ++j) {
        i0[j] = ibase + (k0 + (uint64_t)(j * kWave) + lane) * epc;
        nv[j] = nb[j] / es;
      }
      tile_slow<DT, ND, !COS, U>(va, vb, i0, nv, lane, tol_mode, strict, S.atol, S.rtol, acc, X, permuted, slot);
      continue;
    }
    if (GATHERS && pair2a && pair2b) {
      // the same chunks in the same order, two in flight
#pragma unroll 1
      for (int j = 0; j < U; j += 2) {
        u32x4 va[2], vb[2];
        uint32_t nb[2];
        uint64_t c[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          c[h] = k0 + (uint64_t)((j + h) * kWave) + lane;
          va[h] = u32x4{0u, 0u, 0u, 0u};
          vb[h] = u32x4{0u, 0u, 0u, 0u};
          nb[h] = 0;
          if (c[h] < S.row_chunks) {
            const uint64_t rem = S.row_bytes - c[h] * kChunk;
            nb[h] = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
            load_nd_chunk<DT>(pa, pb, c[h], nb[h], vec, gather, in_sa, in_sb, pair2a, pair2b,
                              c[h] + 1 == S.row_chunks, va[h], vb[h]);
          }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          chunk<DT, ND>(va[h], vb[h], ibase + c[h] * epc, nb[h] / es, tol_mode, strict, S.atol, S.rtol, acc, X,
                        permuted);
          const Cos keep = cs;
          cos_chunk_fast<DT>(va[h], vb[h], cs);
          if (!(__builtin_isfinite(cs.ab) && __builtin_isfinite(cs.aa) && __builtin_isfinite(cs.bb))) {
            cs = keep;
            cos_chunk<DT>(va[h], vb[h], nb[h] / es, cs, nonfinite);
          }
        }
      }
      cos_store(cs, partials + kCosRec * (S.tile_begin + tile), lane);
      continue;
    }
#pragma unroll 1
    for (int j = 0; j < U; ++j) {
      const uint64_t c = k0 + (uint64_t)(j * kWave) + lane;
      u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
      uint32_t nb = 0;
      if (c < S.row_chunks) {
        const uint64_t cb = c * kChunk;
        const uint64_t rem = S.row_bytes - cb;
        nb = rem < (uint64_t)kChunk ? (uint32_t)rem : (uint32_t)kChunk;
        if constexpr (ND)
          load_nd_chunk<DT>(pa, pb, c, nb, vec, gather, in_sa, in_sb, pair2a, pair2b, c + 1 == S.row_chunks,
                            va, vb);
        else load_chunk<DT>(pa + cb, pb + cb, nb, vec, va, vb);
      }
      chunk<DT, ND>(va, vb, ibase + c * epc, nb / es, tol_mode, strict, S.atol, S.rtol, acc, X, permuted);
      if constexpr (kCos && ND) {
        // the unchecked sums first (the elements past nb load as zeros), the
        // checked ones when a NaN or Inf made them non-finite: the same
        // additions in the same order either way
        const Cos keep = cs;
        cos_chunk_fast<DT>(va, vb, cs);
        if (!(__builtin_isfinite(cs.ab) && __builtin_isfinite(cs.aa) && __builtin_isfinite(cs.bb))) {
          cs = keep;
          cos_chunk<DT>(va, vb, nb / es, cs, nonfinite);
        }
      } else if constexpr (kCos) {
        cos_chunk<DT>(va, vb, nb / es, cs, nonfinite);
      }
    }
    if constexpr (kCos) cos_store(cs, partials + kCosRec * (S.tile_begin + tile), lane);
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
// Adds a wave's partials for segment S to its result: counts added, first
// indices min'd, the non-negative maxima max'd as bit patterns, all with
// exact 64-bit atomics; fields with nothing to add are skipped.  VEC: the
// seven fields go as three vector atomics from lanes 0-2 (one per
// operation: counts at words 0, 2, 4, first indices at 1, 3, maxima at 5, 6)
// instead of seven from lane 0 -- on one result's cache line each atomic is
// serialised, and the 2-D kernels' flushes meet there when a difference sits
// in nearly every tile (the N-D variants keep lane 0, for want of
// registers).
__device__ __forceinline__ void add_result(unsigned long long* R, bool vec, uint32_t lane, uint64_t tol,
                                           uint64_t ftol, uint64_t bw, uint64_t fbw, uint64_t nf, uint64_t mab,
                                           uint64_t mre) {
  if (vec) {
    const uint64_t cnt = lane == 0 ? tol : lane == 1 ? bw : nf;
    if (lane < 3u && cnt != 0) atomicAdd(R + 2 * lane, cnt);
    const uint64_t first = lane == 0 ? ftol : fbw;
    if (lane < 2u && first != ~0ull) atomicMin(R + 1 + 2 * lane, first);
    const uint64_t mx = lane == 0 ? mab : mre;
    if (lane < 2u && mx != 0) atomicMax(R + 5 + lane, mx);
  } else if (lane == 0) {
    if (bw) {
      atomicAdd(R + 2, bw);
      atomicMin(R + 3, fbw);
    }
    if (tol) {
      atomicAdd(R + 0, tol);
      atomicMin(R + 1, ftol);
    }
    if (nf) atomicAdd(R + 4, nf);
    if (mab) atomicMax(R + 5, mab);
    if (mre) atomicMax(R + 6, mre);
  }
}

// The cosine variants' count of pairs with a NaN or Inf, added to S's.
__device__ __forceinline__ void flush_nonfinite(const DiffSeg& S, uint32_t lane, uint32_t& nonfinite,
                                                unsigned long long* nonfinite_pairs) {
  if (nonfinite_pairs != nullptr && __ballot(nonfinite != 0u) != 0ull) {
    const uint64_t nfp = wave_sum(nonfinite);
    if (lane == 0) atomicAdd(nonfinite_pairs + S.result_index, (unsigned long long)nfp);
    nonfinite = 0;
  }
}

template <bool VEC>
__device__ __forceinline__ void flush(Acc& acc, const DiffSeg& S, asmevo_segment_result* results,
                                      uint32_t lane, uint32_t& nonfinite,
                                      unsigned long long* nonfinite_pairs) {
  flush_nonfinite(S, lane, nonfinite, nonfinite_pairs);
  if (__ballot((acc.bw | acc.tol) != 0u) == 0ull) return;
  uint64_t bw = wave_sum(acc.bw);
  uint64_t tol = wave_sum(acc.tol);
  const uint64_t nf = wave_sum(acc.nf);
  uint64_t fbw = wave_min(acc.first_bw);
  uint64_t ftol = wave_min(acc.first_tol);
  const uint64_t mab = wave_max(acc.max_abs);
  const uint64_t mre = wave_max(acc.max_rel);
  if (S.mode != ASMEVO_TOLERANCE) {
    tol = bw;
    ftol = fbw;
  }
  add_result(reinterpret_cast<unsigned long long*>(results + S.result_index), VEC, lane, tol, ftol, bw, fbw, nf,
             mab, mre);
  acc_reset(acc);
}

// The workgroup's last flushes, merged: every wave leaves its partials for
// its range's last segment (result index `last`, or -1) in LDS; the first
// wave holding a result adds in the other waves' partials for the same
// result and flushes them with one set of atomics.  Every wave of the
// workgroup must call this.
__device__ __forceinline__ void merge_last(Acc& acc, int last, uint32_t mode, asmevo_segment_result* results,
                                           uint32_t lane) {
  constexpr int kW = kDiffBlock / kWave;
  __shared__ uint64_t fin[kW][8];
  const uint32_t w = threadIdx.x / kWave;
  const bool any = last >= 0 && __ballot((acc.bw | acc.tol) != 0u) != 0ull;
  uint64_t bw = wave_sum(acc.bw), tol = wave_sum(acc.tol), nf = wave_sum(acc.nf);
  uint64_t fbw = wave_min(acc.first_bw), ftol = wave_min(acc.first_tol);
  uint64_t mab = wave_max(acc.max_abs), mre = wave_max(acc.max_rel);
  if (mode != ASMEVO_TOLERANCE) {
    tol = bw;
    ftol = fbw;
  }
  if (lane == 0) {
    fin[w][0] = any ? (uint64_t)last : ~0ull;
    fin[w][1] = tol;
    fin[w][2] = ftol;
    fin[w][3] = bw;
    fin[w][4] = fbw;
    fin[w][5] = nf;
    fin[w][6] = mab;
    fin[w][7] = mre;
  }
  __syncthreads();
  const uint64_t r = fin[w][0];
  bool first_holder = r != ~0ull;
  for (uint32_t k = 0; k < w; ++k) first_holder = first_holder && fin[k][0] != r;
  if (first_holder) {
    for (uint32_t k = w + 1; k < (uint32_t)kW; ++k) {
      if (fin[k][0] != r) continue;
      tol += fin[k][1];
      ftol = fin[k][2] < ftol ? fin[k][2] : ftol;
      bw += fin[k][3];
      fbw = fin[k][4] < fbw ? fin[k][4] : fbw;
      nf += fin[k][5];
      mab = fin[k][6] > mab ? fin[k][6] : mab;
      mre = fin[k][7] > mre ? fin[k][7] : mre;
    }
    add_result(reinterpret_cast<unsigned long long*>(results + r), true, lane, tol, ftol, bw, fbw, nf, mab, mre);
  }
}

__global__ void diff_init_kernel(asmevo_segment_result* results, int n,
                                 unsigned long long* nonfinite_pairs) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  if (nonfinite_pairs != nullptr) nonfinite_pairs[t] = 0;
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


template <bool COS, bool ND>
__global__ __launch_bounds__(kDiffBlock)
__attribute__((amdgpu_waves_per_eu(COS ? ASMEVO_COS_WAVES_PER_EU
                                        : (ND ? ASMEVO_DIFF_ND_WAVES_PER_EU : ASMEVO_DIFF_WAVES_PER_EU))))
void diff_kernel(const DiffSeg* __restrict__ segs, const NdExt* __restrict__ ext, int n,
                 uint64_t total_tiles, asmevo_segment_result* results, double* partials,
                 unsigned long long* nonfinite_pairs) {
  // kStep consecutive waves of a workgroup share their tiles and take them in
  // turn (kStep = 1: every wave has tiles of its own).  With kDeal = 0 the
  // group's tiles are one contiguous range; otherwise blocks of kDeal tiles
  // (fewer when the groups would not all get one) are dealt to the groups
  // round-robin, so every group sees the same mix of segments (and of
  // element types).
  constexpr uint32_t kStep = COS ? ASMEVO_COS_WAVE_STEP : ASMEVO_DIFF_WAVE_STEP;
  constexpr uint64_t kDeal = COS ? ASMEVO_COS_DEAL : ASMEVO_DIFF_DEAL;
  static_assert(kStep >= 1 && (kDiffBlock / kWave) % kStep == 0, "a tile range stays inside a workgroup");
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = (uint64_t)blockIdx.x * (kDiffBlock / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t ngroups = (uint64_t)gridDim.x * (kDiffBlock / kWave) / kStep;
  const uint64_t group = wave / kStep;
  const uint64_t per_group = (total_tiles + ngroups - 1) / ngroups;
  const uint64_t block = kDeal < per_group ? kDeal : per_group;
  // a slot of LDS per wave for the slow path (the cosine variants use none)
  __shared__ __align__(16) uint8_t slow[COS ? 16 : (kDiffBlock / kWave) * kSlotBytes];
  uint8_t* slot = slow + (COS ? 0 : (threadIdx.x / kWave) * kSlotBytes);
  int s = -1;
  Acc acc;
  acc_reset(acc);
  uint32_t nonfinite = 0;
  // each wave's last segment is flushed together with the workgroup's other
  // waves (the 2-D kernels: a workgroup's waves take neighbouring ranges, or
  // share their blocks, so they end in the same or neighbouring segments)
  constexpr bool kMergeLast = !ND;
  int last = -1;
  uint32_t last_mode = 0;
  for (uint64_t j = group;; j += ngroups) {
    uint64_t lo, hi;
    if constexpr (kDeal == 0) {
      lo = total_tiles * group / ngroups;
      hi = total_tiles * (group + 1) / ngroups;
    } else {
      lo = j * block;
      if (lo >= total_tiles) break;
      hi = lo + block < total_tiles ? lo + block : total_tiles;
    }
    uint64_t t = lo + wave % kStep;
    if (t < hi && s < 0) {
      int s_lo = 0, s_hi = n - 1;        // last segment with tile_begin <= t
      while (s_lo < s_hi) {
        const int mid = (s_lo + s_hi + 1) >> 1;
        if (segs[mid].tile_begin <= t) s_lo = mid;
        else s_hi = mid - 1;
      }
      s = s_lo;
    }
    if constexpr (kDeal != 0 && ND) {
      // The group's next block lies ngroups blocks on, past any number of
      // segments: gallop from the next segment, then bisect (a step at a
      // time, a wave re-read hundreds of descriptors per block of a block
      // table).  The 2-D cosine kernel keeps the steps: with the search in
      // it, its pass over the sweep ran 0.6 % slower.
      if (t < hi && s + 1 < n && segs[s + 1].tile_begin <= t) {
        int a = s + 1, d = 1;          // segs[a].tile_begin <= t
        while (a + d < n && segs[a + d].tile_begin <= t) {
          a += d;
          d <<= 1;
        }
        int b = a + d < n ? a + d - 1 : n - 1;
        while (a < b) {
          const int mid = (a + b + 1) >> 1;
          if (segs[mid].tile_begin <= t) a = mid;
          else b = mid - 1;
        }
        s = a;
      }
    }
    while (t < hi) {
      while (s + 1 < n && segs[s + 1].tile_begin <= t) ++s;
      const DiffSeg S = segs[s];
      const uint64_t seg_end = S.tile_begin + S.tile_count;
      const uint64_t t_end = seg_end < hi ? seg_end : hi;
      const uint64_t b = t - S.tile_begin, e = t_end - S.tile_begin;
      const NdExt* X = (ND && S.nd_ext != ~0ull) ? ext + S.nd_ext : nullptr;
      switch (S.dtype) {
        case ASMEVO_F32: diff_range<ASMEVO_F32, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
        case ASMEVO_BF16: diff_range<ASMEVO_BF16, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
        case ASMEVO_F16: diff_range<ASMEVO_F16, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
        case ASMEVO_FP8_E4M3:
          diff_range<ASMEVO_FP8_E4M3, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
          break;
        case ASMEVO_I32: diff_range<ASMEVO_I32, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
        case ASMEVO_I64: diff_range<ASMEVO_I64, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
        default: diff_range<ASMEVO_U8, COS, ND>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot); break;
      }
      // the wave's last segment: its range's (or last block's) end
      const bool final_seg = t_end == hi && (kDeal == 0 || (j + ngroups) * block >= total_tiles);
      if (kMergeLast && final_seg) {
        flush_nonfinite(S, lane, nonfinite, COS ? nonfinite_pairs : nullptr);
        last = (int)S.result_index;    // merged with the workgroup's other waves below
        last_mode = S.mode;
      } else {
        flush<!ND>(acc, S, results, lane, nonfinite, COS ? nonfinite_pairs : nullptr);
      }
      t += (t_end - t + kStep - 1) / kStep * kStep;   // this wave's first tile at or after t_end
    }
    if constexpr (kDeal == 0) break;
  }
  if constexpr (kMergeLast) merge_last(acc, last, last_mode, results, lane);
}

// One level of the cosine's block tree: every workgroup reduces full aligned
// groups of 256 level-(k-1) entries (perfect subtrees) to one level-k entry,
// pairing neighbours level by level in LDS.  Groups are numbered across
// segments by `prefix` (prefix[s] = the groups of segments before s).
constexpr int kCosBlock = 256;

__global__ __launch_bounds__(kCosBlock) void cos_level_kernel(const CosLevels* __restrict__ lv,
                                                              const uint64_t* __restrict__ prefix, int n, int k,
                                                              const double* __restrict__ partials,
                                                              double* __restrict__ levels) {
  __shared__ double v[3][kCosBlock];
  const int t = threadIdx.x;
  const uint64_t total = prefix[n];
  for (uint64_t g = blockIdx.x; g < total; g += gridDim.x) {
    int lo = 0, hi = n - 1;                  // last segment with prefix[s] <= g
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (prefix[mid] <= g) lo = mid;
      else hi = mid - 1;
    }
    const uint64_t j = g - prefix[lo];
    const CosLevels& L = lv[lo];
    const double* src =
        (k == 1 ? partials + kCosRec * L.off[0] : levels + kCosRec * L.off[k - 1]) + kCosRec * (256 * j + t);
    v[0][t] = src[0];
    v[1][t] = src[1];
    v[2][t] = src[2];
    __syncthreads();
    for (int width = kCosBlock / 2; width >= 1; width >>= 1) {
      double ab = 0.0, aa = 0.0, bb = 0.0;
      if (t < width) {
        ab = v[0][2 * t] + v[0][2 * t + 1];
        aa = v[1][2 * t] + v[1][2 * t + 1];
        bb = v[2][2 * t] + v[2][2 * t + 1];
      }
      __syncthreads();
      if (t < width) {
        v[0][t] = ab;
        v[1][t] = aa;
        v[2][t] = bb;
      }
      __syncthreads();
    }
    if (t < kCosRec) {   // one 32-byte record from four lanes
      double* dst = levels + kCosRec * (L.off[k] + j);
      dst[t] = t == 0 ? v[0][0] : t == 1 ? v[1][0] : t == 2 ? v[2][0] : 0.0;
    }
    __syncthreads();
  }
}

// One workgroup per segment.  The entries no level-k group absorbed (m_k <
// 256 per level) are staged in LDS; their binary decomposition -- perfect
// subtrees of sizes given by the set bits of m_k, largest first -- is
// reduced in place in parallel (pairs 2^j apart inside every full aligned
// block of 2^(j+1)).  One thread then pushes those subtree sums -- highest
// level first, left to right -- onto a binary counter of perfect subtrees
// (equal heights merge, left + right).  Folding the counter from the right
// gives exactly the left-complete tree P(x[0..n)) = P(x[0..h)) + P(x[h..n))
// over the segment's blocks.
__global__ __launch_bounds__(kCosBlock) void cosine_kernel(const DiffSeg* __restrict__ segs,
                                                           const CosLevels* __restrict__ lv,
                                                           const double* __restrict__ partials,
                                                           const double* __restrict__ levels,
                                                           const unsigned long long* nonfinite_pairs,
                                                           asmevo_cosine_result* out) {
  constexpr int kLeft = 255;                       // at most 255 leftovers per level
  __shared__ double left[3][kCosLevels * kLeft];
  __shared__ double stack_val[3][64];
  __shared__ int stack_lvl[64];
  const int s = blockIdx.x;
  const int t = threadIdx.x;
  const DiffSeg S = segs[s];
  if (!(S.dtype >= ASMEVO_F32 && S.dtype <= ASMEVO_FP8_E4M3)) {
    if (t == 0) {
      asmevo_cosine_result r;
      r.sum_ab = r.sum_aa = r.sum_bb = 0.0;
      r.cosine = __builtin_nan("");
      r.pairs = 0;
      r.blocks = 0;
      out[S.result_index] = r;
    }
    return;
  }
  const CosLevels L = lv[s];
  int m[kCosLevels];
  for (int k = 0; k < kCosLevels; ++k) {
    const uint64_t first = (k + 1 < kCosLevels) ? 256 * L.cnt[k + 1] : 0;
    m[k] = (int)(L.cnt[k] - first);                // <= 255: first is cnt[k] rounded down to 256
    const double* base = k == 0 ? partials + kCosRec * L.off[0] : levels + kCosRec * L.off[k];
    for (int e = t; e < m[k]; e += kCosBlock) {
      left[0][k * kLeft + e] = base[kCosRec * (first + e) + 0];
      left[1][k * kLeft + e] = base[kCosRec * (first + e) + 1];
      left[2][k * kLeft + e] = base[kCosRec * (first + e) + 2];
    }
  }
  __syncthreads();
  for (int j = 0; j < 8; ++j) {
    const int half = 1 << j, span = 2 << j;
    for (int k = 0; k < kCosLevels; ++k) {
      const int p = t * span;
      if (p + span <= m[k]) {
        const int q = k * kLeft + p;
        left[0][q] = left[0][q] + left[0][q + half];
        left[1][q] = left[1][q] + left[1][q + half];
        left[2][q] = left[2][q] + left[2][q + half];
      }
    }
    __syncthreads();
  }
  if (t != 0) return;
  asmevo_cosine_result r;
  int depth = 0;
  for (int k = kCosLevels - 1; k >= 0; --k) {
    int pos = 0;
    for (int bit = 7; bit >= 0; --bit) {
      if (!((m[k] >> bit) & 1)) continue;
      const int q = k * kLeft + pos;
      pos += 1 << bit;
      double ab = left[0][q], aa = left[1][q], bb = left[2][q];
      int lvl = 8 * k + bit;
      while (depth > 0 && stack_lvl[depth - 1] == lvl) {
        ab = stack_val[0][depth - 1] + ab;
        aa = stack_val[1][depth - 1] + aa;
        bb = stack_val[2][depth - 1] + bb;
        --depth;
        ++lvl;
      }
      stack_val[0][depth] = ab;
      stack_val[1][depth] = aa;
      stack_val[2][depth] = bb;
      stack_lvl[depth] = lvl;
      ++depth;
    }
  }
  double ab = 0.0, aa = 0.0, bb = 0.0;
  if (depth > 0) {
    ab = stack_val[0][depth - 1];
    aa = stack_val[1][depth - 1];
    bb = stack_val[2][depth - 1];
    for (int q = depth - 2; q >= 0; --q) {
      ab = stack_val[0][q] + ab;
      aa = stack_val[1][q] + aa;
      bb = stack_val[2][q] + bb;
    }
  }
  r.sum_ab = ab;
  r.sum_aa = aa;
  r.sum_bb = bb;
  if (aa == 0.0 && bb == 0.0) r.cosine = 1.0;
  else if (aa == 0.0 || bb == 0.0) r.cosine = 0.0;
  else {
    const double na = __builtin_sqrt(aa);
    const double nbb = __builtin_sqrt(bb);
    const double den = na * nbb;
    r.cosine = ab / den;
  }
  r.pairs = S.rows * S.cols - nonfinite_pairs[S.result_index];
  r.blocks = S.tile_count;
  out[S.result_index] = r;
}


// The cosine pass over N-D segments for calls made only of one kind of
// float segment, with the dealing and the segment search of
// diff_kernel<true, true> and one path of its code:
// * narrow_cos_kernel: short rows (at least two rows of at most
//   kNarrowCosChunks chunks each), the short-row path.  Without the other
//   paths it needs 122 VGPRs, four waves per SIMD instead of three (256-byte
//   half rows: 3.95-3.99 against 4.27 ms; four chunks a lane ran slower,
//   4.70 ms spilling at three waves per SIMD and 4.44 ms at two).
// * rows_cos_kernel: long rows, 16-byte aligned and unit-stride (one row, or
//   rows of more than kNarrowCosChunks chunks), the row-tiled whole-tile code:
//   140 VGPRs and no spill instead of 168 and six spilled (sliced rows 5.94
//   against 6.19 ms, transposed and permuted views and a block table 2 %
//   faster).
// * gather_cos_kernel: gathers of long rows with elements 2 apart in both
//   operands, the chunk-by-chunk code with two chunks in flight: four waves
//   per SIMD (the stride-2 gather: 5.68 against 6.07 ms).  Gathers whose
//   elements load one by one stay in diff_kernel<true, true>: in this kernel
//   the stride-3 gather ran 6.29 ms with two chunks in flight (1.8 % more
//   fetched) and 6.56 ms with one, against 5.89.
template <int DT>
__device__ __forceinline__ void narrow_cos_range(const DiffSeg& S, const NdExt* X, uint64_t b, uint64_t e,
                                                 uint32_t step, uint32_t lane, Acc& acc, double* partials,
                                                 uint32_t& nonfinite) {
  const bool permuted = (S.flags & kSegPermuted) != 0;
  diff_range_narrow_cos<DT, true, 2>(S, X, b, e, step, lane, acc, partials, nonfinite, S.mode == ASMEVO_TOLERANCE,
                                     (S.flags & kSegStrict) != 0, (S.flags & kSegVec) != 0,
                                     (S.flags & kSegGather) != 0, (S.flags & kSegPair2A) != 0,
                                     (S.flags & kSegPair2B) != 0, X ? X->in_sa : 0, X ? X->in_sb : 0,
                                     permuted ? 0 : S.nd_index_base, permuted);
}

template <int KIND>   // kCosNdShortRows, kCosNdLongRows or kCosNdGathers
__device__ __forceinline__ void split_cos_ranges(const DiffSeg* __restrict__ segs, const NdExt* __restrict__ ext,
                                                 int n, uint64_t total_tiles, asmevo_segment_result* results,
                                                 double* partials, unsigned long long* nonfinite_pairs,
                                                 uint8_t* slot) {
  constexpr uint32_t kStep = ASMEVO_COS_WAVE_STEP;
  constexpr uint64_t kDeal = ASMEVO_COS_DEAL;
  static_assert(kDeal > 0 && (kDiffBlock / kWave) % kStep == 0, "blocks dealt inside a workgroup");
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = (uint64_t)blockIdx.x * (kDiffBlock / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t ngroups = (uint64_t)gridDim.x * (kDiffBlock / kWave) / kStep;
  const uint64_t group = wave / kStep;
  const uint64_t per_group = (total_tiles + ngroups - 1) / ngroups;
  const uint64_t block = kDeal < per_group ? kDeal : per_group;
  int s = -1;
  Acc acc;
  acc_reset(acc);
  uint32_t nonfinite = 0;
  for (uint64_t j = group;; j += ngroups) {
    const uint64_t lo = j * block;
    if (lo >= total_tiles) break;
    const uint64_t hi = lo + block < total_tiles ? lo + block : total_tiles;
    uint64_t t = lo + wave % kStep;
    if (t < hi && s < 0) {
      int s_lo = 0, s_hi = n - 1;        // last segment with tile_begin <= t
      while (s_lo < s_hi) {
        const int mid = (s_lo + s_hi + 1) >> 1;
        if (segs[mid].tile_begin <= t) s_lo = mid;
        else s_hi = mid - 1;
      }
      s = s_lo;
    }
    if (t < hi && s + 1 < n && segs[s + 1].tile_begin <= t) {
      int a = s + 1, d = 1;              // gallop, then bisect, as in diff_kernel
      while (a + d < n && segs[a + d].tile_begin <= t) {
        a += d;
        d <<= 1;
      }
      int z = a + d < n ? a + d - 1 : n - 1;
      while (a < z) {
        const int mid = (a + z + 1) >> 1;
        if (segs[mid].tile_begin <= t) a = mid;
        else z = mid - 1;
      }
      s = a;
    }
    while (t < hi) {
      while (s + 1 < n && segs[s + 1].tile_begin <= t) ++s;
      const DiffSeg S = segs[s];
      const uint64_t seg_end = S.tile_begin + S.tile_count;
      const uint64_t t_end = seg_end < hi ? seg_end : hi;
      const uint64_t b = t - S.tile_begin, e = t_end - S.tile_begin;
      const NdExt* X = S.nd_ext != ~0ull ? ext + S.nd_ext : nullptr;
      if constexpr (KIND == kCosNdGathers) {
        switch (S.dtype) {
          case ASMEVO_F32:
            diff_range<ASMEVO_F32, true, true, false, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_BF16:
            diff_range<ASMEVO_BF16, true, true, false, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_F16:
            diff_range<ASMEVO_F16, true, true, false, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_FP8_E4M3:
            diff_range<ASMEVO_FP8_E4M3, true, true, false, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite,
                                                                 slot);
            break;
          default: break;                // not launched for other types
        }
      } else if constexpr (KIND == kCosNdLongRows) {
        switch (S.dtype) {
          case ASMEVO_F32:
            diff_range<ASMEVO_F32, true, true, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_BF16:
            diff_range<ASMEVO_BF16, true, true, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_F16:
            diff_range<ASMEVO_F16, true, true, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          case ASMEVO_FP8_E4M3:
            diff_range<ASMEVO_FP8_E4M3, true, true, true>(S, X, b, e, kStep, lane, acc, partials, nonfinite, slot);
            break;
          default: break;                // not launched for other types
        }
      } else {
        switch (S.dtype) {
          case ASMEVO_F32: narrow_cos_range<ASMEVO_F32>(S, X, b, e, kStep, lane, acc, partials, nonfinite); break;
          case ASMEVO_BF16: narrow_cos_range<ASMEVO_BF16>(S, X, b, e, kStep, lane, acc, partials, nonfinite); break;
          case ASMEVO_F16: narrow_cos_range<ASMEVO_F16>(S, X, b, e, kStep, lane, acc, partials, nonfinite); break;
          case ASMEVO_FP8_E4M3:
            narrow_cos_range<ASMEVO_FP8_E4M3>(S, X, b, e, kStep, lane, acc, partials, nonfinite);
            break;
          default: break;                // not launched for other types
        }
      }
      flush<false>(acc, S, results, lane, nonfinite, nonfinite_pairs);
      t += (t_end - t + kStep - 1) / kStep * kStep;   // this wave's first tile at or after t_end
    }
  }
}
__global__ __launch_bounds__(kDiffBlock) __attribute__((amdgpu_waves_per_eu(4)))
void narrow_cos_kernel(const DiffSeg* __restrict__ segs, const NdExt* __restrict__ ext, int n,
                       uint64_t total_tiles, asmevo_segment_result* results, double* partials,
                       unsigned long long* nonfinite_pairs) {
  split_cos_ranges<kCosNdShortRows>(segs, ext, n, total_tiles, results, partials, nonfinite_pairs, nullptr);
}

__global__ __launch_bounds__(kDiffBlock) __attribute__((amdgpu_waves_per_eu(ASMEVO_COS_WAVES_PER_EU)))
void rows_cos_kernel(const DiffSeg* __restrict__ segs, const NdExt* __restrict__ ext, int n,
                     uint64_t total_tiles, asmevo_segment_result* results, double* partials,
                     unsigned long long* nonfinite_pairs) {
  __shared__ __align__(16) uint8_t slot[16];     // unused by the cosine variant's code
  split_cos_ranges<kCosNdLongRows>(segs, ext, n, total_tiles, results, partials, nonfinite_pairs, slot);
}

__global__ __launch_bounds__(kDiffBlock) __attribute__((amdgpu_waves_per_eu(ASMEVO_COS_WAVES_PER_EU)))
void gather_cos_kernel(const DiffSeg* __restrict__ segs, const NdExt* __restrict__ ext, int n,
                       uint64_t total_tiles, asmevo_segment_result* results, double* partials,
                       unsigned long long* nonfinite_pairs) {
  __shared__ __align__(16) uint8_t slot[16];     // unused by the cosine variant's code
  split_cos_ranges<kCosNdGathers>(segs, ext, n, total_tiles, results, partials, nonfinite_pairs, slot);
}

}  // namespace

// Resident workgroups per CU of a diff kernel (one code object: queried once).
template <bool COS, bool ND>
int resident_blocks() {
  static const int blocks = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, diff_kernel<COS, ND>, kDiffBlock, 0) != hipSuccess ||
        b <= 0)
      b = 4;
    return b;
  }();
  return blocks;
}

int cos_blocks_per_cu() { return resident_blocks<true, false>(); }

int diff_nd_blocks_per_cu() { return resident_blocks<false, true>(); }

int cos_nd_blocks_per_cu() { return resident_blocks<true, true>(); }

int split_cos_blocks_per_cu(int variant) {
  static const int narrow = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, narrow_cos_kernel, kDiffBlock, 0) != hipSuccess || b <= 0)
      b = 3;
    return b;
  }();
  static const int rows = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, rows_cos_kernel, kDiffBlock, 0) != hipSuccess || b <= 0)
      b = 3;
    return b;
  }();
  static const int gathers = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, gather_cos_kernel, kDiffBlock, 0) != hipSuccess || b <= 0)
      b = 3;
    return b;
  }();
  return variant == kCosNdShortRows ? narrow : variant == kCosNdLongRows ? rows : gathers;
}

int cos_nd_variant(const DiffSeg* segs, int n) {
  bool any = false, all_short = true, all_long = true, all_gathers = true;
  for (int k = 0; k < n; ++k) {
    const DiffSeg& S = segs[k];
    if (S.tile_count == 0) continue;
    const bool fp = S.dtype == ASMEVO_F32 || S.dtype == ASMEVO_BF16 || S.dtype == ASMEVO_F16 ||
                    S.dtype == ASMEVO_FP8_E4M3;
    if (!fp) return kCosNdMixed;
    const bool short_rows = S.rows > 1 && S.row_chunks <= (uint64_t)kNarrowCosChunks;
    all_short = all_short && short_rows;
    all_long = all_long && !short_rows && (S.flags & kSegVec) != 0 && (S.flags & kSegGather) == 0;
    all_gathers = all_gathers && !short_rows && (S.flags & kSegGather) != 0 && (S.flags & kSegPair2A) != 0 &&
                  (S.flags & kSegPair2B) != 0;
    any = true;
  }
  if (!any) return kCosNdMixed;
  return all_short ? kCosNdShortRows : all_long ? kCosNdLongRows : all_gathers ? kCosNdGathers : kCosNdMixed;
}

hipError_t launch_diff(const DiffSeg* segs, int n, uint64_t total_tiles,
                       asmevo_segment_result* results, int workgroups, hipStream_t stream,
                       double* partials, unsigned long long* nonfinite_pairs,
                       asmevo_cosine_result* cos_results, const CosLevels* levels_of,
                       const uint64_t* level_prefix, const uint64_t* level_groups, double* levels) {
  if (n == 0) return hipSuccess;
  const bool cos = cos_results != nullptr;
  hipLaunchKernelGGL(diff_init_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, results, n,
                     cos ? nonfinite_pairs : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (total_tiles > 0) {
    const uint64_t max_wg = (total_tiles + (kDiffBlock / kWave) - 1) / (kDiffBlock / kWave);
    const int wg = (uint64_t)workgroups > max_wg ? (int)max_wg : workgroups;
    if (cos)
      hipLaunchKernelGGL((diff_kernel<true, false>), dim3(wg), dim3(kDiffBlock), 0, stream, segs, nullptr,
                         n, total_tiles, results, partials, nonfinite_pairs);
    else
      hipLaunchKernelGGL((diff_kernel<false, false>), dim3(wg), dim3(kDiffBlock), 0, stream, segs, nullptr,
                         n, total_tiles, results, nullptr, nullptr);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (cos) {
    // levels 1.. of every segment's block tree, in parallel, then the per-segment fold
    for (int k = 1; k < kCosLevels; ++k) {
      if (level_groups[k] == 0) break;
      const uint64_t grid = level_groups[k] < 65536 ? level_groups[k] : 65536;
      hipLaunchKernelGGL(cos_level_kernel, dim3((unsigned)grid), dim3(kCosBlock), 0, stream, levels_of,
                         level_prefix + (size_t)(k - 1) * (n + 1), n, k, partials, levels);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(cosine_kernel, dim3(n), dim3(kCosBlock), 0, stream, segs, levels_of, partials, levels,
                       nonfinite_pairs, cos_results);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_diff_nd(const DiffSeg* segs, const NdExt* ext, int n, int n_results,
                          uint64_t total_tiles, asmevo_segment_result* results, int workgroups,
                          hipStream_t stream) {
  if (n_results > 0) {
    hipLaunchKernelGGL(diff_init_kernel, dim3((n_results + 255) / 256), dim3(256), 0, stream, results,
                       n_results, nullptr);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (n == 0 || total_tiles == 0) return hipSuccess;
  const uint64_t max_wg = (total_tiles + (kDiffBlock / kWave) - 1) / (kDiffBlock / kWave);
  const int wg = (uint64_t)workgroups > max_wg ? (int)max_wg : workgroups;
  hipLaunchKernelGGL((diff_kernel<false, true>), dim3(wg), dim3(kDiffBlock), 0, stream, segs, ext, n,
                     total_tiles, results, nullptr, nullptr);
  return hipGetLastError();
}

hipError_t launch_diff_cosine_nd(const DiffSeg* segs, const NdExt* ext, int n, const DiffSeg* units,
                                 int n_results, uint64_t total_tiles, asmevo_segment_result* results,
                                 int workgroups, hipStream_t stream, double* partials,
                                 unsigned long long* nonfinite_pairs, asmevo_cosine_result* cos_results,
                                 const CosLevels* levels_of, const uint64_t* level_prefix,
                                 const uint64_t* level_groups, double* levels, int variant) {
  if (n_results == 0) return hipSuccess;
  hipLaunchKernelGGL(diff_init_kernel, dim3((n_results + 255) / 256), dim3(256), 0, stream, results, n_results,
                     nonfinite_pairs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n > 0 && total_tiles > 0) {
    const uint64_t max_wg = (total_tiles + (kDiffBlock / kWave) - 1) / (kDiffBlock / kWave);
    const int wg = (uint64_t)workgroups > max_wg ? (int)max_wg : workgroups;
    if (variant == kCosNdShortRows)
      hipLaunchKernelGGL(narrow_cos_kernel, dim3(wg), dim3(kDiffBlock), 0, stream, segs, ext, n, total_tiles,
                         results, partials, nonfinite_pairs);
    else if (variant == kCosNdLongRows)
      hipLaunchKernelGGL(rows_cos_kernel, dim3(wg), dim3(kDiffBlock), 0, stream, segs, ext, n, total_tiles,
                         results, partials, nonfinite_pairs);
    else if (variant == kCosNdGathers)
      hipLaunchKernelGGL(gather_cos_kernel, dim3(wg), dim3(kDiffBlock), 0, stream, segs, ext, n, total_tiles,
                         results, partials, nonfinite_pairs);
    else
      hipLaunchKernelGGL((diff_kernel<true, true>), dim3(wg), dim3(kDiffBlock), 0, stream, segs, ext, n,
                         total_tiles, results, partials, nonfinite_pairs);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // the block trees run per result (a "unit": the result's segments, whose
  // tiles are consecutive), as the 2-D pass runs them per segment
  for (int k = 1; k < kCosLevels; ++k) {
    if (level_groups[k] == 0) break;
    const uint64_t grid = level_groups[k] < 65536 ? level_groups[k] : 65536;
    hipLaunchKernelGGL(cos_level_kernel, dim3((unsigned)grid), dim3(kCosBlock), 0, stream, levels_of,
                       level_prefix + (size_t)(k - 1) * (n_results + 1), n_results, k, partials, levels);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(cosine_kernel, dim3(n_results), dim3(kCosBlock), 0, stream, units, levels_of, partials,
                     levels, nonfinite_pairs, cos_results);
  return hipGetLastError();
}

}  // namespace asmevo
