// fill.hip -- guarded seeded fill (AsmEvo section 3.4, Tier 1: deterministic
// seeded inputs; every allocation carries canary-initialised guard regions so
// that out-of-bounds writes become visible to the equivalence check).
//
// One pass writes every byte of every allocation in 16-byte vector stores:
// lo canary | data elements | row-pad bytes | hi canary.  Candidate
// differences selected by Bernoulli rules are applied in the same pass; point
// injections and guard writes follow in a second, tiny kernel.
#include "device_math.h"
#include "kernels.h"
#include "layout.h"

namespace asmevo {
namespace {

template <int DT>
struct Elem;
template <> struct Elem<ASMEVO_F32> { static constexpr int es = 4; };
template <> struct Elem<ASMEVO_BF16> { static constexpr int es = 2; };
template <> struct Elem<ASMEVO_F16> { static constexpr int es = 2; };
template <> struct Elem<ASMEVO_FP8_E4M3> { static constexpr int es = 1; };
template <> struct Elem<ASMEVO_I32> { static constexpr int es = 4; };
template <> struct Elem<ASMEVO_I64> { static constexpr int es = 8; };
template <> struct Elem<ASMEVO_U8> { static constexpr int es = 1; };

__device__ __forceinline__ uint64_t emask(uint32_t es) {
  return es == 8 ? ~0ull : ((1ull << (8u * es)) - 1ull);
}

// Boundary pattern k (0..15) of an element type.  Float patterns come from
// the format's exponent and mantissa widths; integer patterns from the width.
__device__ __forceinline__ uint64_t boundary_bits(uint32_t dtype, uint32_t es, uint32_t k) {
  const uint32_t W = 8u * es;
  const uint64_t mask = emask(es);
  const uint64_t sign = 1ull << (W - 1u);
  if (dtype <= ASMEVO_FP8_E4M3) {
    const uint32_t M = dtype == ASMEVO_F32 ? 23u : dtype == ASMEVO_BF16 ? 7u : dtype == ASMEVO_F16 ? 10u : 3u;
    const uint32_t E = W - 1u - M;
    const uint64_t one = ((1ull << (E - 1u)) - 1ull) << M;   // biased exponent of 1.0
    const uint64_t expo = ((1ull << E) - 1ull) << M;         // all-ones exponent field
    const bool fp8 = dtype == ASMEVO_FP8_E4M3;
    const uint64_t maxf = fp8 ? 0x7Eull : expo - 1ull;
    switch (k) {
      case 0: return 0;
      case 1: return sign;
      case 2: return 1;
      case 3: return sign | 1ull;
      case 4: return (1ull << M) - 1ull;
      case 5: return 1ull << M;
      case 6: return one;
      case 7: return sign | one;
      case 8: return one - 1ull;
      case 9: return one + 1ull;
      case 10: return maxf;
      case 11: return sign | maxf;
      case 12: return fp8 ? 0x7Full : expo;
      case 13: return fp8 ? 0xFFull : sign | expo;
      case 14: return fp8 ? 0x7Full : expo | (1ull << (M - 1u));
      default: return fp8 ? maxf - 1ull : expo | 1ull;
    }
  }
  switch (k) {
    case 0: return 0;
    case 1: return 1;
    case 2: return mask;
    case 3: return sign;
    case 4: return mask ^ sign;
    case 5: return sign | 1ull;
    case 6: return (mask ^ sign) - 1ull;
    case 7: return 0x5555555555555555ull & mask;
    case 8: return 0xAAAAAAAAAAAAAAAAull & mask;
    default: break;
  }
  if (es == 1) {
    switch (k) {
      case 9: return 0x0F;
      case 10: return 0xF0;
      case 11: return 0x10;
      case 12: return 0xEF;
      case 13: return 0x40;
      case 14: return 0xBF;
      default: return 2;
    }
  }
  const uint32_t H = W / 2u;                                   // half width
  switch (k) {
    case 9: return 0xFF;
    case 10: return (1ull << H) - 1ull;
    case 11: return 1ull << H;
    case 12: return mask ^ ((1ull << H) - 1ull);
    case 13: return es == 4 ? 0x80ull : 0x80000000ull;
    case 14: return es == 4 ? 0x7F7F7F7Full : 0x7FFFFFFFull;
    default: return 2;
  }
}

// Base value of element i (before any injection), for an element whose
// generator block has already been drawn: X = VALUE block i/4.
__device__ __forceinline__ uint64_t base_from_block(const FillAlloc& A, const U4& X, uint64_t i,
                                                    uint64_t seed) {
  switch (A.dist) {
    case ASMEVO_DIST_NORMAL: {
      const uint32_t pair = (uint32_t)(i >> 1) & 1u;
      double z0, z1;
      box_muller(pair ? X.z : X.x, pair ? X.w : X.y, z0, z1);
      const double z = (i & 1) ? z1 : z0;
      const double scaled = A.p1 * z;
      const double v = A.p0 + scaled;
      return encode_f32(A.dtype, (float)v, A.saturate != 0);
    }
    case ASMEVO_DIST_UNIFORM_INT: {
      const uint64_t span = (uint64_t)(A.i1 - A.i0);
      const uint64_t x = word_of(X, (uint32_t)i & 3u);
      const int64_t v = A.i0 + (int64_t)((x * span) >> 32);
      if (A.dtype <= ASMEVO_FP8_E4M3) return encode_f32(A.dtype, (float)(double)v, A.saturate != 0);
      return (uint64_t)v & emask(A.esize);
    }
    case ASMEVO_DIST_BITS: {
      // bytes [i*es, (i+1)*es) of the VALUE stream; they sit in one block
      const uint64_t q0 = i * A.esize;
      const U4 B = stream(seed, A.alloc_id, kValue, 0, 0, q0 >> 4);
      uint64_t bits = 0;
      for (uint32_t k = 0; k < A.esize; ++k)
        bits |= (uint64_t)byte_of(B, (uint32_t)((q0 + k) & 15u)) << (8u * k);
      return bits;
    }
    case ASMEVO_DIST_BOUNDARY: {
      // its own VALUE block i: x selects (threshold in i0), y picks the pattern
      const U4 B = stream(seed, A.alloc_id, kValue, 0, 0, i);
      if ((uint64_t)B.x < (uint64_t)A.i0) return boundary_bits(A.dtype, A.esize, B.y & 15u);
      if (A.dtype <= ASMEVO_FP8_E4M3) {
        double z0, z1;
        box_muller(B.z, B.w, z0, z1);
        const double v = A.p1 * z0;
        return encode_f32(A.dtype, (float)v, A.saturate != 0);
      }
      return ((uint64_t)B.z | ((uint64_t)B.w << 32)) & emask(A.esize);
    }
    default:  // CONST
      if (A.dtype <= ASMEVO_FP8_E4M3) return encode_f32(A.dtype, (float)A.p0, A.saturate != 0);
      return (uint64_t)A.i0 & emask(A.esize);
  }
}

__device__ __forceinline__ uint64_t base_element(const FillAlloc& A, uint64_t i, uint64_t seed) {
  U4 X{0, 0, 0, 0};
  if (A.dist == ASMEVO_DIST_NORMAL || A.dist == ASMEVO_DIST_UNIFORM_INT)
    X = stream(seed, A.alloc_id, kValue, 0, 0, i >> 2);
  return base_from_block(A, X, i, seed);
}

__device__ __forceinline__ uint64_t max_finite_mag(uint32_t dtype) {
  switch (dtype) {
    case ASMEVO_F32: return 0x7F7FFFFFull;
    case ASMEVO_BF16: return 0x7F7Full;
    case ASMEVO_F16: return 0x7BFFull;
    default: return 0x7Eull;
  }
}

__device__ __forceinline__ uint64_t decode_any(uint32_t dtype, uint64_t raw, double& v, int& cls) {
  switch (dtype) {
    case ASMEVO_F32: cls = decode<ASMEVO_F32>(raw, v); break;
    case ASMEVO_BF16: cls = decode<ASMEVO_BF16>(raw, v); break;
    case ASMEVO_F16: cls = decode<ASMEVO_F16>(raw, v); break;
    default: cls = decode<ASMEVO_FP8_E4M3>(raw, v); break;
  }
  return raw;
}

// The candidate value of an injected element, from its base value.
__device__ __forceinline__ uint64_t apply_injection(const FillAlloc& A, uint32_t kind, uint32_t vsel, uint32_t arg,
                                    double atol, double rtol, uint64_t base, uint64_t seed,
                                    uint64_t i) {
  const uint32_t es = A.esize;
  const uint64_t sign_bit = 1ull << (8u * es - 1u);
  if (kind == ASMEVO_INJ_FLIP_BIT) {
    uint32_t bit = arg;
    if (arg == 0xFFFFFFFFu) bit = stream(seed, A.alloc_id, kInject, 0, vsel, i).x & (8u * es - 1u);
    return base ^ (1ull << bit);
  }
  if (kind == ASMEVO_INJ_STEP_WITHIN) {
    const uint64_t sign = base & sign_bit;
    uint64_t mag = base & ~sign_bit & emask(es);
    const uint64_t maxmag = max_finite_mag(A.dtype);
    if (mag > maxmag) return base;
    const bool grow = (stream(seed, A.alloc_id, kInject, 0, vsel, i).x & 1u) == 0u;
    if ((grow && mag < maxmag) || mag == 0) mag += 1;
    else mag -= 1;
    return sign | mag;
  }
  if (kind == ASMEVO_INJ_SET_BEYOND) {
    double B = 0.0;
    int cls = 0;
    decode_any(A.dtype, base, B, cls);
    if (cls != 0) return base;
    const double scaled = rtol * __builtin_fabs(B);
    const double t = atol + scaled;
    const double four_t = 4.0 * t;
    const double v = (base & sign_bit) ? B + four_t : B - four_t;
    return encode_f32(A.dtype, (float)v, A.saturate != 0);
  }
  if (kind == ASMEVO_INJ_SET_NAN) {
    switch (A.dtype) {
      case ASMEVO_F32: return 0x7FC00000ull;
      case ASMEVO_BF16: return 0x7FC0ull;
      case ASMEVO_F16: return 0x7E00ull;
      default: return 0x7Full;
    }
  }
  if (kind == ASMEVO_INJ_SET_INF) {
    const uint64_t s = (arg & 1u) ? sign_bit : 0ull;
    switch (A.dtype) {
      case ASMEVO_F32: return s | 0x7F800000ull;
      case ASMEVO_BF16: return s | 0x7F80ull;
      default: return s | 0x7C00ull;
    }
  }
  return base;
}

// Applies the allocation's Bernoulli rules to element i (last selecting rule
// wins; each acts on the base value).
__device__ __forceinline__ uint64_t apply_rules(const FillAlloc& A, const FillRule* rules,
                                                uint64_t base, uint64_t seed, uint64_t i) {
  uint64_t v = base;
  for (uint32_t r = 0; r < A.rule_count; ++r) {
    const FillRule R = rules[A.rule_begin + r];
    const U4 S = stream(seed, A.alloc_id, kSelect, R.ordinal, R.vsel, i >> 2);
    if ((uint64_t)word_of(S, (uint32_t)i & 3u) < R.threshold)
      v = apply_injection(A, R.kind, R.vsel, R.arg, R.atol, R.rtol, base, seed, i);
  }
  return v;
}

__device__ __forceinline__ uint64_t element_value(const FillAlloc& A, const FillRule* rules,
                                                  uint64_t i, uint64_t seed) {
  return apply_rules(A, rules, base_element(A, i, seed), seed, i);
}

// Inserts element m (es bytes, little-endian) into a 16-byte chunk held in
// four words, with selects instead of register indexing.
template <int ES>
__device__ __forceinline__ void put_elem(uint32_t w[4], uint32_t m, uint64_t v) {
  if constexpr (ES == 8) {
    const bool hi = m != 0;
    w[0] = hi ? w[0] : (uint32_t)v;
    w[1] = hi ? w[1] : (uint32_t)(v >> 32);
    w[2] = hi ? (uint32_t)v : w[2];
    w[3] = hi ? (uint32_t)(v >> 32) : w[3];
  } else {
    const uint32_t byte = m * ES;
    const uint32_t wi = byte >> 2;
    const uint32_t bits = (uint32_t)(v & ((ES == 4) ? 0xFFFFFFFFull : ((1ull << (8 * ES)) - 1))) << (8u * (byte & 3u));
    w[0] |= wi == 0 ? bits : 0u;
    w[1] |= wi == 1 ? bits : 0u;
    w[2] |= wi == 2 ? bits : 0u;
    w[3] |= wi == 3 ? bits : 0u;
  }
}

// 16 data bytes holding exactly 16/es whole elements starting at logical
// index i0 of one row.  When i0 is a multiple of 4 the chunk is made of whole
// generator blocks: each VALUE and SELECT block is drawn once for its four
// elements.
template <int DT>
__device__ __forceinline__ void data_chunk(const FillAlloc& A, const FillAlloc* Ap, const FillRule* rules,
                                           uint64_t i0, uint64_t seed, uint32_t w[4]) {
  constexpr int es = Elem<DT>::es;
  constexpr int epc = 16 / es;
  w[0] = w[1] = w[2] = w[3] = 0;
  if (es <= 4 && (i0 & 3u) == 0 &&
      (A.dist == ASMEVO_DIST_NORMAL || A.dist == ASMEVO_DIST_UNIFORM_INT)) {
#pragma unroll 1
    for (uint32_t blk = 0; blk < (uint32_t)(epc / 4); ++blk) {
      const uint64_t j = (i0 >> 2) + blk;
      // The value parameters are loaded again for every block (the empty asm
      // hides that the pointer is loop-invariant): held across the loop they
      // would be spilled and read back by v_readlane inside it.
      const FillAlloc* q = Ap;
      asm volatile("" : "+s"(q));
      const U4 X = stream(seed, q->alloc_id, kValue, 0, 0, j);
      uint64_t base[4];
      if (A.dist == ASMEVO_DIST_NORMAL) {
        const double p0 = q->p0, p1 = q->p1;
        const bool sat = q->saturate != 0;
#pragma unroll 1
        for (uint32_t h = 0; h < 2; ++h) {
          double z0, z1;
          box_muller(h ? X.z : X.x, h ? X.w : X.y, z0, z1);
          const double v0 = p0 + p1 * z0;
          const double v1 = p0 + p1 * z1;
          const uint64_t e0 = encode_f32(DT, (float)v0, sat);
          const uint64_t e1 = encode_f32(DT, (float)v1, sat);
          base[0] = h ? base[0] : e0;
          base[1] = h ? base[1] : e1;
          base[2] = h ? e0 : base[2];
          base[3] = h ? e1 : base[3];
        }
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) base[t] = base_from_block(A, X, 4 * j + t, seed);
      }
      uint64_t val[4] = {base[0], base[1], base[2], base[3]};
      for (uint32_t r = 0; r < A.rule_count; ++r) {
        const FillRule R = rules[A.rule_begin + r];
        const U4 S = stream(seed, A.alloc_id, kSelect, R.ordinal, R.vsel, j);
        uint32_t sel = ((uint64_t)S.x < R.threshold ? 1u : 0u) | ((uint64_t)S.y < R.threshold ? 2u : 0u) |
                       ((uint64_t)S.z < R.threshold ? 4u : 0u) | ((uint64_t)S.w < R.threshold ? 8u : 0u);
        while (sel) {                       // rare: the selected elements of this block
          const uint32_t t = (uint32_t)__builtin_ctz(sel);
          sel &= sel - 1u;
          const uint64_t b = t == 0 ? base[0] : t == 1 ? base[1] : t == 2 ? base[2] : base[3];
          const uint64_t v = apply_injection(A, R.kind, R.vsel, R.arg, R.atol, R.rtol, b, seed, 4 * j + t);
          val[0] = t == 0 ? v : val[0];
          val[1] = t == 1 ? v : val[1];
          val[2] = t == 2 ? v : val[2];
          val[3] = t == 3 ? v : val[3];
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) put_elem<es>(w, blk * 4 + t, val[t]);
    }
  } else {
#pragma unroll 1
    for (uint32_t m = 0; m < (uint32_t)epc; ++m)
      put_elem<es>(w, m, element_value(A, rules, i0 + m, seed));
  }
}

__device__ __forceinline__ uint8_t pad_byte(const FillAlloc& A, uint64_t q, uint64_t seed) {
  return byte_of(stream(seed, A.alloc_id, kPad, 0, 0, q >> 4), (uint32_t)(q & 15u));
}

__device__ __forceinline__ uint8_t canary_byte(uint32_t alloc_id, uint32_t side, uint64_t p,
                                               uint64_t seed) {
  return byte_of(stream(seed, alloc_id, kCanary, side, 0, p >> 4), (uint32_t)(p & 15u));
}

// Byte-by-byte general path for chunks that straddle a region boundary or
// the allocation's ends (o may be negative: the first chunk of an
// allocation that does not start on a 16-byte boundary).
__device__ __forceinline__ void general_chunk(const FillAlloc& A, const FillRule* rules, int64_t o,
                              uint64_t seed, uint32_t w[4]) {
  const uint64_t glo = A.guard_lo, D = A.data_bytes, tot = A.total_bytes;
  uint64_t cached_e = ~0ull, cached_v = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) w[k] = 0;
#pragma unroll 1
  for (uint32_t b = 0; b < 16; ++b) {
    if (o + (int64_t)b < 0) continue;
    const uint64_t p = (uint64_t)(o + (int64_t)b);
    if (p >= tot) break;
    uint8_t byte;
    if (p < glo) {
      byte = canary_byte(A.alloc_id, 0, p, seed);
    } else if (p < glo + D) {
      const uint64_t q = p - glo;
      const uint64_t e = q / A.esize;
      const uint64_t r = e / A.stride, c = e - r * A.stride;
      if (c < A.cols) {
        if (e != cached_e) {
          cached_v = element_value(A, rules, r * A.cols + c, seed);
          cached_e = e;
        }
        byte = (uint8_t)(cached_v >> (8u * (uint32_t)(q % A.esize)));
      } else {
        byte = pad_byte(A, q, seed);
      }
    } else {
      byte = canary_byte(A.alloc_id, 1, p - glo - D, seed);
    }
    put_elem<1>(w, b, byte);
  }
}

template <int DT>
__device__ __forceinline__ bool try_data_chunk(const FillAlloc& A, const FillAlloc* Ap, const FillRule* rules,
                                               uint64_t o, uint64_t seed, uint32_t w[4]) {
  constexpr int es = Elem<DT>::es;
  constexpr int epc = 16 / es;
  const uint64_t q = o - A.guard_lo;
  const uint64_t e0 = q / es;
  uint64_t r = 0, c0 = e0;
  if (A.rows > 1) {
    r = e0 / A.stride;
    c0 = e0 - r * A.stride;
  }
  if (c0 + epc > A.cols) return false;
  data_chunk<DT>(A, Ap, rules, r * A.cols + c0, seed, w);
  return true;
}

// Allocation bytes [o, o + 16) (one 16-byte block of memory; o may be
// negative for the first one).  The whole-chunk paths below need the
// allocation to start on a 16-byte boundary (phase 0), where a chunk is one
// generator block of canary bytes or whole elements; otherwise every chunk
// goes byte by byte.
__device__ __forceinline__ void fill_one_chunk(const FillAlloc& A, const FillAlloc* Ap, const FillRule* rules,
                                               int64_t os, uint64_t seed) {
  const uint64_t glo = A.guard_lo, D = A.data_bytes, tot = A.total_bytes;
  const uint64_t o = (uint64_t)os;            // used only where os >= 0
  uint32_t w[4];
  bool done = false;
  if (A.phase != 0) {
    // (no whole-chunk path)
  } else if (o + 16 <= glo) {
    const U4 C = stream(seed, A.alloc_id, kCanary, 0, 0, o >> 4);
    w[0] = C.x; w[1] = C.y; w[2] = C.z; w[3] = C.w;
    done = true;
  } else if (o >= glo + D && o + 16 <= tot && ((o - glo - D) & 15u) == 0) {
    const U4 C = stream(seed, A.alloc_id, kCanary, 1, 0, (o - glo - D) >> 4);
    w[0] = C.x; w[1] = C.y; w[2] = C.z; w[3] = C.w;
    done = true;
  } else if (o >= glo && o + 16 <= glo + D) {
    switch (A.dtype) {
      case ASMEVO_F32: done = try_data_chunk<ASMEVO_F32>(A, Ap, rules, o, seed, w); break;
      case ASMEVO_BF16: done = try_data_chunk<ASMEVO_BF16>(A, Ap, rules, o, seed, w); break;
      case ASMEVO_F16: done = try_data_chunk<ASMEVO_F16>(A, Ap, rules, o, seed, w); break;
      case ASMEVO_FP8_E4M3: done = try_data_chunk<ASMEVO_FP8_E4M3>(A, Ap, rules, o, seed, w); break;
      case ASMEVO_I32: done = try_data_chunk<ASMEVO_I32>(A, Ap, rules, o, seed, w); break;
      case ASMEVO_I64: done = try_data_chunk<ASMEVO_I64>(A, Ap, rules, o, seed, w); break;
      default: done = try_data_chunk<ASMEVO_U8>(A, Ap, rules, o, seed, w); break;
    }
  }
  if (!done) general_chunk(A, rules, os, seed, w);
  if (os >= 0 && o + 16 <= tot) {             // base + o is 16-byte aligned
    // Non-temporal: the state is written once and read next by a full pass
    // over all of it.  With ordinary stores the last ~256 MB written stayed
    // in the memory-side cache and the diff that followed the fill ran 2 %
    // slower over the 64 GiB sweep (20.76 against 20.31 ms).
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = {w[0], w[1], w[2], w[3]};
    __builtin_nontemporal_store(v, gptr_mut<u32x4>(A.base + o));
  } else {                                    // only the allocation's own bytes
    for (uint32_t b = 0; b < 16; ++b) {
      const int64_t p = os + (int64_t)b;
      if (p >= 0 && (uint64_t)p < tot) *gptr_mut<uint8_t>(A.base + (uint64_t)p) = (uint8_t)(w[b >> 2] >> (8u * (b & 3u)));
    }
  }
}

// Tiles of 64 chunks (one chunk per lane) never straddle allocations.  The
// fill is bound by its arithmetic, whose cost per tile depends on the
// element type (a tile of fp8 values draws 4x the normals of an fp32 one),
// so the waves of the resident grid deal the tiles round-robin: every wave
// gets the same mix and all finish together.
__global__ __launch_bounds__(kFillBlock) void fill_kernel(const FillAlloc* __restrict__ allocs,
                                                          int n, const FillRule* __restrict__ rules,
                                                          uint64_t total_tiles, uint64_t seed) {
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = (uint64_t)blockIdx.x * (kFillBlock / kWave) +
                        __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t nwaves = (uint64_t)gridDim.x * (kFillBlock / kWave);
  if (wave >= total_tiles) return;
  int s_lo = 0, s_hi = n - 1;             // last allocation with tile_begin <= wave
  while (s_lo < s_hi) {
    const int mid = (s_lo + s_hi + 1) >> 1;
    if (allocs[mid].tile_begin <= wave) s_lo = mid;
    else s_hi = mid - 1;
  }
  int k = s_lo;
  for (uint64_t t = wave; t < total_tiles; t += nwaves) {
    while (k + 1 < n && allocs[k + 1].tile_begin <= t) ++k;
    const FillAlloc A = allocs[k];
    // chunk c of the allocation is the 16-byte block of memory at
    // base - phase + 16 c, i.e. allocation bytes [16 c - phase, 16 c - phase + 16)
    const int64_t o = (int64_t)(((t - A.tile_begin) * kWave + lane) * kChunk) - (int64_t)A.phase;
    if (o < (int64_t)A.total_bytes) fill_one_chunk(A, allocs + k, rules, o, seed);
  }
}

// Point injections (deduplicated on the host: one entry per element), guard
// writes (bytes set to the complement of their canary) and row-pad writes
// (bytes set to the complement of their pad byte).
__global__ void inject_kernel(const FillAlloc* __restrict__ allocs,
                              const PointEntry* __restrict__ pts, int n_pts, uint64_t seed) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_pts) return;
  const PointEntry P = pts[t];
  const FillAlloc A = allocs[P.alloc];
  if (P.kind == ASMEVO_INJ_GUARD_WRITE_LO || P.kind == ASMEVO_INJ_GUARD_WRITE_HI) {
    const uint32_t side = P.kind == ASMEVO_INJ_GUARD_WRITE_HI;
    AS_GLOBAL uint8_t* g = gptr_mut<uint8_t>(side ? A.base + A.guard_lo + A.data_bytes : A.base);
    for (uint32_t b = 0; b < P.arg; ++b) {
      const uint64_t p = (uint64_t)P.index + b;
      g[p] = (uint8_t)~canary_byte(A.alloc_id, side, p, seed);
    }
    return;
  }
  if (P.kind == ASMEVO_INJ_PAD_WRITE) {
    AS_GLOBAL uint8_t* d = gptr_mut<uint8_t>(A.base + A.guard_lo);
    for (uint32_t b = 0; b < P.arg; ++b) {
      const uint64_t q = (uint64_t)P.index + b;
      d[q] = (uint8_t)~pad_byte(A, q, seed);
    }
    return;
  }
  const uint64_t i = (uint64_t)P.index;
  const uint64_t v = apply_injection(A, P.kind, P.vsel, P.arg, P.atol, P.rtol,
                                     base_element(A, i, seed), seed, i);
  const uint64_t r = i / A.cols, c = i - r * A.cols;
  const uint64_t dst = A.base + A.guard_lo + (r * A.stride + c) * A.esize;
  switch (A.esize) {
    case 1: *gptr_mut<uint8_t>(dst) = (uint8_t)v; break;
    case 2: *gptr_mut<uint16_t>(dst) = (uint16_t)v; break;
    case 4: *gptr_mut<uint32_t>(dst) = (uint32_t)v; break;
    default: *gptr_mut<uint64_t>(dst) = v; break;
  }
}

}  // namespace

int fill_blocks_per_cu() {
  static const int blocks = [] {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, fill_kernel, kFillBlock, 0) != hipSuccess || b <= 0)
      b = 4;
    return b;
  }();
  return blocks;
}

hipError_t launch_fill(const FillAlloc* allocs, int n, const FillRule* rules, uint64_t total_tiles,
                       uint64_t seed, int workgroups, hipStream_t stream) {
  if (total_tiles == 0 || n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3(workgroups), dim3(kFillBlock), 0, stream, allocs, n, rules,
                     total_tiles, seed);
  return hipGetLastError();
}

hipError_t launch_inject(const FillAlloc* allocs, const PointEntry* pts, int n_pts, uint64_t seed,
                         hipStream_t stream) {
  if (n_pts == 0) return hipSuccess;
  const int block = 256;
  hipLaunchKernelGGL(inject_kernel, dim3((n_pts + block - 1) / block), dim3(block), 0, stream,
                     allocs, pts, n_pts, seed);
  return hipGetLastError();
}

}  // namespace asmevo
