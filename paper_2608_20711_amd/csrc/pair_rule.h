// pair_rule.h -- the comparison's element types, and its rule for one pair
// of elements applied to a lane's partial result (AsmEvo section 3.2, Eq. 1:
// Delta = K'(x) - O(x) element by element; section 3.4: floating outputs
// compared within a tolerance, integer and opaque state byte-exactly).
//
// Every pair counts towards the bitwise result when its bits differ.  The
// tolerance rule, for candidate element A and reference element B of a float
// type with raw bits xa, xb:
//  * identical bits match, except a NaN in B under the strict NaN policy;
//  * bits that differ with a NaN on either side fail, unless both are NaN
//    and the policy is EQUAL;
//  * bits that differ with an infinity on either side fail;
//  * finite pairs fail unless |A - B| <= atol + rtol * |B| (fp64, each
//    operation rounded once, no fused multiply-add);
//  * finite pairs whose bits differ report |A - B| and |A - B| / |B| (+Inf
//    when B = 0 and A != 0) for the segment's maxima.
#pragma once
#pragma clang fp contract(off)

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asmevo.h"

namespace asmevo {

template <int DT> struct Et;
template <> struct Et<ASMEVO_F32> { static constexpr int es = 4; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_BF16> { static constexpr int es = 2; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_F16> { static constexpr int es = 2; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_FP8_E4M3> { static constexpr int es = 1; static constexpr bool fp = true; };
template <> struct Et<ASMEVO_I32> { static constexpr int es = 4; static constexpr bool fp = false; };
template <> struct Et<ASMEVO_I64> { static constexpr int es = 8; static constexpr bool fp = false; };
template <> struct Et<ASMEVO_U8> { static constexpr int es = 1; static constexpr bool fp = false; };

template <int DT>
__device__ __forceinline__ bool is_nan_raw(uint64_t r) {
  if constexpr (DT == ASMEVO_F32) return (r & 0x7FFFFFFFu) > 0x7F800000u;
  else if constexpr (DT == ASMEVO_BF16) return (r & 0x7FFFu) > 0x7F80u;
  else if constexpr (DT == ASMEVO_F16) return (r & 0x7FFFu) > 0x7C00u;
  else if constexpr (DT == ASMEVO_FP8_E4M3) return (r & 0x7Fu) == 0x7Fu;
  else return false;
}

// Exact fp64 value of an element given its raw bits (any value for Inf and
// NaN, which the callers test for separately): binary32 and bfloat16 by a
// bit cast, binary16 by v_cvt_f32_f16, fp8 e4m3 by v_cvt_f32_fp8 (both exact,
// subnormals kept), then binary32 -> binary64, which is exact.
template <int DT>
__device__ __forceinline__ double raw_f64(uint32_t r) {
  if constexpr (DT == ASMEVO_F32) return (double)__uint_as_float(r);
  else if constexpr (DT == ASMEVO_BF16) return (double)__uint_as_float(r << 16);
  else if constexpr (DT == ASMEVO_F16) return (double)(float)__builtin_bit_cast(_Float16, (uint16_t)r);
  else return (double)__builtin_amdgcn_cvt_f32_fp8((int)r, 0);
}

template <int DT>
__device__ __forceinline__ bool is_finite_raw(uint32_t r) {
  if constexpr (DT == ASMEVO_F32) return (r & 0x7F800000u) != 0x7F800000u;
  else if constexpr (DT == ASMEVO_BF16) return (r & 0x7F80u) != 0x7F80u;
  else if constexpr (DT == ASMEVO_F16) return (r & 0x7C00u) != 0x7C00u;
  else return (r & 0x7Fu) != 0x7Fu;       // e4m3fn: no infinities, S.1111.111 is NaN
}

// A lane's partial result over the pairs it has compared.
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

// One element pair at logical index i that needs attention (its bits differ,
// or b is a NaN under the strict policy), added to the lane's partials: the
// bitwise count, and in tolerance mode the rule above.  The rule is
// evaluated without branches (every quantity is computed and the outcome
// selected), so lanes of a wave that hold different cases run it together.
template <int DT>
__device__ __forceinline__ void pair_slow(uint64_t ra, uint64_t rb, uint64_t i, bool tol_mode,
                                       bool strict, double atol, double rtol, Acc& acc) {
  const bool bw = ra != rb;
  acc.bw += bw ? 1u : 0u;
  acc.first_bw = (bw && i < acc.first_bw) ? i : acc.first_bw;
  if constexpr (Et<DT>::fp) {
    if (!tol_mode) return;                  // uniform across the wave
    const uint32_t xa = (uint32_t)ra, xb = (uint32_t)rb;
    const bool nan_a = is_nan_raw<DT>(xa), nan_b = is_nan_raw<DT>(xb);
    const bool finite = is_finite_raw<DT>(xa) && is_finite_raw<DT>(xb);
    const double A = raw_f64<DT>(xa), B = raw_f64<DT>(xb);
    const double d = __builtin_fabs(A - B);
    const double mag_b = __builtin_fabs(B);
    const double scaled = rtol * mag_b;
    const double t = atol + scaled;
    // the cases of the rule as 0/1 words combined with bitwise operators,
    // which keeps the compiler from turning them into branches
    const uint32_t w_bw = bw, w_na = nan_a, w_nb = nan_b, w_st = strict;
    const uint32_t w_fail = (uint32_t)(!finite) | (uint32_t)!(d <= t);
    const uint32_t w_nan = w_na | w_nb;
    const bool mism = ((~w_bw & w_nb & w_st) | (w_bw & w_nan & ~(w_na & w_nb & ~w_st)) |
                       (w_bw & ~w_nan & w_fail)) & 1u;
    const double q = d / mag_b;
    const double rel = mag_b != 0.0 ? q : (d == 0.0 ? 0.0 : __builtin_inf());
    const bool upd = bw && finite;          // the maxima cover finite pairs whose bits differ
    const uint64_t db = upd ? (uint64_t)__double_as_longlong(d) : 0ull;
    const uint64_t rlb = upd ? (uint64_t)__double_as_longlong(rel) : 0ull;
    acc.max_abs = db > acc.max_abs ? db : acc.max_abs;
    acc.max_rel = rlb > acc.max_rel ? rlb : acc.max_rel;
    acc.tol += mism ? 1u : 0u;
    acc.first_tol = (mism && i < acc.first_tol) ? i : acc.first_tol;
    acc.nf += (mism && !finite) ? 1u : 0u;
  }
}

}  // namespace asmevo
