/*
 * ref_oracle.h -- the CPU oracle's own interface (test infrastructure only).
 *
 * This header belongs to the plain, slow CPU reference that the GPU library is
 * checked against.  It shares no code, header, table or constant with the GPU
 * library: every struct and constant here is declared independently, from the
 * definitions of the differential oracle (paper section 3.2, Eq. 1 and the
 * predicate iota; section 3.4, "Tier 1" guarded synthesis and the Tier-2
 * byte-exact checks).  Only tests/, the smoke entry point and the bench's
 * cpu_baseline leg load it.
 */
#ifndef REF_ORACLE_H
#define REF_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types */
enum { REF_F32 = 1, REF_BF16 = 2, REF_F16 = 3, REF_FP8E4M3 = 4, REF_I32 = 5, REF_I64 = 6, REF_U8 = 7 };
/* comparison modes and NaN policies */
enum { REF_BITWISE = 0, REF_TOLERANCE = 1 };
enum { REF_NAN_EQUAL = 0, REF_NAN_STRICT = 1 };
/* value distributions of a fill */
enum { REF_NORMAL = 0, REF_UNIFORM_INT = 1, REF_BITS = 2, REF_CONST = 3, REF_BOUNDARY = 4 };
/* injection kinds; REF_RATE is or-ed into the kind of a Bernoulli rule */
enum {
  REF_FLIP_BIT = 1, REF_STEP_WITHIN = 2, REF_SET_BEYOND = 3, REF_SET_NAN = 4, REF_SET_INF = 5,
  REF_GUARD_WRITE_LO = 6, REF_GUARD_WRITE_HI = 7,
  REF_PAD_WRITE = 8        /* invert `arg` row-pad bytes from data byte offset `index` */
};
#define REF_RATE 0x100u
enum { REF_SIDE_CANDIDATE = 0, REF_SIDE_BOTH = 1 };

typedef struct {
  int32_t dtype;
  uint32_t alloc_id;       /* logical buffer id, identical on both sides */
  int64_t rows, cols, stride;   /* elements */
  int64_t guard_lo, guard_hi;   /* bytes */
  int32_t dist;
  int32_t saturate;        /* fp8: clamp to +-448 before rounding */
  double p0, p1;           /* NORMAL mean/std; CONST value; BOUNDARY rate/std */
  int64_t i0, i1;          /* UNIFORM_INT [i0, i1); CONST integer value */
} ref_alloc;

typedef struct {
  uint32_t alloc;          /* index into the allocation array */
  uint32_t kind;           /* REF_* kind, optionally | REF_RATE */
  uint32_t sides;          /* REF_SIDE_* */
  uint32_t arg;            /* bit index (0xffffffff = random) / Inf sign / guard or pad byte count */
  int64_t index;           /* element index, guard byte offset, data byte offset (PAD_WRITE),
                              or (RATE) threshold T */
  double atol, rtol;       /* tolerance targeted by SET_BEYOND */
} ref_inj;

typedef struct {
  int32_t dtype, mode, nan_policy, pad_;
  int64_t rows, cols, stride_a, stride_b;  /* elements */
  double atol, rtol;
} ref_seg;

/* An N-dimensional segment: element (i_0, ..., i_{ndim-1}) of the candidate
 * lies at a + sum_d i_d * stride_a[d] elements (b likewise); its logical
 * index is index_base plus its row-major position (last dimension fastest). */
#define REF_MAX_DIMS 8
typedef struct {
  int32_t dtype, mode, nan_policy, ndim;
  int64_t index_base;
  int64_t shape[REF_MAX_DIMS];
  int64_t stride_a[REF_MAX_DIMS], stride_b[REF_MAX_DIMS];   /* elements, >= 0 */
  double atol, rtol;
} ref_seg_nd;

typedef struct {
  uint64_t mismatches;
  int64_t first_mismatch;
  uint64_t bitwise_mismatches;
  int64_t first_bitwise;
  uint64_t nonfinite_mismatches;
  double max_abs, max_rel;
} ref_seg_result;

typedef struct {
  uint64_t bad_lo, bad_hi;
  int64_t first_bad_lo, first_bad_hi;
  uint64_t bad_pad;          /* row-pad bytes that differ from their canary */
  int64_t first_bad_pad;     /* lowest such byte, as an offset from the first data byte */
} ref_guard_result;

/* Philox4x32-10 block function (Salmon et al., SC'11). */
void ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* element codecs */
int ref_esize(int32_t dtype);
/* class: 0 finite, 1 +Inf, 2 -Inf, 3 NaN; *value = exact fp64 value when finite */
int ref_decode(int32_t dtype, uint64_t raw, double* value);
uint64_t ref_encode_f32(int32_t dtype, float x, int saturate);

/* the fill's own transcendental pieces (exposed for pinning against libm) */
double ref_log_u(uint32_t x);                       /* ln((x + 0.5) * 2^-32) */
void ref_sincos_turns(uint32_t x, double* c, double* s);   /* cos/sin(2*pi*x*2^-32) */
double ref_normal(uint32_t xa, uint32_t xb, int which);    /* Box-Muller: which 0 cos, 1 sin */

/* raw bits of element i of allocation k as written by a fill of `variant` */
uint64_t ref_element(const ref_alloc* allocs, int32_t k, const ref_inj* inj, int64_t n_inj,
                     uint64_t seed, uint32_t variant, int64_t i);
uint8_t ref_canary_byte(uint64_t seed, uint32_t alloc_id, int side, int64_t p);

/* Writes bytes [off, off + nbytes) of allocation k (offsets from its first lo-guard byte). */
int ref_fill_range(const ref_alloc* allocs, int32_t k, const ref_inj* inj, int64_t n_inj,
                   uint64_t seed, uint32_t variant, int64_t off, int64_t nbytes, uint8_t* out);

/* Compares one segment: a, b point at element (0,0) of candidate and reference. */
int ref_diff_segment(const ref_seg* seg, const uint8_t* a, const uint8_t* b, ref_seg_result* res);

/* Compares one N-dimensional segment: a, b point at element (0, ..., 0). */
int ref_diff_segment_nd(const ref_seg_nd* seg, const uint8_t* a, const uint8_t* b, ref_seg_result* res);

/* Guard check of one allocation: lo/hi point at the first byte of each guard (may be NULL if 0).
 * Sets bad_pad = 0 and first_bad_pad = -1. */
int ref_guard_check(uint64_t seed, uint32_t alloc_id, const uint8_t* lo, int64_t n_lo,
                    const uint8_t* hi, int64_t n_hi, ref_guard_result* res);

/* Row-pad check of one allocation: `data` points at its first data byte; every
 * byte of a row's padding (elements cols..stride-1 of rows 0..rows-2) is
 * compared with the PAD byte the fill writes there.  Sets bad_pad and
 * first_bad_pad of `res` only. */
int ref_pad_check(const ref_alloc* A, uint64_t seed, const uint8_t* data, ref_guard_result* res);

/* Exact sum of binary64 values: a fixed-point integer from 2^-1074 up, in
 * base-2^32 digits held in int64 (a carry is needed only every 2^30
 * additions), rounded once to the nearest binary64 value, ties to even. */
#define REF_XACC_DIGITS 70          /* 2240 bits: 2^-1074 .. 2^1024, 64 bits of headroom, sign */
typedef struct {
  int64_t d[REF_XACC_DIGITS];
  int64_t adds;                     /* additions since the last carry */
} ref_xacc;
void ref_xacc_init(ref_xacc* x);
void ref_xacc_add(ref_xacc* x, double v);      /* v finite */
double ref_xacc_round(const ref_xacc* x);
double ref_exact_sum(const double* v, int64_t n);

/* Cosine term of Eq. 1 over one segment (float dtypes): the sums over the
 * element pairs with both values finite, each computed exactly and rounded
 * once; cosine = sum_ab / (sqrt(sum_aa) * sqrt(sum_bb)), each operation
 * rounded (1 when both sums of squares are 0, 0 when exactly one is).
 * sum_abs_ab = sum |a*b| (rounded once), the scale of the error bound of any
 * other summation order.  Integer buffers: sums 0, cosine NaN. */
typedef struct {
  double sum_ab, sum_aa, sum_bb, cosine;
  uint64_t pairs;        /* pairs with both values finite */
  double sum_abs_ab;
} ref_cos_result;
int ref_cosine_segment(const ref_seg* seg, const uint8_t* a, const uint8_t* b, ref_cos_result* res);
/* The same term over the elements of n N-D segments that share one result.
 * a[k], b[k]: element (0, ..., 0) of segment k.  Every segment must have the
 * same dtype.  n = 0: cosine 1 over no pairs. */
int ref_cosine_nd(const ref_seg_nd* segs, int32_t n, const uint8_t* const* a, const uint8_t* const* b,
                  ref_cos_result* res);

/* Restore / snapshot of captured regions: dst[k][0..bytes) = src[k][0..bytes)
 * for each region, in order (regions are host memory here). */
typedef struct {
  uint8_t* dst;
  const uint8_t* src;
  int64_t bytes;
} ref_region;
void ref_copy_regions(const ref_region* regions, int64_t n);

/* bulk loops over the scalar functions above (used by the pin tests) */
void ref_decode_n(int32_t dtype, const uint64_t* raw, int64_t n, int32_t* cls, double* value);
void ref_encode_f32_n(int32_t dtype, const float* x, int64_t n, int saturate, uint64_t* out);
void ref_log_u_n(const uint32_t* x, int64_t n, double* out);
void ref_sincos_turns_n(const uint32_t* x, int64_t n, double* c, double* s);
void ref_normal_n(const uint32_t* xa, const uint32_t* xb, int64_t n, int which, double* out);
void ref_philox_n(const uint32_t* ctr, const uint32_t* key, int64_t n, uint32_t* out);
/* Each pair (ra[k], rb[k]) compared on its own as a one-element segment:
 * flags bit 0 bitwise difference, bit 1 mismatch, bit 2 non-finite mismatch;
 * max_abs / max_rel the segment's maxima (0 unless finite with differing bits). */
void ref_compare_pair_n(int32_t dtype, int32_t mode, int32_t nan_policy, double atol, double rtol,
                        const uint64_t* ra, const uint64_t* rb, int64_t n, uint8_t* flags,
                        double* max_abs, double* max_rel);

#ifdef __cplusplus
}
#endif
#endif
