/*
 * ref_oracle.c -- plain, slow CPU oracle for the differential-oracle hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link or call this
 * file; only tests/, the smoke entry point and the bench's cpu_baseline leg do.
 * It shares no code with the GPU library.  Everything is scalar loops in index
 * order, fp64 where floating point is involved, and it is compiled without
 * fast-math and with floating-point contraction off, so every rounding below
 * is the one written.
 *
 * What it follows:
 *  - the equivalence predicate of the paper (section 3.2, Eq. 1): the element
 *    error Delta = K'(x) - O(x) and its infinity norm, with the reference O(x)
 *    as the operand that scales the relative term; the predicate iota requires
 *    bit-exact integer buffers and intact out-of-bounds guards;
 *  - section 3.4: Tier-1 deterministic seeded inputs whose allocations carry
 *    canary-initialised guard regions, and the Tier-2 rule that floating
 *    outputs are checked by tolerance while integer, opaque and guard bytes are
 *    checked byte-exactly.
 *  The element-wise tolerance |a - b| <= atol + rtol*|b| generalises the
 *  paper's ||Delta||_inf <= tau (atol = tau, rtol = 0 is exactly that test).
 *  The fill is this library's own definition (the paper only asks for
 *  deterministic seeded inputs); its generator is Philox4x32-10 from Salmon,
 *  Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3"
 *  (SC'11).
 *
 *  The cosine term of Eq. 1 has no summation order in its definition, so
 *  its three sums are computed exactly (a fixed-point accumulator) and each
 *  is rounded once.
 *
 * Pins (tests/test_oracle_*.py): Philox known-answer vectors; codecs against
 * numpy/torch casts over every 8- and 16-bit pattern; the tolerance mask
 * against numpy.isclose; the fill's ln/sin/cos against libm; closed-form
 * counts of constructed cases; brute force over every (index, bit) of tiny
 * buffers and every byte of tiny guards; the exact sums against Python's
 * exact rationals and math.fsum; the region copy against numpy slices; the
 * per-pair bulk loop against one-element segments and numpy.
 */
#include "ref_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10, as defined by Salmon et al. (SC'11): ten rounds of two     */
/* 32x32->64 multiplies with the round keys bumped by the Weyl constants.    */
/* ------------------------------------------------------------------------ */
void ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The fill's counter layout: (lo32(j), hi32(j), alloc_id, word3) with key =  */
/* (lo32(seed), hi32(seed)); word3 = purpose<<24 | aux<<16 | variant.         */
enum { PURPOSE_VALUE = 0, PURPOSE_SELECT = 1, PURPOSE_INJECT = 2, PURPOSE_CANARY = 3, PURPOSE_PAD = 5 };

static void stream_block(uint64_t seed, uint32_t alloc_id, uint32_t purpose, uint32_t aux,
                         uint32_t variant, uint64_t j, uint32_t out[4]) {
  uint32_t ctr[4], key[2];
  ctr[0] = (uint32_t)j;
  ctr[1] = (uint32_t)(j >> 32);
  ctr[2] = alloc_id;
  ctr[3] = (purpose << 24) | ((aux & 0xFFu) << 16) | (variant & 0xFFFFu);
  key[0] = (uint32_t)seed;
  key[1] = (uint32_t)(seed >> 32);
  ref_philox4x32_10(ctr, key, out);
}

/* byte q of a stream, little-endian within each 32-bit word */
static uint8_t stream_byte(uint64_t seed, uint32_t alloc_id, uint32_t purpose, uint32_t aux,
                           uint32_t variant, uint64_t q) {
  uint32_t w[4];
  stream_block(seed, alloc_id, purpose, aux, variant, q / 16, w);
  uint32_t word = w[(q % 16) / 4];
  return (uint8_t)(word >> (8 * (q % 4)));
}

uint8_t ref_canary_byte(uint64_t seed, uint32_t alloc_id, int side, int64_t p) {
  return stream_byte(seed, alloc_id, PURPOSE_CANARY, (uint32_t)side, 0, (uint64_t)p);
}

/* ------------------------------------------------------------------------ */
/* Element codecs.                                                           */
/* ------------------------------------------------------------------------ */
int ref_esize(int32_t dtype) {
  switch (dtype) {
    case REF_F32: return 4;
    case REF_BF16: return 2;
    case REF_F16: return 2;
    case REF_FP8E4M3: return 1;
    case REF_I32: return 4;
    case REF_I64: return 8;
    case REF_U8: return 1;
    default: return 0;
  }
}

static int is_float(int32_t dtype) {
  return dtype == REF_F32 || dtype == REF_BF16 || dtype == REF_F16 || dtype == REF_FP8E4M3;
}

/* IEEE binary32 via the C float type. */
static int decode_f32(uint32_t bits, double* value) {
  float f;
  memcpy(&f, &bits, 4);
  if (isnan(f)) return 3;
  if (isinf(f)) return f > 0 ? 1 : 2;
  *value = (double)f;
  return 0;
}

/* Binary16: 1 sign, 5 exponent (bias 15), 10 mantissa bits, subnormals. */
static int decode_f16(uint32_t h, double* value) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1F;
  int m = h & 0x3FF;
  if (e == 31) {
    if (m != 0) return 3;
    return sign ? 2 : 1;
  }
  double mag = (e == 0) ? ldexp((double)m, -24) : ldexp((double)(1024 + m), e - 25);
  *value = sign ? -mag : mag;
  return 0;
}

/* OCP 8-bit E4M3 ("fn" variant): bias 7, no infinities, S.1111.111 is NaN,  */
/* largest finite 1.75*2^8 = 448, subnormals m*2^-9.                         */
static int decode_fp8(uint32_t b, double* value) {
  int sign = (b >> 7) & 1;
  int e = (b >> 3) & 0xF;
  int m = b & 7;
  if (e == 15 && m == 7) return 3;
  double mag = (e == 0) ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
  *value = sign ? -mag : mag;
  return 0;
}

int ref_decode(int32_t dtype, uint64_t raw, double* value) {
  switch (dtype) {
    case REF_F32: return decode_f32((uint32_t)raw, value);
    case REF_BF16: return decode_f32((uint32_t)raw << 16, value);
    case REF_F16: return decode_f16((uint32_t)raw, value);
    case REF_FP8E4M3: return decode_fp8((uint32_t)raw, value);
    default: return -1;
  }
}

/*
 * Round a finite real x (here always an exact binary32 value held in a
 * double) to nearest-even on a binary format with `mbits` stored mantissa
 * bits, minimum normal exponent `emin`, exponent bias `bias`; returns the
 * unsigned magnitude code, or -1 if the rounded magnitude exceeds `maxfin`.
 * Written as the textbook definition: find the quantum of x's binade (or of
 * the subnormal range), scale x by it (exact: both are powers of two apart),
 * split into integer and fraction, and round the fraction half-to-even.
 */
static int64_t round_to_format(double ax, int mbits, int emin, int bias, double maxfin) {
  if (ax == 0.0) return 0;
  int e2;
  (void)frexp(ax, &e2);   /* ax = f * 2^e2, f in [0.5, 1) */
  int e = e2 - 1;         /* ax in [2^e, 2^(e+1)) */
  if (e < emin) e = emin;
  double quantum = ldexp(1.0, e - mbits);
  double n = ax / quantum;          /* exact */
  double n_int = floor(n);
  double frac = n - n_int;          /* exact */
  if (frac > 0.5 || (frac == 0.5 && fmod(n_int, 2.0) == 1.0)) n_int += 1.0;
  double rounded = n_int * quantum;
  if (rounded > maxfin) return -1;
  int64_t ni = (int64_t)n_int;
  int64_t one = (int64_t)1 << mbits;
  if (ni >= 2 * one) {              /* carried into the next binade */
    ni /= 2;
    e += 1;
  }
  if (ni < one) return ni;          /* subnormal (only possible at e == emin) */
  return ((int64_t)(e + bias) << mbits) | (ni - one);
}

uint64_t ref_encode_f32(int32_t dtype, float x, int saturate) {
  uint32_t fbits;
  memcpy(&fbits, &x, 4);
  if (dtype == REF_F32) return fbits;
  int neg = (fbits >> 31) & 1;
  double ax = fabs((double)x);
  if (dtype == REF_BF16) {
    if (isnan(x)) return (uint64_t)(0x7FC0u | (neg << 15));
    if (isinf(x)) return (uint64_t)(0x7F80u | (neg << 15));
    int64_t code = round_to_format(ax, 7, -126, 127, ldexp(255.0, 120));
    if (code < 0) code = 0x7F80;
    return (uint64_t)(code | (neg << 15));
  }
  if (dtype == REF_F16) {
    if (isnan(x)) return (uint64_t)(0x7E00u | (neg << 15));
    if (isinf(x)) return (uint64_t)(0x7C00u | (neg << 15));
    int64_t code = round_to_format(ax, 10, -14, 15, 65504.0);
    if (code < 0) code = 0x7C00;
    return (uint64_t)(code | (neg << 15));
  }
  if (dtype == REF_FP8E4M3) {
    if (isnan(x)) return (uint64_t)(0x7Fu | (neg << 7));
    if (saturate && ax > 448.0) ax = 448.0;
    if (isinf(ax)) return (uint64_t)(0x7Fu | (neg << 7));
    int64_t code = round_to_format(ax, 3, -6, 7, 448.0);
    if (code < 0) code = 0x7F;      /* no infinity in this format: overflow is NaN */
    return (uint64_t)(code | (neg << 7));
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* The fill's normal transform: Box-Muller from two 32-bit uniforms, with    */
/* its own fixed-sequence ln and sin/cos so that the result is one defined   */
/* fp64 number (only + - * / and sqrt, each correctly rounded, appear).      */
/* ------------------------------------------------------------------------ */
static const double LN2 = 0x1.62e42fefa39efp-1;     /* fl(ln 2) */
static const double SQRT2 = 0x1.6a09e667f3bcdp+0;   /* fl(sqrt 2) */
static const double PIO2 = 0x1.921fb54442d18p+0;    /* fl(pi / 2) */

/* ln u for u = (x + 1/2) * 2^-32 = N * 2^-33 with N = 2x + 1 odd.
 * N = m * 2^e with m in (sqrt(2)/2, sqrt(2)], ln m = 2 atanh(s) with
 * s = (m - 1)/(m + 1) = f/(2 + f), and atanh(s) = s + s^3/3 + s^5/5 + ...
 * truncated after s^23 (|s| <= 0.1716, so the next term is below 1e-19). */
double ref_log_u(uint32_t x) {
  uint64_t N = 2 * (uint64_t)x + 1;
  int e = 0;
  while ((N >> (e + 1)) != 0) ++e;           /* e = floor(log2 N) */
  double m = ldexp((double)N, -e);           /* exact, in [1, 2) */
  if (m > SQRT2) {
    m = m * 0.5;
    e = e + 1;
  }
  double f = m - 1.0;                        /* exact (Sterbenz) */
  double s = f / (2.0 + f);
  double z = s * s;
  double p = 1.0 / 23.0;
  for (int k = 10; k >= 1; --k) p = 1.0 / (double)(2 * k + 1) + z * p;
  double r = z * p;
  double lnm = 2.0 * (s + s * r);
  return (double)(e - 33) * LN2 + lnm;
}

/* cos and sin of 2*pi*x*2^-32 (x in turns * 2^32).  The quadrant is x's top
 * two bits; the rest is folded into [0, pi/4] exactly in integers, and sin /
 * cos of phi in [0, pi/4] are their Taylor series up to phi^15 / phi^16. */
void ref_sincos_turns(uint32_t x, double* c_out, double* s_out) {
  uint32_t q = x >> 30;
  uint32_t w = x & 0x3FFFFFFFu;
  int swap = 0;
  if (w > (1u << 29)) {
    w = (1u << 30) - w;
    swap = 1;
  }
  double t = ldexp((double)w, -30);          /* exact */
  double phi = t * PIO2;
  double x2 = phi * phi;
  /* sin: phi + phi*x2*(S1 + x2*(S2 + ... + x2*S7)), S_k = (-1)^k/(2k+1)! */
  double fact_s[8];
  double fa = 1.0;
  for (int n = 1; n <= 15; ++n) {
    fa *= (double)n;
    if (n % 2 == 1) fact_s[(n - 1) / 2] = fa;   /* fact_s[k] = (2k+1)! */
  }
  double ps = ((7 % 2) ? -1.0 : 1.0) / fact_s[7];
  for (int k = 6; k >= 1; --k) ps = ((k % 2) ? -1.0 : 1.0) / fact_s[k] + x2 * ps;
  double sn = phi + (phi * x2) * ps;
  /* cos: 1 + x2*(C1 + x2*(C2 + ... + x2*C8)), C_k = (-1)^k/(2k)! */
  double fact_c[9];
  fa = 1.0;
  for (int n = 1; n <= 16; ++n) {
    fa *= (double)n;
    if (n % 2 == 0) fact_c[n / 2] = fa;         /* fact_c[k] = (2k)! */
  }
  double pc = ((8 % 2) ? -1.0 : 1.0) / fact_c[8];
  for (int k = 7; k >= 1; --k) pc = ((k % 2) ? -1.0 : 1.0) / fact_c[k] + x2 * pc;
  double cs = 1.0 + x2 * pc;
  if (swap) {
    double tmp = sn;
    sn = cs;
    cs = tmp;
  }
  double c, s;
  switch (q) {
    case 0: c = cs; s = sn; break;
    case 1: c = -sn; s = cs; break;
    case 2: c = -cs; s = -sn; break;
    default: c = sn; s = -cs; break;
  }
  *c_out = c;
  *s_out = s;
}

double ref_normal(uint32_t xa, uint32_t xb, int which) {
  double ell = ref_log_u(xa);
  double rho = sqrt(-2.0 * ell);
  double c, s;
  ref_sincos_turns(xb, &c, &s);
  return which ? rho * s : rho * c;
}

/* ------------------------------------------------------------------------ */
/* Fill: base value, Bernoulli rules, point injections.                      */
/* ------------------------------------------------------------------------ */
static uint64_t esize_mask(int es) {
  return es == 8 ? ~(uint64_t)0 : (((uint64_t)1 << (8 * es)) - 1);
}

/* Boundary patterns per element type (16 each): signed zeros, the smallest
 * and largest subnormals, the smallest normal, +-1 and the neighbours of 1,
 * +-largest finite, +-Inf and NaNs (fp8 e4m3 has no Inf: NaN instead);
 * for integers the extremes and alternating bit patterns. */
static uint64_t boundary_pattern(int32_t dtype, uint32_t k) {
  static const uint32_t f32[16] = {0x00000000u, 0x80000000u, 0x00000001u, 0x80000001u,
                                   0x007FFFFFu, 0x00800000u, 0x3F800000u, 0xBF800000u,
                                   0x3F7FFFFFu, 0x3F800001u, 0x7F7FFFFFu, 0xFF7FFFFFu,
                                   0x7F800000u, 0xFF800000u, 0x7FC00000u, 0x7F800001u};
  static const uint16_t bf16[16] = {0x0000, 0x8000, 0x0001, 0x8001, 0x007F, 0x0080, 0x3F80, 0xBF80,
                                    0x3F7F, 0x3F81, 0x7F7F, 0xFF7F, 0x7F80, 0xFF80, 0x7FC0, 0x7F81};
  static const uint16_t f16[16] = {0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x0400, 0x3C00, 0xBC00,
                                   0x3BFF, 0x3C01, 0x7BFF, 0xFBFF, 0x7C00, 0xFC00, 0x7E00, 0x7C01};
  static const uint8_t fp8[16] = {0x00, 0x80, 0x01, 0x81, 0x07, 0x08, 0x38, 0xB8,
                                  0x37, 0x39, 0x7E, 0xFE, 0x7F, 0xFF, 0x7F, 0x7D};
  static const uint32_t i32[16] = {0x00000000u, 0x00000001u, 0xFFFFFFFFu, 0x80000000u,
                                   0x7FFFFFFFu, 0x80000001u, 0x7FFFFFFEu, 0x55555555u,
                                   0xAAAAAAAAu, 0x000000FFu, 0x0000FFFFu, 0x00010000u,
                                   0xFFFF0000u, 0x00000080u, 0x7F7F7F7Fu, 0x00000002u};
  static const uint64_t i64[16] = {0x0ull, 0x1ull, 0xFFFFFFFFFFFFFFFFull, 0x8000000000000000ull,
                                   0x7FFFFFFFFFFFFFFFull, 0x8000000000000001ull, 0x7FFFFFFFFFFFFFFEull,
                                   0x5555555555555555ull, 0xAAAAAAAAAAAAAAAAull, 0xFFull, 0xFFFFFFFFull,
                                   0x100000000ull, 0xFFFFFFFF00000000ull, 0x80000000ull, 0x7FFFFFFFull,
                                   0x2ull};
  static const uint8_t u8[16] = {0x00, 0x01, 0xFF, 0x80, 0x7F, 0x81, 0x7E, 0x55,
                                 0xAA, 0x0F, 0xF0, 0x10, 0xEF, 0x40, 0xBF, 0x02};
  k &= 15u;
  switch (dtype) {
    case REF_F32: return f32[k];
    case REF_BF16: return bf16[k];
    case REF_F16: return f16[k];
    case REF_FP8E4M3: return fp8[k];
    case REF_I32: return i32[k];
    case REF_I64: return i64[k];
    default: return u8[k];
  }
}

/* BOUNDARY threshold: element is a boundary pattern iff its draw is below
 * floor(rate * 2^32 + 1/2), the rate clamped to [0, 1]. */
static uint64_t boundary_threshold(double rate) {
  if (!(rate > 0.0)) return 0;
  if (rate >= 1.0) return (uint64_t)1 << 32;
  return (uint64_t)floor(rate * 4294967296.0 + 0.5);
}

static uint64_t base_element(const ref_alloc* A, uint64_t seed, int64_t i) {
  int es = ref_esize(A->dtype);
  uint32_t X[4];
  if (A->dist == REF_NORMAL) {
    stream_block(seed, A->alloc_id, PURPOSE_VALUE, 0, 0, (uint64_t)i / 4, X);
    int pair = (int)((i / 2) % 2);
    double z = ref_normal(X[2 * pair], X[2 * pair + 1], (int)(i % 2));
    double scaled = A->p1 * z;
    double v = A->p0 + scaled;
    return ref_encode_f32(A->dtype, (float)v, A->saturate);
  }
  if (A->dist == REF_UNIFORM_INT) {
    stream_block(seed, A->alloc_id, PURPOSE_VALUE, 0, 0, (uint64_t)i / 4, X);
    uint64_t span = (uint64_t)(A->i1 - A->i0);
    int64_t v = A->i0 + (int64_t)(((uint64_t)X[i % 4] * span) >> 32);
    if (is_float(A->dtype)) return ref_encode_f32(A->dtype, (float)(double)v, A->saturate);
    return (uint64_t)v & esize_mask(es);
  }
  if (A->dist == REF_BITS) {
    uint64_t bits = 0;
    for (int k = 0; k < es; ++k) {
      uint64_t q = (uint64_t)i * (uint64_t)es + (uint64_t)k;
      bits |= (uint64_t)stream_byte(seed, A->alloc_id, PURPOSE_VALUE, 0, 0, q) << (8 * k);
    }
    return bits;
  }
  if (A->dist == REF_BOUNDARY) {
    /* one VALUE block per element: x selects, y picks the pattern, (z, w)
     * give a Box-Muller cosine value of standard deviation p1 otherwise */
    stream_block(seed, A->alloc_id, PURPOSE_VALUE, 0, 0, (uint64_t)i, X);
    if ((uint64_t)X[0] < boundary_threshold(A->p0)) return boundary_pattern(A->dtype, X[1]);
    if (is_float(A->dtype)) {
      double z = ref_normal(X[2], X[3], 0);
      double v = A->p1 * z;
      return ref_encode_f32(A->dtype, (float)v, A->saturate);
    }
    return ((uint64_t)X[2] | ((uint64_t)X[3] << 32)) & esize_mask(es);
  }
  /* REF_CONST */
  if (is_float(A->dtype)) return ref_encode_f32(A->dtype, (float)A->p0, A->saturate);
  return (uint64_t)A->i0 & esize_mask(es);
}

static uint64_t max_finite_mag(int32_t dtype) {
  switch (dtype) {
    case REF_F32: return 0x7F7FFFFFu;
    case REF_BF16: return 0x7F7Fu;
    case REF_F16: return 0x7BFFu;
    default: return 0x7Eu;   /* fp8 e4m3 */
  }
}

static uint64_t apply_injection(const ref_alloc* A, const ref_inj* J, uint64_t base, uint64_t seed,
                                uint32_t vsel, int64_t i) {
  int es = ref_esize(A->dtype);
  uint32_t R[4];
  stream_block(seed, A->alloc_id, PURPOSE_INJECT, 0, vsel, (uint64_t)i, R);
  uint32_t kind = J->kind & 0xFFu;
  uint64_t sign_bit = (uint64_t)1 << (8 * es - 1);
  if (kind == REF_FLIP_BIT) {
    uint32_t bit = (J->arg == 0xFFFFFFFFu) ? (R[0] & (uint32_t)(8 * es - 1)) : J->arg;
    return base ^ ((uint64_t)1 << bit);
  }
  if (kind == REF_STEP_WITHIN) {
    uint64_t sign = base & sign_bit;
    uint64_t mag = base & ~sign_bit & esize_mask(es);
    uint64_t maxmag = max_finite_mag(A->dtype);
    if (mag > maxmag) return base;                 /* NaN or Inf: left alone */
    int grow = (R[0] & 1) == 0;
    if ((grow && mag < maxmag) || mag == 0) mag = mag + 1;
    else mag = mag - 1;
    return sign | mag;
  }
  if (kind == REF_SET_BEYOND) {
    double B;
    if (ref_decode(A->dtype, base, &B) != 0) return base;
    double t = J->atol + J->rtol * fabs(B);
    double four_t = 4.0 * t;
    double v = (base & sign_bit) ? B + four_t : B - four_t;
    return ref_encode_f32(A->dtype, (float)v, A->saturate);
  }
  if (kind == REF_SET_NAN) {
    switch (A->dtype) {
      case REF_F32: return 0x7FC00000u;
      case REF_BF16: return 0x7FC0u;
      case REF_F16: return 0x7E00u;
      default: return 0x7Fu;
    }
  }
  if (kind == REF_SET_INF) {
    uint64_t s = (J->arg & 1) ? sign_bit : 0;
    switch (A->dtype) {
      case REF_F32: return s | 0x7F800000u;
      case REF_BF16: return s | 0x7F80u;
      default: return s | 0x7C00u;   /* F16; fp8 e4m3 has no infinity (rejected) */
    }
  }
  return base;
}

static int applies(const ref_inj* J, uint32_t variant) {
  return variant != 0 || J->sides == REF_SIDE_BOTH;
}

uint64_t ref_element(const ref_alloc* allocs, int32_t k, const ref_inj* inj, int64_t n_inj,
                     uint64_t seed, uint32_t variant, int64_t i) {
  const ref_alloc* A = &allocs[k];
  uint64_t base = base_element(A, seed, i);
  uint64_t value = base;
  /* Bernoulli rules, in list order; the last one that selects i wins. */
  uint32_t ordinal = 0;
  for (int64_t t = 0; t < n_inj; ++t) {
    const ref_inj* J = &inj[t];
    if (J->alloc != (uint32_t)k || !(J->kind & REF_RATE)) continue;
    uint32_t this_ordinal = ordinal++;
    if (!applies(J, variant)) continue;
    uint32_t vsel = (J->sides == REF_SIDE_BOTH) ? 0 : variant;
    uint32_t S[4];
    stream_block(seed, A->alloc_id, PURPOSE_SELECT, this_ordinal, vsel, (uint64_t)i / 4, S);
    if ((uint64_t)S[i % 4] < (uint64_t)J->index) value = apply_injection(A, J, base, seed, vsel, i);
  }
  /* Point entries, in list order; the last one naming i wins. */
  for (int64_t t = 0; t < n_inj; ++t) {
    const ref_inj* J = &inj[t];
    if (J->alloc != (uint32_t)k || (J->kind & REF_RATE)) continue;
    uint32_t kind = J->kind & 0xFFu;
    if (kind == REF_GUARD_WRITE_LO || kind == REF_GUARD_WRITE_HI || kind == REF_PAD_WRITE) continue;
    if (J->index != i || !applies(J, variant)) continue;
    uint32_t vsel = (J->sides == REF_SIDE_BOTH) ? 0 : variant;
    value = apply_injection(A, J, base, seed, vsel, i);
  }
  return value;
}

static int64_t data_bytes(const ref_alloc* A) {
  if (A->rows <= 0 || A->cols <= 0) return 0;
  return ((A->rows - 1) * A->stride + A->cols) * ref_esize(A->dtype);
}

static int guard_written(const ref_inj* inj, int64_t n_inj, int32_t k, uint32_t variant, int side,
                         int64_t p) {
  int hit = 0;
  for (int64_t t = 0; t < n_inj; ++t) {
    const ref_inj* J = &inj[t];
    if (J->alloc != (uint32_t)k || (J->kind & REF_RATE)) continue;
    uint32_t kind = J->kind & 0xFFu;
    int s = (kind == REF_GUARD_WRITE_LO) ? 0 : (kind == REF_GUARD_WRITE_HI) ? 1 : -1;
    if (s != side || !applies(J, variant)) continue;
    if (p >= J->index && p < J->index + (int64_t)J->arg) hit = 1;
  }
  return hit;
}

/* Is data byte q of allocation k (a pad byte) inverted by a PAD_WRITE entry? */
static int pad_written(const ref_inj* inj, int64_t n_inj, int32_t k, uint32_t variant, int64_t q) {
  int hit = 0;
  for (int64_t t = 0; t < n_inj; ++t) {
    const ref_inj* J = &inj[t];
    if (J->alloc != (uint32_t)k || (J->kind & REF_RATE) || (J->kind & 0xFFu) != REF_PAD_WRITE) continue;
    if (!applies(J, variant)) continue;
    if (q >= J->index && q < J->index + (int64_t)J->arg) hit = 1;
  }
  return hit;
}

int ref_fill_range(const ref_alloc* allocs, int32_t k, const ref_inj* all_inj, int64_t n_all,
                   uint64_t seed, uint32_t variant, int64_t off, int64_t nbytes, uint8_t* out) {
  const ref_alloc* A = &allocs[k];
  int es = ref_esize(A->dtype);
  if (es == 0 || off < 0 || nbytes < 0) return -1;
  if (A->rows > 0 && A->cols > 0 && A->stride < A->cols) return -1;
  int64_t D = data_bytes(A);
  int64_t total = A->guard_lo + D + A->guard_hi;
  if (off + nbytes > total) return -1;
  /* only allocation k's entries, in list order (the others are skipped for
   * every byte anyway; a workload with an entry per allocation would
   * otherwise scan them all for every element) */
  ref_inj* inj = (ref_inj*)malloc(sizeof(ref_inj) * (size_t)(n_all > 0 ? n_all : 1));
  if (!inj) return -1;
  int64_t n_inj = 0;
  for (int64_t t = 0; t < n_all; ++t)
    if (all_inj[t].alloc == (uint32_t)k) inj[n_inj++] = all_inj[t];
  int64_t cached_e = -1;
  uint64_t cached_bits = 0;
  for (int64_t n = 0; n < nbytes; ++n) {
    int64_t p = off + n;
    uint8_t byte;
    if (p < A->guard_lo) {
      byte = ref_canary_byte(seed, A->alloc_id, 0, p);
      if (guard_written(inj, n_inj, k, variant, 0, p)) byte = (uint8_t)~byte;
    } else if (p < A->guard_lo + D) {
      int64_t q = p - A->guard_lo;
      int64_t e = q / es;
      int64_t r = e / A->stride;
      int64_t c = e % A->stride;
      if (c < A->cols) {
        if (e != cached_e) {
          cached_bits = ref_element(allocs, k, inj, n_inj, seed, variant, r * A->cols + c);
          cached_e = e;
        }
        byte = (uint8_t)(cached_bits >> (8 * (q % es)));
      } else {
        byte = stream_byte(seed, A->alloc_id, PURPOSE_PAD, 0, 0, (uint64_t)q);
        if (pad_written(inj, n_inj, k, variant, q)) byte = (uint8_t)~byte;
      }
    } else {
      int64_t ph = p - A->guard_lo - D;
      byte = ref_canary_byte(seed, A->alloc_id, 1, ph);
      if (guard_written(inj, n_inj, k, variant, 1, ph)) byte = (uint8_t)~byte;
    }
    out[n] = byte;
  }
  free(inj);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Comparison of one segment (Eq. 1's Delta and iota's bit-exactness).       */
/* ------------------------------------------------------------------------ */
static uint64_t load_raw(const uint8_t* p, int es) {
  uint64_t v = 0;
  for (int k = 0; k < es; ++k) v |= (uint64_t)p[k] << (8 * k);
  return v;
}

static void result_reset(ref_seg_result* res) {
  res->mismatches = 0;
  res->first_mismatch = -1;
  res->bitwise_mismatches = 0;
  res->first_bitwise = -1;
  res->nonfinite_mismatches = 0;
  res->max_abs = 0.0;
  res->max_rel = 0.0;
}

/* One element pair at logical index i: the tolerance rule of the header, and
 * the bitwise count.  Pairs are visited in increasing i, so the first index
 * seen is the lowest. */
static void compare_pair(int32_t dtype, int32_t mode, int32_t nan_policy, double atol, double rtol,
                         uint64_t ra, uint64_t rb, int64_t i, ref_seg_result* res) {
  int bitwise = ra != rb;
  if (bitwise) {
    res->bitwise_mismatches += 1;
    if (res->first_bitwise < 0) res->first_bitwise = i;
  }
  int mismatch;
  int nonfinite = 0;
  if (mode == REF_BITWISE) {
    mismatch = bitwise;
  } else {
    double A = 0.0, B = 0.0;
    int ca = ref_decode(dtype, ra, &A);
    int cb = ref_decode(dtype, rb, &B);
    nonfinite = (ca != 0) || (cb != 0);
    if (!bitwise) {
      /* identical bits: a match, except a NaN under the strict policy */
      mismatch = (cb == 3 && nan_policy == REF_NAN_STRICT);
    } else if (ca == 3 || cb == 3) {
      mismatch = !(ca == 3 && cb == 3 && nan_policy == REF_NAN_EQUAL);
    } else if (nonfinite) {
      mismatch = 1;   /* an infinity against anything with other bits */
    } else {
      double d = fabs(A - B);
      double scaled = rtol * fabs(B);
      double t = atol + scaled;
      mismatch = !(d <= t);
      double rel;
      if (B != 0.0) rel = d / fabs(B);
      else rel = (d == 0.0) ? 0.0 : INFINITY;
      if (d > res->max_abs) res->max_abs = d;
      if (rel > res->max_rel) res->max_rel = rel;
    }
  }
  if (mismatch) {
    res->mismatches += 1;
    if (res->first_mismatch < 0) res->first_mismatch = i;
    if (nonfinite) res->nonfinite_mismatches += 1;
  }
}

int ref_diff_segment(const ref_seg* seg, const uint8_t* a, const uint8_t* b, ref_seg_result* res) {
  int es = ref_esize(seg->dtype);
  if (es == 0) return -1;
  if (seg->mode == REF_TOLERANCE && !is_float(seg->dtype)) return -1;
  result_reset(res);
  for (int64_t r = 0; r < seg->rows; ++r) {
    for (int64_t c = 0; c < seg->cols; ++c) {
      int64_t i = r * seg->cols + c;
      uint64_t ra = load_raw(a + (r * seg->stride_a + c) * es, es);
      uint64_t rb = load_raw(b + (r * seg->stride_b + c) * es, es);
      compare_pair(seg->dtype, seg->mode, seg->nan_policy, seg->atol, seg->rtol, ra, rb, i, res);
    }
  }
  return 0;
}

int ref_diff_segment_nd(const ref_seg_nd* seg, const uint8_t* a, const uint8_t* b, ref_seg_result* res) {
  int es = ref_esize(seg->dtype);
  if (es == 0 || seg->ndim < 0 || seg->ndim > REF_MAX_DIMS) return -1;
  if (seg->mode == REF_TOLERANCE && !is_float(seg->dtype)) return -1;
  result_reset(res);
  int64_t total = 1;
  for (int d = 0; d < seg->ndim; ++d) {
    if (seg->shape[d] < 0 || seg->stride_a[d] < 0 || seg->stride_b[d] < 0) return -1;
    total *= seg->shape[d];
  }
  for (int64_t i = 0; i < total; ++i) {
    /* row-major multi-index of i: the last dimension varies fastest */
    int64_t rest = i, off_a = 0, off_b = 0;
    for (int d = seg->ndim - 1; d >= 0; --d) {
      int64_t idx = rest % seg->shape[d];
      rest /= seg->shape[d];
      off_a += idx * seg->stride_a[d];
      off_b += idx * seg->stride_b[d];
    }
    uint64_t ra = load_raw(a + off_a * es, es);
    uint64_t rb = load_raw(b + off_b * es, es);
    compare_pair(seg->dtype, seg->mode, seg->nan_policy, seg->atol, seg->rtol, ra, rb,
                 seg->index_base + i, res);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Cosine term of Eq. 1: c = cos(K'(x), O(x)) = sum a*b / (|a| * |b|) over  */
/* the element pairs of a buffer with both values finite.  The definition   */
/* fixes no order of summation, so the oracle computes each of the three    */
/* sums exactly and rounds it once (to nearest, ties to even).  Every       */
/* product is exact in fp64: the float element types have at most 24        */
/* significant bits and exponents in [-149, 127], so a product has at most  */
/* 48 significant bits and lies in [2^-298, 2^256].                         */
/* ------------------------------------------------------------------------ */

/* The exact sum is a signed fixed-point integer with one bit for every power
 * of two a binary64 value can carry: bit 0 weighs 2^-1074 (the smallest
 * subnormal), the largest finite value ends below bit 2098, and 64 more bits
 * leave room for 2^64 terms.  It is held as base-2^32 digits in int64, so an
 * addition changes at most three digits by less than 2^32 each and no carry
 * has to move until 2^30 additions have been made. */
void ref_xacc_init(ref_xacc* x) { memset(x, 0, sizeof(*x)); }

/* floor(v / 2^32) for any int64 v, without relying on how C shifts a
 * negative value */
static int64_t floor_div_2p32(int64_t v) {
  const int64_t q = v / 4294967296LL;           /* truncates toward zero */
  return (v < 0 && q * 4294967296LL != v) ? q - 1 : q;
}

/* Moves every digit's excess into the next one: digits 0..N-2 end in
 * [0, 2^32) and the top digit carries the sign. */
static void xacc_carry(ref_xacc* x) {
  for (int i = 0; i + 1 < REF_XACC_DIGITS; ++i) {
    const int64_t c = floor_div_2p32(x->d[i]);
    x->d[i] -= c * 4294967296LL;
    x->d[i + 1] += c;
  }
  x->adds = 0;
}

/* Adds a finite binary64 value exactly.  From its IEEE 754 encoding: a normal
 * value with biased exponent E >= 1 and fraction F is (2^52 + F) * 2^(E-1075),
 * i.e. the integer 2^52 + F placed at bit E - 1 of the accumulator; a
 * subnormal one (E = 0) is F * 2^-1074, i.e. F at bit 0. */
void ref_xacc_add(ref_xacc* x, double v) {
  uint64_t bits;
  memcpy(&bits, &v, sizeof(bits));
  const int neg = (int)(bits >> 63);
  const int E = (int)((bits >> 52) & 0x7FF);
  const uint64_t F = bits & 0xFFFFFFFFFFFFFull;
  if (E == 0x7FF) return;                       /* not finite: callers never pass one */
  const uint64_t m = E == 0 ? F : (F | (1ull << 52));
  if (m == 0) return;
  const int p = E == 0 ? 0 : E - 1;             /* bit position of m's bit 0 */
  const unsigned __int128 w = (unsigned __int128)m << (p % 32);   /* below 2^85 */
  const int k = p / 32;
  const int64_t d0 = (int64_t)(uint32_t)w;
  const int64_t d1 = (int64_t)(uint32_t)(w >> 32);
  const int64_t d2 = (int64_t)(uint32_t)(w >> 64);
  if (neg) {
    x->d[k] -= d0;
    x->d[k + 1] -= d1;
    x->d[k + 2] -= d2;
  } else {
    x->d[k] += d0;
    x->d[k + 1] += d1;
    x->d[k + 2] += d2;
  }
  if (++x->adds >= (1LL << 30)) xacc_carry(x);
}

/* Bit i of a non-negative normalised accumulator. */
static int xacc_bit(const ref_xacc* x, int i) { return (int)((x->d[i / 32] >> (i % 32)) & 1); }

/* The binary64 value nearest to the exact sum, ties to even; an exact zero
 * gives +0.0. */
double ref_xacc_round(const ref_xacc* in) {
  ref_xacc x = *in;
  xacc_carry(&x);
  const int neg = x.d[REF_XACC_DIGITS - 1] < 0;
  if (neg) {                                    /* work with the magnitude */
    for (int i = 0; i < REF_XACC_DIGITS; ++i) x.d[i] = -x.d[i];
    xacc_carry(&x);
  }
  int top = -1;                                 /* highest set bit */
  for (int i = REF_XACC_DIGITS * 32 - 1; i >= 0 && top < 0; --i)
    if (xacc_bit(&x, i)) top = i;
  if (top < 0) return 0.0;
  double r;
  if (top < 53) {                               /* at most 53 bits above 2^-1074: exact */
    uint64_t m = 0;
    for (int i = top; i >= 0; --i) m = (m << 1) | (uint64_t)xacc_bit(&x, i);
    r = ldexp((double)m, -1074);
  } else {
    uint64_t m = 0;                             /* the 53 leading bits */
    for (int i = top; i > top - 53; --i) m = (m << 1) | (uint64_t)xacc_bit(&x, i);
    const int round = xacc_bit(&x, top - 53);
    int sticky = 0;
    for (int i = top - 54; i >= 0 && !sticky; --i) sticky = xacc_bit(&x, i);
    int e = top - 52 - 1074;                    /* weight of m's last bit */
    if (round && (sticky || (m & 1))) {
      m += 1;
      if (m == (1ull << 53)) {
        m >>= 1;
        e += 1;
      }
    }
    r = ldexp((double)m, e);                    /* +Inf beyond the largest finite value */
  }
  return neg ? -r : r;
}

double ref_exact_sum(const double* v, int64_t n) {
  ref_xacc x;
  ref_xacc_init(&x);
  for (int64_t k = 0; k < n; ++k) ref_xacc_add(&x, v[k]);
  return ref_xacc_round(&x);
}

/* Exact running sums of one cosine term. */
typedef struct {
  ref_xacc ab, aa, bb, abs_ab;
  uint64_t pairs;
} cos_sums;

static void cos_sums_init(cos_sums* s) {
  ref_xacc_init(&s->ab);
  ref_xacc_init(&s->aa);
  ref_xacc_init(&s->bb);
  ref_xacc_init(&s->abs_ab);
  s->pairs = 0;
}

/* One element pair: excluded when either value is NaN or infinite. */
static void cos_pair(int32_t dtype, uint64_t ra, uint64_t rb, cos_sums* s) {
  double A, B;
  if (ref_decode(dtype, ra, &A) != 0 || ref_decode(dtype, rb, &B) != 0) return;
  ref_xacc_add(&s->ab, A * B);
  ref_xacc_add(&s->aa, A * A);
  ref_xacc_add(&s->bb, B * B);
  ref_xacc_add(&s->abs_ab, fabs(A * B));
  s->pairs += 1;
}

/* c = S_ab / (sqrt(S_aa) * sqrt(S_bb)) from the rounded sums, each operation
 * rounded; 1 when both vectors are zero, 0 when exactly one is. */
static void cos_finish(const cos_sums* s, ref_cos_result* res) {
  res->sum_ab = ref_xacc_round(&s->ab);
  res->sum_aa = ref_xacc_round(&s->aa);
  res->sum_bb = ref_xacc_round(&s->bb);
  res->sum_abs_ab = ref_xacc_round(&s->abs_ab);
  res->pairs = s->pairs;
  if (res->sum_aa == 0.0 && res->sum_bb == 0.0) {
    res->cosine = 1.0;
  } else if (res->sum_aa == 0.0 || res->sum_bb == 0.0) {
    res->cosine = 0.0;
  } else {
    const double na = sqrt(res->sum_aa);
    const double nb = sqrt(res->sum_bb);
    const double den = na * nb;
    res->cosine = res->sum_ab / den;
  }
}

static void cos_undefined(ref_cos_result* res) {
  res->sum_ab = res->sum_aa = res->sum_bb = res->sum_abs_ab = 0.0;
  res->cosine = NAN;                            /* not defined for integer buffers */
  res->pairs = 0;
}

int ref_cosine_segment(const ref_seg* seg, const uint8_t* a, const uint8_t* b, ref_cos_result* res) {
  const int es = ref_esize(seg->dtype);
  if (es == 0) return -1;
  cos_undefined(res);
  if (!is_float(seg->dtype)) return 0;
  cos_sums s;
  cos_sums_init(&s);
  for (int64_t r = 0; r < seg->rows && seg->cols > 0; ++r)
    for (int64_t c = 0; c < seg->cols; ++c)
      cos_pair(seg->dtype, load_raw(a + (r * seg->stride_a + c) * es, es),
               load_raw(b + (r * seg->stride_b + c) * es, es), &s);
  cos_finish(&s, res);
  return 0;
}

int ref_cosine_nd(const ref_seg_nd* segs, int32_t n, const uint8_t* const* a, const uint8_t* const* b,
                  ref_cos_result* res) {
  cos_undefined(res);
  if (n <= 0) {
    res->cosine = 1.0;                          /* no elements: both vectors are zero */
    res->sum_ab = res->sum_aa = res->sum_bb = res->sum_abs_ab = 0.0;
    return 0;
  }
  const int32_t dtype = segs[0].dtype;
  const int es = ref_esize(dtype);
  if (es == 0) return -1;
  for (int32_t k = 0; k < n; ++k)
    if (segs[k].dtype != dtype || segs[k].ndim < 0 || segs[k].ndim > REF_MAX_DIMS) return -1;
  if (!is_float(dtype)) return 0;
  cos_sums s;
  cos_sums_init(&s);
  for (int32_t k = 0; k < n; ++k) {
    const ref_seg_nd* seg = &segs[k];
    int64_t count = 1;
    for (int d = 0; d < seg->ndim; ++d) count *= seg->shape[d];
    for (int64_t i = 0; i < count; ++i) {       /* logical order; any order gives the same sums */
      int64_t rest = i, off_a = 0, off_b = 0;
      for (int d = seg->ndim - 1; d >= 0; --d) {
        const int64_t idx = rest % seg->shape[d];
        rest /= seg->shape[d];
        off_a += idx * seg->stride_a[d];
        off_b += idx * seg->stride_b[d];
      }
      cos_pair(dtype, load_raw(a[k] + off_a * es, es), load_raw(b[k] + off_b * es, es), &s);
    }
  }
  cos_finish(&s, res);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Tier-2 state restore: plain byte copies.                                  */
/* ------------------------------------------------------------------------ */
void ref_copy_regions(const ref_region* regions, int64_t n) {
  for (int64_t k = 0; k < n; ++k)
    for (int64_t p = 0; p < regions[k].bytes; ++p) regions[k].dst[p] = regions[k].src[p];
}

/* ------------------------------------------------------------------------ */
/* Guard check: every guard byte against the regenerated canary.             */
/* ------------------------------------------------------------------------ */
int ref_guard_check(uint64_t seed, uint32_t alloc_id, const uint8_t* lo, int64_t n_lo,
                    const uint8_t* hi, int64_t n_hi, ref_guard_result* res) {
  res->bad_lo = 0;
  res->bad_hi = 0;
  res->first_bad_lo = -1;
  res->first_bad_hi = -1;
  res->bad_pad = 0;
  res->first_bad_pad = -1;
  for (int64_t p = 0; p < n_lo; ++p) {
    if (lo[p] != ref_canary_byte(seed, alloc_id, 0, p)) {
      res->bad_lo += 1;
      if (res->first_bad_lo < 0) res->first_bad_lo = p;
    }
  }
  for (int64_t p = 0; p < n_hi; ++p) {
    if (hi[p] != ref_canary_byte(seed, alloc_id, 1, p)) {
      res->bad_hi += 1;
      if (res->first_bad_hi < 0) res->first_bad_hi = p;
    }
  }
  return 0;
}

int ref_pad_check(const ref_alloc* A, uint64_t seed, const uint8_t* data, ref_guard_result* res) {
  res->bad_pad = 0;
  res->first_bad_pad = -1;
  if (A->rows < 2 || A->stride <= A->cols) return 0;
  int es = ref_esize(A->dtype);
  if (es == 0) return -1;
  int64_t D = data_bytes(A);
  for (int64_t q = 0; q < D; ++q) {
    int64_t e = q / es;
    if (e % A->stride < A->cols) continue;        /* a data element, not padding */
    if (data[q] != stream_byte(seed, A->alloc_id, PURPOSE_PAD, 0, 0, (uint64_t)q)) {
      res->bad_pad += 1;
      if (res->first_bad_pad < 0) res->first_bad_pad = q;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Bulk loops for the pin tests.                                             */
/* ------------------------------------------------------------------------ */
void ref_decode_n(int32_t dtype, const uint64_t* raw, int64_t n, int32_t* cls, double* value) {
  for (int64_t k = 0; k < n; ++k) {
    double v = 0.0;
    cls[k] = ref_decode(dtype, raw[k], &v);
    value[k] = v;
  }
}

void ref_encode_f32_n(int32_t dtype, const float* x, int64_t n, int saturate, uint64_t* out) {
  for (int64_t k = 0; k < n; ++k) out[k] = ref_encode_f32(dtype, x[k], saturate);
}

void ref_log_u_n(const uint32_t* x, int64_t n, double* out) {
  for (int64_t k = 0; k < n; ++k) out[k] = ref_log_u(x[k]);
}

void ref_sincos_turns_n(const uint32_t* x, int64_t n, double* c, double* s) {
  for (int64_t k = 0; k < n; ++k) ref_sincos_turns(x[k], &c[k], &s[k]);
}

void ref_normal_n(const uint32_t* xa, const uint32_t* xb, int64_t n, int which, double* out) {
  for (int64_t k = 0; k < n; ++k) out[k] = ref_normal(xa[k], xb[k], which);
}

void ref_philox_n(const uint32_t* ctr, const uint32_t* key, int64_t n, uint32_t* out) {
  for (int64_t k = 0; k < n; ++k) ref_philox4x32_10(ctr + 4 * k, key + 2 * k, out + 4 * k);
}

void ref_compare_pair_n(int32_t dtype, int32_t mode, int32_t nan_policy, double atol, double rtol,
                        const uint64_t* ra, const uint64_t* rb, int64_t n, uint8_t* flags,
                        double* max_abs, double* max_rel) {
  for (int64_t k = 0; k < n; ++k) {
    ref_seg_result r;
    result_reset(&r);
    compare_pair(dtype, mode, nan_policy, atol, rtol, ra[k], rb[k], 0, &r);
    flags[k] = (uint8_t)((r.bitwise_mismatches != 0) | ((r.mismatches != 0) << 1) |
                         ((r.nonfinite_mismatches != 0) << 2));
    max_abs[k] = r.max_abs;
    max_rel[k] = r.max_rel;
  }
}
