/*
 * asmevo.h -- C ABI of the MI355X (gfx950) differential-oracle library.
 *
 * The differential oracle decides whether a candidate kernel K' is
 * functionally equivalent to the original code object K0 on an input x
 * (AsmEvo, section 3.2, Eq. 1): its output state K'(x) is compared against the
 * reference state O(x) = run(K0, x) under the same launch.  Floating-point
 * outputs are checked against a tolerance, integer buffers, opaque state and
 * guard regions byte-exactly (section 3.4, Tier 2), and the predicate iota
 * additionally requires intact out-of-bounds guards, which Tier-1 synthesis
 * places around every allocation as canary-initialised regions (section 3.4,
 * Tier 1).  This library provides the data-parallel part of that check:
 *
 *   asmevo_fill_guarded   seeded guarded states (canaries, values, pads,
 *                         injected candidate differences)        (sec. 3.4)
 *   asmevo_diff_segments  element-wise compare of many buffers in one launch,
 *                         per-buffer counts / first index / max abs / max rel
 *                                                          (sec. 3.2, Eq. 1)
 *                         (2-D segments; _nd: N-D shapes and strides)
 *   asmevo_guard_check    canary integrity of every guard region and of
 *                         the row padding                 (sec. 3.2 iota,
 *                                                          sec. 3.4)
 *
 * Conventions for every call:
 *  - All addresses inside descriptors and all result pointers are HIP device
 *    addresses on the current device.  Descriptor arrays (`allocs`, `inj`,
 *    `segs`) are host memory: they are read and copied during the call, so the
 *    caller may free or reuse them on return.
 *  - `workspace` is device memory of at least asmevo_workspace_bytes(...)
 *    bytes, owned by the caller, starting on a 256-byte boundary (as hipMalloc
 *    and torch allocations do; otherwise ASMEVO_E_INVALID); the call stages
 *    its descriptor tables there.
 *    It must not be reused by another call until this call's work on `stream`
 *    has completed.  The library allocates no memory of its own, apart from
 *    the asmevo_va_alloc calls, which exist to allocate.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *    asynchronously; results are defined once the stream has been
 *    synchronised.  The descriptor upload is a host-to-device copy from
 *    pageable memory, which HIP performs synchronously with the host.
 *  - Return value: ASMEVO_OK (0) or a negative status.  Argument errors are
 *    detected before anything is enqueued.  A failing HIP call returns
 *    ASMEVO_E_HIP and asmevo_last_hip_error() gives the hipError_t code.
 *  - Element indices are logical row-major: i = r * cols + c, independent of
 *    row strides; -1 means "none".
 *  - Results are exact (integer counts, minimum indices, maxima of correctly
 *    rounded fp64 values), so they do not depend on launch geometry or
 *    scheduling and repeat bit-for-bit (the paper repeats each check three
 *    times, section 4.1).
 */
#ifndef ASMEVO_H
#define ASMEVO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ASMEVO_ABI_VERSION 2

typedef int32_t asmevo_status;
enum {
  ASMEVO_OK = 0,
  ASMEVO_E_INVALID = -1,      /* malformed descriptor or argument */
  ASMEVO_E_UNSUPPORTED = -2,  /* valid but not supported (e.g. +-Inf in fp8 e4m3) */
  ASMEVO_E_WORKSPACE = -3,    /* workspace missing or smaller than required */
  ASMEVO_E_HIP = -4,          /* a HIP runtime call failed */
  ASMEVO_E_CAPACITY = -5      /* more descriptors than a fixed-size call holds */
};

/* element types */
enum {
  ASMEVO_F32 = 1,        /* IEEE binary32 */
  ASMEVO_BF16 = 2,       /* bfloat16: the top half of a binary32 */
  ASMEVO_F16 = 3,        /* IEEE binary16 */
  ASMEVO_FP8_E4M3 = 4,   /* OCP 8-bit E4M3 (fn): bias 7, no Inf, 0x7F/0xFF NaN, max 448 */
  ASMEVO_I32 = 5,
  ASMEVO_I64 = 6,
  ASMEVO_U8 = 7          /* opaque bytes */
};

/* comparison mode of a segment */
enum {
  ASMEVO_BITWISE = 0,    /* raw bits must be equal (any dtype) */
  ASMEVO_TOLERANCE = 1   /* float dtypes only: |a - b| <= atol + rtol * |b| */
};

/* NaN policy of a TOLERANCE segment */
enum {
  ASMEVO_NAN_EQUAL = 0,  /* NaN matches NaN (sign and payload ignored) */
  ASMEVO_NAN_STRICT = 1  /* a NaN never matches, not even identical bits */
};

/* value distribution of an allocation's data elements */
enum {
  ASMEVO_DIST_NORMAL = 0,       /* N(p0, p1^2): Box-Muller, then fp32 (RNE), then dtype (RNE) */
  ASMEVO_DIST_UNIFORM_INT = 1,  /* integers uniform in [i0, i1), 0 < i1 - i0 <= 2^32 */
  ASMEVO_DIST_BITS = 2,         /* raw generator bytes */
  ASMEVO_DIST_CONST = 3,        /* p0 (float dtypes, via fp32) or i0 (integer dtypes) */
  ASMEVO_DIST_BOUNDARY = 4      /* boundary values at rate p0 (0 <= p0 <= 1), else N(0, p1^2)
                                   (float dtypes) or raw generator bits (integer dtypes); below */
};

/*
 * ASMEVO_DIST_BOUNDARY (section 3.4, Tier 1: inputs that cover boundary
 * values).  Element i draws one VALUE block (x, y, z, w).  If x < T, with
 * T = 2^32 for p0 = 1 and floor(p0 * 2^32 + 1/2) otherwise, the element is
 * boundary pattern (y mod 16) of its type; otherwise it is p1 * rho * cos
 * from the Box-Muller pair (z, w), rounded to fp32 and then to the dtype
 * (float dtypes), or the bits of z | w << 32 (integer dtypes).
 * Float patterns 0..15: +0, -0, +min subnormal, -min subnormal, max
 * subnormal, min normal, +1, -1, the float below 1, the float above 1, +max
 * finite, -max finite, +Inf, -Inf, quiet NaN (the canonical one), signalling
 * NaN (payload 1).  fp8 e4m3 has no infinities and one NaN per sign: 12 and
 * 14 are 0x7F, 13 is 0xFF, 15 is the largest finite below max (0x7D).
 * Integer patterns (s = the sign bit, m = all ones of the width): 0, 1, m,
 * s, m^s, s|1, (m^s)-1, 0x55.., 0xAA.., then per width
 *   u8:  0x0F, 0xF0, 0x10, 0xEF, 0x40, 0xBF, 2
 *   i32: 0xFF, 0xFFFF, 0x10000, 0xFFFF0000, 0x80, 0x7F7F7F7F, 2
 *   i64: 0xFF, 0xFFFFFFFF, 2^32, 0xFFFFFFFF00000000, 0x80000000, 0x7FFFFFFF, 2.
 */
#define ASMEVO_FILL_SATURATE 1u  /* fp8: clamp to +-448 before rounding */

/*
 * One guarded allocation (section 3.4, Tier 1: allocations carry guard
 * regions initialised with canaries).  Memory layout from `base`:
 *   [guard_lo bytes][data: rows rows of `stride` elements, the last row
 *   holding only `cols`][guard_hi bytes]
 * i.e. data bytes = ((rows - 1) * stride + cols) * element size (0 if rows
 * or cols is 0).  Requirements: base non-null and a multiple of the element
 * size (an allocation that does not start on a 16-byte boundary is filled
 * byte by byte, several times slower); rows, cols >= 0; stride >= cols;
 * guard_lo a multiple of the element size; guard sizes >= 0.  `alloc_id` is
 * the logical buffer id and must be the same for the candidate's and the
 * reference's copy of a buffer: it keys the generator, so both copies get
 * identical values, pads and canaries.
 */
typedef struct {
  uint64_t base;
  int64_t rows, cols, stride;   /* elements */
  int64_t guard_lo, guard_hi;   /* bytes */
  uint32_t dtype, alloc_id;
  uint32_t dist, flags;         /* ASMEVO_DIST_*, ASMEVO_FILL_* */
  double p0, p1;
  int64_t i0, i1;
} asmevo_alloc;

/* kinds of injected differences; ASMEVO_INJ_RATE is or-ed into `kind` to make
 * a Bernoulli rule over every element instead of one element */
enum {
  ASMEVO_INJ_FLIP_BIT = 1,       /* flip bit `arg` (0xFFFFFFFF: a random bit) */
  ASMEVO_INJ_STEP_WITHIN = 2,    /* move the magnitude one unit in the last place (float dtypes) */
  ASMEVO_INJ_SET_BEYOND = 3,     /* a = b - sign(b) * 4 * (atol + rtol*|b|) (float dtypes) */
  ASMEVO_INJ_SET_NAN = 4,        /* canonical quiet NaN (float dtypes) */
  ASMEVO_INJ_SET_INF = 5,        /* +Inf (arg 0) or -Inf (arg 1); not for fp8 e4m3 */
  ASMEVO_INJ_GUARD_WRITE_LO = 6, /* invert `arg` canary bytes of the lo guard from byte `index` */
  ASMEVO_INJ_GUARD_WRITE_HI = 7, /* same for the hi guard (an out-of-bounds write) */
  ASMEVO_INJ_PAD_WRITE = 8       /* invert `arg` row-pad bytes from data byte offset `index`
                                    (a write past the end of a row); every byte named
                                    must be padding of one row */
};
#define ASMEVO_INJ_RATE 0x100u
enum { ASMEVO_SIDE_CANDIDATE = 0, ASMEVO_SIDE_BOTH = 1 };

/*
 * One injected difference.  A fill with variant 0 (the reference) applies only
 * entries with sides == ASMEVO_SIDE_BOTH; a fill with variant v > 0 applies
 * every entry.  Element entries act on the element's base value; when several
 * entries hit one element the last in the array wins, and element entries
 * override Bernoulli rules.  For a RATE rule `index` holds the threshold T
 * (0 <= T <= 2^32): element i is selected iff its SELECT draw is below T.
 * The caller converts a rate r in [0, 1] into T; the rule this library's
 * bindings use is T = floor(r * 2^32 + 1/2) (2^32 for r = 1), the same as
 * the library applies to the rate p0 of ASMEVO_DIST_BOUNDARY.
 */
typedef struct {
  uint32_t alloc;      /* index into the allocation array of the call */
  uint32_t kind;
  uint32_t sides;
  uint32_t arg;
  int64_t index;       /* element index, guard byte offset, or RATE threshold */
  double atol, rtol;   /* tolerance targeted by SET_BEYOND */
} asmevo_injection;

/*
 * asmevo_fill_guarded -- writes every byte of each allocation: lo canary,
 * data elements from the allocation's distribution, row-pad bytes, hi
 * canary; then applies the injections that `variant` selects (section 3.4,
 * Tier 1: deterministic seeded inputs with canary-initialised guards).
 * Deterministic: a pure function of (descriptors, seed, variant).
 * variant: 0 = reference state, 1..65535 = candidate state number.
 * Allocations must not overlap.  Errors: ASMEVO_E_INVALID for malformed
 * descriptors, overlapping allocations, NORMAL/BITS on integer dtypes mixed
 * with fp-only injections, out-of-range indices; ASMEVO_E_UNSUPPORTED for
 * SET_INF on fp8 e4m3 or more than 16 RATE rules on one allocation.
 */
asmevo_status asmevo_fill_guarded(const asmevo_alloc* allocs, int32_t n,
                                  const asmevo_injection* inj, int64_t n_inj,
                                  uint64_t seed, uint32_t variant,
                                  void* workspace, size_t ws_bytes, void* stream);

/*
 * One compared buffer pair: `a` is the candidate state K'(x), `b` the
 * reference O(x) (section 3.2: Delta = K'(x) - O(x); the relative term is
 * scaled by the reference).  a and b address element (0,0); row r starts at
 * a + r * stride_a elements (b likewise); strides >= cols; a and b aligned to
 * the element size.  TOLERANCE requires a float dtype and finite
 * atol, rtol >= 0.
 */
typedef struct {
  uint64_t a, b;
  uint32_t dtype, mode, nan_policy, reserved;
  int64_t rows, cols, stride_a, stride_b;   /* elements */
  double atol, rtol;
} asmevo_segment;

/*
 * Per-segment result (56 bytes).  TOLERANCE mode, per element pair:
 *   identical bits: match, unless b is NaN under NAN_STRICT;
 *   a or b NaN: match iff both are NaN and the policy is NAN_EQUAL;
 *   a or b infinite (bits differ): mismatch;
 *   both finite: d = |A - B| and t = atol + rtol*|B| in fp64 with two
 *     roundings (no fused multiply-add), match iff d <= t.
 * `nonfinite_mismatches` counts mismatches where a or b is NaN or Inf.
 * max_abs = max d and max_rel = max d/|B| (d > 0 and B = 0 give +Inf, d = 0
 * and B = 0 give 0) over all pairs with both values finite; +0.0 if none.
 * BITWISE mode: mismatches/first_mismatch equal the bitwise fields, the
 * other fields are 0 / +0.0.
 */
typedef struct {
  uint64_t mismatches;
  int64_t first_mismatch;        /* logical index, -1 if none */
  uint64_t bitwise_mismatches;   /* raw bits differ (always reported) */
  int64_t first_bitwise;
  uint64_t nonfinite_mismatches;
  double max_abs, max_rel;
} asmevo_segment_result;

/*
 * asmevo_diff_segments -- compares all n segments in one launch and writes
 * results[0..n) (device memory).  Results are initialised in-stream, so n = 0
 * and empty segments are fine.  Errors: ASMEVO_E_INVALID for null pointers,
 * negative sizes, stride < cols, misaligned a/b, TOLERANCE on an integer
 * dtype, negative or non-finite tolerances; ASMEVO_E_WORKSPACE.
 */
asmevo_status asmevo_diff_segments(const asmevo_segment* segs, int32_t n,
                                   asmevo_segment_result* results,
                                   void* workspace, size_t ws_bytes, void* stream);

/* As asmevo_diff_segments with an explicit number of workgroups (0 = the
 * library's choice); results are identical for every value. */
asmevo_status asmevo_diff_segments_ex(const asmevo_segment* segs, int32_t n,
                                      asmevo_segment_result* results,
                                      void* workspace, size_t ws_bytes, void* stream,
                                      int32_t workgroups);

/*
 * asmevo_diff_segments_noalloc -- asmevo_diff_segments for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): no workspace argument; the
 * descriptor table goes to a static device array of the library that holds
 * ASMEVO_NOALLOC_MAX_SEGMENTS descriptors (512 KiB; each GPU the library runs
 * on keeps its own copy until the process ends).  The call allocates nothing
 * (no hipMalloc, no hipFree, no allocating library routine).  Results are
 * identical to asmevo_diff_segments'.  Every call on one GPU shares that
 * GPU's array: calls whose work overlaps on one GPU (other streams, other
 * threads before their stream has drained) race and give undefined results;
 * calls in one stream are ordered.  Errors as for asmevo_diff_segments, and
 * ASMEVO_E_CAPACITY for n > ASMEVO_NOALLOC_MAX_SEGMENTS.
 */
#define ASMEVO_NOALLOC_MAX_SEGMENTS 4096
asmevo_status asmevo_diff_segments_noalloc(const asmevo_segment* segs, int32_t n,
                                           asmevo_segment_result* results, void* stream);

/*
 * One N-dimensional compared buffer pair (section 3.4: captured dispatch
 * states hold non-contiguous tensors and block-table layouts; Tier-1 inputs
 * span shapes and strides).  Element (i_0, ..., i_{ndim-1}) of the candidate
 * lies at a + sum_d i_d * stride_a[d] elements (b likewise); its logical
 * index is index_base plus its row-major position (the last dimension
 * varies fastest).  0 <= ndim <= ASMEVO_MAX_DIMS (ndim 0: one element);
 * shape[d] >= 0; strides >= 0 in elements (0 broadcasts; overlapping views
 * are allowed, the operands are only read); a and b aligned to the element
 * size; index_base >= 0.  `result` selects the entry of the results array
 * this segment accumulates into: several segments may share one (a
 * block-table layout: one segment per block, each with index_base = the
 * block's logical start), and the shared entry then holds the summed
 * counts, the lowest first indices and the largest maxima.  dtype, mode,
 * nan_policy, atol and rtol as in asmevo_segment.
 */
#define ASMEVO_MAX_DIMS 8
typedef struct {
  uint64_t a, b;
  uint32_t dtype, mode, nan_policy, ndim;
  uint32_t result, reserved;
  int64_t index_base;
  int64_t shape[ASMEVO_MAX_DIMS];
  int64_t stride_a[ASMEVO_MAX_DIMS];
  int64_t stride_b[ASMEVO_MAX_DIMS];
  double atol, rtol;
} asmevo_segment_nd;

/* Workspace bytes asmevo_diff_segments_nd needs for n segments. */
size_t asmevo_diff_nd_workspace_bytes(int32_t n);

/*
 * asmevo_diff_segments_nd -- as asmevo_diff_segments for N-D segments, in one
 * launch.  results[0..n_results) (device memory) are cleared first, then
 * every segment accumulates into results[segs[k].result].  The planner drops
 * unit dimensions and merges dimensions that are contiguous in both
 * operands, so a contiguous tensor of any shape is one row and runs at the
 * speed of the 1-D path.  asmevo_diff_cosine_nd adds the cosine term.
 * Errors: ASMEVO_E_INVALID (also: result >= n_results, ndim out of range,
 * negative shape, stride or index_base, an element offset beyond 2^52
 * bytes), ASMEVO_E_WORKSPACE.
 */
asmevo_status asmevo_diff_segments_nd(const asmevo_segment_nd* segs, int32_t n,
                                      asmevo_segment_result* results, int32_t n_results,
                                      void* workspace, size_t ws_bytes, void* stream);

/*
 * Cosine term of Eq. 1 (section 3.2): c_x = cos(K'(x), O(x)) per buffer,
 * over the element pairs with both values finite.  The products of two
 * values of any float element type are exact in fp64, so only the additions
 * round, and they follow one defined order, independent of launch geometry:
 *   - rows: a segment whose operands are both contiguous (rows == 1, or
 *     stride_a == stride_b == cols) is one row of rows*cols elements;
 *     otherwise every row is separate;
 *   - each row is cut into blocks of 4096 bytes (4096/esize elements, the
 *     last block of a row shorter);
 *   - in a block, element t belongs to lane (t / (16/esize)) mod 64; each lane
 *     adds its products in increasing t, starting from +0.0;
 *   - the 64 lane sums combine by an xor butterfly: for m = 32, 16, 8, 4, 2, 1
 *     every lane adds the lane m apart; the block sum is lane 0's value;
 *   - the blocks of the segment (row-major) combine by the left-complete
 *     pairwise tree P(x[0..n)) = P(x[0..h)) + P(x[h..n)), h the largest power
 *     of two below n, P of one value = that value, P of none = +0.0.
 * cosine = sum_ab / (sqrt(sum_aa) * sqrt(sum_bb)), each operation rounded;
 * 1.0 when both sums of squares are 0, 0.0 when exactly one is.  Integer and
 * opaque buffers: sums 0, pairs 0, cosine NaN (not defined).
 */
typedef struct {
  double sum_ab, sum_aa, sum_bb, cosine;
  uint64_t pairs;    /* element pairs with both values finite */
  uint64_t blocks;   /* 4096-byte blocks summed */
} asmevo_cosine_result;

/*
 * asmevo_diff_cosine -- asmevo_diff_segments plus the cosine term of every
 * float segment, from the same single pass over the operands (a second, small
 * kernel folds the per-block sums).  `results` as for asmevo_diff_segments;
 * `cos_results[0..n)` device memory.  The workspace must hold
 * asmevo_diff_cosine_workspace_bytes(segs, n) bytes (it keeps 32 bytes per
 * 4096-byte block).  Errors as for asmevo_diff_segments.
 */
asmevo_status asmevo_diff_cosine(const asmevo_segment* segs, int32_t n,
                                 asmevo_segment_result* results,
                                 asmevo_cosine_result* cos_results,
                                 void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes asmevo_diff_cosine needs for these segments (0 if they are
 * invalid). */
size_t asmevo_diff_cosine_workspace_bytes(const asmevo_segment* segs, int32_t n);

/*
 * asmevo_diff_cosine_nd -- asmevo_diff_segments_nd plus the cosine term of
 * every result, from the same single pass.  The order of the additions is
 * that of asmevo_diff_cosine, along each segment's walk: the dimensions of
 * extent > 1 ordered by decreasing stride of a (stride 0 first), ties by
 * decreasing stride of b, then neighbours contiguous in both operands merged;
 * the innermost merged dimension forms the rows (cut into 4096-byte blocks),
 * the other dimensions order the rows, last fastest; the blocks of all the
 * segments of a result, in array order, combine by one pairwise tree.  (A
 * 2-D segment of asmevo_diff_cosine walks the same way.)  The segments of a
 * result must be consecutive in `segs` and of one element type, else
 * ASMEVO_E_UNSUPPORTED; a result with no segments has cosine 1.0 over no
 * blocks.  cos_results[0..n_results) device memory; the workspace must hold
 * asmevo_diff_cosine_nd_workspace_bytes(segs, n, n_results) bytes.  Other
 * errors as for asmevo_diff_segments_nd.
 */
asmevo_status asmevo_diff_cosine_nd(const asmevo_segment_nd* segs, int32_t n,
                                    asmevo_segment_result* results, int32_t n_results,
                                    asmevo_cosine_result* cos_results,
                                    void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes asmevo_diff_cosine_nd needs (0 if the segments are invalid
 * or unsupported, or n_results <= 0). */
size_t asmevo_diff_cosine_nd_workspace_bytes(const asmevo_segment_nd* segs, int32_t n, int32_t n_results);

/* Per-allocation guard result (48 bytes): counts of corrupted bytes and the
 * lowest corrupted byte offset within each guard (-1 if intact), and the same
 * for the row padding, whose offsets count from the first data byte. */
typedef struct {
  uint64_t bad_lo, bad_hi;
  int64_t first_bad_lo, first_bad_hi;
  uint64_t bad_pad;
  int64_t first_bad_pad;
} asmevo_guard_result;

/*
 * asmevo_guard_check -- compares every guard byte of the n allocations
 * against the canary regenerated from (seed, alloc_id) (the predicate iota
 * of section 3.2 requires intact out-of-bounds guards), and every row-pad
 * byte (elements cols..stride-1 of rows 0..rows-2, interior guards between
 * rows) against the pad byte the fill wrote there, writing results[0..n)
 * (device memory).  Only the allocation geometry (base, rows, cols, stride,
 * guards, dtype, alloc_id) is used.  Errors: ASMEVO_E_INVALID,
 * ASMEVO_E_WORKSPACE.
 */
asmevo_status asmevo_guard_check(const asmevo_alloc* allocs, int32_t n, uint64_t seed,
                                 asmevo_guard_result* results,
                                 void* workspace, size_t ws_bytes, void* stream);

/*
 * Staged plans (section 3.7, Algorithm 1: eq(c, x) runs for every input x of
 * every candidate, and section 4.1 repeats each check three times): a diff
 * or a guard check whose descriptors do not change between calls is planned,
 * validated and uploaded once, then launched as often as it is repeated with
 * no host planning and no host-to-device copy per launch.  The plan records
 * the device addresses its descriptors name: it stays valid while those
 * buffers and the workspace it was staged in stay allocated and unchanged.
 *
 * asmevo_plan_diff / asmevo_plan_guard -- validate exactly as asmevo_diff_
 * segments / asmevo_guard_check, stage the descriptor table in `workspace`
 * (at least asmevo_plan_bytes(n) bytes, caller-owned; stream-ordered upload
 * from pageable memory, synchronous with the host) and fill *plan (host
 * memory).  Errors as for the unplanned calls; ASMEVO_E_INVALID for a null
 * plan.
 * asmevo_plan_diff_nd -- the same for asmevo_diff_segments_nd's segments
 * and n_results results.
 * asmevo_diff_planned / asmevo_guard_planned -- enqueue the planned check:
 * results as the unplanned call's (asmevo_segment_result per result or
 * asmevo_guard_result per allocation, device memory, initialised
 * in-stream).  The staged table is only read: launches of one plan may
 * overlap, each with results of its own.  ASMEVO_E_INVALID for a null or
 * mismatched plan.
 */
enum { ASMEVO_PLAN_DIFF = 1, ASMEVO_PLAN_GUARD = 2, ASMEVO_PLAN_DIFF_ND = 3 };
typedef struct {
  uint64_t table;       /* device address of the staged table, inside the plan's workspace */
  uint64_t units;       /* tiles of the diff, or 16-byte chunks of the guard check */
  int32_t n;            /* descriptors in the table */
  int32_t n_results;    /* results one launch writes */
  int32_t kind;         /* ASMEVO_PLAN_DIFF, ASMEVO_PLAN_DIFF_ND or ASMEVO_PLAN_GUARD */
  int32_t workgroups;   /* launch width of the diff */
} asmevo_plan;

size_t asmevo_plan_bytes(int32_t n_descs);
asmevo_status asmevo_plan_diff(const asmevo_segment* segs, int32_t n, void* workspace, size_t ws_bytes,
                               void* stream, asmevo_plan* plan);
asmevo_status asmevo_plan_diff_nd(const asmevo_segment_nd* segs, int32_t n, int32_t n_results, void* workspace,
                                  size_t ws_bytes, void* stream, asmevo_plan* plan);
asmevo_status asmevo_diff_planned(const asmevo_plan* plan, asmevo_segment_result* results, void* stream);
asmevo_status asmevo_plan_guard(const asmevo_alloc* allocs, int32_t n, void* workspace, size_t ws_bytes,
                                void* stream, asmevo_plan* plan);
asmevo_status asmevo_guard_planned(const asmevo_plan* plan, uint64_t seed, asmevo_guard_result* results,
                                   void* stream);

/*
 * One region of a captured pre-dispatch state (section 3.4, Tier 2: the
 * dispatch's referenced device-memory regions and their pre-state are
 * recorded once; every candidate replays with identical memory contents).
 */
typedef struct {
  uint64_t dst, src;   /* device addresses */
  uint64_t bytes;
} asmevo_region;

/*
 * asmevo_copy_regions -- copies every region (dst <- src, `bytes` bytes) in
 * one launch: a snapshot (live -> backup) or a restore (backup -> live) of a
 * captured state, in place so that absolute device pointers inside the state
 * stay valid.  Any alignment is accepted; regions whose source and
 * destination share their address modulo 16 move in 16-byte chunks.
 * Requirements: non-null addresses for non-empty regions; no destination
 * range may overlap another destination or any source range.  Errors:
 * ASMEVO_E_INVALID, ASMEVO_E_WORKSPACE (needs asmevo_workspace_bytes(n, 0)).
 */
asmevo_status asmevo_copy_regions(const asmevo_region* regions, int32_t n,
                                  void* workspace, size_t ws_bytes, void* stream);

/*
 * Device memory at a chosen virtual address (section 3.4, Tier 2: a captured
 * pre-dispatch state holds absolute device pointers, so replaying it, here or
 * in another process, needs its regions back at the addresses they were
 * captured at).  These are the library's only allocating calls; everything
 * else works on caller-owned memory.
 *
 * asmevo_va_granularity -- the size and address granularity of the calls
 * below for the current device, in bytes; 0 if the device has no virtual
 * memory management (HIP's hipMemAddressReserve family).
 *
 * asmevo_va_alloc -- reserves `bytes` of device address space starting at
 * `addr` (0: wherever the driver chooses), backs it with memory of the
 * current device, maps it readable and writable, and stores its address in
 * *out.  Contents are undefined.  `addr` and `bytes` must be multiples of
 * asmevo_va_granularity().  A range that cannot be placed at `addr` (already
 * in use, or outside the device's address aperture) is released again and the
 * call returns ASMEVO_E_UNSUPPORTED.  A range freed in this process can be
 * requested again.  A state meant for replay in another process is best
 * placed at an explicit address: the addresses the driver picks lie near the
 * top of the device aperture, where a new process's runtime places its own
 * allocations (on MI355X under ROCm 7 explicit addresses from 2^44 to
 * 0x4F00'0000'0000 were honoured in fresh processes; 0x7F00'0000'0000 lies
 * outside the aperture).  Errors: ASMEVO_E_INVALID (null out, zero or
 * unaligned size or address), ASMEVO_E_UNSUPPORTED, ASMEVO_E_HIP.
 * Synchronous.
 *
 * asmevo_va_free -- unmaps and releases a range returned by asmevo_va_alloc
 * (its start address).  The caller makes sure no queued work still uses it.
 * Errors: ASMEVO_E_INVALID (not a live range of this process), ASMEVO_E_HIP.
 */
size_t asmevo_va_granularity(void);
asmevo_status asmevo_va_alloc(uint64_t addr, uint64_t bytes, uint64_t* out);
asmevo_status asmevo_va_free(uint64_t addr);

/* Workspace bytes sufficient for any of the three calls with up to n_descs
 * descriptors and n_inj injections. */
size_t asmevo_workspace_bytes(int32_t n_descs, int64_t n_inj);
const char* asmevo_status_string(asmevo_status status);
int32_t asmevo_abi_version(void);
/* hipError_t code of the last failing HIP call on this thread (0 if none). */
int32_t asmevo_last_hip_error(void);

/*
 * Code objects under test (section 3.7, Algorithm 1: a candidate is built
 * into a code object and, once its static checks pass, run under the same
 * device and launch conditions as the original K0 for the equivalence check
 * and the timing).  The caller builds the code objects; these calls load one,
 * launch it with explicit arguments, and time it.
 */
typedef struct {
  uint64_t module, function;     /* hipModule_t / hipFunction_t */
  int32_t num_regs;              /* from the runtime's function attributes */
  int32_t shared_bytes;          /* static LDS */
  int32_t max_threads;           /* largest workgroup the code object accepts */
  int32_t local_bytes;           /* scratch per work-item */
} asmevo_kernel;

/* Loads a code object image (an AMDGPU ELF, host memory, size image_bytes)
 * and finds kernel `name`.  The caller owns the returned handle and frees it
 * with asmevo_kernel_unload.  Errors: ASMEVO_E_INVALID for null arguments,
 * ASMEVO_E_HIP when the runtime rejects the image or does not find the
 * kernel (asmevo_last_hip_error gives the code). */
asmevo_status asmevo_kernel_load(const void* image, size_t image_bytes, const char* name,
                                 asmevo_kernel* out);
asmevo_status asmevo_kernel_unload(asmevo_kernel* k);

/* Enqueues one launch: grid in workgroups, block in work-items, dynamic LDS
 * bytes, params[i] pointing at the value of explicit argument i (laid out by
 * the runtime from the code object's metadata).  Errors: ASMEVO_E_INVALID
 * for zero dimensions or a block larger than the kernel allows, ASMEVO_E_HIP. */
asmevo_status asmevo_kernel_launch(const asmevo_kernel* k, const uint32_t grid[3],
                                   const uint32_t block[3], uint32_t lds_bytes, void** params,
                                   void* stream);

/* `warmup` untimed launches, then `reps` launches each bracketed by HIP
 * events on `stream`; waits for the stream and writes the reps durations in
 * milliseconds to ms_out[0..reps). */
asmevo_status asmevo_kernel_time(const asmevo_kernel* k, const uint32_t grid[3],
                                 const uint32_t block[3], uint32_t lds_bytes, void** params,
                                 int32_t warmup, int32_t reps, float* ms_out, void* stream);

#ifdef __cplusplus
}
#endif
#endif
