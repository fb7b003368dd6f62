// layout.h -- device-side descriptor tables staged by the host planner into
// the caller's workspace.  Internal to the library (not part of the C ABI).
#pragma once
#include <stdint.h>

namespace asmevo {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kChunk = 16;         // bytes per lane per load (dwordx4)

// ---------------------------------------------------------------- diff
#ifndef ASMEVO_DIFF_UNROLL
#define ASMEVO_DIFF_UNROLL 4
#endif
constexpr int kDiffUnroll = ASMEVO_DIFF_UNROLL;      // chunks per lane per tile
#ifndef ASMEVO_DIFF_WAVES_PER_EU                     // occupancy target of the plain 2-D diff kernel
#define ASMEVO_DIFF_WAVES_PER_EU 2                   // (it runs 1-2 waves per SIMD: the register budget
#endif                                               // goes to the deferred slow path)
#ifndef ASMEVO_DIFF_ND_WAVES_PER_EU                  // ... of the N-D diff kernel (its resident set)
#define ASMEVO_DIFF_ND_WAVES_PER_EU 4
#endif
#ifndef ASMEVO_COS_WAVES_PER_EU                      // ... and of its cosine variant
#define ASMEVO_COS_WAVES_PER_EU 3
#endif
#ifndef ASMEVO_DIFF_WAVE_STEP                        // waves of a workgroup sharing one tile range
#define ASMEVO_DIFF_WAVE_STEP 1
#endif
#ifndef ASMEVO_COS_WAVE_STEP                         // ... in the cosine variant (4 resident
#define ASMEVO_COS_WAVE_STEP 4                       // workgroups per CU: 4x fewer read streams)
#endif
#ifndef ASMEVO_DIFF_DEAL                             // tiles per block dealt round-robin (0: ranges)
#define ASMEVO_DIFF_DEAL 0
#endif
#ifndef ASMEVO_COS_DEAL                              // ... in the cosine variant, whose cost per
#define ASMEVO_COS_DEAL 256                          // tile depends on the element type
#endif
constexpr int kTileChunks = kWave * kDiffUnroll;     // 256 chunks = 4 KiB per operand
constexpr int kDiffBlock = 256;                      // 4 waves per workgroup

enum : uint32_t {
  kSegVec = 1u,       // a, b and both row pitches are 16-byte aligned
  kSegStrict = 4u,    // TOLERANCE with the strict NaN policy
  kSegNarrow = 8u,    // short 2-D rows: tiles run over the flattened chunk space
  kSegGather = 16u,   // N-D: the innermost dimension is not unit-stride in a or b
  kSegPermuted = 32u, // N-D: visited in memory order, not logical order (see NdExt)
  kSegPair2A = 64u,   // N-D gather: a's elements are 2 apart and its rows start 16-byte aligned
  kSegPair2B = 128u,  // ... the same for b
  kSegSpan = 256u,    // N-D: a gather read as its rows' covering bytes; only the elements at
                      // multiples of `span` compare (the others are masked to zero on both sides)
};

// A segment is either "row-tiled" (every tile lies inside one row: contiguous
// segments are one long row) or "narrow" (rows shorter than half a tile; tiles
// run over the row-major chunk space and each lane finds its own row).
struct DiffSeg {                // 128 bytes
  uint64_t a, b;                // element (0,0) of candidate / reference
  union {
    uint64_t a_pitch;           // 2-D: bytes between row starts
    uint64_t nd_index_base;     // N-D: added to every reported index
  };
  union {
    uint64_t b_pitch;
    uint64_t nd_ext;            // N-D: index of the segment's NdExt; ~0 if it needs none
  };
  uint64_t rows;                // 1 when the segment is contiguous in both operands
  uint64_t cols;                // logical elements per (possibly flattened) row
  uint64_t row_bytes;           // cols * esize
  uint64_t row_chunks;          // ceil(row_bytes / 16)
  uint64_t full_chunks;         // row_bytes / 16
  uint64_t tile_begin;          // first tile of this segment in the global tile space
  uint64_t tile_count;
  double atol, rtol;
  uint32_t dtype, mode, flags, esize;
  uint32_t result_index;
  union {
    uint32_t tiles_per_row;     // 2-D: tiles of one row
    uint32_t span;              // N-D: 0, or a span row (kSegSpan): bits 0-7 the element
                                // stride s, bits 8-23 bit k set iff k mod s == 0 (k < 16)
  };
};
static_assert(sizeof(DiffSeg) == 128, "DiffSeg layout");

// N-D segments.  The planner orders the dimensions by decreasing stride of
// `a` (broadcast dimensions outermost) so that the walk follows memory, then
// drops unit dimensions and merges dimensions contiguous in both operands.
// The DiffSeg describes rows of `cols` elements of the innermost remaining
// dimension; this extension places row r: r is decomposed over the outer
// dimensions (last one fastest) and each index is scaled by that
// dimension's byte pitch.  Within a row, element j lies at j * in_sa (in_sb)
// bytes.  The walk position q = r * cols + j is the element's logical
// (row-major) index when the order was not changed; otherwise (kSegPermuted)
// q is decomposed over the ordered, unmerged dimensions ishape (last one
// fastest) and the logical index is sum idx_d * lpitch[d].  Either way
// index_base is added.  A segment that is one row in memory order (rows == 1,
// unit stride, no reordering) needs no extension.
constexpr int kMaxOuter = 7;
constexpr int kMaxDims = 8;
struct NdExt {                  // 328 bytes
  uint64_t index_base;
  uint64_t in_sa, in_sb;        // innermost-dimension strides in bytes
  uint32_t nouter, ni;          // outer (merged) dimensions; ordered unmerged dimensions
  uint64_t oshape[kMaxOuter];   // outer dimensions, outermost first
  uint64_t opa[kMaxOuter], opb[kMaxOuter];
  uint64_t ishape[kMaxDims];    // kSegPermuted: walk order, outermost first
  uint64_t lpitch[kMaxDims];    // logical index pitch of each of them
};
static_assert(sizeof(NdExt) == 328, "NdExt layout");

// The cosine's block tree per segment, by levels: level 0 holds the block
// sums (cnt[0] = the segment's tiles, at partials + kCosRec * off[0]); level
// k >= 1 holds one sum per full aligned group of 256 level-(k-1) entries
// (cnt[k] = cnt[k-1] / 256, at levels + kCosRec * off[k]).  Such a group is a perfect
// subtree of the left-complete tree, so the levels are reduced in parallel
// and only the entries no group absorbed are folded per segment.
constexpr int kCosLevels = 6;
// doubles per block-sum record: {sum a*b, sum a*a, sum b*b, 0}, 32 bytes, so
// one store from four lanes writes a whole 32-byte memory sector
constexpr int kCosRec = 4;
struct CosLevels {              // 96 bytes
  uint64_t off[kCosLevels];
  uint64_t cnt[kCosLevels];
};
static_assert(sizeof(CosLevels) == 96, "CosLevels layout");

// ---------------------------------------------------------------- fill
constexpr int kMaxRules = 16;      // Bernoulli rules per allocation
constexpr int kFillBlock = 256;

struct FillAlloc {              // 128 bytes
  uint64_t base;                // first lo-guard byte (element-aligned)
  uint64_t total_bytes;         // guard_lo + data + guard_hi
  uint64_t guard_lo, data_bytes;
  uint64_t rows, cols, stride;  // elements
  uint64_t tile_begin;          // first 64-chunk tile of this allocation
  double p0, p1;
  int64_t i0, i1;
  uint32_t dtype, esize, alloc_id, dist;
  uint32_t saturate, rule_begin, rule_count;
  uint32_t phase;               // base mod 16: the chunks are the 16-byte blocks of memory
};
static_assert(sizeof(FillAlloc) == 128, "FillAlloc layout");

struct FillRule {               // a Bernoulli rule (or a point entry)
  uint32_t kind, vsel, arg, ordinal;   // vsel: variant field used in SELECT/INJECT counters
  uint64_t threshold;           // RATE: selected iff draw < threshold
  double atol, rtol;
};
static_assert(sizeof(FillRule) == 40, "FillRule layout");

struct PointEntry {             // one deduplicated point injection
  uint32_t alloc, kind, vsel, arg;
  int64_t index;
  double atol, rtol;
};
static_assert(sizeof(PointEntry) == 40, "PointEntry layout");

// ---------------------------------------------------------------- copy
struct CopyRegion {             // 64 bytes
  uint64_t dst, src, bytes;
  uint64_t head;                // bytes before src/dst reach 16-byte alignment (vec regions)
  uint64_t body_bytes;          // bytes - head; moved in whole 16-byte chunks, the rest by the last tile
  uint64_t tile_begin, tile_count;
  uint32_t vec, pad0;           // vec: src and dst have the same address phase modulo 16
};
static_assert(sizeof(CopyRegion) == 64, "CopyRegion layout");

// ---------------------------------------------------------------- guard
// One guard side of one allocation, or (side 2) all row paddings of one
// allocation: `runs` runs of `bytes` bytes, run r starting at data byte
// r * pitch + pad_off; every run is cut into run_chunks 16-byte chunks.
struct GuardRegion {            // 64 bytes
  uint64_t addr;                // first guard byte; side 2: first data byte
  uint64_t bytes;               // guard bytes; side 2: pad bytes per row
  uint64_t chunk_begin;         // first 16-byte chunk in the global chunk space
  uint64_t pitch, pad_off;      // side 2: row pitch and pad start within a row, in bytes
  uint64_t run_chunks;          // side 2: ceil(bytes / 16)
  uint32_t alloc_id, side;      // side 0 = lo, 1 = hi, 2 = row padding
  uint32_t result_index, pad0;
};
static_assert(sizeof(GuardRegion) == 64, "GuardRegion layout");

}  // namespace asmevo
