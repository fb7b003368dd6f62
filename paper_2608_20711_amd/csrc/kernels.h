// kernels.h -- host-side launchers of the library's kernels (internal).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asmevo.h"
#include "layout.h"

namespace asmevo {

// Resident fill workgroups per compute unit.
int fill_blocks_per_cu();
hipError_t launch_fill(const FillAlloc* allocs, int n, const FillRule* rules, uint64_t total_tiles,
                       uint64_t seed, int workgroups, hipStream_t stream);
hipError_t launch_inject(const FillAlloc* allocs, const PointEntry* pts, int n_pts, uint64_t seed,
                         hipStream_t stream);

// Resident workgroups per compute unit of the diff's cosine variant (from the
// occupancy calculator).
int cos_blocks_per_cu();
// Diff of all segments; with cos_results, also the cosine term (partials:
// one block-sum record of kCosRec doubles per tile; nonfinite_pairs: one
// counter per segment; the block tree by levels: levels_of[n] (device),
// level_prefix[(kCosLevels-1) x (n+1)] (device: groups of the segments
// before s, per level), level_groups[kCosLevels] (host: groups per level),
// levels: one record per level entry).
hipError_t launch_diff(const DiffSeg* segs, int n, uint64_t total_tiles,
                       asmevo_segment_result* results, int workgroups, hipStream_t stream,
                       double* partials = nullptr, unsigned long long* nonfinite_pairs = nullptr,
                       asmevo_cosine_result* cos_results = nullptr, const CosLevels* levels_of = nullptr,
                       const uint64_t* level_prefix = nullptr, const uint64_t* level_groups = nullptr,
                       double* levels = nullptr);

// Resident N-D diff workgroups per compute unit.
int diff_nd_blocks_per_cu();
// Diff of N-D segments (descriptor k extended by ext[k]); zeroes results[0, n_results) first.
hipError_t launch_diff_nd(const DiffSeg* segs, const NdExt* ext, int n, int n_results,
                          uint64_t total_tiles, asmevo_segment_result* results, int workgroups,
                          hipStream_t stream);

// The N-D cosine pass's kernel for a call: the general one, or a variant for
// calls whose segments (those with tiles) are all of a float type and all
// short rows, all long 16-byte-aligned unit-stride rows, or all gathers of
// long rows with elements 2 apart in both operands.
enum { kCosNdMixed = 0, kCosNdShortRows = 1, kCosNdLongRows = 2, kCosNdGathers = 3 };
// The variant for these descriptors (host copies of the device descriptors).
int cos_nd_variant(const DiffSeg* segs, int n);
// Resident workgroups per CU of the general N-D cosine kernel, and of a variant.
int cos_nd_blocks_per_cu();
int split_cos_blocks_per_cu(int variant);
// Diff and cosine term of N-D segments: the diff as launch_diff_nd, the block
// sums per tile as launch_diff; the block trees run over `units`, one
// descriptor per result (its first tile, its tile count, dtype, element
// count), so the tables (levels_of, level_prefix, counters) are per result.
// variant: the kernel to launch (cos_nd_variant).
hipError_t launch_diff_cosine_nd(const DiffSeg* segs, const NdExt* ext, int n, const DiffSeg* units,
                                 int n_results, uint64_t total_tiles, asmevo_segment_result* results,
                                 int workgroups, hipStream_t stream, double* partials,
                                 unsigned long long* nonfinite_pairs, asmevo_cosine_result* cos_results,
                                 const CosLevels* levels_of, const uint64_t* level_prefix,
                                 const uint64_t* level_groups, double* levels, int variant);

hipError_t launch_copy(const CopyRegion* regs, int n, uint64_t total_tiles, int workgroups,
                       hipStream_t stream);

hipError_t launch_guard(const GuardRegion* regs, int n_regs, uint64_t total_chunks, uint64_t seed,
                        asmevo_guard_result* results, int n_results, hipStream_t stream);

}  // namespace asmevo
