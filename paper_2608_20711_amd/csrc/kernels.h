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

// Resident workgroups per CU of the N-D cosine pass, and of its variant for
// calls whose segments all have short rows of a float type.
int cos_nd_blocks_per_cu();
int narrow_cos_blocks_per_cu();
// Whether every segment with tiles (host copies of the device descriptors)
// has short rows of a float type, so the N-D cosine pass may take the variant.
bool cos_nd_short_rows_only(const DiffSeg* segs, int n);
// Diff and cosine term of N-D segments: the diff as launch_diff_nd, the block
// sums per tile as launch_diff; the block trees run over `units`, one
// descriptor per result (its first tile, its tile count, dtype, element
// count), so the tables (levels_of, level_prefix, counters) are per result.
// short_rows: launch the short-row variant (cos_nd_short_rows_only).
hipError_t launch_diff_cosine_nd(const DiffSeg* segs, const NdExt* ext, int n, const DiffSeg* units,
                                 int n_results, uint64_t total_tiles, asmevo_segment_result* results,
                                 int workgroups, hipStream_t stream, double* partials,
                                 unsigned long long* nonfinite_pairs, asmevo_cosine_result* cos_results,
                                 const CosLevels* levels_of, const uint64_t* level_prefix,
                                 const uint64_t* level_groups, double* levels, bool short_rows);

hipError_t launch_copy(const CopyRegion* regs, int n, uint64_t total_tiles, int workgroups,
                       hipStream_t stream);

hipError_t launch_guard(const GuardRegion* regs, int n_regs, uint64_t total_chunks, uint64_t seed,
                        asmevo_guard_result* results, int n_results, hipStream_t stream);

}  // namespace asmevo
