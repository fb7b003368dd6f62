// api.hip -- the C ABI (include/asmevo.h): argument validation, planning of
// the device descriptor tables, one host-to-device copy into the caller's
// workspace, kernel launches.  Validation finishes before anything is
// enqueued, so an argument error leaves the stream untouched.  The tables are
// built in pageable host vectors that die with the call: hipMemcpyAsync from
// pageable memory is synchronous (HIP stages it through a pinned buffer before
// returning), so the copy has its bytes by then.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "asmevo.h"
#include "kernels.h"
#include "layout.h"

using namespace asmevo;

namespace {

thread_local int32_t g_last_hip = 0;

#define HIP_TRY(expr)                        \
  do {                                       \
    hipError_t e_ = (expr);                  \
    if (e_ != hipSuccess) {                  \
      g_last_hip = (int32_t)e_;              \
      return ASMEVO_E_HIP;                   \
    }                                        \
  } while (0)

int esize_of(uint32_t dtype) {
  switch (dtype) {
    case ASMEVO_F32: return 4;
    case ASMEVO_BF16: return 2;
    case ASMEVO_F16: return 2;
    case ASMEVO_FP8_E4M3: return 1;
    case ASMEVO_I32: return 4;
    case ASMEVO_I64: return 8;
    case ASMEVO_U8: return 1;
    default: return 0;
  }
}

bool is_float(uint32_t dtype) { return dtype >= ASMEVO_F32 && dtype <= ASMEVO_FP8_E4M3; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspaces start on a 256-byte boundary (as hipMalloc and torch
// allocations do): the kernels' 64-bit atomics on counters and accumulators
// staged there need natural alignment.
bool ws_aligned(const void* workspace) { return (reinterpret_cast<uintptr_t>(workspace) & 255u) == 0; }

uint64_t data_bytes(const asmevo_alloc& A) {
  if (A.rows <= 0 || A.cols <= 0) return 0;
  return (uint64_t)((A.rows - 1) * A.stride + A.cols) * (uint64_t)esize_of(A.dtype);
}

// Geometry checks shared by the fill and the guard check.
asmevo_status check_alloc_geometry(const asmevo_alloc& A) {
  const int es = esize_of(A.dtype);
  if (es == 0) return ASMEVO_E_INVALID;
  if (A.rows < 0 || A.cols < 0 || A.guard_lo < 0 || A.guard_hi < 0) return ASMEVO_E_INVALID;
  if (A.rows > 0 && A.cols > 0 && A.stride < A.cols) return ASMEVO_E_INVALID;
  if (A.guard_lo % es != 0) return ASMEVO_E_INVALID;
  // keep every byte offset well inside 63 bits
  const double approx = ((double)A.rows * (double)(A.stride > A.cols ? A.stride : A.cols) + 1.0) * es +
                        (double)A.guard_lo + (double)A.guard_hi;
  if (approx > 0x1p52) return ASMEVO_E_INVALID;
  return ASMEVO_OK;
}

// Compute units of the current device, queried once per device.
int device_cus() {
  constexpr int kDevices = 64;
  static std::atomic<int> known[kDevices];   // 0 until queried
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  const bool cached = dev >= 0 && dev < kDevices;
  if (cached && (cus = known[dev].load(std::memory_order_relaxed)) > 0) return cus;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  if (cached) known[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

// Workgroups of the plain diff: persistent, one (4 waves) per CU when the
// state is large -- on the 64 GiB sweep that streams 1.5-2 % faster than the
// full resident set, whose more concurrent read streams cost DRAM locality --
// and two per CU below 4 GiB of operands, where the second wave per SIMD
// hides the slow path of states with many differences (decode state +4 %).
// Workgroups of the plain 2-D diff: one per CU once the operands hold 4 GiB
// (fewer read streams are faster there), two below, and two whenever short
// rows (the flattened walk, a division per lane and tile) hold 2 % of the
// tiles or more: rows of 64 of every 128 fp32 over 2 x 16 GiB took 2.61 ms
// at two workgroups per CU against 3.66 ms at one.
int diff_workgroups(const DiffSeg* dev, int32_t n, uint64_t tiles) {
  uint64_t narrow = 0;
  for (int32_t k = 0; k < n; ++k)
    if (dev[k].flags & kSegNarrow) narrow += dev[k].tile_count;
  const uint64_t operand_bytes = tiles * (uint64_t)kTileChunks * kChunk * 2;
  return device_cus() * (operand_bytes < (4ull << 30) || narrow * 50 >= tiles ? 2 : 1);
}

// Workgroups of the plain N-D diff.  Tiles other than whole 16-byte aligned
// 4 KiB runs of a row (short rows, the last tile of a row, gathers) cost the
// kernel more per byte, and more resident waves hide that; whole tiles
// stream fastest from one workgroup per CU once the operands hold 4 GiB, as
// in the 2-D diff.  Measured on 2 x 16 GiB views, one workgroup per CU
// against the resident set: transposed 5.14 against 5.42 ms, a block table
// of 2 MiB blocks 5.34 against 5.55 ms; 256-byte half rows 6.20 against
// 2.65 ms, rows of 4032 elements 8.00 against 5.23 ms.
int nd_workgroups(const std::vector<DiffSeg>& dev, uint64_t tiles) {
  uint64_t other = 0;
  for (const DiffSeg& D : dev) {
    if (D.tile_count == 0) continue;
    if ((D.flags & kSegNarrow) || !(D.flags & kSegVec) || (D.flags & kSegGather)) {
      other += D.tile_count;
      continue;
    }
    const uint64_t tpr = (D.row_chunks + kTileChunks - 1) / kTileChunks;
    other += D.rows * (tpr - D.full_chunks / kTileChunks);
  }
  const uint64_t operand_bytes = tiles * (uint64_t)kTileChunks * kChunk * 2;
  const bool stream = operand_bytes >= (4ull << 30) && other * 50 < tiles;   // under 2 % of the tiles
  return device_cus() * (stream ? 1 : diff_nd_blocks_per_cu());
}

template <typename T>
void put(std::vector<uint8_t>& buf, size_t off, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(buf.data() + off, v.data(), v.size() * sizeof(T));
}

}  // namespace

extern "C" {

int32_t asmevo_abi_version(void) { return ASMEVO_ABI_VERSION; }

int32_t asmevo_last_hip_error(void) { return g_last_hip; }

const char* asmevo_status_string(asmevo_status s) {
  switch (s) {
    case ASMEVO_OK: return "ok";
    case ASMEVO_E_INVALID: return "invalid argument";
    case ASMEVO_E_UNSUPPORTED: return "unsupported";
    case ASMEVO_E_WORKSPACE: return "workspace missing or too small";
    case ASMEVO_E_HIP: return "HIP runtime error";
    case ASMEVO_E_CAPACITY: return "more descriptors than the static scratch array holds";
    default: return "unknown status";
  }
}

size_t asmevo_workspace_bytes(int32_t n_descs, int64_t n_inj) {
  const size_t n = n_descs > 0 ? (size_t)n_descs : 0;
  const size_t m = n_inj > 0 ? (size_t)n_inj : 0;
  return align256(n * sizeof(FillAlloc)) + align256(m * sizeof(FillRule)) +
         align256(m * sizeof(PointEntry)) + align256(3 * n * sizeof(GuardRegion)) + 256;
}

// ---------------------------------------------------------------------------
asmevo_status asmevo_fill_guarded(const asmevo_alloc* allocs, int32_t n,
                                  const asmevo_injection* inj, int64_t n_inj, uint64_t seed,
                                  uint32_t variant, void* workspace, size_t ws_bytes,
                                  void* stream) {
  if (n < 0 || n_inj < 0 || (n > 0 && !allocs) || (n_inj > 0 && !inj)) return ASMEVO_E_INVALID;
  if (variant > 0xFFFFu) return ASMEVO_E_INVALID;
  if (n == 0) return n_inj == 0 ? ASMEVO_OK : ASMEVO_E_INVALID;

  // allocations
  std::vector<FillAlloc> dev(n);
  std::vector<std::pair<uint64_t, uint64_t>> spans;
  uint64_t tiles = 0;
  for (int32_t k = 0; k < n; ++k) {
    const asmevo_alloc& A = allocs[k];
    asmevo_status st = check_alloc_geometry(A);
    if (st != ASMEVO_OK) return st;
    const int es = esize_of(A.dtype);
    const uint64_t D = data_bytes(A);
    const uint64_t total = (uint64_t)A.guard_lo + D + (uint64_t)A.guard_hi;
    if (total > 0 && (A.base == 0 || A.base % (uint64_t)es != 0)) return ASMEVO_E_INVALID;
    if ((A.flags & ~ASMEVO_FILL_SATURATE) != 0) return ASMEVO_E_INVALID;
    switch (A.dist) {
      case ASMEVO_DIST_NORMAL:
        if (!is_float(A.dtype) || !std::isfinite(A.p0) || !std::isfinite(A.p1)) return ASMEVO_E_INVALID;
        break;
      case ASMEVO_DIST_UNIFORM_INT:
        if (A.i1 <= A.i0 || (uint64_t)(A.i1 - A.i0) > (1ull << 32)) return ASMEVO_E_INVALID;
        break;
      case ASMEVO_DIST_BITS:
        break;
      case ASMEVO_DIST_CONST:
        if (is_float(A.dtype) && !std::isfinite(A.p0)) return ASMEVO_E_INVALID;
        break;
      case ASMEVO_DIST_BOUNDARY:
        if (!(A.p0 >= 0.0 && A.p0 <= 1.0) || (is_float(A.dtype) && !std::isfinite(A.p1)))
          return ASMEVO_E_INVALID;
        break;
      default:
        return ASMEVO_E_INVALID;
    }
    FillAlloc& F = dev[k];
    std::memset(&F, 0, sizeof(F));
    F.base = A.base;
    F.total_bytes = total;
    F.guard_lo = (uint64_t)A.guard_lo;
    F.data_bytes = D;
    F.rows = (uint64_t)A.rows;
    F.cols = (uint64_t)A.cols;
    F.stride = (uint64_t)A.stride;
    F.tile_begin = tiles;
    F.p0 = A.p0;
    F.p1 = A.p1;
    F.i0 = A.i0;
    F.i1 = A.i1;
    if (A.dist == ASMEVO_DIST_BOUNDARY)   // selection threshold on a 32-bit draw
      F.i0 = A.p0 >= 1.0 ? (int64_t)(1ll << 32) : (int64_t)std::floor(A.p0 * 4294967296.0 + 0.5);
    F.dtype = A.dtype;
    F.esize = (uint32_t)es;
    F.alloc_id = A.alloc_id;
    F.dist = A.dist;
    F.saturate = (A.flags & ASMEVO_FILL_SATURATE) ? 1u : 0u;
    F.phase = (uint32_t)(A.base % kChunk);
    const uint64_t chunks = (F.phase + total + kChunk - 1) / kChunk;   // 16-byte blocks of memory touched
    tiles += (chunks + kWave - 1) / kWave;
    if (total) spans.emplace_back(A.base, A.base + total);
  }
  std::sort(spans.begin(), spans.end());
  for (size_t s = 1; s < spans.size(); ++s)
    if (spans[s].first < spans[s - 1].second) return ASMEVO_E_INVALID;

  // injections: Bernoulli rules per allocation, deduplicated point entries
  std::vector<std::vector<FillRule>> rules_of(n);
  std::vector<uint32_t> rate_seen(n, 0);
  std::vector<PointEntry> points;
  std::map<std::pair<uint32_t, int64_t>, size_t> slot;   // (alloc, element) -> index in points
  for (int64_t t = 0; t < n_inj; ++t) {
    const asmevo_injection& J = inj[t];
    if (J.alloc >= (uint32_t)n || J.sides > ASMEVO_SIDE_BOTH) return ASMEVO_E_INVALID;
    const asmevo_alloc& A = allocs[J.alloc];
    const int es = esize_of(A.dtype);
    const bool rate = (J.kind & ASMEVO_INJ_RATE) != 0;
    const uint32_t kind = J.kind & ~ASMEVO_INJ_RATE;
    if (kind < ASMEVO_INJ_FLIP_BIT || kind > ASMEVO_INJ_PAD_WRITE) return ASMEVO_E_INVALID;
    const bool guard = kind == ASMEVO_INJ_GUARD_WRITE_LO || kind == ASMEVO_INJ_GUARD_WRITE_HI;
    const bool pad = kind == ASMEVO_INJ_PAD_WRITE;
    if ((guard || pad) && rate) return ASMEVO_E_INVALID;
    if (!guard && !pad && kind != ASMEVO_INJ_FLIP_BIT && !is_float(A.dtype)) return ASMEVO_E_INVALID;
    if (kind == ASMEVO_INJ_SET_INF && A.dtype == ASMEVO_FP8_E4M3) return ASMEVO_E_UNSUPPORTED;
    if (kind == ASMEVO_INJ_FLIP_BIT && J.arg != 0xFFFFFFFFu && J.arg >= (uint32_t)(8 * es))
      return ASMEVO_E_INVALID;
    if (kind == ASMEVO_INJ_SET_BEYOND &&
        (!std::isfinite(J.atol) || !std::isfinite(J.rtol) || J.atol < 0 || J.rtol < 0))
      return ASMEVO_E_INVALID;
    const bool applies = variant != 0 || J.sides == ASMEVO_SIDE_BOTH;
    const uint32_t vsel = J.sides == ASMEVO_SIDE_BOTH ? 0u : variant;
    if (rate) {
      if (J.index < 0 || J.index > (int64_t)(1ll << 32)) return ASMEVO_E_INVALID;
      const uint32_t ordinal = rate_seen[J.alloc]++;
      if (ordinal >= (uint32_t)kMaxRules) return ASMEVO_E_UNSUPPORTED;
      if (applies)
        rules_of[J.alloc].push_back(FillRule{kind, vsel, J.arg, ordinal, (uint64_t)J.index, J.atol, J.rtol});
      continue;
    }
    if (guard) {
      const int64_t gsize = kind == ASMEVO_INJ_GUARD_WRITE_LO ? A.guard_lo : A.guard_hi;
      if (J.index < 0 || J.index + (int64_t)J.arg > gsize) return ASMEVO_E_INVALID;
      if (applies && J.arg > 0)
        points.push_back(PointEntry{J.alloc, kind, vsel, J.arg, J.index, J.atol, J.rtol});
      continue;
    }
    if (pad) {
      // the bytes must be padding of one row: [cols, stride) elements of a row below the last
      const int64_t pitch = A.stride * es, row_data = A.cols * es;
      if (J.index < 0 || pitch == 0) return ASMEVO_E_INVALID;
      const int64_t r = J.index / pitch, off = J.index - r * pitch;
      if (J.arg > 0 && (A.cols == 0 || r >= A.rows - 1 || off < row_data ||
                        off + (int64_t)J.arg > pitch || J.index + (int64_t)J.arg > (int64_t)data_bytes(A)))
        return ASMEVO_E_INVALID;
      if (applies && J.arg > 0)
        points.push_back(PointEntry{J.alloc, kind, vsel, J.arg, J.index, J.atol, J.rtol});
      continue;
    }
    if (J.index < 0 || J.index >= A.rows * A.cols) return ASMEVO_E_INVALID;
    if (!applies) continue;
    const PointEntry P{J.alloc, kind, vsel, J.arg, J.index, J.atol, J.rtol};
    const auto key = std::make_pair(J.alloc, J.index);
    auto it = slot.find(key);
    if (it != slot.end()) {
      points[it->second] = P;                       // a later entry overrides
    } else {
      slot.emplace(key, points.size());
      points.push_back(P);
    }
  }
  std::vector<FillRule> rules;
  for (int32_t k = 0; k < n; ++k) {
    dev[k].rule_begin = (uint32_t)rules.size();
    dev[k].rule_count = (uint32_t)rules_of[k].size();
    rules.insert(rules.end(), rules_of[k].begin(), rules_of[k].end());
  }

  // staging
  const size_t off_rules = align256(dev.size() * sizeof(FillAlloc));
  const size_t off_pts = off_rules + align256(rules.size() * sizeof(FillRule));
  const size_t bytes = off_pts + points.size() * sizeof(PointEntry);
  if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  std::vector<uint8_t> host(bytes, 0);
  put(host, 0, dev);
  put(host, off_rules, rules);
  put(host, off_pts, points);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(hipMemcpyAsync(workspace, host.data(), bytes, hipMemcpyHostToDevice, s));
  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  const FillAlloc* d_allocs = reinterpret_cast<const FillAlloc*>(ws);
  const FillRule* d_rules = reinterpret_cast<const FillRule*>(ws + off_rules);
  const PointEntry* d_pts = reinterpret_cast<const PointEntry*>(ws + off_pts);
  // the resident grid, no more: every wave deals itself tiles to the end
  const uint64_t resident = (uint64_t)device_cus() * fill_blocks_per_cu() * (kFillBlock / kWave);
  const uint64_t waves = std::max<uint64_t>(1, std::min<uint64_t>(tiles, resident));
  const int wg = (int)((waves + (kFillBlock / kWave) - 1) / (kFillBlock / kWave));
  HIP_TRY(launch_fill(d_allocs, n, d_rules, tiles, seed, wg, s));
  HIP_TRY(launch_inject(d_allocs, d_pts, (int)points.size(), seed, s));
  return ASMEVO_OK;
}

// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

// Validates the segments and builds their device descriptors dev[0..n).
// `row_tiled` keeps every tile inside one row (the cosine's 4096-byte blocks).
asmevo_status plan_diff(const asmevo_segment* segs, int32_t n, bool row_tiled, DiffSeg* dev, uint64_t& tiles) {
  if (n < 0 || (n > 0 && !segs)) return ASMEVO_E_INVALID;
  tiles = 0;
  for (int32_t k = 0; k < n; ++k) {
    const asmevo_segment& S = segs[k];
    const int es = esize_of(S.dtype);
    if (es == 0) return ASMEVO_E_INVALID;
    if (S.mode != ASMEVO_BITWISE && S.mode != ASMEVO_TOLERANCE) return ASMEVO_E_INVALID;
    if (S.nan_policy != ASMEVO_NAN_EQUAL && S.nan_policy != ASMEVO_NAN_STRICT) return ASMEVO_E_INVALID;
    if (S.rows < 0 || S.cols < 0) return ASMEVO_E_INVALID;
    const bool empty = S.rows == 0 || S.cols == 0;
    if (!empty) {
      if (S.stride_a < S.cols || S.stride_b < S.cols) return ASMEVO_E_INVALID;
      if (!S.a || !S.b || (S.a % (uint64_t)es) != 0 || (S.b % (uint64_t)es) != 0) return ASMEVO_E_INVALID;
      const double span = (double)S.rows * (double)std::max(S.stride_a, S.stride_b) * es;
      if (span > 0x1p52) return ASMEVO_E_INVALID;
    }
    if (S.mode == ASMEVO_TOLERANCE) {
      if (!is_float(S.dtype)) return ASMEVO_E_INVALID;
      if (!std::isfinite(S.atol) || !std::isfinite(S.rtol) || S.atol < 0 || S.rtol < 0)
        return ASMEVO_E_INVALID;
    }
    DiffSeg& D = dev[k];
    std::memset(&D, 0, sizeof(D));
    D.a = S.a;
    D.b = S.b;
    D.atol = S.atol;
    D.rtol = S.rtol;
    D.dtype = S.dtype;
    D.mode = S.mode;
    D.esize = (uint32_t)es;
    D.result_index = (uint32_t)k;
    D.tile_begin = tiles;
    if (empty) continue;
    const bool flat = S.rows == 1 || (S.stride_a == S.cols && S.stride_b == S.cols);
    D.rows = flat ? 1 : (uint64_t)S.rows;
    D.cols = flat ? (uint64_t)(S.rows * S.cols) : (uint64_t)S.cols;
    D.a_pitch = (uint64_t)S.stride_a * es;
    D.b_pitch = (uint64_t)S.stride_b * es;
    D.row_bytes = D.cols * es;
    D.row_chunks = (D.row_bytes + kChunk - 1) / kChunk;
    D.full_chunks = D.row_bytes / kChunk;
    const bool aligned = (S.a % 16 == 0) && (S.b % 16 == 0) &&
                         (D.rows == 1 || (D.a_pitch % 16 == 0 && D.b_pitch % 16 == 0));
    const bool narrow = !row_tiled && D.rows > 1 && D.row_chunks < (uint64_t)kTileChunks / 2;
    D.flags = (aligned ? kSegVec : 0u) | (narrow ? kSegNarrow : 0u) |
              ((S.mode == ASMEVO_TOLERANCE && S.nan_policy == ASMEVO_NAN_STRICT) ? kSegStrict : 0u);
    if (narrow) {
      D.tiles_per_row = 0;
      D.tile_count = (D.rows * D.row_chunks + kTileChunks - 1) / kTileChunks;
    } else {
      const uint64_t tpr = (D.row_chunks + kTileChunks - 1) / kTileChunks;
      D.tile_count = D.rows * tpr;
      // 2-D row-tiled segments index tiles in 32 bits
      if (D.rows > 1 && (D.tile_count >> 32) != 0) return ASMEVO_E_INVALID;
      D.tiles_per_row = (uint32_t)(tpr > 0xFFFFFFFFull ? 0xFFFFFFFFull : tpr);
    }
    tiles += D.tile_count;
  }
  return ASMEVO_OK;
}

// Validates N-D segments and builds their descriptors.  The dimensions are
// ordered by decreasing stride of `a` (broadcast dimensions outermost), so the
// walk follows memory; unit dimensions are dropped and dimensions contiguous
// in both operands merged; the innermost remaining dimension forms the rows
// and the others place them.  When the order differs from the logical one
// the kernel maps walk positions back to logical indices on a mismatch.
asmevo_status plan_diff_nd(const asmevo_segment_nd* segs, int32_t n, int32_t n_results,
                           std::vector<DiffSeg>& dev, std::vector<NdExt>& ext, uint64_t& tiles,
                           bool row_tiled = false) {
  if (n < 0 || (n > 0 && !segs)) return ASMEVO_E_INVALID;
  dev.assign((size_t)n, DiffSeg{});
  ext.clear();
  tiles = 0;
  struct Dim {
    uint64_t n;
    int64_t sa, sb;   // elements
    uint64_t lpitch;  // logical index pitch
  };
  uint64_t n_ext = 0;
  for (int32_t k = 0; k < n; ++k) {
    const asmevo_segment_nd& S = segs[k];
    const int es = esize_of(S.dtype);
    if (es == 0) return ASMEVO_E_INVALID;
    if (S.mode != ASMEVO_BITWISE && S.mode != ASMEVO_TOLERANCE) return ASMEVO_E_INVALID;
    if (S.nan_policy != ASMEVO_NAN_EQUAL && S.nan_policy != ASMEVO_NAN_STRICT) return ASMEVO_E_INVALID;
    if (S.mode == ASMEVO_TOLERANCE) {
      if (!is_float(S.dtype)) return ASMEVO_E_INVALID;
      if (!std::isfinite(S.atol) || !std::isfinite(S.rtol) || S.atol < 0 || S.rtol < 0)
        return ASMEVO_E_INVALID;
    }
    if (S.ndim > (uint32_t)ASMEVO_MAX_DIMS || S.result >= (uint32_t)n_results || S.index_base < 0)
      return ASMEVO_E_INVALID;
    bool empty = false;
    double count = 1.0, span_a = 0.0, span_b = 0.0;   // range checks in fp64, exact below
    for (uint32_t d = 0; d < S.ndim; ++d) {
      if (S.shape[d] < 0 || S.stride_a[d] < 0 || S.stride_b[d] < 0) return ASMEVO_E_INVALID;
      if (S.shape[d] == 0) empty = true;
      count *= (double)S.shape[d];
      if (S.shape[d] > 0) {
        span_a += (double)(S.shape[d] - 1) * (double)S.stride_a[d];
        span_b += (double)(S.shape[d] - 1) * (double)S.stride_b[d];
      }
    }
    DiffSeg& D = dev[k];
    NdExt X;
    std::memset(&D, 0, sizeof(D));
    std::memset(&X, 0, sizeof(X));
    D.a = S.a;
    D.b = S.b;
    D.atol = S.atol;
    D.rtol = S.rtol;
    D.dtype = S.dtype;
    D.mode = S.mode;
    D.esize = (uint32_t)es;
    D.result_index = S.result;
    D.tile_begin = tiles;
    D.nd_index_base = (uint64_t)S.index_base;
    D.nd_ext = ~0ull;
    X.index_base = (uint64_t)S.index_base;
    if (empty) continue;
    if (!S.a || !S.b || (S.a % (uint64_t)es) != 0 || (S.b % (uint64_t)es) != 0) return ASMEVO_E_INVALID;
    if ((span_a + 1.0) * es > 0x1p52 || (span_b + 1.0) * es > 0x1p52) return ASMEVO_E_INVALID;
    if ((double)S.index_base + count > 0x1p62) return ASMEVO_E_INVALID;
    // fixed-size arrays: planning many small segments (block tables) stays cheap
    Dim dims[ASMEVO_MAX_DIMS], walk[ASMEVO_MAX_DIMS], m[ASMEVO_MAX_DIMS];
    int nd = 0;
    uint64_t pitch = 1;
    uint64_t pitches[ASMEVO_MAX_DIMS];
    for (int d = (int)S.ndim - 1; d >= 0; --d) {
      pitches[d] = pitch;
      pitch *= (uint64_t)S.shape[d];
    }
    for (uint32_t d = 0; d < S.ndim; ++d)   // logical order, outermost first
      if (S.shape[d] > 1) dims[nd++] = Dim{(uint64_t)S.shape[d], S.stride_a[d], S.stride_b[d], pitches[d]};
    // walk order: decreasing stride of a, then of b; broadcast (stride 0) dimensions outermost;
    // a stable insertion sort
    auto key = [](int64_t v) { return v == 0 ? INT64_MAX : v; };
    auto before = [&](const Dim& x, const Dim& y) {
      if (key(x.sa) != key(y.sa)) return key(x.sa) > key(y.sa);
      return key(x.sb) > key(y.sb);
    };
    for (int d = 0; d < nd; ++d) {
      const Dim v = dims[d];
      int j = d;
      while (j > 0 && before(v, walk[j - 1])) {
        walk[j] = walk[j - 1];
        --j;
      }
      walk[j] = v;
    }
    bool permuted = false;
    for (int d = 0; d < nd; ++d) permuted = permuted || walk[d].lpitch != dims[d].lpitch;
    X.ni = (uint32_t)nd;
    for (int d = 0; d < nd; ++d) {
      X.ishape[d] = walk[d].n;
      X.lpitch[d] = walk[d].lpitch;
    }
    int nm = 0;   // merged, innermost first
    for (int d = nd - 1; d >= 0; --d) {
      if (nm > 0 && walk[d].sa == (int64_t)m[nm - 1].n * m[nm - 1].sa &&
          walk[d].sb == (int64_t)m[nm - 1].n * m[nm - 1].sb)
        m[nm - 1].n *= walk[d].n;
      else
        m[nm++] = walk[d];
    }
    std::reverse(m, m + nm);   // outermost first
    if (nm == 0) m[nm++] = Dim{1, 1, 1, 1};
    const Dim inner = m[nm - 1];
    bool unit = inner.sa == 1 && inner.sb == 1;
    X.in_sa = (uint64_t)inner.sa * es;
    X.in_sb = (uint64_t)inner.sb * es;
    X.nouter = (uint32_t)(nm - 1);
    uint64_t rows = 1;
    bool pitches16 = true;
    for (int d = 0; d + 1 < nm; ++d) {
      X.oshape[d] = m[d].n;
      X.opa[d] = (uint64_t)m[d].sa * es;
      X.opb[d] = (uint64_t)m[d].sb * es;
      pitches16 = pitches16 && X.opa[d] % 16 == 0 && X.opb[d] % 16 == 0;
      rows *= m[d].n;
    }
    D.rows = rows;
    D.cols = inner.n;
    D.row_bytes = D.cols * es;
    D.row_chunks = (D.row_bytes + kChunk - 1) / kChunk;
    D.full_chunks = D.row_bytes / kChunk;
    const bool aligned = unit && S.a % 16 == 0 && S.b % 16 == 0 && pitches16;
    const bool narrow = !row_tiled && D.rows > 1 && D.row_chunks < (uint64_t)kTileChunks / 2;
    // gathers of every other element: rows that start 16-byte aligned load whole 32-byte windows
    bool pitches16a = true, pitches16b = true;
    for (int d = 0; d + 1 < nm; ++d) {
      pitches16a = pitches16a && X.opa[d] % 16 == 0;
      pitches16b = pitches16b && X.opb[d] % 16 == 0;
    }
    // A gather whose elements are s apart in both operands, s * esize <= 64 bytes, rows 16-byte
    // aligned (the plain diff only: the cosine's order follows the logical elements): its rows are
    // read as their covering bytes, whole 16-byte chunks like a contiguous row, and only the
    // elements at multiples of s compare.  The walk then counts covering positions: a last
    // dimension of s positions with logical pitch 0 maps a position back to its element.  (A
    // 64-byte memory sector holds at least one element, so the covering bytes are what the
    // element loads fetch anyway.)
    const uint64_t s_el = (uint64_t)inner.sa;
    const bool span = !row_tiled && !unit && inner.sa == inner.sb && inner.sa >= 2 && s_el * es <= 64 &&
                      S.a % 16 == 0 && S.b % 16 == 0 && pitches16a && pitches16b && nd < ASMEVO_MAX_DIMS;
    if (span) {
      X.ishape[nd] = s_el;
      X.lpitch[nd] = 0;
      X.ni = (uint32_t)nd + 1;
      X.in_sa = X.in_sb = (uint64_t)es;
      D.cols = inner.n * s_el;
      D.row_bytes = ((inner.n - 1) * s_el + 1) * es;
      D.row_chunks = (D.row_bytes + kChunk - 1) / kChunk;
      D.full_chunks = D.row_bytes / kChunk;
      uint32_t pattern = 0;
      for (uint32_t k = 0; k < 16; k += (uint32_t)s_el) pattern |= 1u << k;
      D.span = (uint32_t)s_el | (pattern << 8);
      permuted = true;
      unit = true;
    }
    const bool narrow_s = !row_tiled && D.rows > 1 && D.row_chunks < (uint64_t)kTileChunks / 2;
    const bool pair2a = !unit && inner.sa == 2 && S.a % 16 == 0 && pitches16a;
    const bool pair2b = !unit && inner.sb == 2 && S.b % 16 == 0 && pitches16b;
    D.flags = ((aligned || span) ? kSegVec : 0u) | ((span ? narrow_s : narrow) ? kSegNarrow : 0u) |
              (unit ? 0u : kSegGather) | (span ? kSegSpan : 0u) |
              (pair2a ? kSegPair2A : 0u) | (pair2b ? kSegPair2B : 0u) |
              (permuted ? kSegPermuted : 0u) |
              ((S.mode == ASMEVO_TOLERANCE && S.nan_policy == ASMEVO_NAN_STRICT) ? kSegStrict : 0u);
    if (D.rows > 1 || !unit || permuted) {   // only these segments read an extension
      D.nd_ext = n_ext++;
      ext.push_back(X);
    }
    if (D.flags & kSegNarrow) {
      D.tile_count = (D.rows * D.row_chunks + kTileChunks - 1) / kTileChunks;
    } else {
      const uint64_t tpr = (D.row_chunks + kTileChunks - 1) / kTileChunks;
      D.tile_count = D.rows * tpr;
    }
    tiles += D.tile_count;
  }
  // the kernel reads an extension exactly for these segments: it must exist
  for (int32_t k = 0; k < n; ++k) {
    const DiffSeg& D = dev[k];
    const bool needs = D.tile_count > 0 && (D.rows > 1 || (D.flags & (kSegGather | kSegPermuted)) != 0);
    if (needs && D.nd_ext >= ext.size()) return ASMEVO_E_INVALID;
  }
  return ASMEVO_OK;
}

// Cosine workspace: descriptors | one non-finite pair counter per segment |
// one block-sum record (kCosRec doubles) per tile | one record per level
// entry of the block trees | CosLevels per segment | for each level k >= 1,
// n + 1 group prefix counts.
struct CosPlan {
  size_t off_counters = 0, off_partials = 0, off_levels = 0, off_lv = 0, off_prefix = 0, bytes = 0;
  std::vector<CosLevels> lv;
  std::vector<uint64_t> prefix;         // (kCosLevels - 1) x (n + 1)
  uint64_t groups[kCosLevels] = {};     // groups per level (index 0 unused)
};

CosPlan cos_plan(const std::vector<DiffSeg>& dev, uint64_t tiles) {
  const size_t n = dev.size();
  CosPlan P;
  P.lv.assign(n, CosLevels{});
  P.prefix.assign((size_t)(kCosLevels - 1) * (n + 1), 0);
  uint64_t entries = 0;
  for (size_t s = 0; s < n; ++s) {
    CosLevels& L = P.lv[s];
    L.off[0] = dev[s].tile_begin;
    L.cnt[0] = is_float(dev[s].dtype) ? dev[s].tile_count : 0;   // integer segments store no block sums
    for (int k = 1; k < kCosLevels; ++k) {
      L.cnt[k] = L.cnt[k - 1] / 256;
      L.off[k] = entries;
      entries += L.cnt[k];
    }
  }
  for (int k = 1; k < kCosLevels; ++k) {
    uint64_t* pre = P.prefix.data() + (size_t)(k - 1) * (n + 1);
    for (size_t s = 0; s < n; ++s) pre[s + 1] = pre[s] + P.lv[s].cnt[k];
    P.groups[k] = pre[n];
  }
  P.off_counters = align256(n * sizeof(DiffSeg));
  P.off_partials = P.off_counters + align256(n * sizeof(uint64_t));
  P.off_levels = P.off_partials + align256((size_t)tiles * kCosRec * sizeof(double));
  P.off_lv = P.off_levels + align256((size_t)entries * kCosRec * sizeof(double));
  P.off_prefix = P.off_lv + align256(n * sizeof(CosLevels));
  P.bytes = P.off_prefix + P.prefix.size() * sizeof(uint64_t);
  return P;
}

// The cosine's tree units of an N-D pass: one per result, spanning the tiles
// of the result's segments, which must be consecutive in the array (so their
// tiles are) and of one element type.  A result without segments is an empty
// float unit (cosine 1.0 over no blocks).
asmevo_status cos_units(const std::vector<DiffSeg>& dev, int32_t n_results, std::vector<DiffSeg>& units) {
  units.assign((size_t)n_results, DiffSeg{});
  std::vector<int64_t> last((size_t)n_results, -1);
  for (int32_t r = 0; r < n_results; ++r) {
    std::memset(&units[r], 0, sizeof(DiffSeg));
    units[r].dtype = ASMEVO_F32;
    units[r].result_index = (uint32_t)r;
    units[r].rows = 1;
  }
  for (size_t k = 0; k < dev.size(); ++k) {
    const DiffSeg& D = dev[k];
    DiffSeg& U = units[D.result_index];
    if (last[D.result_index] < 0) {
      U.dtype = D.dtype;
      U.tile_begin = D.tile_begin;
    } else if (last[D.result_index] != (int64_t)k - 1 || U.dtype != D.dtype) {
      return ASMEVO_E_UNSUPPORTED;
    }
    U.tile_count += D.tile_count;
    U.cols += D.rows * D.cols;
    last[D.result_index] = (int64_t)k;
  }
  return ASMEVO_OK;
}

// Workspace of the N-D cosine pass: the cosine tables of the units (as for
// the 2-D pass, units in place of segments), then the segment descriptors and
// their extensions.
struct CosNdPlan {
  std::vector<DiffSeg> dev, units;
  std::vector<NdExt> ext;
  uint64_t tiles = 0;
  CosPlan cos;
  size_t off_segs = 0, off_ext = 0, bytes = 0;
};

asmevo_status cos_nd_plan(const asmevo_segment_nd* segs, int32_t n, int32_t n_results, CosNdPlan& P) {
  asmevo_status st = plan_diff_nd(segs, n, n_results, P.dev, P.ext, P.tiles, true);
  if (st != ASMEVO_OK) return st;
  st = cos_units(P.dev, n_results, P.units);
  if (st != ASMEVO_OK) return st;
  P.cos = cos_plan(P.units, P.tiles);
  for (const CosLevels& L : P.cos.lv)
    if (L.cnt[kCosLevels - 1] > 255) return ASMEVO_E_UNSUPPORTED;
  P.off_segs = align256(P.cos.bytes);
  P.off_ext = P.off_segs + align256(P.dev.size() * sizeof(DiffSeg));
  P.bytes = P.off_ext + P.ext.size() * sizeof(NdExt);
  return ASMEVO_OK;
}

}  // namespace

extern "C" {

asmevo_status asmevo_diff_segments_ex(const asmevo_segment* segs, int32_t n,
                                      asmevo_segment_result* results, void* workspace,
                                      size_t ws_bytes, void* stream, int32_t workgroups) {
  if (n < 0 || (n > 0 && (!segs || !results)) || workgroups < 0) return ASMEVO_E_INVALID;
  if (n == 0) return ASMEVO_OK;
  std::vector<DiffSeg> dev((size_t)n);
  uint64_t tiles = 0;
  asmevo_status st = plan_diff(segs, n, false, dev.data(), tiles);
  if (st != ASMEVO_OK) return st;
  const size_t bytes = dev.size() * sizeof(DiffSeg);
  if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(hipMemcpyAsync(workspace, dev.data(), bytes, hipMemcpyHostToDevice, s));
  int wg = workgroups;
  if (wg == 0) wg = diff_workgroups(dev.data(), n, tiles);
  HIP_TRY(launch_diff(reinterpret_cast<const DiffSeg*>(workspace), n, tiles, results, wg, s));
  return ASMEVO_OK;
}

asmevo_status asmevo_diff_segments(const asmevo_segment* segs, int32_t n,
                                   asmevo_segment_result* results, void* workspace,
                                   size_t ws_bytes, void* stream) {
  return asmevo_diff_segments_ex(segs, n, results, workspace, ws_bytes, stream, 0);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The diff for callers that cannot allocate: its descriptor table, the only
// scratch the plain diff uses, lives in a static device array instead of a
// workspace.  Each device holds its own copy of `scratch` until the process
// ends; host code never names the array itself (in host code it is a
// stand-in, not a device address) but the address that hipGetSymbolAddress
// gives for the current device, looked up on the first call on that device.
// The host-side table is planned into a static array too, under a mutex.
namespace {

__attribute__((used)) static __device__ __align__(256) DiffSeg scratch[ASMEVO_NOALLOC_MAX_SEGMENTS];

constexpr int kMaxDevices = 64;
std::atomic<uint64_t> g_scratch_addr[kMaxDevices];   // 0 until looked up
std::mutex g_noalloc_mutex;                          // guards g_noalloc_host
DiffSeg g_noalloc_host[ASMEVO_NOALLOC_MAX_SEGMENTS];

asmevo_status scratch_of_current_device(DiffSeg** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return ASMEVO_E_UNSUPPORTED;
  uint64_t a = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (a == 0) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return ASMEVO_E_HIP;
    a = reinterpret_cast<uint64_t>(p);
    g_scratch_addr[dev].store(a, std::memory_order_release);
  }
  *out = reinterpret_cast<DiffSeg*>(a);
  return ASMEVO_OK;
}

}  // namespace

extern "C" {

asmevo_status asmevo_diff_segments_noalloc(const asmevo_segment* segs, int32_t n,
                                           asmevo_segment_result* results, void* stream) {
  if (n < 0 || (n > 0 && (!segs || !results))) return ASMEVO_E_INVALID;
  if (n > ASMEVO_NOALLOC_MAX_SEGMENTS) return ASMEVO_E_CAPACITY;
  if (n == 0) return ASMEVO_OK;
  std::lock_guard<std::mutex> lock(g_noalloc_mutex);
  uint64_t tiles = 0;
  asmevo_status st = plan_diff(segs, n, false, g_noalloc_host, tiles);
  if (st != ASMEVO_OK) return st;
  DiffSeg* table = nullptr;
  st = scratch_of_current_device(&table);
  if (st != ASMEVO_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // pageable source: HIP has read it when the call returns, so the host
  // table may be planned again by the next call
  HIP_TRY(hipMemcpyAsync(table, g_noalloc_host, (size_t)n * sizeof(DiffSeg), hipMemcpyHostToDevice, s));
  HIP_TRY(launch_diff(table, n, tiles, results, diff_workgroups(g_noalloc_host, n, tiles), s));
  return ASMEVO_OK;
}

size_t asmevo_diff_nd_workspace_bytes(int32_t n) {
  const size_t m = n > 0 ? (size_t)n : 0;
  return align256(m * sizeof(DiffSeg)) + align256(m * sizeof(NdExt)) + 256;
}

asmevo_status asmevo_diff_segments_nd(const asmevo_segment_nd* segs, int32_t n,
                                      asmevo_segment_result* results, int32_t n_results,
                                      void* workspace, size_t ws_bytes, void* stream) {
  if (n < 0 || n_results < 0 || (n > 0 && !segs) || (n_results > 0 && !results)) return ASMEVO_E_INVALID;
  std::vector<DiffSeg> dev;
  std::vector<NdExt> ext;
  uint64_t tiles = 0;
  asmevo_status st = plan_diff_nd(segs, n, n_results, dev, ext, tiles);
  if (st != ASMEVO_OK) return st;
  if (n_results == 0) return ASMEVO_OK;
  const size_t off_ext = align256(dev.size() * sizeof(DiffSeg));
  const size_t bytes = off_ext + ext.size() * sizeof(NdExt);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  if (n > 0) {
    if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
    if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
    std::vector<uint8_t> host(bytes, 0);
    put(host, 0, dev);
    put(host, off_ext, ext);
    HIP_TRY(hipMemcpyAsync(ws, host.data(), bytes, hipMemcpyHostToDevice, s));
  }
  const int wg = nd_workgroups(dev, tiles);
  HIP_TRY(launch_diff_nd(reinterpret_cast<const DiffSeg*>(ws), reinterpret_cast<const NdExt*>(ws + off_ext),
                         n, n_results, tiles, results, wg, s));
  return ASMEVO_OK;
}

size_t asmevo_diff_cosine_workspace_bytes(const asmevo_segment* segs, int32_t n) {
  if (n <= 0 || !segs) return 0;
  std::vector<DiffSeg> dev((size_t)n);
  uint64_t tiles = 0;
  if (plan_diff(segs, n, true, dev.data(), tiles) != ASMEVO_OK) return 0;
  return cos_plan(dev, tiles).bytes;
}

asmevo_status asmevo_diff_cosine(const asmevo_segment* segs, int32_t n,
                                 asmevo_segment_result* results, asmevo_cosine_result* cos_results,
                                 void* workspace, size_t ws_bytes, void* stream) {
  if (n < 0 || (n > 0 && (!segs || !results || !cos_results))) return ASMEVO_E_INVALID;
  if (n == 0) return ASMEVO_OK;
  std::vector<DiffSeg> dev((size_t)n);
  uint64_t tiles = 0;
  asmevo_status st = plan_diff(segs, n, true, dev.data(), tiles);
  if (st != ASMEVO_OK) return st;
  const CosPlan P = cos_plan(dev, tiles);
  for (const CosLevels& L : P.lv)     // the final fold stages at most 255 entries per level
    if (L.cnt[kCosLevels - 1] > 255) return ASMEVO_E_UNSUPPORTED;
  if (!workspace || ws_bytes < P.bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  HIP_TRY(hipMemcpyAsync(ws, dev.data(), dev.size() * sizeof(DiffSeg), hipMemcpyHostToDevice, s));
  std::vector<uint8_t> tables(P.bytes - P.off_lv, 0);   // CosLevels | prefix counts, one upload
  std::memcpy(tables.data(), P.lv.data(), P.lv.size() * sizeof(CosLevels));
  std::memcpy(tables.data() + (P.off_prefix - P.off_lv), P.prefix.data(), P.prefix.size() * sizeof(uint64_t));
  HIP_TRY(hipMemcpyAsync(ws + P.off_lv, tables.data(), tables.size(), hipMemcpyHostToDevice, s));
  const int wg = device_cus() * cos_blocks_per_cu();   // the resident set
  HIP_TRY(launch_diff(reinterpret_cast<const DiffSeg*>(ws), n, tiles, results, wg, s,
                      reinterpret_cast<double*>(ws + P.off_partials),
                      reinterpret_cast<unsigned long long*>(ws + P.off_counters), cos_results,
                      reinterpret_cast<const CosLevels*>(ws + P.off_lv),
                      reinterpret_cast<const uint64_t*>(ws + P.off_prefix), P.groups,
                      reinterpret_cast<double*>(ws + P.off_levels)));
  return ASMEVO_OK;
}

size_t asmevo_diff_cosine_nd_workspace_bytes(const asmevo_segment_nd* segs, int32_t n, int32_t n_results) {
  if (n < 0 || n_results <= 0 || (n > 0 && !segs)) return 0;
  CosNdPlan P;
  if (cos_nd_plan(segs, n, n_results, P) != ASMEVO_OK) return 0;
  return P.bytes;
}

asmevo_status asmevo_diff_cosine_nd(const asmevo_segment_nd* segs, int32_t n, asmevo_segment_result* results,
                                    int32_t n_results, asmevo_cosine_result* cos_results, void* workspace,
                                    size_t ws_bytes, void* stream) {
  if (n < 0 || n_results < 0 || (n > 0 && !segs) || (n_results > 0 && (!results || !cos_results)))
    return ASMEVO_E_INVALID;
  CosNdPlan P;
  asmevo_status st = cos_nd_plan(segs, n, n_results, P);
  if (st != ASMEVO_OK) return st;
  if (n_results == 0) return ASMEVO_OK;
  if (!workspace || ws_bytes < P.bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  const CosPlan& C = P.cos;
  HIP_TRY(hipMemcpyAsync(ws, P.units.data(), P.units.size() * sizeof(DiffSeg), hipMemcpyHostToDevice, s));
  std::vector<uint8_t> tables(C.bytes - C.off_lv, 0);   // CosLevels | prefix counts
  std::memcpy(tables.data(), C.lv.data(), C.lv.size() * sizeof(CosLevels));
  std::memcpy(tables.data() + (C.off_prefix - C.off_lv), C.prefix.data(), C.prefix.size() * sizeof(uint64_t));
  HIP_TRY(hipMemcpyAsync(ws + C.off_lv, tables.data(), tables.size(), hipMemcpyHostToDevice, s));
  if (n > 0) {
    std::vector<uint8_t> host(P.bytes - P.off_segs, 0);  // descriptors | extensions
    put(host, 0, P.dev);
    put(host, P.off_ext - P.off_segs, P.ext);
    HIP_TRY(hipMemcpyAsync(ws + P.off_segs, host.data(), host.size(), hipMemcpyHostToDevice, s));
  }
  const int variant = cos_nd_variant(P.dev.data(), (int)P.dev.size());
  const int wg = device_cus() * (variant == kCosNdMixed ? cos_nd_blocks_per_cu() : split_cos_blocks_per_cu(variant));
  HIP_TRY(launch_diff_cosine_nd(reinterpret_cast<const DiffSeg*>(ws + P.off_segs),
                                reinterpret_cast<const NdExt*>(ws + P.off_ext), n,
                                reinterpret_cast<const DiffSeg*>(ws), n_results, P.tiles, results, wg, s,
                                reinterpret_cast<double*>(ws + C.off_partials),
                                reinterpret_cast<unsigned long long*>(ws + C.off_counters), cos_results,
                                reinterpret_cast<const CosLevels*>(ws + C.off_lv),
                                reinterpret_cast<const uint64_t*>(ws + C.off_prefix), C.groups,
                                reinterpret_cast<double*>(ws + C.off_levels), variant));
  return ASMEVO_OK;
}

// ---------------------------------------------------------------------------
asmevo_status asmevo_copy_regions(const asmevo_region* regions, int32_t n, void* workspace,
                                  size_t ws_bytes, void* stream) {
  if (n < 0 || (n > 0 && !regions)) return ASMEVO_E_INVALID;
  if (n == 0) return ASMEVO_OK;
  std::vector<CopyRegion> dev((size_t)n);
  std::vector<std::pair<uint64_t, uint64_t>> dsts, srcs;
  uint64_t tiles = 0;
  const uint64_t tile_bytes = (uint64_t)kTileChunks * kChunk;
  for (int32_t k = 0; k < n; ++k) {
    const asmevo_region& R = regions[k];
    CopyRegion& C = dev[k];
    std::memset(&C, 0, sizeof(C));
    C.tile_begin = tiles;
    if (R.bytes == 0) continue;
    if (!R.dst || !R.src || R.bytes > (1ull << 52)) return ASMEVO_E_INVALID;
    if (R.dst + R.bytes < R.dst || R.src + R.bytes < R.src) return ASMEVO_E_INVALID;
    if (R.dst < R.src + R.bytes && R.src < R.dst + R.bytes) return ASMEVO_E_INVALID;   // memcpy semantics
    dsts.emplace_back(R.dst, R.dst + R.bytes);
    srcs.emplace_back(R.src, R.src + R.bytes);
    C.dst = R.dst;
    C.src = R.src;
    C.bytes = R.bytes;
    C.vec = (R.dst % kChunk) == (R.src % kChunk);
    if (C.vec) {
      const uint64_t head = (kChunk - R.src % kChunk) % kChunk;
      C.head = head < R.bytes ? head : R.bytes;
      C.body_bytes = R.bytes - C.head;
      const uint64_t body_chunks = C.body_bytes / kChunk;
      C.tile_count = std::max<uint64_t>(1, (body_chunks + kTileChunks - 1) / kTileChunks);
    } else {
      C.tile_count = (R.bytes + tile_bytes - 1) / tile_bytes;
    }
    tiles += C.tile_count;
  }
  // destinations pairwise disjoint, and disjoint from every source
  std::sort(dsts.begin(), dsts.end());
  for (size_t i = 1; i < dsts.size(); ++i)
    if (dsts[i].first < dsts[i - 1].second) return ASMEVO_E_INVALID;
  for (const auto& sr : srcs) {
    auto it = std::lower_bound(dsts.begin(), dsts.end(), std::make_pair(sr.second, (uint64_t)0));
    if (it != dsts.begin() && std::prev(it)->second > sr.first) return ASMEVO_E_INVALID;
  }
  const size_t bytes = dev.size() * sizeof(CopyRegion);
  if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(hipMemcpyAsync(workspace, dev.data(), bytes, hipMemcpyHostToDevice, s));
  // two workgroups per CU, each streaming one range with its four waves: of
  // 1-8 workgroups per CU and 1-4 waves per range, the fastest on the 64 GiB
  // restore (by 2-9 %, on allocations where the copy is not bound elsewhere)
  HIP_TRY(launch_copy(reinterpret_cast<const CopyRegion*>(workspace), n, tiles, device_cus() * 2, s));
  return ASMEVO_OK;
}

// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

// Validates the allocations and builds the guard regions: each guard side,
// and the row padding of a strided allocation as one region of runs.
asmevo_status plan_guard(const asmevo_alloc* allocs, int32_t n, std::vector<GuardRegion>& regs,
                         uint64_t& chunks) {
  regs.clear();
  chunks = 0;
  for (int32_t k = 0; k < n; ++k) {
    const asmevo_alloc& A = allocs[k];
    asmevo_status st = check_alloc_geometry(A);
    if (st != ASMEVO_OK) return st;
    if ((A.guard_lo > 0 || A.guard_hi > 0) && A.base == 0) return ASMEVO_E_INVALID;
    const uint64_t D = data_bytes(A);
    for (uint32_t side = 0; side < 2; ++side) {
      const uint64_t g = (uint64_t)(side ? A.guard_hi : A.guard_lo);
      if (g == 0) continue;
      GuardRegion R;
      std::memset(&R, 0, sizeof(R));
      R.addr = side ? A.base + (uint64_t)A.guard_lo + D : A.base;
      R.bytes = g;
      R.chunk_begin = chunks;
      R.alloc_id = A.alloc_id;
      R.side = side;
      R.result_index = (uint32_t)k;
      regs.push_back(R);
      chunks += (g + kChunk - 1) / kChunk;
    }
    if (A.rows >= 2 && A.cols > 0 && A.stride > A.cols) {   // row padding: interior guards
      if (A.base == 0) return ASMEVO_E_INVALID;
      const uint64_t es = (uint64_t)esize_of(A.dtype);
      GuardRegion R;
      std::memset(&R, 0, sizeof(R));
      R.addr = A.base + (uint64_t)A.guard_lo;
      R.bytes = (uint64_t)(A.stride - A.cols) * es;
      R.chunk_begin = chunks;
      R.pitch = (uint64_t)A.stride * es;
      R.pad_off = (uint64_t)A.cols * es;
      R.run_chunks = (R.bytes + kChunk - 1) / kChunk;
      R.alloc_id = A.alloc_id;
      R.side = 2;
      R.result_index = (uint32_t)k;
      regs.push_back(R);
      chunks += (uint64_t)(A.rows - 1) * R.run_chunks;
    }
  }
  return ASMEVO_OK;
}

}  // namespace

extern "C" {

asmevo_status asmevo_guard_check(const asmevo_alloc* allocs, int32_t n, uint64_t seed,
                                 asmevo_guard_result* results, void* workspace, size_t ws_bytes,
                                 void* stream) {
  if (n < 0 || (n > 0 && (!allocs || !results))) return ASMEVO_E_INVALID;
  if (n > (1 << 29)) return ASMEVO_E_INVALID;   // result index and guard side share a 32-bit key
  if (n == 0) return ASMEVO_OK;
  std::vector<GuardRegion> regs;
  uint64_t chunks = 0;
  asmevo_status st = plan_guard(allocs, n, regs, chunks);
  if (st != ASMEVO_OK) return st;
  const size_t bytes = std::max<size_t>(regs.size(), 1) * sizeof(GuardRegion);
  if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
  if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!regs.empty())
    HIP_TRY(hipMemcpyAsync(workspace, regs.data(), regs.size() * sizeof(GuardRegion),
                           hipMemcpyHostToDevice, s));
  HIP_TRY(launch_guard(reinterpret_cast<const GuardRegion*>(workspace), (int)regs.size(), chunks,
                       seed, results, n, s));
  return ASMEVO_OK;
}

// ---------------------------------------------------------------------------
// Staged plans: the descriptor table of a diff or guard check is planned and
// uploaded once, then launched as often as the check is repeated.

size_t asmevo_plan_bytes(int32_t n_descs) {
  const size_t n = n_descs > 0 ? (size_t)n_descs : 0;
  // the largest table: N-D segments with extensions, or up to 3 guard regions per allocation
  return align256(std::max(n * sizeof(DiffSeg), 3 * n * sizeof(GuardRegion))) + align256(n * sizeof(NdExt)) + 256;
}

asmevo_status asmevo_plan_diff(const asmevo_segment* segs, int32_t n, void* workspace, size_t ws_bytes,
                               void* stream, asmevo_plan* plan) {
  if (!plan || n < 0 || (n > 0 && !segs)) return ASMEVO_E_INVALID;
  std::vector<DiffSeg> dev((size_t)n);
  uint64_t tiles = 0;
  asmevo_status st = plan_diff(segs, n, false, dev.data(), tiles);
  if (st != ASMEVO_OK) return st;
  const size_t bytes = dev.size() * sizeof(DiffSeg);
  if (n > 0) {
    if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
    if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
    HIP_TRY(hipMemcpyAsync(workspace, dev.data(), bytes, hipMemcpyHostToDevice,
                           reinterpret_cast<hipStream_t>(stream)));
  }
  std::memset(plan, 0, sizeof(*plan));
  plan->table = reinterpret_cast<uint64_t>(workspace);
  plan->units = tiles;
  plan->n = n;
  plan->n_results = n;
  plan->kind = ASMEVO_PLAN_DIFF;
  plan->workgroups = diff_workgroups(dev.data(), n, tiles);
  return ASMEVO_OK;
}

asmevo_status asmevo_plan_diff_nd(const asmevo_segment_nd* segs, int32_t n, int32_t n_results, void* workspace,
                                  size_t ws_bytes, void* stream, asmevo_plan* plan) {
  if (!plan || n < 0 || n_results < 0 || (n > 0 && !segs)) return ASMEVO_E_INVALID;
  std::vector<DiffSeg> dev;
  std::vector<NdExt> ext;
  uint64_t tiles = 0;
  asmevo_status st = plan_diff_nd(segs, n, n_results, dev, ext, tiles);
  if (st != ASMEVO_OK) return st;
  const size_t off_ext = align256(dev.size() * sizeof(DiffSeg));
  const size_t bytes = off_ext + ext.size() * sizeof(NdExt);
  if (n > 0) {
    if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
    if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
    std::vector<uint8_t> host(bytes, 0);
    put(host, 0, dev);
    put(host, off_ext, ext);
    HIP_TRY(hipMemcpyAsync(workspace, host.data(), bytes, hipMemcpyHostToDevice,
                           reinterpret_cast<hipStream_t>(stream)));
  }
  std::memset(plan, 0, sizeof(*plan));
  plan->table = reinterpret_cast<uint64_t>(workspace);
  plan->units = tiles;
  plan->n = n;
  plan->n_results = n_results;
  plan->kind = ASMEVO_PLAN_DIFF_ND;
  plan->workgroups = nd_workgroups(dev, tiles);
  return ASMEVO_OK;
}

asmevo_status asmevo_diff_planned(const asmevo_plan* plan, asmevo_segment_result* results, void* stream) {
  if (!plan || plan->n < 0 || plan->n_results < 0) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (plan->kind == ASMEVO_PLAN_DIFF) {
    if (plan->n != plan->n_results || (plan->n > 0 && (!results || !plan->table))) return ASMEVO_E_INVALID;
    if (plan->n == 0) return ASMEVO_OK;
    HIP_TRY(launch_diff(reinterpret_cast<const DiffSeg*>(plan->table), plan->n, plan->units, results,
                        plan->workgroups, s));
    return ASMEVO_OK;
  }
  if (plan->kind == ASMEVO_PLAN_DIFF_ND) {
    if ((plan->n_results > 0 && !results) || (plan->n > 0 && !plan->table)) return ASMEVO_E_INVALID;
    if (plan->n_results == 0) return ASMEVO_OK;
    const uint8_t* ws = reinterpret_cast<const uint8_t*>(plan->table);
    const size_t off_ext = align256((size_t)plan->n * sizeof(DiffSeg));
    HIP_TRY(launch_diff_nd(reinterpret_cast<const DiffSeg*>(ws), reinterpret_cast<const NdExt*>(ws + off_ext),
                           plan->n, plan->n_results, plan->units, results, plan->workgroups, s));
    return ASMEVO_OK;
  }
  return ASMEVO_E_INVALID;
}

asmevo_status asmevo_plan_guard(const asmevo_alloc* allocs, int32_t n, void* workspace, size_t ws_bytes,
                                void* stream, asmevo_plan* plan) {
  if (!plan || n < 0 || (n > 0 && !allocs)) return ASMEVO_E_INVALID;
  if (n > (1 << 29)) return ASMEVO_E_INVALID;
  std::vector<GuardRegion> regs;
  uint64_t chunks = 0;
  asmevo_status st = plan_guard(allocs, n, regs, chunks);
  if (st != ASMEVO_OK) return st;
  const size_t bytes = regs.size() * sizeof(GuardRegion);
  if (!regs.empty()) {
    if (!workspace || ws_bytes < bytes) return ASMEVO_E_WORKSPACE;
    if (!ws_aligned(workspace)) return ASMEVO_E_INVALID;
    HIP_TRY(hipMemcpyAsync(workspace, regs.data(), bytes, hipMemcpyHostToDevice,
                           reinterpret_cast<hipStream_t>(stream)));
  }
  std::memset(plan, 0, sizeof(*plan));
  plan->table = reinterpret_cast<uint64_t>(workspace);
  plan->units = chunks;
  plan->n = (int32_t)regs.size();
  plan->n_results = n;
  plan->kind = ASMEVO_PLAN_GUARD;
  return ASMEVO_OK;
}

asmevo_status asmevo_guard_planned(const asmevo_plan* plan, uint64_t seed, asmevo_guard_result* results,
                                   void* stream) {
  if (!plan || plan->kind != ASMEVO_PLAN_GUARD || plan->n < 0 || plan->n_results < 0 ||
      (plan->n_results > 0 && !results) || (plan->n > 0 && !plan->table))
    return ASMEVO_E_INVALID;
  if (plan->n_results == 0) return ASMEVO_OK;
  HIP_TRY(launch_guard(reinterpret_cast<const GuardRegion*>(plan->table), plan->n, plan->units, seed, results,
                       plan->n_results, reinterpret_cast<hipStream_t>(stream)));
  return ASMEVO_OK;
}

// ---------------------------------------------------------------------------
// Code objects: the kernel under test and its candidates are built into code
// objects and run under the same launch (section 3.7, Algorithm 1).
asmevo_status asmevo_kernel_load(const void* image, size_t image_bytes, const char* name,
                                 asmevo_kernel* out) {
  if (!image || image_bytes == 0 || !name || !out) return ASMEVO_E_INVALID;
  std::memset(out, 0, sizeof(*out));
  hipModule_t mod = nullptr;
  HIP_TRY(hipModuleLoadData(&mod, image));
  hipFunction_t fn = nullptr;
  hipError_t e = hipModuleGetFunction(&fn, mod, name);
  if (e != hipSuccess) {
    g_last_hip = (int32_t)e;
    (void)hipModuleUnload(mod);
    return ASMEVO_E_HIP;
  }
  int regs = 0, shared = 0, threads = 0, local = 0;
  (void)hipFuncGetAttribute(&regs, HIP_FUNC_ATTRIBUTE_NUM_REGS, fn);
  (void)hipFuncGetAttribute(&shared, HIP_FUNC_ATTRIBUTE_SHARED_SIZE_BYTES, fn);
  (void)hipFuncGetAttribute(&threads, HIP_FUNC_ATTRIBUTE_MAX_THREADS_PER_BLOCK, fn);
  (void)hipFuncGetAttribute(&local, HIP_FUNC_ATTRIBUTE_LOCAL_SIZE_BYTES, fn);
  out->module = reinterpret_cast<uint64_t>(mod);
  out->function = reinterpret_cast<uint64_t>(fn);
  out->num_regs = regs;
  out->shared_bytes = shared;
  out->max_threads = threads;
  out->local_bytes = local;
  return ASMEVO_OK;
}

asmevo_status asmevo_kernel_unload(asmevo_kernel* k) {
  if (!k) return ASMEVO_E_INVALID;
  if (k->module) HIP_TRY(hipModuleUnload(reinterpret_cast<hipModule_t>(k->module)));
  k->module = 0;
  k->function = 0;
  return ASMEVO_OK;
}

namespace {
asmevo_status check_launch(const asmevo_kernel* k, const uint32_t grid[3], const uint32_t block[3],
                           void** params) {
  if (!k || !k->function || !grid || !block || !params) return ASMEVO_E_INVALID;
  for (int d = 0; d < 3; ++d)
    if (grid[d] == 0 || block[d] == 0) return ASMEVO_E_INVALID;
  const uint64_t threads = (uint64_t)block[0] * block[1] * block[2];
  if (k->max_threads > 0 && threads > (uint64_t)k->max_threads) return ASMEVO_E_INVALID;
  return ASMEVO_OK;
}
}  // namespace

asmevo_status asmevo_kernel_launch(const asmevo_kernel* k, const uint32_t grid[3], const uint32_t block[3],
                                   uint32_t lds_bytes, void** params, void* stream) {
  asmevo_status st = check_launch(k, grid, block, params);
  if (st != ASMEVO_OK) return st;
  HIP_TRY(hipModuleLaunchKernel(reinterpret_cast<hipFunction_t>(k->function), grid[0], grid[1], grid[2],
                                block[0], block[1], block[2], lds_bytes,
                                reinterpret_cast<hipStream_t>(stream), params, nullptr));
  return ASMEVO_OK;
}

asmevo_status asmevo_kernel_time(const asmevo_kernel* k, const uint32_t grid[3], const uint32_t block[3],
                                 uint32_t lds_bytes, void** params, int32_t warmup, int32_t reps,
                                 float* ms_out, void* stream) {
  asmevo_status st = check_launch(k, grid, block, params);
  if (st != ASMEVO_OK) return st;
  if (warmup < 0 || reps <= 0 || !ms_out) return ASMEVO_E_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipFunction_t fn = reinterpret_cast<hipFunction_t>(k->function);
  for (int32_t w = 0; w < warmup; ++w)
    HIP_TRY(hipModuleLaunchKernel(fn, grid[0], grid[1], grid[2], block[0], block[1], block[2], lds_bytes, s,
                                  params, nullptr));
  std::vector<hipEvent_t> ev(2 * (size_t)reps, nullptr);
  asmevo_status result = ASMEVO_OK;
  for (auto& e : ev) {
    const hipError_t c = hipEventCreate(&e);
    if (c != hipSuccess) {
      e = nullptr;
      g_last_hip = (int32_t)c;
      result = ASMEVO_E_HIP;
    }
  }
  for (int32_t r = 0; r < reps && result == ASMEVO_OK; ++r) {
    hipError_t e = hipEventRecord(ev[2 * r], s);
    if (e == hipSuccess)
      e = hipModuleLaunchKernel(fn, grid[0], grid[1], grid[2], block[0], block[1], block[2], lds_bytes, s,
                                params, nullptr);
    if (e == hipSuccess) e = hipEventRecord(ev[2 * r + 1], s);
    if (e != hipSuccess) {
      g_last_hip = (int32_t)e;
      result = ASMEVO_E_HIP;
    }
  }
  if (result == ASMEVO_OK) {
    const hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      g_last_hip = (int32_t)e;
      result = ASMEVO_E_HIP;
    }
  }
  for (int32_t r = 0; r < reps && result == ASMEVO_OK; ++r) {
    const hipError_t e = hipEventElapsedTime(&ms_out[r], ev[2 * r], ev[2 * r + 1]);
    if (e != hipSuccess) {
      g_last_hip = (int32_t)e;
      result = ASMEVO_E_HIP;
    }
  }
  for (auto& e : ev)
    if (e) (void)hipEventDestroy(e);
  return result;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Device memory at chosen virtual addresses (Tier-2 replay of captured state).

namespace {

struct VaRange {
  uint64_t bytes;
  hipMemGenericAllocationHandle_t handle;
};
std::mutex g_va_mutex;
std::map<uint64_t, VaRange> g_va;   // live ranges of this process, by start address

hipMemAllocationProp va_prop(int dev) {
  hipMemAllocationProp prop;
  std::memset(&prop, 0, sizeof(prop));
  prop.type = hipMemAllocationTypePinned;
  prop.location.type = hipMemLocationTypeDevice;
  prop.location.id = dev;
  return prop;
}

size_t va_granularity_of(int dev) {
  int vmm = 0;
  if (hipDeviceGetAttribute(&vmm, hipDeviceAttributeVirtualMemoryManagementSupported, dev) != hipSuccess || !vmm)
    return 0;
  const hipMemAllocationProp prop = va_prop(dev);
  size_t gran = 0;
  if (hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityMinimum) != hipSuccess) return 0;
  return gran;
}

}  // namespace

extern "C" {

size_t asmevo_va_granularity(void) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  return va_granularity_of(dev);
}

asmevo_status asmevo_va_alloc(uint64_t addr, uint64_t bytes, uint64_t* out) {
  if (!out || bytes == 0) return ASMEVO_E_INVALID;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  const size_t gran = va_granularity_of(dev);
  if (gran == 0) return ASMEVO_E_UNSUPPORTED;
  if (bytes % gran != 0 || addr % gran != 0) return ASMEVO_E_INVALID;
  const hipMemAllocationProp prop = va_prop(dev);
  void* p = nullptr;
  const hipError_t er = hipMemAddressReserve(&p, (size_t)bytes, gran, reinterpret_cast<void*>(addr), 0);
  if (er != hipSuccess) {
    g_last_hip = (int32_t)er;
    return addr != 0 ? ASMEVO_E_UNSUPPORTED : ASMEVO_E_HIP;
  }
  if (addr != 0 && reinterpret_cast<uint64_t>(p) != addr) {
    (void)hipMemAddressFree(p, (size_t)bytes);
    return ASMEVO_E_UNSUPPORTED;
  }
  hipMemGenericAllocationHandle_t h;
  hipError_t e = hipMemCreate(&h, (size_t)bytes, &prop, 0);
  if (e != hipSuccess) {
    (void)hipMemAddressFree(p, (size_t)bytes);
    g_last_hip = (int32_t)e;
    return ASMEVO_E_HIP;
  }
  e = hipMemMap(p, (size_t)bytes, 0, h, 0);
  if (e == hipSuccess) {
    hipMemAccessDesc acc;
    std::memset(&acc, 0, sizeof(acc));
    acc.location = prop.location;
    acc.flags = hipMemAccessFlagsProtReadWrite;
    e = hipMemSetAccess(p, (size_t)bytes, &acc, 1);
    if (e != hipSuccess) (void)hipMemUnmap(p, (size_t)bytes);
  }
  if (e != hipSuccess) {
    (void)hipMemRelease(h);
    (void)hipMemAddressFree(p, (size_t)bytes);
    g_last_hip = (int32_t)e;
    // a requested address the driver reserved but cannot map lies outside the
    // device's aperture
    return addr != 0 ? ASMEVO_E_UNSUPPORTED : ASMEVO_E_HIP;
  }
  {
    std::lock_guard<std::mutex> lock(g_va_mutex);
    g_va[reinterpret_cast<uint64_t>(p)] = VaRange{bytes, h};
  }
  *out = reinterpret_cast<uint64_t>(p);
  return ASMEVO_OK;
}

asmevo_status asmevo_va_free(uint64_t addr) {
  std::lock_guard<std::mutex> lock(g_va_mutex);
  auto it = g_va.find(addr);
  if (it == g_va.end()) return ASMEVO_E_INVALID;
  void* p = reinterpret_cast<void*>(addr);
  const VaRange r = it->second;
  HIP_TRY(hipMemUnmap(p, (size_t)r.bytes));
  g_va.erase(it);                       // unmapped: the range is no longer usable
  HIP_TRY(hipMemRelease(r.handle));
  HIP_TRY(hipMemAddressFree(p, (size_t)r.bytes));
  return ASMEVO_OK;
}

}  // extern "C"
