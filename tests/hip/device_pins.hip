// device_pins.hip -- test-only kernels that run the library's per-element
// device functions over large input sets, so that the tests can compare every
// output, bit for bit, with the CPU oracle:
//  * the fill's encoder from binary32 to each element type (encode_f32);
//  * the fill's normal transform: log_u, sincos_turns and box_muller;
//  * the comparison's rule for one pair of elements (pair_slow), whose fp64
//    quantities include the division |A - B| / |B|.
// Built from the library's own headers into a library of its own; nothing in
// the product loads it.
#include "device_math.h"
#include "pair_rule.h"

using namespace asmevo;

namespace {

constexpr int kThreads = 256;
constexpr uint64_t kMaxBlocks = 8192;

__device__ __forceinline__ uint64_t first_index() { return blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; }
__device__ __forceinline__ uint64_t grid_stride() { return (uint64_t)gridDim.x * blockDim.x; }

__global__ void __launch_bounds__(kThreads) encode_kernel(uint32_t x0, uint64_t n, uint16_t* bf16, uint16_t* f16,
                                                          uint8_t* fp8_sat, uint8_t* fp8) {
  for (uint64_t i = first_index(); i < n; i += grid_stride()) {
    const float f = __uint_as_float((uint32_t)(x0 + i));
    bf16[i] = (uint16_t)encode_f32(ASMEVO_BF16, f, false);
    f16[i] = (uint16_t)encode_f32(ASMEVO_F16, f, false);
    fp8_sat[i] = (uint8_t)encode_f32(ASMEVO_FP8_E4M3, f, true);
    fp8[i] = (uint8_t)encode_f32(ASMEVO_FP8_E4M3, f, false);
  }
}

__global__ void __launch_bounds__(kThreads) log_kernel(uint32_t x0, uint64_t n, double* out) {
  for (uint64_t i = first_index(); i < n; i += grid_stride()) out[i] = log_u((uint32_t)(x0 + i));
}

__global__ void __launch_bounds__(kThreads) sincos_kernel(uint32_t x0, uint64_t n, double* c, double* s) {
  for (uint64_t i = first_index(); i < n; i += grid_stride()) {
    double cv, sv;
    sincos_turns((uint32_t)(x0 + i), cv, sv);
    c[i] = cv;
    s[i] = sv;
  }
}

__global__ void __launch_bounds__(kThreads) normal_kernel(const uint32_t* xa, const uint32_t* xb, uint64_t n,
                                                          double* z0, double* z1) {
  for (uint64_t i = first_index(); i < n; i += grid_stride()) {
    double a, b;
    box_muller(xa[i], xb[i], a, b);
    z0[i] = a;
    z1[i] = b;
  }
}

// Each pair on its own: a lane's partials reset, then the pair added.
template <int DT>
__global__ void __launch_bounds__(kThreads) pair_kernel(const uint32_t* ra, const uint32_t* rb, uint64_t n,
                                                        bool strict, double atol, double rtol, uint8_t* flags,
                                                        uint64_t* max_abs, uint64_t* max_rel) {
  for (uint64_t i = first_index(); i < n; i += grid_stride()) {
    Acc acc;
    acc_reset(acc);
    pair_slow<DT>(ra[i], rb[i], 0, true, strict, atol, rtol, acc);
    flags[i] = (uint8_t)((acc.bw ? 1u : 0u) | (acc.tol ? 2u : 0u) | (acc.nf ? 4u : 0u));
    max_abs[i] = acc.max_abs;
    max_rel[i] = acc.max_rel;
  }
}

unsigned blocks_for(uint64_t n) {
  const uint64_t b = (n + kThreads - 1) / kThreads;
  return (unsigned)(b < kMaxBlocks ? b : kMaxBlocks);
}

int launched() { return (int)hipGetLastError(); }

struct PairArgs {
  const uint32_t* ra;
  const uint32_t* rb;
  uint64_t n;
  bool strict;
  double atol, rtol;
  uint8_t* flags;
  uint64_t* max_abs;
  uint64_t* max_rel;
};

template <int DT>
int launch_pairs(const PairArgs& p, hipStream_t s) {
  hipLaunchKernelGGL(pair_kernel<DT>, dim3(blocks_for(p.n)), dim3(kThreads), 0, s, p.ra, p.rb, p.n, p.strict,
                     p.atol, p.rtol, p.flags, p.max_abs, p.max_rel);
  return launched();
}

}  // namespace

// Every entry point: n outputs (or pairs) written to device arrays of n
// elements each, on the given stream; returns a hipError_t value, or -1 for
// an unknown element type.
extern "C" {

int pins_encode(uint32_t x0, uint64_t n, void* bf16, void* f16, void* fp8_sat, void* fp8, void* stream) {
  if (n == 0) return 0;
  hipLaunchKernelGGL(encode_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, (hipStream_t)stream, x0, n,
                     (uint16_t*)bf16, (uint16_t*)f16, (uint8_t*)fp8_sat, (uint8_t*)fp8);
  return launched();
}

int pins_log_u(uint32_t x0, uint64_t n, void* out, void* stream) {
  if (n == 0) return 0;
  hipLaunchKernelGGL(log_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, (hipStream_t)stream, x0, n,
                     (double*)out);
  return launched();
}

int pins_sincos(uint32_t x0, uint64_t n, void* c, void* s, void* stream) {
  if (n == 0) return 0;
  hipLaunchKernelGGL(sincos_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, (hipStream_t)stream, x0, n,
                     (double*)c, (double*)s);
  return launched();
}

int pins_normal(const void* xa, const void* xb, uint64_t n, void* z0, void* z1, void* stream) {
  if (n == 0) return 0;
  hipLaunchKernelGGL(normal_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, (hipStream_t)stream,
                     (const uint32_t*)xa, (const uint32_t*)xb, n, (double*)z0, (double*)z1);
  return launched();
}

int pins_pairs(int32_t dtype, int32_t strict, double atol, double rtol, const void* ra, const void* rb, uint64_t n,
               void* flags, void* max_abs, void* max_rel, void* stream) {
  if (n == 0) return 0;
  const PairArgs p{(const uint32_t*)ra, (const uint32_t*)rb, n, strict != 0, atol, rtol,
                   (uint8_t*)flags, (uint64_t*)max_abs, (uint64_t*)max_rel};
  switch (dtype) {
    case ASMEVO_F32: return launch_pairs<ASMEVO_F32>(p, (hipStream_t)stream);
    case ASMEVO_BF16: return launch_pairs<ASMEVO_BF16>(p, (hipStream_t)stream);
    case ASMEVO_F16: return launch_pairs<ASMEVO_F16>(p, (hipStream_t)stream);
    case ASMEVO_FP8_E4M3: return launch_pairs<ASMEVO_FP8_E4M3>(p, (hipStream_t)stream);
    default: return -1;
  }
}

}  // extern "C"
