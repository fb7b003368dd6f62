// k0_rmsnorm.hip -- the original kernel K0 whose compiled code object the
// gated verification harness evaluates candidates against (AsmEvo section
// 3.7, Algorithm 1).  A fused residual add + RMS normalisation with a
// per-row argmax, the shape of a decode-time normalisation kernel:
//
//   h        = bf16(x + residual)                  (res_out, bf16)
//   rstd     = 1 / sqrt(mean(h^2) + eps)            (rstd, fp32, one per row)
//   out      = h * rstd * weight                    (out, fp32)
//   amax     = the lowest index of max |h| in the row (amax, int32)
//
// One workgroup of 256 threads per row.  This is the straightforward
// version: each thread walks its own contiguous run of hidden / 256 elements
// with 2-byte loads, so the lanes of a wave touch addresses 2 * hidden / 256
// bytes apart.  Requires hidden to be a multiple of 256.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
constexpr float kEps = 1e-5f;

__device__ __forceinline__ float bf16_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f32_bf16(float f) {   // round to nearest even; NaN stays NaN
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

}  // namespace

extern "C" __global__ __launch_bounds__(kBlock) void rmsnorm_k0(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ residual,
    const uint16_t* __restrict__ weight, float* __restrict__ out, uint16_t* __restrict__ res_out,
    float* __restrict__ rstd, int32_t* __restrict__ amax, int hidden, int in_stride, int out_stride) {
  __shared__ float s_sum[kBlock];
  __shared__ float s_best[kBlock];
  __shared__ int s_idx[kBlock];
  const int row = blockIdx.x;
  const int t = threadIdx.x;
  const int per = hidden / kBlock;
  const size_t in_off = (size_t)row * in_stride;
  const size_t out_off = (size_t)row * out_stride;
  float ss = 0.0f, best = -1.0f;
  int bi = 0;
  for (int k = 0; k < per; ++k) {
    const int i = t * per + k;
    const uint16_t hb = f32_bf16(bf16_f32(x[in_off + i]) + bf16_f32(residual[in_off + i]));
    res_out[in_off + i] = hb;
    const float h = bf16_f32(hb);
    ss += h * h;
    const float a = fabsf(h);
    if (a > best) {
      best = a;
      bi = i;
    }
  }
  s_sum[t] = ss;
  s_best[t] = best;
  s_idx[t] = bi;
  __syncthreads();
  for (int s = kBlock / 2; s > 0; s >>= 1) {
    if (t < s) {
      s_sum[t] += s_sum[t + s];
      const float ob = s_best[t + s];
      const int oi = s_idx[t + s];
      if (ob > s_best[t] || (ob == s_best[t] && oi < s_idx[t])) {
        s_best[t] = ob;
        s_idx[t] = oi;
      }
    }
    __syncthreads();
  }
  const float r = 1.0f / sqrtf(s_sum[0] / (float)hidden + kEps);
  if (t == 0) {
    rstd[row] = r;
    amax[row] = s_idx[0];
  }
  for (int k = 0; k < per; ++k) {
    const int i = t * per + k;
    const float h = bf16_f32(res_out[in_off + i]);
    out[out_off + i] = h * r * bf16_f32(weight[i]);
  }
}
