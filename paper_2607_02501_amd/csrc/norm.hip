// norm.hip -- the RMS-normalisation prologue for projections on the MFMA
// path (paper section 3.2, operator fusion; the decoder backbones of section
// 2.1 normalise the residual stream before their attention and feed-forward
// projections).  The MFMA kernels copy activation tiles straight from memory
// into LDS, so the normalised activations are written once, in the 16-bit
// type the product consumes, by this row kernel; the GEMV path normalises
// while it stages x instead (gemv.hip).
//
//   x_hat[i][j] = round_xt(h[i][j] * g[j] * r_i),  r_i = 1 / sqrt(eps + mean_j h[i][j]^2)
//
// One workgroup of 256 threads per row: each thread sums the squares of its
// float4 columns j = t, t + 256, ... in fp32, the 64 lanes of a wave and then
// the four waves are added in a fixed order, and the same threads write their
// columns.  HBM traffic: 4 k bytes read and 2 k written per row (the weights g
// stay in cache).
#include <hip/hip_runtime.h>

#include "eb_internal.h"

namespace eb {
namespace {

constexpr int kThreads = 256;

template <int XT>
__device__ inline uint32_t pack2(float a, float b) {
  if (XT == EB_F16)
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) |
           ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)b) << 16);
}

template <int XT>
__global__ void __launch_bounds__(kThreads)
    rmsnorm_kernel(const float *__restrict__ h, const float *__restrict__ g, float eps, int64_t k,
                   uint32_t *__restrict__ out) {
  __shared__ float red[kThreads / 64];
  const int64_t row = blockIdx.x;
  const float4 *src = reinterpret_cast<const float4 *>(h + row * k);
  const float4 *gs = reinterpret_cast<const float4 *>(g);
  const int64_t k4 = k / 4;
  float ss = 0.f;
  for (int64_t i = threadIdx.x; i < k4; i += kThreads) {
    const float4 v = src[i];
    ss = __builtin_fmaf(v.x, v.x, ss);
    ss = __builtin_fmaf(v.y, v.y, ss);
    ss = __builtin_fmaf(v.z, v.z, ss);
    ss = __builtin_fmaf(v.w, v.w, ss);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) tot += red[w];
  const float r = 1.0f / __builtin_sqrtf(tot / (float)k + eps);
  uint2 *dst = reinterpret_cast<uint2 *>(out + row * (k / 2));
  for (int64_t i = threadIdx.x; i < k4; i += kThreads) {
    const float4 v = src[i], w = gs[i];
    dst[i] = make_uint2(pack2<XT>(v.x * w.x * r, v.y * w.y * r), pack2<XT>(v.z * w.z * r, v.w * w.w * r));
  }
}

}  // namespace

hipError_t launch_rmsnorm(const float *h, const float *gamma, float eps, int64_t m, int64_t k,
                          int32_t xt, void *out, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  if (m > 0x7fffffff || k % 4 != 0) return hipErrorInvalidValue;
  if (xt == EB_F16)
    rmsnorm_kernel<EB_F16><<<(unsigned)m, kThreads, 0, s>>>(h, gamma, eps, k, static_cast<uint32_t *>(out));
  else
    rmsnorm_kernel<EB_BF16><<<(unsigned)m, kThreads, 0, s>>>(h, gamma, eps, k, static_cast<uint32_t *>(out));
  return hipGetLastError();
}

}  // namespace eb
