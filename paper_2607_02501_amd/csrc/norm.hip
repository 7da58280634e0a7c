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

// The rest of a row's normalisation once every thread holds the sum of the
// squares of its float4 columns j = t, t + 256, ... (summed in that order):
// the 64 lanes of a wave, then the four waves in order, then the row written
// from h.  Both row kernels below end here, so the split-K reduction with the
// normalisation fused writes the same bits as its reduction followed by
// rmsnorm_kernel.
__device__ inline float row_factor(float ss, float *red, float eps, int64_t k) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) tot += red[w];
  return 1.0f / __builtin_sqrtf(tot / (float)k + eps);
}

template <int XT>
__device__ inline uint2 norm4(const float4 &v, const float4 &w, float r) {
  return make_uint2(pack2<XT>(v.x * w.x * r, v.y * w.y * r), pack2<XT>(v.z * w.z * r, v.w * w.w * r));
}

template <int XT>
__device__ inline void finish_row(float ss, float *red, const float *__restrict__ h,
                                  const float *__restrict__ g, float eps, int64_t k,
                                  uint32_t *__restrict__ out) {
  const float r = row_factor(ss, red, eps, k);
  const float4 *src = reinterpret_cast<const float4 *>(h);
  const float4 *gs = reinterpret_cast<const float4 *>(g);
  uint2 *dst = reinterpret_cast<uint2 *>(out);
  for (int64_t i = threadIdx.x; i < k / 4; i += kThreads) dst[i] = norm4<XT>(src[i], gs[i], r);
}

__device__ inline float sum_sq(float ss, const float4 &v) {
  ss = __builtin_fmaf(v.x, v.x, ss);
  ss = __builtin_fmaf(v.y, v.y, ss);
  ss = __builtin_fmaf(v.z, v.z, ss);
  return __builtin_fmaf(v.w, v.w, ss);
}

template <int XT>
__global__ void __launch_bounds__(kThreads)
    rmsnorm_kernel(const float *__restrict__ h, const float *__restrict__ g, float eps, int64_t k,
                   uint32_t *__restrict__ out) {
  __shared__ float red[kThreads / 64];
  const int64_t row = blockIdx.x;
  const float4 *src = reinterpret_cast<const float4 *>(h + row * k);
  float ss = 0.f;
  for (int64_t i = threadIdx.x; i < k / 4; i += kThreads) ss = sum_sq(ss, src[i]);
  finish_row<XT>(ss, red, h + row * k, g, eps, k, out + row * (k / 2));
}

// Sum of the partials of flat element o (float4 at o) in split order, plus
// the residual.
__device__ inline float4 reduce4(const float *__restrict__ ws, int splits, int64_t ws_stride,
                                 int64_t o, const float *r) {
  float4 v = *reinterpret_cast<const float4 *>(ws + o);
  // unrolled so several partial loads are in flight; the sum stays in split order
#pragma unroll 4
  for (int p = 1; p < splits; ++p) {
    const float4 b = *reinterpret_cast<const float4 *>(ws + p * ws_stride + o);
    v.x += b.x;
    v.y += b.y;
    v.z += b.z;
    v.w += b.w;
  }
  if (r) {
    const float4 a = *reinterpret_cast<const float4 *>(r + o);
    v.x += a.x;
    v.y += a.y;
    v.z += a.z;
    v.w += a.w;
  }
  return v;
}

// The same for rows of at most R * 1024 outputs: each thread keeps its R
// float4 of h in registers for the normalisation instead of reading them
// back (same values, same operations, same bits).
template <int XT, int R>
__global__ void __launch_bounds__(kThreads)
    reduce_rmsnorm_reg_kernel(const float *__restrict__ ws, int splits, int64_t ws_stride, int64_t n,
                              float *y, const float *r, const float *__restrict__ g, float eps,
                              uint32_t *__restrict__ out) {
  __shared__ float red[kThreads / 64];
  const int64_t row = blockIdx.x;
  float ss = 0.f;
  float4 v[R];
#pragma unroll
  for (int c = 0; c < R; ++c) {
    const int64_t i = threadIdx.x + (int64_t)c * kThreads;
    if (i < n / 4) {
      const int64_t o = row * n + 4 * i;
      v[c] = reduce4(ws, splits, ws_stride, o, r);
      *reinterpret_cast<float4 *>(y + o) = v[c];
      ss = sum_sq(ss, v[c]);
    }
  }
  const float rf = row_factor(ss, red, eps, n);
  const float4 *gs = reinterpret_cast<const float4 *>(g);
  uint2 *dst = reinterpret_cast<uint2 *>(out + row * (n / 2));
#pragma unroll
  for (int c = 0; c < R; ++c) {
    const int64_t i = threadIdx.x + (int64_t)c * kThreads;
    if (i < n / 4) dst[i] = norm4<XT>(v[c], gs[i], rf);
  }
}

// Split-K reduction of a projection with n outputs per row whose fp32 output
// row h is the next projection's input under a normalisation prologue: row
// `row` of y = the partials summed in split order (+ the residual), as the
// plain reduction computes each element, then the row is normalised into
// `out` for the next projection.  One workgroup per row; every thread reads
// back only the y elements it wrote itself.
template <int XT>
__global__ void __launch_bounds__(kThreads)
    reduce_rmsnorm_kernel(const float *__restrict__ ws, int splits, int64_t ws_stride, int64_t n,
                          float *y, const float *r, const float *__restrict__ g, float eps,
                          uint32_t *__restrict__ out) {
  __shared__ float red[kThreads / 64];
  const int64_t row = blockIdx.x;
  float ss = 0.f;
  for (int64_t i = threadIdx.x; i < n / 4; i += kThreads) {
    const int64_t o = row * n + 4 * i;
    const float4 v = reduce4(ws, splits, ws_stride, o, r);
    *reinterpret_cast<float4 *>(y + o) = v;
    ss = sum_sq(ss, v);
  }
  finish_row<XT>(ss, red, y + row * n, g, eps, n, out + row * (n / 2));
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

hipError_t launch_splitk_reduce_rmsnorm(const float *ws, int splits, int64_t ws_stride, int64_t m,
                                        int64_t n, float *y, const float *residual,
                                        const NormOut &no, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  if (m > 0x7fffffff || n % 4 != 0 || ws_stride % 4 != 0 || splits < 1) return hipErrorInvalidValue;
  uint32_t *out = static_cast<uint32_t *>(no.xout);
  const unsigned grid = (unsigned)m;
  const int64_t per = (n / 4 + kThreads - 1) / kThreads;  // float4 per thread
#define EB_REDUCE_REG(R)                                                                         \
  if (per <= R) {                                                                                \
    if (no.xt == EB_F16)                                                                         \
      reduce_rmsnorm_reg_kernel<EB_F16, R><<<grid, kThreads, 0, s>>>(ws, splits, ws_stride, n, y, \
                                                                     residual, no.gamma, no.eps, out); \
    else                                                                                         \
      reduce_rmsnorm_reg_kernel<EB_BF16, R><<<grid, kThreads, 0, s>>>(ws, splits, ws_stride, n, y, \
                                                                      residual, no.gamma, no.eps, out); \
    return hipGetLastError();                                                                    \
  }
  EB_REDUCE_REG(1)
  EB_REDUCE_REG(2)
  EB_REDUCE_REG(4)
#undef EB_REDUCE_REG
  if (no.xt == EB_F16)
    reduce_rmsnorm_kernel<EB_F16><<<(unsigned)m, kThreads, 0, s>>>(ws, splits, ws_stride, n, y, residual,
                                                                  no.gamma, no.eps, out);
  else
    reduce_rmsnorm_kernel<EB_BF16><<<(unsigned)m, kThreads, 0, s>>>(ws, splits, ws_stride, n, y, residual,
                                                                   no.gamma, no.eps, out);
  return hipGetLastError();
}

}  // namespace eb
