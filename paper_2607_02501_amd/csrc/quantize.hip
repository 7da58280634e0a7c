// quantize.hip -- fp32 weights -> Q8_0 / Q4_0 planar layout, and conversion
// between the planar device layout and the canonical array-of-blocks bytes.
//
// One thread per 32-weight block.  Quantization runs once when a model is
// loaded, so these kernels favour exactness over speed: the scale is
// fl32(amax / 127) or fl32(m / -8) (IEEE binary32 division), rounded to
// binary16 ties-to-even by the hardware conversion, and each code is decided
// on the binary64 quotient w / d16 (w has 24 significant bits and d16 at most
// 11, so that quotient is never rounded onto or off a rounding tie).
// Block formats: paper section 4, Table 3 (8-bit / 4-bit configurations).
#include <hip/hip_runtime.h>
#include <math.h>

#include "eb_internal.h"

namespace eb {
namespace {

__device__ inline uint16_t f32_to_f16_bits(float f) {
  _Float16 h = (_Float16)f;  // v_cvt_f16_f32, round to nearest even
  return __builtin_bit_cast(uint16_t, h);
}

__device__ inline double f16_bits_to_f64(uint16_t b) {
  return (double)__builtin_bit_cast(_Float16, b);
}

// Zero the alignment gaps of the planar layout: [qs_end, d_off) and
// [d_end, round_up(d_end, 256)), so that equal weights give equal buffers.
__device__ inline void zero_gaps(uint8_t *out, int64_t qs_end, int64_t d_off, int64_t d_end) {
  const int64_t end = round_up(d_end, 256);
  for (int64_t i = qs_end + threadIdx.x; i < d_off; i += blockDim.x) out[i] = 0;
  for (int64_t i = d_end + threadIdx.x; i < end; i += blockDim.x) out[i] = 0;
}

// One block of 32 fp32 weights -> d16 bits and 32 signed codes.
template <int QT>
__device__ inline uint16_t quantize_block(const float *src, int codes[kQK]) {
  float v[kQK];
#pragma unroll
  for (int i = 0; i < kQK; i += 4) {
    float4 t = *reinterpret_cast<const float4 *>(src + i);
    v[i] = t.x;
    v[i + 1] = t.y;
    v[i + 2] = t.z;
    v[i + 3] = t.w;
  }
  float amax = 0.0f, smax = 0.0f;
#pragma unroll
  for (int j = 0; j < kQK; ++j) {
    float a = fabsf(v[j]);
    if (a > amax) {
      amax = a;
      smax = v[j];
    }
  }
  float d32 = (QT == EB_Q8_0) ? amax / 127.0f : smax / -8.0f;
  uint16_t d16 = f32_to_f16_bits(d32);
  // All-zero block: the scale is +0 / 127 = +0 (Q8_0) or +0 / -8 = -0 (Q4_0).
  // Written out because the compiler may fuse the product into a mixed-precision
  // FMA with a +0 addend, which loses the sign of an exact zero.
  if (amax == 0.0f) d16 = (QT == EB_Q8_0) ? 0x0000 : 0x8000;
  double d = f16_bits_to_f64(d16);
#pragma unroll
  for (int j = 0; j < kQK; ++j) {
    int c = 0;
    if (d != 0.0) {
      double t = (double)v[j] / d;
      if (QT == EB_Q8_0) {
        t = round(t);  // half away from zero
        t = fmin(fmax(t, -127.0), 127.0);
      } else {
        t = floor(t + 0.5);  // half up
        t = fmin(fmax(t, -8.0), 7.0);
      }
      c = (int)t;
    }
    codes[j] = c;
  }
  return d16;
}

template <int QT>
__global__ void __launch_bounds__(256) quantize_kernel(const float *__restrict__ w, int64_t n,
                                                       int64_t k, uint8_t *__restrict__ out) {
  const int64_t nb = k / kQK;
  const int64_t ds = round_up(nb, 8);
  const int64_t qsb = (QT == EB_Q8_0) ? 32 : 16;
  const int64_t d_off = round_up(n * nb * qsb, 256);
  const int64_t total = n * ds;  // one thread per scale-plane slot (incl. padding)
  if (blockIdx.x == 0) zero_gaps(out, n * nb * qsb, d_off, d_off + total * 2);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / ds, b = t % ds;
    uint16_t *dplane = reinterpret_cast<uint16_t *>(out + d_off);
    if (b >= nb) {
      dplane[r * ds + b] = 0;
      continue;
    }
    int codes[kQK];
    uint16_t d16 = quantize_block<QT>(w + r * k + b * kQK, codes);
    dplane[r * ds + b] = d16;
    uint8_t *qs = out + (r * nb + b) * qsb;
    if (QT == EB_Q8_0) {
      uint32_t words[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        words[i] = (uint32_t)(uint8_t)(int8_t)codes[4 * i] |
                   ((uint32_t)(uint8_t)(int8_t)codes[4 * i + 1] << 8) |
                   ((uint32_t)(uint8_t)(int8_t)codes[4 * i + 2] << 16) |
                   ((uint32_t)(uint8_t)(int8_t)codes[4 * i + 3] << 24);
      uint4 *dst = reinterpret_cast<uint4 *>(qs);
      dst[0] = make_uint4(words[0], words[1], words[2], words[3]);
      dst[1] = make_uint4(words[4], words[5], words[6], words[7]);
    } else {
      uint32_t words[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t wv = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int e = 4 * i + j;
          uint32_t byte = (uint32_t)(codes[e] + 8) | ((uint32_t)(codes[e + 16] + 8) << 4);
          wv |= byte << (8 * j);
        }
        words[i] = wv;
      }
      *reinterpret_cast<uint4 *>(qs) = make_uint4(words[0], words[1], words[2], words[3]);
    }
  }
}

// planar -> canonical: one thread per block, byte stores (no alignment on dst).
template <int QT>
__global__ void __launch_bounds__(256) to_canonical_kernel(const uint8_t *__restrict__ planar,
                                                           int64_t n, int64_t k,
                                                           uint8_t *__restrict__ dst) {
  const int64_t nb = k / kQK;
  const int64_t ds = round_up(nb, 8);
  const int64_t qsb = (QT == EB_Q8_0) ? 32 : 16;
  const int64_t d_off = round_up(n * nb * qsb, 256);
  const uint16_t *dplane = reinterpret_cast<const uint16_t *>(planar + d_off);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * nb;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / nb, b = t % nb;
    uint8_t *o = dst + t * (2 + qsb);
    uint16_t d16 = dplane[r * ds + b];
    o[0] = (uint8_t)(d16 & 0xff);
    o[1] = (uint8_t)(d16 >> 8);
    const uint8_t *q = planar + t * qsb;
    for (int i = 0; i < qsb; ++i) o[2 + i] = q[i];
  }
}

// canonical -> planar (scale-plane padding written as zero).
template <int QT>
__global__ void __launch_bounds__(256) from_canonical_kernel(const uint8_t *__restrict__ src,
                                                             int64_t n, int64_t k,
                                                             uint8_t *__restrict__ out) {
  const int64_t nb = k / kQK;
  const int64_t ds = round_up(nb, 8);
  const int64_t qsb = (QT == EB_Q8_0) ? 32 : 16;
  const int64_t d_off = round_up(n * nb * qsb, 256);
  uint16_t *dplane = reinterpret_cast<uint16_t *>(out + d_off);
  if (blockIdx.x == 0) zero_gaps(out, n * nb * qsb, d_off, d_off + n * ds * 2);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * ds;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / ds, b = t % ds;
    if (b >= nb) {
      dplane[t] = 0;
      continue;
    }
    const uint8_t *c = src + (r * nb + b) * (2 + qsb);
    dplane[t] = (uint16_t)(c[0] | (c[1] << 8));
    uint8_t *q = out + (r * nb + b) * qsb;
    for (int i = 0; i < qsb; ++i) q[i] = c[2 + i];
  }
}

inline unsigned grid_for(int64_t threads) {
  int64_t g = (threads + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (unsigned)g;
}

}  // namespace

hipError_t launch_quantize(int32_t type, const float *w, int64_t n, int64_t k, void *out,
                           hipStream_t s) {
  const int64_t threads = n * round_up(k / kQK, 8);
  if (threads == 0) return hipSuccess;
  if (type == EB_Q8_0)
    quantize_kernel<EB_Q8_0><<<grid_for(threads), 256, 0, s>>>(w, n, k, (uint8_t *)out);
  else
    quantize_kernel<EB_Q4_0><<<grid_for(threads), 256, 0, s>>>(w, n, k, (uint8_t *)out);
  return hipGetLastError();
}

hipError_t launch_to_canonical(int32_t type, const void *planar, int64_t n, int64_t k, void *dst,
                               hipStream_t s) {
  const int64_t threads = n * (k / kQK);
  if (threads == 0) return hipSuccess;
  if (type == EB_Q8_0)
    to_canonical_kernel<EB_Q8_0>
        <<<grid_for(threads), 256, 0, s>>>((const uint8_t *)planar, n, k, (uint8_t *)dst);
  else
    to_canonical_kernel<EB_Q4_0>
        <<<grid_for(threads), 256, 0, s>>>((const uint8_t *)planar, n, k, (uint8_t *)dst);
  return hipGetLastError();
}

hipError_t launch_from_canonical(int32_t type, const void *src, int64_t n, int64_t k, void *out,
                                 hipStream_t s) {
  const int64_t threads = n * round_up(k / kQK, 8);
  if (threads == 0) return hipSuccess;
  if (type == EB_Q8_0)
    from_canonical_kernel<EB_Q8_0>
        <<<grid_for(threads), 256, 0, s>>>((const uint8_t *)src, n, k, (uint8_t *)out);
  else
    from_canonical_kernel<EB_Q4_0>
        <<<grid_for(threads), 256, 0, s>>>((const uint8_t *)src, n, k, (uint8_t *)out);
  return hipGetLastError();
}

}  // namespace eb
