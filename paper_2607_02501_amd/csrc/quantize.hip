// quantize.hip -- fp32 weights -> Q8_0 / Q4_0 / Q6_S planar layout, and
// conversion between the planar device layout and the canonical
// array-of-blocks bytes.
//
// One thread per 32-weight block.  Quantization runs once when a model is
// loaded, so these kernels favour exactness over speed: the scale is
// fl32(amax / 127) or fl32(m / -8) (IEEE binary32 division), rounded to
// binary16 ties-to-even by the hardware conversion, and each code is decided
// on the binary64 quotient w / d16 (w has 24 significant bits and d16 at most
// 11, so that quotient is never rounded onto or off a rounding tie).
// Q6_S takes one thread per 256-weight super-block: the sub-block scales
// s_j = fl32(m_j / -32), the binary16 super-scale from fl32(max |s_j| / 127),
// the int8 sub-scales decided on the binary64 quotient s_j / d16 and the
// 6-bit codes on x / (d16 sc_j) (at most 18 significant bits in the divisor,
// so again no quotient is rounded onto or off a tie).
// Block formats: paper section 4, Table 3 (8-, 6- and 4-bit configurations).
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

// ---- Q6_S ----

// Zero [a, b) of the buffer (workgroup 0's threads).
__device__ inline void zero_range(uint8_t *out, int64_t a, int64_t b) {
  for (int64_t i = a + threadIdx.x; i < b; i += blockDim.x) out[i] = 0;
}

// The gaps of the Q6_S planar layout: after the code plane, after the
// sub-scale plane and after the scale plane, up to each next 256-byte start.
__device__ inline void zero_gaps_q6(uint8_t *out, int64_t n, const Layout &L) {
  zero_range(out, n * L.qs_row, L.sc_off);
  zero_range(out, L.sc_off + n * L.ss, L.d_off);
  zero_range(out, L.d_off + n * L.ds * 2, L.total);
}

__device__ inline Layout layout_q6(int64_t n, int64_t k) {
  Layout L;
  L.nb = k / kQK;
  L.qs_row = L.nb * 24;
  L.sc_off = round_up(n * L.qs_row, 256);
  L.ss = k / 16;
  L.d_off = round_up(L.sc_off + n * L.ss, 256);
  L.ds = round_up(k / kQK6, 8);
  L.total = round_up(L.d_off + n * L.ds * 2, 256);
  return L;
}

// 32 codes u (0..63) -> the 24 bytes of a chunk: byte i (0..15) holds the low
// nibbles of u_i and u_{i+16}, byte 16 + t the top two bits of u_t, u_{t+8},
// u_{t+16}, u_{t+24} (two bits each, from the least significant end).
__device__ inline void pack_chunk_q6(const int u[32], uint8_t *dst) {
  uint32_t w[6];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t v = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = 4 * i + j;
      v |= ((uint32_t)(u[e] & 15) | (uint32_t)(u[e + 16] & 15) << 4) << (8 * j);
    }
    w[i] = v;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    uint32_t v = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = 4 * i + j;
      const uint32_t b = (uint32_t)(u[t] >> 4) | (uint32_t)(u[t + 8] >> 4) << 2 |
                         (uint32_t)(u[t + 16] >> 4) << 4 | (uint32_t)(u[t + 24] >> 4) << 6;
      v |= b << (8 * j);
    }
    w[4 + i] = v;
  }
  uint2 *d = reinterpret_cast<uint2 *>(dst);  // chunks are 8-byte aligned
  d[0] = make_uint2(w[0], w[1]);
  d[1] = make_uint2(w[2], w[3]);
  d[2] = make_uint2(w[4], w[5]);
}

__global__ void __launch_bounds__(256) quantize_q6_kernel(const float *__restrict__ w, int64_t n,
                                                          int64_t k, uint8_t *__restrict__ out) {
  const Layout L = layout_q6(n, k);
  const int64_t nsb = k / kQK6;
  if (blockIdx.x == 0) zero_gaps_q6(out, n, L);
  uint16_t *dplane = reinterpret_cast<uint16_t *>(out + L.d_off);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * L.ds;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / L.ds, sb = t % L.ds;
    if (sb >= nsb) {
      dplane[t] = 0;
      continue;
    }
    const float *src = w + r * k + sb * kQK6;
    // sub-block scales: the signed element of largest magnitude (first index) / -32
    float s[16];
    float amax = 0.0f;
    for (int j = 0; j < 16; ++j) {
      float mag = 0.0f, m = 0.0f;
      for (int i = 0; i < 16; ++i) {
        const float v = src[16 * j + i];
        if (fabsf(v) > mag) {
          mag = fabsf(v);
          m = v;
        }
      }
      s[j] = m / -32.0f;
      amax = fmaxf(amax, fabsf(s[j]));
    }
    uint16_t d16 = f32_to_f16_bits(amax / 127.0f);
    if (amax == 0.0f) d16 = 0x0000;  // +0 / 127
    dplane[t] = d16;
    const double d = f16_bits_to_f64(d16);
    int sc[16];
    uint8_t *scp = out + L.sc_off + r * L.ss + sb * 16;
    for (int j = 0; j < 16; ++j) {
      double v = 0.0;
      if (d != 0.0) v = fmin(fmax(round((double)s[j] / d), -127.0), 127.0);  // half away from zero
      sc[j] = (int)v;
      scp[j] = (uint8_t)(int8_t)sc[j];
    }
    // codes, one 32-weight chunk at a time
    for (int c = 0; c < kQK6 / kQK; ++c) {
      int u[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const double e = d * (double)sc[(32 * c + i) / 16];  // exact
        double q = 0.0;
        if (e != 0.0) q = fmin(fmax(floor((double)src[32 * c + i] / e + 0.5), -32.0), 31.0);
        u[i] = (int)q + 32;
      }
      pack_chunk_q6(u, out + (r * L.nb + sb * 8 + c) * 24);
    }
  }
}

// planar -> canonical: one thread per super-block, byte stores.
__global__ void __launch_bounds__(256) to_canonical_q6_kernel(const uint8_t *__restrict__ planar,
                                                              int64_t n, int64_t k,
                                                              uint8_t *__restrict__ dst) {
  const Layout L = layout_q6(n, k);
  const int64_t nsb = k / kQK6;
  const uint16_t *dplane = reinterpret_cast<const uint16_t *>(planar + L.d_off);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * nsb;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / nsb, sb = t % nsb;
    uint8_t *o = dst + t * 210;
    const uint16_t d16 = dplane[r * L.ds + sb];
    o[0] = (uint8_t)(d16 & 0xff);
    o[1] = (uint8_t)(d16 >> 8);
    const uint8_t *scp = planar + L.sc_off + r * L.ss + sb * 16;
    for (int j = 0; j < 16; ++j) o[2 + j] = scp[j];
    const uint8_t *q = planar + (r * L.nb + sb * 8) * 24;
    for (int i = 0; i < 192; ++i) o[18 + i] = q[i];
  }
}

// canonical -> planar (padding and gaps written as zero).
__global__ void __launch_bounds__(256) from_canonical_q6_kernel(const uint8_t *__restrict__ src,
                                                                int64_t n, int64_t k,
                                                                uint8_t *__restrict__ out) {
  const Layout L = layout_q6(n, k);
  const int64_t nsb = k / kQK6;
  uint16_t *dplane = reinterpret_cast<uint16_t *>(out + L.d_off);
  if (blockIdx.x == 0) zero_gaps_q6(out, n, L);
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * L.ds;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / L.ds, sb = t % L.ds;
    if (sb >= nsb) {
      dplane[t] = 0;
      continue;
    }
    const uint8_t *c = src + (r * nsb + sb) * 210;
    dplane[t] = (uint16_t)(c[0] | (c[1] << 8));
    uint8_t *scp = out + L.sc_off + r * L.ss + sb * 16;
    for (int j = 0; j < 16; ++j) scp[j] = c[2 + j];
    uint8_t *q = out + (r * L.nb + sb * 8) * 24;
    for (int i = 0; i < 192; ++i) q[i] = c[18 + i];
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
  if (type == EB_Q6_S) {
    const int64_t threads = n * round_up(k / kQK6, 8);
    if (threads == 0) return hipSuccess;
    quantize_q6_kernel<<<grid_for(threads), 256, 0, s>>>(w, n, k, (uint8_t *)out);
    return hipGetLastError();
  }
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
  if (type == EB_Q6_S) {
    const int64_t threads = n * (k / kQK6);
    if (threads == 0) return hipSuccess;
    to_canonical_q6_kernel<<<grid_for(threads), 256, 0, s>>>((const uint8_t *)planar, n, k,
                                                             (uint8_t *)dst);
    return hipGetLastError();
  }
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
  if (type == EB_Q6_S) {
    const int64_t threads = n * round_up(k / kQK6, 8);
    if (threads == 0) return hipSuccess;
    from_canonical_q6_kernel<<<grid_for(threads), 256, 0, s>>>((const uint8_t *)src, n, k,
                                                               (uint8_t *)out);
    return hipGetLastError();
  }
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
