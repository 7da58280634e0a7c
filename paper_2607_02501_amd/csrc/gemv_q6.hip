// gemv_q6.hip -- batch-1 / few-row (m <= 8) linear layers on Q6_S weights:
// the bandwidth-bound decode case of the 6-bit configuration (paper section
// 4, Table 3; section 3.2, latency-first batch-1 execution).
//
// A wave owns a pair of weight rows (so a gate/up pair's product is formed in
// the wave) and its lanes walk the rows' 24-byte code chunks (32 weights
// each) in lane order: one wave load covers 64 consecutive chunks of a row,
// 1536 contiguous bytes, read as three 8-byte loads per lane.  A chunk
// decodes to u = low nibble | top bits << 4, and the lane accumulates
// (u - 32) x in fp32 per 16-weight sub-block (every product exact: 6-bit code
// times 16-bit activation), then e_j times that sum (e_j = d16 sc_j, exact in
// fp32) into its row sum; the wave's lanes are added by a butterfly.  x (all
// m rows, normalised first when the op has the RMS-normalisation prologue)
// is staged in LDS as 16-bit values by the whole workgroup.
#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"

namespace eb {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;

__device__ inline float x_to_f32(uint16_t v, int xt) {
  return xt == EB_F16 ? (float)__builtin_bit_cast(_Float16, v) : __uint_as_float((uint32_t)v << 16);
}

__device__ inline uint16_t f32_to_x(float v, int xt) {
  return xt == EB_F16 ? __builtin_bit_cast(uint16_t, (_Float16)v) : __builtin_bit_cast(uint16_t, (__bf16)v);
}

// Stage the MT rows of x (rows past m as zeros) into xs[MT][k] as 16-bit
// values of type xt; with the prologue, x is the fp32 stream h and each row is
// normalised: r = 1 / sqrt(sum h^2 / k + eps) (each thread's columns
// j = t, t + 512, ... summed in order, then the 64 lanes of a wave, then the
// waves in order), x_hat = round(h g r).
template <int MT>
__device__ void stage_q6(const void *x, int64_t m, int64_t k, int xt, const Fuse &f, uint16_t *xs,
                         float *red) {
  const int t = threadIdx.x;
  if (f.pro == EB_PRO_RMSNORM) {
    const float *h = static_cast<const float *>(x);
    for (int mm = 0; mm < MT; ++mm) {
      if (mm >= m) {
        for (int64_t j = t; j < k; j += kThreads) xs[mm * k + j] = 0;
        continue;
      }
      float ss = 0.f;
      for (int64_t j = t; j < k; j += kThreads) {
        const float v = h[mm * k + j];
        ss = __builtin_fmaf(v, v, ss);
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
      __syncthreads();  // red is reused row after row
      if ((t & 63) == 0) red[t >> 6] = ss;
      __syncthreads();
      float tot = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) tot += red[w];
      const float r = 1.0f / __builtin_sqrtf(tot / (float)k + f.eps);
      for (int64_t j = t; j < k; j += kThreads) xs[mm * k + j] = f32_to_x(h[mm * k + j] * f.gamma[j] * r, xt);
    }
  } else {
    // 16-byte pieces (k is a multiple of 256, so a row is a whole number of them)
    const uint4 *src = static_cast<const uint4 *>(x);
    uint4 *dst = reinterpret_cast<uint4 *>(xs);
    const int64_t per_row = k / 8;
    for (int64_t i = t; i < MT * per_row; i += kThreads)
      dst[i] = (i / per_row < m) ? src[i] : make_uint4(0, 0, 0, 0);
  }
  __syncthreads();
}

// u codes of a chunk, 4 per word: word w holds weights 4w .. 4w + 3.
__device__ inline void decode_chunk(const uint2 a, const uint2 b, const uint2 c, uint32_t u[8]) {
  const uint32_t L0 = a.x, L1 = a.y, L2 = b.x, L3 = b.y, H0 = c.x, H1 = c.y;
  constexpr uint32_t N = 0x0f0f0f0fu, T = 0x03030303u;
  u[0] = (L0 & N) | ((H0 & T) << 4);
  u[1] = (L1 & N) | ((H1 & T) << 4);
  u[2] = (L2 & N) | (((H0 >> 2) & T) << 4);
  u[3] = (L3 & N) | (((H1 >> 2) & T) << 4);
  u[4] = ((L0 >> 4) & N) | (((H0 >> 4) & T) << 4);
  u[5] = ((L1 >> 4) & N) | (((H1 >> 4) & T) << 4);
  u[6] = ((L2 >> 4) & N) | (((H0 >> 6) & T) << 4);
  u[7] = ((L3 >> 4) & N) | (((H1 >> 6) & T) << 4);
}

// sum over 4 weights of word w: (u - 32) x, x from 4 consecutive 16-bit values
// (each byte to float is one v_cvt_f32_ubyte; u - 32 and the product are exact)
__device__ inline float dot4(uint32_t w, uint2 xv, int xt, float acc) {
  const float x0 = x_to_f32((uint16_t)(xv.x & 0xffffu), xt), x1 = x_to_f32((uint16_t)(xv.x >> 16), xt);
  const float x2 = x_to_f32((uint16_t)(xv.y & 0xffffu), xt), x3 = x_to_f32((uint16_t)(xv.y >> 16), xt);
  acc = __builtin_fmaf((float)((w >> 0) & 0xffu) - 32.0f, x0, acc);
  acc = __builtin_fmaf((float)((w >> 8) & 0xffu) - 32.0f, x1, acc);
  acc = __builtin_fmaf((float)((w >> 16) & 0xffu) - 32.0f, x2, acc);
  acc = __builtin_fmaf((float)((w >> 24) & 0xffu) - 32.0f, x3, acc);
  return acc;
}

template <int MT>
__global__ void __launch_bounds__(kThreads)
    gemv_q6_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t sc_off,
                   int64_t d_off, int64_t ds, const void *__restrict__ x, int64_t m, int xt,
                   void *__restrict__ y, int yt, Fuse f) {
  extern __shared__ uint16_t xs[];  // [MT][k]
  __shared__ float red[kWaves];
  stage_q6<MT>(x, m, k, xt, f, xs, red);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t pair = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t r0 = 2 * pair;
  if (r0 >= n) return;
  const bool two = r0 + 1 < n;
  const int64_t nc = k / kQK;              // chunks per row
  const int64_t qrow = nc * 24, srow = k / 16;
  float acc[2][MT];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) acc[rr][mm] = 0.f;

  for (int64_t c = lane; c < nc; c += 64) {
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      if (rr == 1 && !two) break;
      const int64_t row = r0 + rr;
      const uint2 *q = reinterpret_cast<const uint2 *>(wdata + row * qrow + c * 24);
      const uint2 a = q[0], b = q[1], h = q[2];
      const uint16_t sc2 = *reinterpret_cast<const uint16_t *>(wdata + sc_off + row * srow + 2 * c);
      const uint16_t d16 = *reinterpret_cast<const uint16_t *>(wdata + d_off + (row * ds + c / 8) * 2);
      const float d = (float)__builtin_bit_cast(_Float16, d16);
      const float e0 = d * (float)(int8_t)(sc2 & 0xff), e1 = d * (float)(int8_t)(sc2 >> 8);  // exact
      uint32_t u[8];
      decode_chunk(a, b, h, u);
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        const uint4 *xv = reinterpret_cast<const uint4 *>(xs + mm * k + c * 32);
        const uint4 x0 = xv[0], x1 = xv[1], x2 = xv[2], x3 = xv[3];
        // weights 0..15 (sub-block 2c), then 16..31 (sub-block 2c + 1)
        float s0 = 0.f, s1 = 0.f;
        s0 = dot4(u[0], make_uint2(x0.x, x0.y), xt, s0);
        s0 = dot4(u[1], make_uint2(x0.z, x0.w), xt, s0);
        s0 = dot4(u[2], make_uint2(x1.x, x1.y), xt, s0);
        s0 = dot4(u[3], make_uint2(x1.z, x1.w), xt, s0);
        s1 = dot4(u[4], make_uint2(x2.x, x2.y), xt, s1);
        s1 = dot4(u[5], make_uint2(x2.z, x2.w), xt, s1);
        s1 = dot4(u[6], make_uint2(x3.x, x3.y), xt, s1);
        s1 = dot4(u[7], make_uint2(x3.z, x3.w), xt, s1);
        acc[rr][mm] = __builtin_fmaf(e0, s0, acc[rr][mm]);
        acc[rr][mm] = __builtin_fmaf(e1, s1, acc[rr][mm]);
      }
    }
  }
#pragma unroll
  for (int rr = 0; rr < 2; ++rr)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm)
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) acc[rr][mm] += __shfl_xor(acc[rr][mm], o);
  if (lane != 0) return;
  for (int mm = 0; mm < MT && mm < m; ++mm) {
    if (f.epi == EB_EPI_GLU) {  // n even: rows r0, r0 + 1 are a gate/up pair
      store_y(y, (int64_t)mm * (n / 2) + pair, silu_mul(acc[0][mm], acc[1][mm]), yt);
      continue;
    }
    put_y(y, (int64_t)mm * n + r0, acc[0][mm], yt, f);
    if (two) put_y(y, (int64_t)mm * n + r0 + 1, acc[1][mm], yt, f);
  }
}

template <int MT>
hipError_t launch_mt(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt, int64_t m,
                     void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(EB_Q6_S, n, k);
  const int64_t pairs = (n + 1) / 2;
  const unsigned grid = (unsigned)((pairs + kWaves - 1) / kWaves);
  const size_t lds = (size_t)MT * k * 2;
  auto kern = gemv_q6_kernel<MT>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<grid, kThreads, lds, s>>>(static_cast<const uint8_t *>(wdata), n, k, L.sc_off,
                                                 L.d_off, L.ds, x, m, xt, y, yt, f);
  return hipGetLastError();
}

}  // namespace

bool gemv_q6_fits(int64_t m, int64_t n, int64_t k) {
  const int64_t mt = m <= 1 ? 1 : (m <= 2 ? 2 : (m <= 4 ? 4 : 8));
  return m >= 1 && m <= kGemvMaxM && mt * k <= kGemvMaxMK && k % kQK6 == 0 &&
         (n + 1) / 2 <= (int64_t)0x7fffffff * kWaves;
}

hipError_t launch_gemv_q6(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt,
                          int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  if (!gemv_q6_fits(m, n, k)) return hipErrorInvalidValue;
  if (m <= 1) return launch_mt<1>(wdata, n, k, x, xt, m, y, yt, f, s);
  if (m <= 2) return launch_mt<2>(wdata, n, k, x, xt, m, y, yt, f, s);
  if (m <= 4) return launch_mt<4>(wdata, n, k, x, xt, m, y, yt, f, s);
  return launch_mt<8>(wdata, n, k, x, xt, m, y, yt, f, s);
}

}  // namespace eb
