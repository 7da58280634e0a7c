// mfma.hip -- matrix-core path of the quantized linear layer for m > 4
// activation rows: prefill of image/text tokens, action-chunk denoising and
// video-latent tokens (paper section 2.1 / Table 1 model families; section 3.2
// "operator fusion, backend-specific dispatch").
//
// y[m][n] = sum_k x[m][k] * w_hat[n][k], w_hat = code * d16 rounded once to
// the activation type (bfloat16 or binary16), fp32 accumulation.
//
// Each workgroup computes a BM x BN tile of y.  Per K-tile of 64:
//   global -> registers: the x tile (16-bit, 16-byte loads) and the packed
//   weight tile (16-byte loads of codes + binary16 scales), prefetched one
//   K-tile ahead while the matrix cores work on the current one;
//   registers -> LDS: x copied, weights dequantized (code * d16 exact in fp32,
//   then one round-to-nearest-even to 16 bits) -- the dequantization is fused
//   into the tile load, no dequantized weight ever reaches HBM;
//   LDS -> MFMA: v_mfma_f32_32x32x16_{bf16,f16}, A = x rows, B = w_hat rows.
#include <hip/hip_runtime.h>

#include "eb_internal.h"

namespace eb {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;        // K elements per tile (2 blocks)
constexpr int kPad = 8;        // LDS row padding in 16-bit elements
constexpr int kLds = kBK + kPad;

template <int XT>
__device__ inline uint16_t to16(float f) {
  if (XT == EB_BF16) return __builtin_bit_cast(uint16_t, (__bf16)f);
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

template <int XT>
__device__ inline uint32_t pack2(float a, float b) {
  return (uint32_t)to16<XT>(a) | ((uint32_t)to16<XT>(b) << 16);
}

template <int XT>
__device__ inline f32x16_t mfma32(const uint4 a, const uint4 b, f32x16_t c) {
  if (XT == EB_BF16)
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

template <int QT>
struct WTile {
  // 16-byte weight chunks per row per K-tile: Q8_0 four half-blocks, Q4_0 two blocks
  static constexpr int kChunksPerRow = (QT == EB_Q8_0) ? 4 : 2;
};

template <int QT, int XT, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(WM *WN * 64)
    mfma_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off, int64_t ds,
                const uint16_t *__restrict__ x, int64_t m, void *__restrict__ y, int yt) {
  constexpr int T = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int ACH = BM * (kBK / 8) / T;                    // x chunks per thread
  constexpr int WCPR = WTile<QT>::kChunksPerRow;
  constexpr int BCH = BN * WCPR / T;                         // weight chunks per thread
  static_assert(ACH * T == BM * (kBK / 8), "x tile must split evenly");
  static_assert(BCH * T == BN * WCPR, "weight tile must split evenly");

  __shared__ __attribute__((aligned(16))) uint16_t As[BM * kLds];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * kLds];

  const int64_t tiles_m = (m + BM - 1) / BM;
  const int64_t tm = blockIdx.x % tiles_m;
  const int64_t tn = blockIdx.x / tiles_m;
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t nb = k / kQK;
  const int64_t qsb = (QT == EB_Q8_0) ? 32 : 16;
  const uint16_t *__restrict__ dplane = reinterpret_cast<const uint16_t *>(wdata + d_off);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  uint4 areg[ACH];
  uint4 breg[BCH];
  uint16_t dreg[BCH];

  auto load_tile = [&](int64_t kt) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int idx = tid + i * T;
      const int r = idx / (kBK / 8), c8 = idx % (kBK / 8);
      const int64_t gm = m0 + r, gk = kt * kBK + c8 * 8;
      areg[i] = (gm < m && gk < k)
                    ? *reinterpret_cast<const uint4 *>(x + gm * k + gk)
                    : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int idx = tid + i * T;
      const int r = idx / WCPR, c = idx % WCPR;
      int64_t gn = n0 + r;
      if (gn >= n) gn = n - 1;  // clamped rows produce columns that are never stored
      const int64_t blk = kt * 2 + ((QT == EB_Q8_0) ? (c >> 1) : c);
      if (blk < nb) {
        const uint8_t *src = wdata + (gn * nb + blk) * qsb + ((QT == EB_Q8_0) ? (c & 1) * 16 : 0);
        breg[i] = *reinterpret_cast<const uint4 *>(src);
        dreg[i] = dplane[gn * ds + blk];
      } else {
        breg[i] = make_uint4(0, 0, 0, 0);
        dreg[i] = 0;
      }
    }
  };

  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int idx = tid + i * T;
      const int r = idx / (kBK / 8), c8 = idx % (kBK / 8);
      *reinterpret_cast<uint4 *>(&As[r * kLds + c8 * 8]) = areg[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int idx = tid + i * T;
      const int r = idx / WCPR, c = idx % WCPR;
      const float d = (float)__builtin_bit_cast(_Float16, dreg[i]);
      const uint32_t w[4] = {breg[i].x, breg[i].y, breg[i].z, breg[i].w};
      if (QT == EB_Q8_0) {
        // 16 int8 codes -> 16 values at k offset 16*c
        uint32_t o[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float q0 = (float)(int8_t)(w[j] & 0xff), q1 = (float)(int8_t)((w[j] >> 8) & 0xff);
          const float q2 = (float)(int8_t)((w[j] >> 16) & 0xff), q3 = (float)(int8_t)(w[j] >> 24);
          o[2 * j] = pack2<XT>(q0 * d, q1 * d);
          o[2 * j + 1] = pack2<XT>(q2 * d, q3 * d);
        }
        uint4 *dst = reinterpret_cast<uint4 *>(&Bs[r * kLds + c * 16]);
        dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
        dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
      } else {
        // 16 bytes: low nibbles are elements 0..15, high nibbles 16..31 of block c
        uint32_t lo[8], hi[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float l[4], h[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const uint32_t byte = (w[j] >> (8 * b)) & 0xff;
            l[b] = (float)((int)(byte & 0xf) - 8) * d;
            h[b] = (float)((int)(byte >> 4) - 8) * d;
          }
          lo[2 * j] = pack2<XT>(l[0], l[1]);
          lo[2 * j + 1] = pack2<XT>(l[2], l[3]);
          hi[2 * j] = pack2<XT>(h[0], h[1]);
          hi[2 * j + 1] = pack2<XT>(h[2], h[3]);
        }
        uint4 *dst = reinterpret_cast<uint4 *>(&Bs[r * kLds + c * 32]);
        dst[0] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        dst[1] = make_uint4(lo[4], lo[5], lo[6], lo[7]);
        dst[2] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        dst[3] = make_uint4(hi[4], hi[5], hi[6], hi[7]);
      }
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int64_t nk = (k + kBK - 1) / kBK;
  load_tile(0);
  for (int64_t kt = 0; kt < nk; ++kt) {
    store_tile();
    __syncthreads();
    if (kt + 1 < nk) load_tile(kt + 1);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int koff = ks * 16 + 8 * (lane >> 5);
      uint4 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(&As[(wm * TM + i * 32 + (lane & 31)) * kLds + koff]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const uint4 *>(&Bs[(wn * TN + j * 32 + (lane & 31)) * kLds + koff]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[i], bfr[j], acc[i][j]);
    }
    __syncthreads();
  }

  // epilogue: lane holds column (lane & 31), rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t col = n0 + wn * TN + j * 32 + (lane & 31);
      if (col >= n) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row >= m) continue;
        if (yt == EB_F32)
          reinterpret_cast<float *>(y)[row * n + col] = acc[i][j][r];
        else
          reinterpret_cast<__bf16 *>(y)[row * n + col] = (__bf16)acc[i][j][r];
      }
    }
}

template <int QT, int XT, int BM, int BN, int WM, int WN>
hipError_t launch_t(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, hipStream_t s) {
  const Layout L = layout_of(QT, n, k);
  const int64_t tiles = ((m + BM - 1) / BM) * ((n + BN - 1) / BN);
  if (tiles > 0x7fffffff) return hipErrorInvalidValue;
  mfma_kernel<QT, XT, BM, BN, WM, WN><<<(unsigned)tiles, WM * WN * 64, 0, s>>>(
      (const uint8_t *)wdata, n, k, L.d_off, L.ds, (const uint16_t *)x, m, y, yt);
  return hipGetLastError();
}

template <int QT, int XT>
hipError_t launch_q(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, hipStream_t s) {
  if (m <= 64) return launch_t<QT, XT, 64, 128, 2, 2>(wdata, n, k, x, m, y, yt, s);
  return launch_t<QT, XT, 128, 128, 2, 2>(wdata, n, k, x, m, y, yt, s);
}

}  // namespace

hipError_t launch_mfma(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                       int32_t xt, int64_t m, void *y, int32_t yt, hipStream_t s) {
  if (type == EB_Q4_0) {
    if (xt == EB_F16) return launch_q<EB_Q4_0, EB_F16>(wdata, n, k, x, m, y, yt, s);
    return launch_q<EB_Q4_0, EB_BF16>(wdata, n, k, x, m, y, yt, s);
  }
  if (xt == EB_F16) return launch_q<EB_Q8_0, EB_F16>(wdata, n, k, x, m, y, yt, s);
  return launch_q<EB_Q8_0, EB_BF16>(wdata, n, k, x, m, y, yt, s);
}

}  // namespace eb
