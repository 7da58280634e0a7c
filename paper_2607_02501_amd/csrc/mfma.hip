// mfma.hip -- matrix-core path of the quantized linear layer for m > 4
// activation rows: prefill of image/text tokens, action-chunk denoising and
// video-latent tokens (paper section 2.1 / Table 1 model families; section 3.2
// "operator fusion, backend-specific dispatch").
//
// y[m][n] = sum_k x[m][k] * w_hat[n][k], w_hat = code * d16 rounded once to
// the activation type (bfloat16 or binary16), fp32 accumulation.
//
// A workgroup of WM x WN waves computes a BM x BN tile of y; each wave owns a
// (BM/WM) x (BN/WN) sub-tile held in fp32 accumulators (AGPRs).  Per K-tile of 64:
//   * global -> registers: the x tile (16-byte loads) and the packed weight
//     tile (16-byte loads of codes + binary16 scales), one K-tile ahead;
//   * registers -> LDS: x copied, weights dequantized (code * d16 exact in
//     fp32, one round-to-nearest-even to 16 bits) -- fused into the tile load,
//     no dequantized weight ever reaches HBM;
//   * LDS -> MFMA: v_mfma_f32_32x32x16_{bf16,f16}, A = x rows, B = w_hat rows.
// LDS is double-buffered, so one barrier per K-tile separates the MFMAs on
// buffer i from the dequantizing stores into buffer i+1; the stores are
// interleaved with the MFMA chain so VALU work overlaps the matrix cores.
//
// Tiles are ordered for the 8 XCDs of MI355X (workgroups are dispatched to
// XCDs round-robin, each XCD has its own L2): each XCD gets a contiguous range
// of tiles, N-tile fastest, so the workgroups sharing an L2 mostly share one
// block of x rows.
#include <hip/hip_runtime.h>

#include <cstdlib>

#include "eb_internal.h"

namespace eb {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;        // K elements per tile (2 blocks)
constexpr int kPad = 8;        // LDS row padding in 16-bit elements
constexpr int kLds = kBK + kPad;
constexpr int kXcds = 8;

template <int XT>
__device__ inline uint32_t pack2(float a, float b) {
  if (XT == EB_BF16) {
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    bf2 v = {(__bf16)a, (__bf16)b};  // v_cvt_pk_bf16_f32, round to nearest even
    return __builtin_bit_cast(uint32_t, v);
  }
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
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
  static constexpr int kElemsPerChunk = (QT == EB_Q8_0) ? 16 : 32;
};

// Dequantize one 16-byte chunk into LDS row `dst` (16-bit elements).
// Q8_0: 16 int8 codes.  u = q + 128 converts exactly with v_cvt_f32_ubyte and
// fma(u, d, -128 d) = q d exactly (all terms fit in fp32), then one RNE.
// Q4_0: 16 bytes, low nibbles = elements 0..15, high nibbles = 16..31, value
// (n - 8) d = fma(n, d, -8 d) exactly.
template <int QT, int XT>
__device__ inline void dequant_chunk(const uint4 q, float d, uint16_t *dst) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  if (QT == EB_Q8_0) {
    const float off = -128.0f * d;
    uint32_t o[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t u = w[j] ^ 0x80808080u;
      const float f0 = __builtin_fmaf((float)(u & 0xffu), d, off);
      const float f1 = __builtin_fmaf((float)((u >> 8) & 0xffu), d, off);
      const float f2 = __builtin_fmaf((float)((u >> 16) & 0xffu), d, off);
      const float f3 = __builtin_fmaf((float)(u >> 24), d, off);
      o[2 * j] = pack2<XT>(f0, f1);
      o[2 * j + 1] = pack2<XT>(f2, f3);
    }
    uint4 *p = reinterpret_cast<uint4 *>(dst);
    p[0] = make_uint4(o[0], o[1], o[2], o[3]);
    p[1] = make_uint4(o[4], o[5], o[6], o[7]);
  } else {
    const float off = -8.0f * d;
    uint32_t lo[8], hi[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t l = w[j] & 0x0f0f0f0fu, h = (w[j] >> 4) & 0x0f0f0f0fu;
      lo[2 * j] = pack2<XT>(__builtin_fmaf((float)(l & 0xffu), d, off),
                            __builtin_fmaf((float)((l >> 8) & 0xffu), d, off));
      lo[2 * j + 1] = pack2<XT>(__builtin_fmaf((float)((l >> 16) & 0xffu), d, off),
                                __builtin_fmaf((float)(l >> 24), d, off));
      hi[2 * j] = pack2<XT>(__builtin_fmaf((float)(h & 0xffu), d, off),
                            __builtin_fmaf((float)((h >> 8) & 0xffu), d, off));
      hi[2 * j + 1] = pack2<XT>(__builtin_fmaf((float)((h >> 16) & 0xffu), d, off),
                                __builtin_fmaf((float)(h >> 24), d, off));
    }
    uint4 *p = reinterpret_cast<uint4 *>(dst);
    p[0] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    p[1] = make_uint4(lo[4], lo[5], lo[6], lo[7]);
    p[2] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    p[3] = make_uint4(hi[4], hi[5], hi[6], hi[7]);
  }
}

template <int QT, int XT, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(WM *WN * 64)
    mfma_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off, int64_t ds,
                const uint16_t *__restrict__ x, int64_t m, void *__restrict__ y, int yt) {
  constexpr int T = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;        // wave sub-tile
  constexpr int FM = TM / 32, FN = TN / 32;        // 32x32 fragments per wave
  constexpr int ACH = BM * (kBK / 8) / T;          // x chunks per thread
  constexpr int WCPR = WTile<QT>::kChunksPerRow;
  constexpr int BCH = BN * WCPR / T;               // weight chunks per thread
  constexpr int KSTEPS = kBK / 16;
  static_assert(ACH * T == BM * (kBK / 8), "x tile must split evenly");
  static_assert(BCH * T == BN * WCPR, "weight tile must split evenly");
  static_assert(BCH % KSTEPS == 0 || KSTEPS % BCH == 0, "dequant interleave");

  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  // buffer b: A tile at lds + b * (BM + BN) * kLds, B tile right after it
  auto Abuf = [&](int b) { return lds + b * (BM + BN) * kLds; };
  auto Bbuf = [&](int b) { return lds + b * (BM + BN) * kLds + BM * kLds; };

  // XCD-aware tile order
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int64_t tiles = tiles_m * tiles_n;
  const int64_t bid = blockIdx.x;
  int64_t t = bid;
  if (tiles % kXcds == 0) t = (bid % kXcds) * (tiles / kXcds) + bid / kXcds;
  const int64_t tm = t / tiles_n, tn = t % tiles_n;
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
      areg[i] = (gm < m && gk < k) ? *reinterpret_cast<const uint4 *>(x + gm * k + gk)
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

  auto store_x = [&](uint16_t *A) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int idx = tid + i * T;
      const int r = idx / (kBK / 8), c8 = idx % (kBK / 8);
      *reinterpret_cast<uint4 *>(&A[r * kLds + c8 * 8]) = areg[i];
    }
  };
  auto store_w = [&](uint16_t *B, int i) {
    const int idx = tid + i * T;
    const int r = idx / WCPR, c = idx % WCPR;
    dequant_chunk<QT, XT>(breg[i], (float)__builtin_bit_cast(_Float16, dreg[i]),
                          &B[r * kLds + c * WTile<QT>::kElemsPerChunk]);
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
  store_x(Abuf(0));
#pragma unroll
  for (int i = 0; i < BCH; ++i) store_w(Bbuf(0), i);
  if (nk > 1) load_tile(1);
  __syncthreads();

  for (int64_t kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const uint16_t *A = Abuf(cur), *B = Bbuf(cur);
    const bool more = kt + 1 < nk;
    if (more) store_x(Abuf(cur ^ 1));
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int koff = ks * 16 + 8 * (lane >> 5);
      uint4 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(&A[(wm * TM + i * 32 + (lane & 31)) * kLds + koff]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const uint4 *>(&B[(wn * TN + j * 32 + (lane & 31)) * kLds + koff]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[i], bfr[j], acc[i][j]);
      // a share of the next tile's dequantization between MFMA groups
      if (more) {
        if constexpr (BCH >= KSTEPS) {
#pragma unroll
          for (int i = ks * (BCH / KSTEPS); i < (ks + 1) * (BCH / KSTEPS); ++i) store_w(Bbuf(cur ^ 1), i);
        } else {
          if (ks % (KSTEPS / BCH) == 0) store_w(Bbuf(cur ^ 1), ks / (KSTEPS / BCH));
        }
      }
    }
    if (kt + 2 < nk) load_tile(kt + 2);
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
  const size_t lds = (size_t)2 * (BM + BN) * kLds * sizeof(uint16_t);
  auto kern = mfma_kernel<QT, XT, BM, BN, WM, WN>;
  static bool attr_set = false;  // idempotent; a race only repeats the same call
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  kern<<<(unsigned)tiles, WM * WN * 64, lds, s>>>((const uint8_t *)wdata, n, k, L.d_off, L.ds,
                                                  (const uint16_t *)x, m, y, yt);
  return hipGetLastError();
}

// Tile configuration; EB_MFMA_CFG=<index> forces one (tuning).
int mfma_cfg_override() {
  static const int v = [] {
    const char *e = getenv("EB_MFMA_CFG");
    return e ? atoi(e) : -1;
  }();
  return v;
}

template <int QT, int XT>
hipError_t launch_q(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, hipStream_t s) {
  int cfg = mfma_cfg_override();
  if (cfg < 0) cfg = m <= 64 ? 0 : (m <= 128 ? 1 : 2);
  switch (cfg) {
    case 0: return launch_t<QT, XT, 64, 128, 2, 2>(wdata, n, k, x, m, y, yt, s);
    case 1: return launch_t<QT, XT, 128, 128, 2, 2>(wdata, n, k, x, m, y, yt, s);
    case 2: return launch_t<QT, XT, 256, 256, 2, 2>(wdata, n, k, x, m, y, yt, s);
    case 3: return launch_t<QT, XT, 256, 256, 2, 4>(wdata, n, k, x, m, y, yt, s);
    case 4: return launch_t<QT, XT, 128, 256, 2, 2>(wdata, n, k, x, m, y, yt, s);
    case 5: return launch_t<QT, XT, 256, 128, 2, 2>(wdata, n, k, x, m, y, yt, s);
    case 6: return launch_t<QT, XT, 128, 256, 2, 4>(wdata, n, k, x, m, y, yt, s);
    default: return launch_t<QT, XT, 256, 256, 4, 2>(wdata, n, k, x, m, y, yt, s);
  }
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
