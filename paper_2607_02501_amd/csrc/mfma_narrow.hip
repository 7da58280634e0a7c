// mfma_narrow.hip -- lone small-m projections (m <= 64) on the matrix cores
// in one launch: a workgroup owns 16 weight rows and the whole of k, its
// waves split k between them and add their partial tiles through LDS, so no
// second kernel reduces a split of k (paper section 3.2: latency-first
// batch-1 execution; the action-expert projections of section 2.1 / Table 1
// run one after another, m = 50 rows, 1-9 MB of weights each, and a
// dependent chain of them pays every launch).
//
// Per 32-weight block (one MFMA k-step, v_mfma_f32_16x16x32): lane l holds
// the 8 weights k = 8 (l / 16) .. + 7 of row l % 16 of the block (A operand,
// dequantized in registers) and the 8 activations of the same k of row
// 16 mb + l % 16 of x for each 16-row block mb of m (B operands, loaded from
// global memory, where x stays in cache for the whole launch).  A lane's
// accumulators then hold rows 4 (l / 16) + i of the tile, i = 0..3, of
// column 16 mb + l % 16.  Blocks of a wave's share of k are loaded four
// ahead of their MFMAs.
#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"

namespace eb {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int XT>
__device__ inline f32x4_t mfma16(const uint4 a, const uint4 b, f32x4_t c) {
  if (XT == EB_BF16)
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

constexpr int kNT = 16;     // weight rows per workgroup
constexpr int kWaves = 8;   // waves per workgroup, splitting k
constexpr int kAhead = 4;   // blocks loaded ahead of their MFMAs

// 8 codes of one block (Q8_0: 8 int8 bytes; Q4_0: the nibble `hi` of 8
// bytes) with scale d -> 8 weights in MFMA operand order, rounded once to
// the activation type, or as hi/lo bfloat16 pairs (HL).
template <int QT, int XT, bool HL>
__device__ inline void deq8(uint2 q, bool hi, float d, uint4 &wh, uint4 &wl) {
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  uint32_t a, b;
  float c;
  if constexpr (QT == EB_Q8_0) {
    a = q.x ^ 0x80808080u;
    b = q.y ^ 0x80808080u;
    c = -1152.0f * d;
  } else {
    const int sh = hi ? 4 : 0;
    a = (q.x >> sh) & 0x0f0f0f0fu;
    b = (q.y >> sh) & 0x0f0f0f0fu;
    c = -1032.0f * d;
  }
  if constexpr (HL) {
    deq_pair_hl(under_1024(a, kSelLo), d, c, wh.x, wl.x);
    deq_pair_hl(under_1024(a, kSelHi), d, c, wh.y, wl.y);
    deq_pair_hl(under_1024(b, kSelLo), d, c, wh.z, wl.z);
    deq_pair_hl(under_1024(b, kSelHi), d, c, wh.w, wl.w);
  } else {
    wh = make_uint4(deq_pair<XT>(under_1024(a, kSelLo), d, c), deq_pair<XT>(under_1024(a, kSelHi), d, c),
                    deq_pair<XT>(under_1024(b, kSelLo), d, c), deq_pair<XT>(under_1024(b, kSelHi), d, c));
  }
}

// MB: 16-row blocks of m (m <= 16 MB).  YT: EB_F32, or EB_BF16 for either
// 16-bit output type (the op's type decides).
template <int QT, int XT, int YT, int MB, bool HL>
__global__ void __launch_bounds__(kWaves * 64)
    mm_narrow_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off,
                     int64_t ds, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int yt,
                     Fuse f) {
  static_assert(!HL || XT == EB_BF16, "hi/lo pairs are for bfloat16 activations");
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;  // code bytes per block
  __shared__ f32x4_t red[kWaves][MB][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g4 = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * kNT;
  const int rows_n = (int)min((int64_t)kNT, n - n0);
  const int nb = (int)(k / kQK);
  const int b0 = (int)((int64_t)nb * wave / kWaves), b1 = (int)((int64_t)nb * (wave + 1) / kWaves);

  // Raw buffer descriptors over this workgroup's rows (rows past n read
  // zeros) and over x's m rows (rows past m read zeros).
  const uint32_t qrow = (uint32_t)nb * QSB, drow = (uint32_t)ds * 2;
  const auto qr = rsrc(wdata + n0 * qrow, (uint32_t)rows_n * qrow);
  const auto dr = rsrc(wdata + d_off + n0 * drow, (uint32_t)rows_n * drow);
  const uint32_t xrow = (uint32_t)k * 2;
  const auto xr = rsrc(x, (uint32_t)m * xrow);
  // lane parts of the offsets: Q8_0 codes 8 g4 .. + 7 of the block, Q4_0 the
  // bytes 8 (g4 & 1) .. + 7 (nibble g4 >> 1)
  const uint32_t qlane = (uint32_t)r16 * qrow + (QT == EB_Q8_0 ? 8u * g4 : 8u * (g4 & 1));
  const uint32_t dlane = (uint32_t)r16 * drow;
  const uint32_t xlane = (uint32_t)r16 * xrow + 16u * g4;
  const bool nib_hi = (g4 >> 1) != 0;

  struct Blk {
    uint2 q;
    uint16_t d;
    uint4 xb[MB];
  };
  auto load = [&](Blk &B, int b) __attribute__((always_inline)) {
    const uint32_t qo = qlane + (uint32_t)b * QSB;
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(qr, (int)qo, 0, 0);
    B.q = make_uint2(v[0], v[1]);
    B.d = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)(dlane + 2u * b), 0, 0);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      B.xb[mb] = bload(xr, xlane + (uint32_t)mb * 16u * xrow + (uint32_t)b * 64u);
  };

  f32x4_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  Blk S0, S1, S2, S3;
  int b = b0;
  if (b0 + 0 < b1) load(S0, b0 + 0);
  if (b0 + 1 < b1) load(S1, b0 + 1);
  if (b0 + 2 < b1) load(S2, b0 + 2);
  if (b0 + 3 < b1) load(S3, b0 + 3);
  // one block: its MFMAs, then its registers take the block kAhead further
  auto step = [&](Blk &B) __attribute__((always_inline)) -> bool {
    if (b >= b1) return false;
    uint4 wh, wl;
    deq8<QT, XT, HL>(B.q, nib_hi, (float)__builtin_bit_cast(_Float16, B.d), wh, wl);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16<XT>(wh, B.xb[mb], acc[mb]);
    if constexpr (HL) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16<XT>(wl, B.xb[mb], acc[mb]);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (b + kAhead < b1) load(B, b + kAhead);
    ++b;
    return true;
  };
  while (step(S0) && step(S1) && step(S2) && step(S3)) {
  }

  // partial tiles of the waves, added in wave order
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) red[wave][mb][lane] = acc[mb];
  __syncthreads();
  // thread t: output pair (rows 2 p, 2 p + 1 of the tile) of one column:
  // flat index e = t over (mb, lane, pair), pair p in 0..1 of the lane's 4 rows
  const int t = threadIdx.x;
  if (t >= MB * 64 * 2) return;
  const int mb = t / 128, rest = t % 128, l = rest / 2, p = rest % 2;
  float v0 = 0.f, v1 = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const f32x4_t a = red[w][mb][l];
    v0 += p ? a[2] : a[0];
    v1 += p ? a[3] : a[1];
  }
  const int col = 16 * mb + (l & 15);         // row of x / y
  const int nl = 4 * (l >> 4) + 2 * p;         // first of the two tile rows
  if (col >= m || nl >= rows_n) return;
  if (f.epi == EB_EPI_GLU) {  // n even: the pair (gate, up) is complete
    store_y(y, (int64_t)col * (n / 2) + (n0 + nl) / 2, silu_mul(v0, v1), yt);
    return;
  }
  const int64_t o = (int64_t)col * n + n0 + nl;
  put_y(y, o, v0, yt, f);
  if (nl + 1 < rows_n) put_y(y, o + 1, v1, yt, f);
}

template <int QT, int XT, int YT, bool HL>
hipError_t launch_mb(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                     int32_t yt, const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(QT, n, k);
  const unsigned grid = (unsigned)((n + kNT - 1) / kNT);
  const auto *xp = static_cast<const uint16_t *>(x);
  const auto *wp = static_cast<const uint8_t *>(wdata);
  if (m <= 16)
    mm_narrow_kernel<QT, XT, YT, 1, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f);
  else if (m <= 32)
    mm_narrow_kernel<QT, XT, YT, 2, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f);
  else
    mm_narrow_kernel<QT, XT, YT, 4, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f);
  return hipGetLastError();
}

template <int QT, int XT, bool HL>
hipError_t launch_y(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, hipStream_t s) {
  if (yt == EB_F32) return launch_mb<QT, XT, EB_F32, HL>(wdata, n, k, x, m, y, yt, f, s);
  return launch_mb<QT, XT, EB_BF16, HL>(wdata, n, k, x, m, y, yt, f, s);
}

template <int QT>
hipError_t launch_x(int32_t xt, bool hl, const void *wdata, int64_t n, int64_t k, const void *x,
                    int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  if (xt == EB_F16) return launch_y<QT, EB_F16, false>(wdata, n, k, x, m, y, yt, f, s);
  if (hl) return launch_y<QT, EB_BF16, true>(wdata, n, k, x, m, y, yt, f, s);
  return launch_y<QT, EB_BF16, false>(wdata, n, k, x, m, y, yt, f, s);
}

}  // namespace

bool narrow_fits(int64_t m, int64_t n, int64_t k) {
  // Every workgroup reads all of x (up to 64 rows of k), which for long k
  // costs more than it saves: measured on the action-expert chain, k = 1024
  // projections take 8-10 us instead of about 16 us (tiled kernel split along
  // k plus its reduction), but the k = 4096 down projection 22 us instead of
  // 16.  Every byte span of a workgroup stays within 32-bit buffer offsets.
  return m >= 1 && m <= kNarrowMaxM && k <= kNarrowMaxK && (int64_t)m * k * 2 <= 0x7fffffffLL &&
         (int64_t)kNT * (k / kQK) * 34 <= 0x7fffffffLL && (n + kNT - 1) / kNT <= 0x7fffffffLL;
}

hipError_t launch_mfma_narrow(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                              int32_t xt, bool hl, int64_t m, void *y, int32_t yt, const Fuse &f,
                              hipStream_t s) {
  if (!narrow_fits(m, n, k)) return hipErrorInvalidValue;
  if (type == EB_Q4_0) return launch_x<EB_Q4_0>(xt, hl, wdata, n, k, x, m, y, yt, f, s);
  return launch_x<EB_Q8_0>(xt, hl, wdata, n, k, x, m, y, yt, f, s);
}

}  // namespace eb
