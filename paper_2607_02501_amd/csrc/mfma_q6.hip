// mfma_q6.hip -- linear layers on Q6_S weights (the 6-bit configuration of
// paper section 4, Table 3) on the matrix cores, in one launch: the path for
// m <= 128 (and for any m the tile kernel cannot address); larger m takes the
// tile kernel of the other formats (mfma_tile.h).
//
// Q6_S: super-blocks of 256 weights along k, 16 int8 sub-block scales sc_j
// under one binary16 scale d16, 6-bit codes u (w_hat = (u - 32) d16 sc_j).
// Planar device layout: a code plane of 24-byte chunks per 32 weights (16
// bytes of low nibbles as in Q4_0, byte i = lo(u_i) | lo(u_{i+16}) << 4, then
// 8 bytes of top bits, byte t = the top two bits of u_t, u_{t+8}, u_{t+16},
// u_{t+24}), a sub-scale plane (k / 16 bytes per row) and a binary16 scale
// plane (round_up(k / 256, 8) entries per row).
//
// A workgroup owns 16 weight rows and up to 64 rows of x (16 MB rows,
// MB = 1, 2, 4), the whole of k, split over its 8 waves; the waves' partial
// tiles are added through LDS in slice order.  Per 32-weight chunk (one
// v_mfma_f32_16x16x32 k-step) lane l holds the 8 weights k = 8 (l / 16) ..
// + 7 of row l % 16 (A operand, dequantized in registers) and the same 8
// activations of row 16 mb + l % 16 of the x tile for each mb (B operands).
// Dequantization places u under 1024 in binary16 and computes
// fma(1024 + u, e, -1056 e) = (u - 32) e exactly in fp32 (e = d16 sc_j has at
// most 18 significant bits), then rounds once to binary16 for binary16
// activations or splits into bfloat16 hi/lo pairs (w_hat to within 2^-16)
// for bfloat16 ones.
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

constexpr int kWaves = 8;  // waves per workgroup, splitting k
constexpr int kAhead = 4;  // chunks loaded ahead of their MFMAs

// 8 codes of a lane (low nibbles `lo` selected by nib_hi, top bits `hi`
// shifted by 2 g4) with e = d16 sc -> 8 weights in MFMA operand order.
template <int XT, bool HL>
__device__ inline void deq8_q6(uint2 lo, uint2 hi, int sh_lo, int sh_hi, float e, uint4 &wh,
                               uint4 &wl) {
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  const uint32_t a = ((lo.x >> sh_lo) & 0x0f0f0f0fu) | (((hi.x >> sh_hi) & 0x03030303u) << 4);
  const uint32_t b = ((lo.y >> sh_lo) & 0x0f0f0f0fu) | (((hi.y >> sh_hi) & 0x03030303u) << 4);
  const float c = -1056.0f * e;
  if constexpr (HL) {
    deq_pair_hl(under_1024(a, kSelLo), e, c, wh.x, wl.x);
    deq_pair_hl(under_1024(a, kSelHi), e, c, wh.y, wl.y);
    deq_pair_hl(under_1024(b, kSelLo), e, c, wh.z, wl.z);
    deq_pair_hl(under_1024(b, kSelHi), e, c, wh.w, wl.w);
  } else {
    wh = make_uint4(deq_pair<XT>(under_1024(a, kSelLo), e, c), deq_pair<XT>(under_1024(a, kSelHi), e, c),
                    deq_pair<XT>(under_1024(b, kSelLo), e, c), deq_pair<XT>(under_1024(b, kSelHi), e, c));
  }
}

// YT: EB_F32, or EB_BF16 for either 16-bit output type (the op's type decides).
template <int XT, int YT, int MB, bool HL>
__global__ void __launch_bounds__(kWaves * 64)
    mm_q6_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t sc_off,
                 int64_t d_off, int64_t ds, const uint16_t *__restrict__ x, int64_t m,
                 void *__restrict__ y, int yt, Fuse f) {
  static_assert(!HL || XT == EB_BF16, "hi/lo pairs are for bfloat16 activations");
  constexpr int PAIRS = MB * 64 * 2;  // output pairs per workgroup
  constexpr int PPT = (PAIRS + kWaves * 64 - 1) / (kWaves * 64);
  constexpr uint32_t kPast = 0x80000000u;  // past every descriptor here: reads zero
  __shared__ f32x4_t red[kWaves][MB][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // consecutive workgroups start on different slices of k
  const int slice = (wave + (int)(blockIdx.x % kWaves)) % kWaves;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t m0 = (int64_t)blockIdx.y * (16 * MB);
  const int rows_n = (int)min((int64_t)16, n - n0);
  const int rows_m = (int)min((int64_t)(16 * MB), m - m0);
  const int nb = (int)(k / kQK);
  const int b0 = (int)((int64_t)nb * slice / kWaves), b1 = (int)((int64_t)nb * (slice + 1) / kWaves);

  // descriptors over this workgroup's weight rows and x rows (rows past the
  // end read zeros)
  const uint32_t qrow = (uint32_t)nb * 24, srow = (uint32_t)(k / 16), drow = (uint32_t)ds * 2;
  const auto qr = rsrc(wdata + n0 * qrow, (uint32_t)rows_n * qrow);
  const auto sr = rsrc(wdata + sc_off + n0 * srow, (uint32_t)rows_n * srow);
  const auto dr = rsrc(wdata + d_off + n0 * drow, (uint32_t)rows_n * drow);
  const uint32_t xrow = (uint32_t)k * 2;
  const auto xr = rsrc(x + m0 * k, (uint32_t)rows_m * xrow);
  const uint32_t qlane = (uint32_t)r16 * qrow + 8u * (g4 & 1);
  const uint32_t slane = (uint32_t)r16 * srow + (uint32_t)(g4 >> 1);
  const uint32_t dlane = (uint32_t)r16 * drow;
  const uint32_t xlane = (uint32_t)r16 * xrow + 16u * g4;
  const int sh_lo = (g4 >> 1) * 4, sh_hi = 2 * g4;

  // residuals of this thread's outputs, loaded before the product
  const int t = threadIdx.x;
  float res[PPT][2];
  if (f.epi == EB_EPI_ADD) {
    constexpr uint32_t es = (YT == EB_F32) ? 4 : 2;
    const auto rr = rsrc(static_cast<const uint8_t *>(f.r) + m0 * n * es,
                         (uint32_t)(rows_m * n) * es);
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int e = t + i * kWaves * 64;
      const int mb = e / 128, l = (e % 128) / 2, p = e % 2;
      const int col = 16 * mb + (l & 15), nl = 4 * (l >> 4) + 2 * p;
      const uint32_t o = (uint32_t)((int64_t)col * n + n0 + nl) * es;
      const bool ok0 = e < PAIRS && col < rows_m && nl < rows_n, ok1 = ok0 && nl + 1 < rows_n;
      if constexpr (YT == EB_F32) {
        res[i][0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (int)(ok0 ? o : kPast), 0, 0));
        res[i][1] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (int)(ok1 ? o + 4 : kPast), 0, 0));
      } else {
        res[i][0] = from_y16(__builtin_amdgcn_raw_buffer_load_b16(rr, (int)(ok0 ? o : kPast), 0, 0), yt);
        res[i][1] = from_y16(__builtin_amdgcn_raw_buffer_load_b16(rr, (int)(ok1 ? o + 2 : kPast), 0, 0), yt);
      }
    }
  }

  struct Blk {
    uint2 lo, hi;
    uint16_t d;
    uint8_t sc;
    uint4 xb[MB];
  };
  // chunk j of this wave's slice; past the slice, zeros (code 0 under scale 0
  // and activations 0 add exactly nothing)
  const int nbw = b1 - b0;
  auto load = [&](Blk &B, int j) __attribute__((always_inline)) {
    const bool ok = j < nbw;
    const uint32_t b = (uint32_t)(b0 + j);
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(qr, (int)(ok ? qlane + b * 24u : kPast), 0, 0);
    const auto h = __builtin_amdgcn_raw_buffer_load_b64(qr, (int)(ok ? (uint32_t)r16 * qrow + b * 24u + 16u : kPast), 0, 0);
    B.lo = make_uint2(v[0], v[1]);
    B.hi = make_uint2(h[0], h[1]);
    B.sc = __builtin_amdgcn_raw_buffer_load_b8(sr, (int)(ok ? slane + 2u * b : kPast), 0, 0);
    B.d = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)(ok ? dlane + 2u * (b >> 3) : kPast), 0, 0);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      B.xb[mb] = bload(xr, ok ? xlane + (uint32_t)mb * 16u * xrow + b * 64u : kPast);
  };

  f32x4_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  Blk S0, S1, S2, S3;
  load(S0, 0);
  __builtin_amdgcn_sched_barrier(0);
  load(S1, 1);
  __builtin_amdgcn_sched_barrier(0);
  load(S2, 2);
  __builtin_amdgcn_sched_barrier(0);
  load(S3, 3);
  __builtin_amdgcn_sched_barrier(0);
  auto step = [&](Blk &B, int j) __attribute__((always_inline)) {
    const float e = (float)__builtin_bit_cast(_Float16, B.d) * (float)(int8_t)B.sc;  // exact
    uint4 wh, wl;
    deq8_q6<XT, HL>(B.lo, B.hi, sh_lo, sh_hi, e, wh, wl);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16<XT>(wh, B.xb[mb], acc[mb]);
    if constexpr (HL) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma16<XT>(wl, B.xb[mb], acc[mb]);
    }
    __builtin_amdgcn_sched_barrier(0);
    load(B, j + kAhead);
    __builtin_amdgcn_sched_barrier(0);
  };
  static_assert(kAhead == 4, "four register sets");
  for (int j = 0; j < nbw; j += 4) {
    step(S0, j);
    step(S1, j + 1);
    step(S2, j + 2);
    step(S3, j + 3);
  }

  // partial tiles of the slices, added in slice order
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) red[slice][mb][lane] = acc[mb];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int e = t + i * kWaves * 64;
    if (e >= PAIRS) break;
    const int mb = e / 128, l = (e % 128) / 2, p = e % 2;
    float v0 = 0.f, v1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const f32x4_t a = red[w][mb][l];
      v0 += p ? a[2] : a[0];
      v1 += p ? a[3] : a[1];
    }
    const int col = 16 * mb + (l & 15);               // row of the x tile
    const int nl = 4 * (l >> 4) + 2 * p;              // first of the two weight rows
    if (col >= rows_m || nl >= rows_n) continue;
    const int64_t row = m0 + col;
    if (f.epi == EB_EPI_GLU) {  // n even: the pair (gate, up) is complete
      store_y(y, row * (n / 2) + (n0 + nl) / 2, silu_mul(v0, v1), yt);
      continue;
    }
    const int64_t o = row * n + n0 + nl;
    if (f.epi == EB_EPI_ADD) {  // the residual shares the output's type
      v0 += res[i][0];
      v1 += res[i][1];
    }
    store_y(y, o, v0, yt);
    if (nl + 1 < rows_n) store_y(y, o + 1, v1, yt);
  }
}

template <int XT, int YT, bool HL>
hipError_t launch_mb(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                     int32_t yt, const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(EB_Q6_S, n, k);
  const auto *xp = static_cast<const uint16_t *>(x);
  const auto *wp = static_cast<const uint8_t *>(wdata);
  const unsigned gx = (unsigned)((n + 15) / 16);
  if (m <= 16) {
    mm_q6_kernel<XT, YT, 1, HL><<<dim3(gx, 1), kWaves * 64, 0, s>>>(wp, n, k, L.sc_off, L.d_off, L.ds, xp, m, y, yt, f);
  } else if (m <= 32) {
    mm_q6_kernel<XT, YT, 2, HL><<<dim3(gx, 1), kWaves * 64, 0, s>>>(wp, n, k, L.sc_off, L.d_off, L.ds, xp, m, y, yt, f);
  } else {
    const unsigned gy = (unsigned)((m + 63) / 64);
    mm_q6_kernel<XT, YT, 4, HL><<<dim3(gx, gy), kWaves * 64, 0, s>>>(wp, n, k, L.sc_off, L.d_off, L.ds, xp, m, y, yt, f);
  }
  return hipGetLastError();
}

}  // namespace

bool q6_fits(int64_t m, int64_t n, int64_t k) {
  // 32-bit offsets: a 64-row x tile, a workgroup's 16 weight rows, a 64-row
  // residual tile; the grid's y dimension
  return m >= 1 && k % kQK6 == 0 && 64 * k * 2 < 0x7fff0000LL && 16 * (k / kQK) * 24 < 0x7fff0000LL &&
         64 * n * 4 < 0x7fff0000LL && (m + 63) / 64 <= 65535;
}

hipError_t launch_mfma_q6(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt,
                          int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  if (!q6_fits(m, n, k)) return hipErrorInvalidValue;
  if (xt == EB_F16) {
    if (yt == EB_F32) return launch_mb<EB_F16, EB_F32, false>(wdata, n, k, x, m, y, yt, f, s);
    return launch_mb<EB_F16, EB_BF16, false>(wdata, n, k, x, m, y, yt, f, s);
  }
  if (yt == EB_F32) return launch_mb<EB_BF16, EB_F32, true>(wdata, n, k, x, m, y, yt, f, s);
  return launch_mb<EB_BF16, EB_BF16, true>(wdata, n, k, x, m, y, yt, f, s);
}

}  // namespace eb
