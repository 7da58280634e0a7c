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

#include <algorithm>
#include <cstdlib>

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
// 16-bit output type (the op's type decides).  Measured on 50-row chains,
// more weight rows per workgroup (32 or 64, the waves split between row
// groups and slices of k) were slower: a workgroup's time grows with the
// blocks each wave walks, at about 1.2 us per block, since every workgroup
// also reads all of x through its compute unit.
template <int QT, int XT, int YT, int MB, bool HL>
__global__ void __launch_bounds__(kWaves * 64)
    mm_narrow_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off,
                     int64_t ds, const uint16_t *__restrict__ x, int m, void *__restrict__ y, int yt,
                     Fuse f, int splits, float *__restrict__ ws, int64_t ws_stride) {
  static_assert(!HL || XT == EB_BF16, "hi/lo pairs are for bfloat16 activations");
  constexpr int KS = kWaves;                        // slices of k
  constexpr int NT = 16;                            // weight rows per workgroup
  constexpr int PAIRS = MB * 64 * 2;                // output pairs per workgroup
  constexpr int PPT = (PAIRS + kWaves * 64 - 1) / (kWaves * 64);
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;  // code bytes per block
  __shared__ f32x4_t red[KS][MB][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // consecutive workgroups start on different slices, so that they do not
  // all read the same activations at once
  const int slice = (wave + (int)(blockIdx.x % KS)) % KS;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * NT;
  const int rows_n = (int)min((int64_t)NT, n - n0);
  // split blockIdx.y of `splits` takes blocks [sb0, sb1) of k; its waves
  // split that range further
  const int nb = (int)(k / kQK);
  const int sp = (int)blockIdx.y;
  const int sb0 = (int)((int64_t)nb * sp / splits), sb1 = (int)((int64_t)nb * (sp + 1) / splits);
  const int b0 = sb0 + (int)((int64_t)(sb1 - sb0) * slice / KS);
  const int b1 = sb0 + (int)((int64_t)(sb1 - sb0) * (slice + 1) / KS);

  // Raw buffer descriptors over this workgroup's rows (rows past n read
  // zeros) and over x's m rows (rows past m read zeros).
  const uint32_t qrow = (uint32_t)nb * QSB, drow = (uint32_t)ds * 2;
  const auto qr = rsrc(wdata + n0 * qrow, (uint32_t)rows_n * qrow);
  const auto dr = rsrc(wdata + d_off + n0 * drow, (uint32_t)rows_n * drow);
  const uint32_t xrow = (uint32_t)k * 2;
  const auto xr = rsrc(x, (uint32_t)m * xrow);
  // lane parts of the offsets: row r16 of the workgroup; Q8_0 codes 8 g4 ..
  // + 7 of the block, Q4_0 the bytes 8 (g4 & 1) .. + 7 (nibble g4 >> 1)
  const uint32_t wr = (uint32_t)r16;
  const uint32_t qlane = wr * qrow + (QT == EB_Q8_0 ? 8u * g4 : 8u * (g4 & 1));
  const uint32_t dlane = wr * drow;
  const uint32_t xlane = (uint32_t)r16 * xrow + 16u * g4;
  const bool nib_hi = (g4 >> 1) != 0;

  // The residuals of this thread's outputs are loaded first, so that their
  // latency passes under the product's.  Every load below is issued
  // unconditionally (an offset past the end of its buffer reads zero without
  // touching memory), so that each wait counts only the loads it needs.
  constexpr uint32_t kPast = 0x80000000u;  // past every descriptor here
  const int t = threadIdx.x;
  float res[PPT][2];
  if (f.epi == EB_EPI_ADD && !ws) {  // (a split's reduction adds the residual)
    constexpr uint32_t es = (YT == EB_F32) ? 4 : 2;
    const auto rr = rsrc(f.r, (uint32_t)(m * n) * es);
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int e = t + i * kWaves * 64;
      const int mb = e / 128, l = (e % 128) / 2, p = e % 2;
      const int col = 16 * mb + (l & 15), nl = 4 * (l >> 4) + 2 * p;
      const uint32_t o = (uint32_t)((int64_t)col * n + n0 + nl) * es;
      const bool ok0 = e < PAIRS && col < m && nl < rows_n, ok1 = ok0 && nl + 1 < rows_n;
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
    uint2 q;
    uint16_t d;
    uint4 xb[MB];
  };
  // block j of this wave's slice; past the slice, zeros (code 0 with scale 0
  // and activations 0 add exactly nothing to the accumulators)
  const int nbw = b1 - b0;
  auto load = [&](Blk &B, int j) __attribute__((always_inline)) {
    const bool ok = j < nbw;
    const uint32_t b = (uint32_t)(b0 + j);
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(qr, (int)(ok ? qlane + b * QSB : kPast), 0, 0);
    B.q = make_uint2(v[0], v[1]);
    B.d = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)(ok ? dlane + 2u * b : kPast), 0, 0);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      B.xb[mb] = bload(xr, ok ? xlane + (uint32_t)mb * 16u * xrow + b * 64u : kPast);
  };

  f32x4_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // issued block by block, each one's loads together, so that the wait
  // before a block's MFMAs leaves the later blocks' loads in flight
  Blk S0, S1, S2, S3;
  load(S0, 0);
  __builtin_amdgcn_sched_barrier(0);
  load(S1, 1);
  __builtin_amdgcn_sched_barrier(0);
  load(S2, 2);
  __builtin_amdgcn_sched_barrier(0);
  load(S3, 3);
  __builtin_amdgcn_sched_barrier(0);
  // one block: its MFMAs, then its registers take the block kAhead further
  auto step = [&](Blk &B, int j) __attribute__((always_inline)) {
    uint4 wh, wl;
    deq8<QT, XT, HL>(B.q, nib_hi, (float)__builtin_bit_cast(_Float16, B.d), wh, wl);
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
  // element e of this thread: output pair (rows 2 p, 2 p + 1 of the lane's 4
  // rows) of one column; e runs over (mb, lane, pair)
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int e = t + i * kWaves * 64;
    if (e >= PAIRS) break;
    const int mb = e / 128, l = (e % 128) / 2, p = e % 2;
    float v0 = 0.f, v1 = 0.f;
#pragma unroll
    for (int w = 0; w < KS; ++w) {
      const f32x4_t a = red[w][mb][l];
      v0 += p ? a[2] : a[0];
      v1 += p ? a[3] : a[1];
    }
    const int col = 16 * mb + (l & 15);               // row of x / y
    const int nl = 4 * (l >> 4) + 2 * p;              // first of the two rows
    if (col >= m || nl >= rows_n) continue;
    if (ws) {  // a split of k: the raw partial sums, for the ordered reduction
      float *w = ws + (int64_t)sp * ws_stride + (int64_t)col * n + n0 + nl;
      w[0] = v0;
      if (nl + 1 < rows_n) w[1] = v1;
      continue;
    }
    if (f.epi == EB_EPI_GLU) {  // n even: the pair (gate, up) is complete
      store_y(y, (int64_t)col * (n / 2) + (n0 + nl) / 2, silu_mul(v0, v1), yt);
      continue;
    }
    const int64_t o = (int64_t)col * n + n0 + nl;
    if (f.epi == EB_EPI_ADD) {  // the residual shares the output's type
      v0 += res[i][0];
      v1 += res[i][1];
    }
    store_y(y, o, v0, yt);
    if (nl + 1 < rows_n) store_y(y, o + 1, v1, yt);
  }
}

struct Split {
  int splits;
  float *ws;
  int64_t stride;
};

template <int QT, int XT, int YT, bool HL>
hipError_t launch_mb(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                     int32_t yt, const Fuse &f, const Split &sp, hipStream_t s) {
  const Layout L = layout_of(QT, n, k);
  const dim3 grid((unsigned)((n + 15) / 16), (unsigned)sp.splits);
  const auto *xp = static_cast<const uint16_t *>(x);
  const auto *wp = static_cast<const uint8_t *>(wdata);
  if (m <= 16)
    mm_narrow_kernel<QT, XT, YT, 1, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f, sp.splits, sp.ws, sp.stride);
  else if (m <= 32)
    mm_narrow_kernel<QT, XT, YT, 2, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f, sp.splits, sp.ws, sp.stride);
  else
    mm_narrow_kernel<QT, XT, YT, 4, HL><<<grid, kWaves * 64, 0, s>>>(wp, n, k, L.d_off, L.ds, xp, (int)m, y, yt, f, sp.splits, sp.ws, sp.stride);
  return hipGetLastError();
}

template <int QT, int XT, bool HL>
hipError_t launch_y(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, const Split &sp, hipStream_t s) {
  if (yt == EB_F32) return launch_mb<QT, XT, EB_F32, HL>(wdata, n, k, x, m, y, yt, f, sp, s);
  return launch_mb<QT, XT, EB_BF16, HL>(wdata, n, k, x, m, y, yt, f, sp, s);
}

template <int QT>
hipError_t launch_x(int32_t xt, bool hl, const void *wdata, int64_t n, int64_t k, const void *x,
                    int64_t m, void *y, int32_t yt, const Fuse &f, const Split &sp, hipStream_t s) {
  if (xt == EB_F16) return launch_y<QT, EB_F16, false>(wdata, n, k, x, m, y, yt, f, sp, s);
  if (hl) return launch_y<QT, EB_BF16, true>(wdata, n, k, x, m, y, yt, f, sp, s);
  return launch_y<QT, EB_BF16, false>(wdata, n, k, x, m, y, yt, f, sp, s);
}

}  // namespace

bool narrow_fits(int64_t m, int64_t n, int64_t k, int splits) {
  // Every workgroup reads all of x for its share of k (up to 64 rows), which
  // for a long share costs more than it saves: measured on the action-expert
  // chain, k = 1024 projections take 8-10 us instead of about 16 us (tiled
  // kernel split along k plus its reduction), but an unsplit k = 4096 down
  // projection 22 us instead of 16.  Offsets in x, a workgroup's weights and
  // y stay below 2^31 (an offset of 2^31 reads zero).
  return m >= 1 && m <= kNarrowMaxM && splits >= 1 && splits <= kNarrowMaxSplits &&
         (splits == 1 || k / kQK >= (int64_t)splits * 8) && k / splits <= kNarrowMaxK &&
         (int64_t)m * k * 2 < 0x7fff0000LL && (int64_t)64 * (k / kQK) * 34 < 0x7fff0000LL &&
         (int64_t)m * n * 4 < 0x7fff0000LL;
}

// Splits of k for a lone small-m projection: when its 16-row workgroups do not
// fill the GPU, k is split so that they do (about one workgroup per CU), each
// split writing partial sums for the ordered reduction -- a narrow launch's
// time follows the activation bytes each workgroup reads through its CU.
int narrow_splits(int64_t n, int64_t k, int cus) {
  static const int env = [] {
    const char *e = std::getenv("EB_NARROW_SPLITS");
    return e ? std::atoi(e) : 0;
  }();
  const int64_t wgs = (n + 15) / 16, nb = k / kQK;
  int sp = env > 0 ? env : (int)std::max<int64_t>(1, cus / std::max<int64_t>(1, wgs));
  sp = (int)std::min<int64_t>({(int64_t)sp, (int64_t)kNarrowMaxSplits, nb / 8});
  // a split of 2 saves each wave half its blocks (about 1.2 us each) but adds
  // the reduction launch: on the 50-row chains the 2048-wide QKV projection
  // (4 blocks per wave) ran faster unsplit
  if (env <= 0 && sp == 2) sp = 1;
  if (k / std::max(sp, 1) > kNarrowMaxK)  // shares of at most kNarrowMaxK
    sp = (int)std::min<int64_t>(kNarrowMaxSplits, (k + kNarrowMaxK - 1) / kNarrowMaxK);
  return std::max(sp, 1);
}

hipError_t launch_mfma_narrow(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                              int32_t xt, bool hl, int64_t m, void *y, int32_t yt, const Fuse &f,
                              int splits, float *ws, int64_t ws_stride, hipStream_t s) {
  if (!narrow_fits(m, n, k, splits) || (splits > 1 && !ws)) return hipErrorInvalidValue;
  const Split sp{splits, splits > 1 ? ws : nullptr, ws_stride};
  if (type == EB_Q4_0) return launch_x<EB_Q4_0>(xt, hl, wdata, n, k, x, m, y, yt, f, sp, s);
  return launch_x<EB_Q8_0>(xt, hl, wdata, n, k, x, m, y, yt, f, sp, s);
}

}  // namespace eb
