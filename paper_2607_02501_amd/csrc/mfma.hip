// mfma.hip -- host side of the matrix-core path of the quantized linear
// layer (paper section 3.2, backend-specific dispatch): the tile
// configurations and the cost model that picks one per problem (and a split
// of k when a problem has too few tiles to fill the GPU), the grouped-launch
// planner, the ordered split-K reduction kernel, and the dispatch to the tile
// kernel's per-format instantiations (mfma_tile.h, mfma_<format>_<x>.hip).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdlib>
#include <iterator>
#include <vector>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"


namespace eb {

bool mfma_fits_offsets(int32_t type, int64_t n, int64_t k, int bm, int bn) {
  const Layout L = layout_of(type, n, k);
  const int64_t qsb = qs_bytes_per_block(type);
  const int64_t lim = 0xffffffffLL;
  return (int64_t)bm * k * 2 <= lim && (int64_t)bn * (k / kQK) * qsb <= lim &&
         (int64_t)bn * L.ds * 2 <= lim && (int64_t)bn * L.ss <= lim;
}

namespace {

// y = sum over s of ws[s] (in order s = 0, 1, ..., so the result does not
// depend on scheduling), converted to the output type, with the op's
// epilogue.  Four outputs per thread; ws_stride is a multiple of 4 so every
// float4 access is aligned; with the gate/up epilogue n is even, so the four
// (a multiple of 4 into the flat [m][n] index) are two gate/up pairs.
__global__ void __launch_bounds__(256)
    splitk_reduce(const float *__restrict__ ws, int splits, int64_t ws_stride, int64_t count,
                  void *__restrict__ y, int yt, Fuse f) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= count) return;
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  const int e = (int)(count - i < 4 ? count - i : 4);
  if (e == 4) {
    float4 v = *reinterpret_cast<const float4 *>(ws + i);
    // unrolled so several partial loads are in flight; the sum stays in split order
#pragma unroll 4
    for (int p = 1; p < splits; ++p) {
      const float4 b = *reinterpret_cast<const float4 *>(ws + p * ws_stride + i);
      v.x += b.x;
      v.y += b.y;
      v.z += b.z;
      v.w += b.w;
    }
    if (f.epi == EB_EPI_NONE && yt == EB_F32) {
      *reinterpret_cast<float4 *>(reinterpret_cast<float *>(y) + i) = v;
      return;
    }
    a[0] = v.x;
    a[1] = v.y;
    a[2] = v.z;
    a[3] = v.w;
  } else {
    for (int t = 0; t < e; ++t) {
      float v = ws[i + t];
      for (int p = 1; p < splits; ++p) v += ws[p * ws_stride + i + t];
      a[t] = v;
    }
  }
  if (f.epi == EB_EPI_GLU) {
    for (int t = 0; t + 1 < e; t += 2) store_y(y, (i + t) / 2, silu_mul(a[t], a[t + 1]), yt);
  } else if (f.epi == EB_EPI_ADD) {  // the residuals read together
    // offsets from the workgroup's first element (the same in every lane)
    const int64_t b0 = (int64_t)blockIdx.x * 1024;
    const int64_t span = count - b0 < 1024 ? count - b0 : 1024;
    const uint32_t t0 = (uint32_t)(i - b0);
    const uint32_t rel[4] = {t0, t0 + 1, t0 + 2, t0 + 3};
    const bool ok[4] = {true, e > 1, e > 2, e > 3};
    put_y_add(y, f.r, b0, span, rel, ok, a, yt);
  } else {
    for (int t = 0; t < e; ++t) store_y(y, i + t, a[t], yt);
  }
}

// Tile configurations: {BM, BN, WM, WN, workgroups per CU (LDS-bound),
// full-chip rate in TFLOP/s on large problems (measured), weight formats it
// is planned for (bit 0: Q8_0, bit 1: Q4_0)}.  The rate only ranks
// configurations against each other.  512 x 128 (two x buffers) halves the
// dequantization per flop of the 256-row tiles; with Q4_0 only half of its
// threads have a 32-weight chunk to dequantize per K-tile, which made it
// slower than 256 x 256 there (measured), so it is planned for Q8_0 only.
// Q6_S (two 32-weight chunks per row per K-tile, like Q4_0) takes Q4_0's set.
struct Cfg {
  int bm, bn, wm, wn, per_cu;
  double rate;
  int formats;
};
constexpr Cfg kCfgs[] = {
    {64, 128, 2, 2, 2, 546, 3},  {128, 128, 2, 2, 2, 769, 3}, {128, 256, 2, 4, 1, 773, 3},
    {256, 128, 4, 2, 1, 812, 3}, {256, 192, 4, 2, 1, 900, 3}, {256, 256, 4, 2, 1, 902, 3},
    {256, 256, 2, 4, 1, 977, 3}, {256, 256, 2, 2, 1, 835, 3}, {512, 128, 4, 2, 1, 1035, 1},
};
bool planned_for(const Cfg &g, int32_t type) { return g.formats & (type == EB_Q8_0 ? 1 : 2); }

// canonical weight bytes per 32 weights
double bytes_per_32(int32_t type) { return type == EB_Q8_0 ? 34.0 : (type == EB_Q6_S ? 26.25 : 18.0); }
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);

// Tile configurations that also come with hi/lo weight tiles (bfloat16
// activations, m <= kHLMaxM): {configuration, workgroups per CU with hi/lo}.
constexpr int kHLCfgs[][2] = {{0, 2}, {1, 1}};
constexpr int64_t kHLMaxM = 128;

constexpr int kMinSplitTiles = 4;                      // K-tiles per split, at least

// Estimated time (s) of one configuration and split count.  Workgroups run in
// rounds over the CUs; a CU holding w of a configuration's per_cu workgroups
// delivers rate/cus * sqrt(w / per_cu) (fewer resident waves hide less
// latency), each round also pays a fixed cost for pipeline fill and epilogue,
// the whole call is at least as long as streaming the weights from HBM, and
// splits > 1 add the traffic and launch of the reduction.
double estimate(int32_t type, const Cfg &g, int64_t m, int64_t n, int64_t k, int splits, int cus) {
  const int64_t nk = (k + kBK - 1) / kBK;
  const int64_t tiles = ((m + g.bm - 1) / g.bm) * ((n + g.bn - 1) / g.bn);
  const int64_t kts = (nk + splits - 1) / splits;
  const int64_t units = tiles * splits;
  const int64_t slots = (int64_t)cus * g.per_cu;
  const double cu_rate = g.rate * 1e12 / cus;
  const double wg_flops = 2.0 * g.bm * g.bn * kts * kBK;
  double t = 0;
  for (int64_t left = units; left > 0; left -= std::min(left, slots)) {
    const int64_t w = std::min<int64_t>(g.per_cu, (std::min(left, slots) + cus - 1) / cus);
    t += w * wg_flops / (cu_rate * std::sqrt((double)w / g.per_cu)) + 1e-6;
  }
  const double wbytes = (double)n * k * bytes_per_32(type) / 32.0;
  t = std::max(t, wbytes / 5e12);
  if (splits > 1) t += (2.0 * splits + 1.0) * (double)m * n * 4 / 4e12 + 3e-6;
  return t;
}
}  // namespace

int mfma_tile_count() { return kNumCfgs; }
int mfma_cfg_bm(int cfg) { return kCfgs[cfg].bm; }
double mfma_cfg_rate(int cfg) { return kCfgs[cfg].rate; }

bool needs_hl(int32_t xt, int64_t m) { return xt == EB_BF16 && m <= kHLMaxM; }

MfmaPlan plan_mfma(int32_t type, int32_t xt, int64_t m, int64_t n, int64_t k, size_t max_ws,
                   int force_cfg, int force_splits) {
  const int64_t nk = (k + kBK - 1) / kBK;
  const int cus = device_cu_count();
  const bool hl = needs_hl(xt, m);
  int fc = force_cfg;
  const int fs = force_splits;
  if (hl) {  // a forced tile without hi/lo tiles does not apply here
    bool ok = false;
    for (const auto &h : kHLCfgs) ok = ok || h[0] == fc;
    if (!ok) fc = -1;
  }
  MfmaPlan best;
  best.hl = hl;
  // Q6_S: its own kernel up to 128 rows (hi/lo weights for bfloat16 x), the
  // tile kernel beyond (measured at 816 and 4096 rows: 10x faster)
  if (type == EB_Q6_S && (m <= kHLMaxM || !mfma_fits_offsets(type, n, k, 64, 128))) {
    best.q6 = true;
    best.hl = xt == EB_BF16;
    best.kts = (int)nk;
    return best;
  }
  // a lone small-m projection: the narrow kernel (16 weight rows per
  // workgroup), k split only when its workgroups do not fill the GPU
  // (measured on the action-expert chain: the tiled kernel split along k
  // plus its reduction took about 16 us per projection)
  if (fc < 0 && fs <= 0 && m <= kNarrowMaxM) {
    int sp = narrow_splits(n, k, cus);
    const int64_t stride = (m * n + 63) / 64 * 64;
    if (sp > 1 && (size_t)(stride * sp * 4) > max_ws) sp = 1;
    if (narrow_fits(m, n, k, sp)) {
      best.narrow = true;
      best.splits = sp;
      best.kts = (int)nk;
      best.ws_stride = sp > 1 ? stride : 0;
      best.ws_bytes = sp > 1 ? (size_t)(stride * sp * 4) : 0;
      return best;
    }
  }
  double best_t = 0;
  bool have = false;
  for (int c = 0; c < kNumCfgs; ++c) {
    if (fc >= 0 && fc < kNumCfgs && c != fc) continue;
    Cfg g = kCfgs[c];
    if (c != fc && !planned_for(g, type)) continue;
    if (hl) {
      int per_cu = 0;
      for (const auto &h : kHLCfgs)
        if (h[0] == c) per_cu = h[1];
      if (!per_cu) continue;
      g.per_cu = per_cu;
    }
    if (!mfma_fits_offsets(type, n, k, g.bm, g.bn)) continue;
    for (int sp = 1; sp <= 16; ++sp) {
      if (sp > 1 && max_ws == 0) break;
      if (fs > 0 && sp != fs) continue;
      const int64_t kts = (nk + sp - 1) / sp;
      if (sp > 1 && (kts < kMinSplitTiles || (nk + kts - 1) / kts != sp)) continue;
      const int64_t stride = (m * n + 63) / 64 * 64;
      const int64_t wsb = sp > 1 ? stride * sp * 4 : 0;
      if ((size_t)wsb > max_ws) continue;
      const double t = estimate(type, g, m, n, k, sp, cus);
      if (!have || t < best_t * 0.999) {
        have = true;
        best_t = t;
        best.cfg = c;
        best.splits = sp;
        best.kts = (int)kts;
        best.ws_stride = sp > 1 ? stride : 0;
        best.ws_bytes = (size_t)wsb;
      }
    }
  }
  if (!have) {  // every accepted shape fits the first configuration unsplit
    best.cfg = 0;
    best.splits = 1;
    best.kts = (int)nk;
    best.ws_stride = 0;
    best.ws_bytes = 0;
  }
  return best;
}

// Configurations a grouped launch may use (instantiated with G = true).
constexpr int kGroupCfgs[] = {1, 2, 4, 6};

int plan_grouped(int32_t type, const std::vector<GOp> &ops, std::vector<int2> &order) {
  const int cus = device_cu_count();
  int best = -1;
  double best_t = 0;
  for (int c : kGroupCfgs) {
    const Cfg &g = kCfgs[c];
    bool fits = true;
    double work = 0, longest = 0;
    for (const GOp &o : ops) {
      fits = fits && mfma_fits_offsets(type, o.n, o.k, g.bm, g.bn);
      const double nk = (double)((o.k + kBK - 1) / kBK);
      work += (double)(((o.m + g.bm - 1) / g.bm) * ((o.n + g.bn - 1) / g.bn)) * nk;
      longest = std::max(longest, nk);
    }
    if (!fits) continue;
    // padded tile work at the configuration's rate, plus half a longest tile of tail
    const double step_s = 2.0 * g.bm * g.bn * kBK / (g.rate * 1e12);
    const double t = work * step_s + 0.5 * longest * step_s * cus * g.per_cu;
    if (best < 0 || t < best_t) {
      best = c;
      best_t = t;
    }
  }
  if (best < 0) return -1;
  const Cfg &g = kCfgs[best];
  // longest tiles first; each op's tiles start at a multiple of 8 entries and
  // run in the XCD-aware order of the single-op launch
  std::vector<int> idx(ops.size());
  for (size_t i = 0; i < ops.size(); ++i) idx[i] = (int)i;
  std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) { return ops[a].k > ops[b].k; });
  order.clear();
  for (int oi : idx) {
    const GOp &o = ops[oi];
    const int64_t tiles = ((o.m + g.bm - 1) / g.bm) * ((o.n + g.bn - 1) / g.bn);
    for (int64_t b = 0; b < tiles; ++b) {
      const int64_t t = tiles % kXcds == 0 ? (b % kXcds) * (tiles / kXcds) + b / kXcds : b;
      order.push_back(make_int2(oi, (int)t));
    }
    while (order.size() % kXcds) order.push_back(make_int2(-1, 0));
  }
  return best;
}

namespace {

template <int QT, int XT>
hipError_t launch_q(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, const MfmaPlan &P, float *ws, hipStream_t s,
                    const NormOut *no) {
  const int sp = ws ? P.splits : 1;
  const int kts = ws ? P.kts : (int)((k + kBK - 1) / kBK);
  const int64_t st = P.ws_stride;
  const hipError_t e =
      P.narrow ? launch_mfma_narrow(QT, wdata, n, k, x, XT, P.hl, m, y, yt, f, sp, ws, st, s)
               : mfma_tile_launch<QT, XT>(P.cfg, P.hl, wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
  if (e != hipSuccess || sp == 1) return e;
  if (no) {
    if (yt != EB_F32 || f.epi == EB_EPI_GLU) return hipErrorInvalidValue;
    return launch_splitk_reduce_rmsnorm(ws, sp, st, m, n, static_cast<float *>(y),
                                        f.epi == EB_EPI_ADD ? static_cast<const float *>(f.r) : nullptr,
                                        *no, s);
  }
  const int64_t count = m * n;
  const int64_t blocks = (count + 1023) / 1024;
  splitk_reduce<<<(unsigned)blocks, 256, 0, s>>>(ws, sp, st, count, y, yt, f);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mfma(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                       int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f,
                       const MfmaPlan &plan, float *ws, hipStream_t s, const NormOut *no) {
  if (type == EB_Q6_S) {
    if (plan.q6) {
      if (no) return hipErrorInvalidValue;  // no split, so no reduction to fuse into
      return launch_mfma_q6(wdata, n, k, x, xt, m, y, yt, f, s);
    }
    if (xt == EB_F16) return launch_q<EB_Q6_S, EB_F16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
    return launch_q<EB_Q6_S, EB_BF16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
  }
  if (type == EB_Q4_0) {
    if (xt == EB_F16) return launch_q<EB_Q4_0, EB_F16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
    return launch_q<EB_Q4_0, EB_BF16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
  }
  if (xt == EB_F16) return launch_q<EB_Q8_0, EB_F16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
  return launch_q<EB_Q8_0, EB_BF16>(wdata, n, k, x, m, y, yt, f, plan, ws, s, no);
}

hipError_t launch_mfma_grouped(int32_t type, int32_t xt, int cfg, const GOp *ops, const int2 *order,
                                int64_t entries, hipStream_t s) {
  if (type == EB_Q6_S) {
    if (xt == EB_F16) return mfma_tile_launch_grouped<EB_Q6_S, EB_F16>(cfg, ops, order, entries, s);
    return mfma_tile_launch_grouped<EB_Q6_S, EB_BF16>(cfg, ops, order, entries, s);
  }
  if (type == EB_Q4_0) {
    if (xt == EB_F16) return mfma_tile_launch_grouped<EB_Q4_0, EB_F16>(cfg, ops, order, entries, s);
    return mfma_tile_launch_grouped<EB_Q4_0, EB_BF16>(cfg, ops, order, entries, s);
  }
  if (xt == EB_F16) return mfma_tile_launch_grouped<EB_Q8_0, EB_F16>(cfg, ops, order, entries, s);
  return mfma_tile_launch_grouped<EB_Q8_0, EB_BF16>(cfg, ops, order, entries, s);
}

}  // namespace eb
