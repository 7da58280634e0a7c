// mfma_multi.hip -- fused MFMA launch over many independent small-m ops of
// a stack (paper section 3.2: operator fusion and graph replay for batch-1
// execution; the action-chunk denoising steps of section 2.1 / Table 1 run
// hundreds of such layers per pass).  Built with the MFMA accumulators in
// VGPRs: its persistent loop otherwise moves them between register files on
// every trip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <vector>

#include "eb_internal.h"
#include "mfma_common.h"
#include "mm_common.h"

namespace eb {
namespace {

// ---------------------------------------------------------------------------
// Fused launch over many independent ops (small m).  The tiles (units) of
// the op table are split into one contiguous range per workgroup, balanced by
// K-tile steps; consecutive ranges go to workgroups on the same XCD (shared
// L2).  A workgroup runs its units as one stream of K-tile steps, with the
// pipeline of mfma_kernel one step deeper (x copies three steps ahead, weight
// loads four), running across unit and op boundaries; a unit's epilogue is
// written when its last step is done.  Cursors walk the stream: the step being
// computed, the x copy ahead and the weight loads ahead.  Loads past the end
// of the range are issued with an empty range (they read zeros and touch no
// memory), so every step issues the same instructions.  The deeper pipeline
// suits a launch that keeps every CU streaming weights, where memory latency
// is longer than in a single-op launch.
// ---------------------------------------------------------------------------
template <int QT, int XT, int YT, int BM, int BN, int WM, int WN, int D>
__global__ void __launch_bounds__(WM *WN * 64)
    mfma_multi_kernel(const MMOp *__restrict__ ops, int nops, const int64_t *__restrict__ wg,
                      int groups) {
  // The body is device code only: the host pass (which only needs the launch
  // stub) does not see it.
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int T = WM * WN * 64;
  constexpr int WAVES = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int ADMA = BM / (8 * WAVES);
  constexpr int WCPR = WTile<QT>::kChunksPerRow;
  constexpr int WCH = BN * WCPR;
  constexpr int BCH = (WCH + T - 1) / T;
  constexpr int KSTEPS = kBK / 16;
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;
  constexpr int NV = Deq<QT>::kVecs;
  constexpr int ABYTES = BM * kBK * 2, BBYTES = BN * kBK * 2;
  constexpr int YSZ = (YT == EB_F32) ? 4 : 2;
  constexpr int NX = ADMA, NW = 2 * BCH;
  static_assert(ADMA >= 1 && ADMA * 8 * WAVES == BM, "x tile must split into 8-row copies");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave sub-tile must be whole fragments");
  // Pipeline depth D: x copies run D steps ahead (D + 1 x buffers), weight
  // loads D + 1 (D + 1 register sets); a step waits at its barrier for the x
  // copy issued D - 1 steps before it.  D = 3 for the small tiles; the large
  // tiles take D = 2, which is what fits in 160 KB of LDS.
  static_assert(D == 2 || D == 3, "pipeline depth");
  constexpr int NWAIT = (D - 1) * NX + D * NW;
  static_assert(NWAIT <= 63, "vmcnt range");

  __shared__ __attribute__((aligned(1024))) uint8_t sA0[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA2[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA3[D == 3 ? ABYTES : 16];
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[BBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB1[BBYTES];

  // workgroups are dispatched to the XCDs round-robin (g % 8 is the XCD):
  // range p goes to XCD p / (groups / 8)
  const int g = blockIdx.x;
  const int p = (g % kXcds) * (groups / kXcds) + g / kXcds;
  const int64_t u_begin = wg[p], u_end = wg[p + 1];
  if (u_begin >= u_end) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // first op of the range: binary search over the ascending unit_end (the
  // last op's unit_end is the total, which exceeds u_begin)
  int lo = 0, hi = nops - 1;
  while (lo < hi) {
    const int mid = (lo + hi) / 2;
    if (ops[mid].unit_end <= u_begin) lo = mid + 1; else hi = mid;
  }
  // steps of the range, rounded up to whole groups of 4 (D = 3) or 6 (D = 2)
  // by the loops below (the extra steps run on zeros, their loads are empty,
  // and write nothing)
  int64_t nsteps = 0;
  for (int o = lo;; ++o) {
    const int64_t first = o ? ops[o - 1].unit_end : 0;
    nsteps += (min(ops[o].unit_end, u_end) - max(first, u_begin)) * ops[o].nk;
    if (ops[o].unit_end >= u_end) break;
  }

  // per-thread tile-local parts of the x copies and weight loads
  uint32_t xr_[ADMA], xc_[ADMA];
#pragma unroll
  for (int i = 0; i < ADMA; ++i) {
    const uint32_t r = 8 * (i * WAVES + wave) + (lane >> 3);
    xr_[i] = r;
    xc_[i] = ((lane & 7) ^ swz(r)) << 4;
  }
  uint32_t wr_[BCH], wq_[BCH], wd_[BCH], wl[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int idx = min(tid + i * T, WCH), r = idx / WCPR, c = idx % WCPR;
    const int blk = (QT == EB_Q8_0) ? (c >> 1) : c;
    wr_[i] = r;
    wq_[i] = blk * QSB + ((QT == EB_Q8_0) ? (c & 1) * 16 : 0);
    wd_[i] = blk * 2;
    wl[i] = (uint32_t)(r * (kBK * 2) + (((NV * c) ^ swz(r)) << 4));
  }

  // --- x copies: base and byte count advance by one K-tile per step ---------
  struct XState {
    MMPos p;
    const uint8_t *base;
    uint32_t rec;
    uint32_t v[ADMA];
  };
  auto x_enter = [&](XState &s) __attribute__((always_inline)) {
    if (!s.p.valid) {
      s.rec = 0;
      return;
    }
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, s.p, m0, n0, rm, rn);
    const MMOp &o = ops[s.p.op];
    const uint32_t row = (uint32_t)o.k * 2;
    s.base = reinterpret_cast<const uint8_t *>(o.x) + m0 * row;
    s.rec = (uint32_t)rm * row;
#pragma unroll
    for (int i = 0; i < ADMA; ++i) s.v[i] = xr_[i] * row + xc_[i];
  };
  auto x_issue = [&](uint8_t *sA, XState &s) __attribute__((always_inline)) {
    const auto r = ursrc(s.base, s.rec);
#pragma unroll
    for (int i = 0; i < ADMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(sA + (i * WAVES + wave) * 1024), 16,
                                               (int)s.v[i], 0, 0, 0);
    if (mm_step(ops, s.p, u_end)) {
      x_enter(s);
    } else if (s.p.valid) {
      s.base += kBK * 2;
      s.rec -= kBK * 2;
    }
  };

  // --- weight loads --------------------------------------------------------
  struct Raw {
    uint4 b[BCH];
    uint16_t d[BCH];
  };
  struct WState {
    MMPos p;
    const uint8_t *qb, *db;
    uint32_t qrec, drec;
    uint32_t qv[BCH], dv[BCH];
  };
  auto w_enter = [&](WState &s) __attribute__((always_inline)) {
    if (!s.p.valid) {
      s.qrec = s.drec = 0;
      return;
    }
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, s.p, m0, n0, rm, rn);
    const MMOp &o = ops[s.p.op];
    const uint32_t qrow = (uint32_t)(o.k / kQK) * QSB, drow = (uint32_t)o.ds * 2;
    s.qb = o.w + n0 * qrow;
    s.db = o.w + o.d_off + n0 * drow;
    s.qrec = (uint32_t)rn * qrow;
    s.drec = (uint32_t)rn * drow;
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      s.qv[i] = wr_[i] * qrow + wq_[i];
      s.dv[i] = wr_[i] * drow + wd_[i];
    }
  };
  auto w_issue = [&](Raw &S, WState &s) __attribute__((always_inline)) {
    const auto qr = ursrc(s.qb, s.qrec);
    const auto dr = ursrc(s.db, s.drec);
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      S.b[i] = bload(qr, s.qv[i]);
      S.d[i] = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)s.dv[i], 0, 0);
    }
    if (mm_step(ops, s.p, u_end)) {
      w_enter(s);
    } else if (s.p.valid) {
      s.qb += 2 * QSB;
      s.qrec -= 2 * QSB;
      s.db += 4;
      s.drec -= 4;
    }
  };
  auto store_w = [&](const Raw &S, uint8_t *sB, int i) __attribute__((always_inline)) {
    if (WCH % T != 0 && i == BCH - 1 && tid + i * T >= WCH) return;
    uint4 v[NV];
    dequant_chunk<QT, XT>(S.b[i], (float)__builtin_bit_cast(_Float16, S.d[i]), v);
#pragma unroll
    for (int q = 0; q < NV; ++q) *reinterpret_cast<uint4 *>(sB + (wl[i] ^ (16u * q))) = v[q];
  };

  // --- MFMAs -----------------------------------------------------------------
  uint32_t abase[FM], bbase[FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t r = wm * TM + i * 32 + (lane & 31);
    abase[i] = r * (kBK * 2) + ((((uint32_t)lane >> 5) ^ swz(r)) << 4);
  }
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const uint32_t r = wn * TN + j * 32 + (lane & 31);
    bbase[j] = r * (kBK * 2) + ((((uint32_t)lane >> 5) ^ swz(r)) << 4);
  }
  f32x16_t acc[FM][FN];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  };
  zero_acc();
  auto compute = [&](const uint8_t *sA, const uint8_t *sB, const Raw &nxt, uint8_t *sBn)
                     __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      uint4 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(sA + (abase[i] ^ (32u * ks)));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const uint4 *>(sB + (bbase[j] ^ (32u * ks)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[i], bfr[j], acc[i][j]);
      constexpr int per = (BCH + KSTEPS - 1) / KSTEPS;
#pragma unroll
      for (int i = ks * per; i < ks * per + per && i < BCH; ++i) store_w(nxt, sBn, i);
    }
  };

  // --- epilogue: buffer stores whose range check drops rows past m; lanes of
  // columns past n use an offset past the range ---------------------------
  auto epilogue = [&](const MMPos &c) __attribute__((always_inline)) {
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, c, m0, n0, rm, rn);
    const MMOp &o = ops[c.op];
    const uint32_t n = (uint32_t)o.n;
    const auto yr = ursrc(o.y, (uint32_t)o.m * n * YSZ);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int cl = wn * TN + j * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint32_t row0 = (uint32_t)m0 + wm * TM + i * 32 + 4 * (lane >> 5);
        const uint32_t base = cl < rn ? (row0 * n + (uint32_t)n0 + cl) * YSZ : 0x80000000u;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t off = base + (uint32_t)(8 * (r >> 2) + (r & 3)) * n * YSZ;
          // copy the element out first: a bit cast of a vector element lvalue
          // reads the wrong element
          const float v = acc[i][j][r];
          if constexpr (YT == EB_F32)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), yr, (int)off, 0, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, (__bf16)v), yr,
                                                  (int)off, 0, 0);
        }
      }
    }
  };

  {
    constexpr int Z = ABYTES / 16 / T;
    static_assert(Z * T * 16 == ABYTES, "zero fill must cover the x buffers");
#pragma unroll
    for (int i = 0; i < Z; ++i) {
      const int o = (tid + i * T) * 16;
      *reinterpret_cast<uint4 *>(sA0 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA1 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA2 + o) = make_uint4(0, 0, 0, 0);
      if constexpr (D == 3) *reinterpret_cast<uint4 *>(sA3 + o) = make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();

  MMPos C;
  C.op = lo;
  C.u = u_begin;
  C.valid = true;
  mm_seek(ops, C, u_end);
  XState X;
  X.p = C;
  x_enter(X);
  WState Wc;
  Wc.p = C;
  w_enter(Wc);

  // prologue: x of steps 0..D-1 and weights of steps 0..D
  Raw S0, S1, S2, S3;
  x_issue(sA0, X);
  x_issue(sA1, X);
  if constexpr (D == 3) x_issue(sA2, X);
  w_issue(S0, Wc);
  w_issue(S1, Wc);
  w_issue(S2, Wc);
  if constexpr (D == 3) w_issue(S3, Wc);
#pragma unroll
  for (int i = 0; i < BCH; ++i) store_w(S0, sB0, i);
  __syncthreads();

  auto step = [&](const uint8_t *A, uint8_t *Anew, const uint8_t *B, uint8_t *Bn, const Raw &deq,
                  Raw &ld) __attribute__((always_inline)) {
    x_issue(Anew, X);
    w_issue(ld, Wc);
    compute(A, B, deq, Bn);
    if (C.valid && C.kt == C.nk - 1) {
      epilogue(C);
      zero_acc();
      wait_vm_barrier<0>();
    } else {
      wait_vm_barrier<NWAIT>();
    }
    mm_step(ops, C, u_end);
  };
  if constexpr (D == 3) {
    for (int64_t j = 0; j < nsteps; j += 4) {
      step(sA0, sA3, sB0, sB1, S1, S0);
      step(sA1, sA0, sB1, sB0, S2, S1);
      step(sA2, sA1, sB0, sB1, S3, S2);
      step(sA3, sA2, sB1, sB0, S0, S3);
    }
  } else {
    for (int64_t j = 0; j < nsteps; j += 6) {
      step(sA0, sA2, sB0, sB1, S1, S0);
      step(sA1, sA0, sB1, sB0, S2, S1);
      step(sA2, sA1, sB0, sB1, S0, S2);
      step(sA0, sA2, sB1, sB0, S1, S0);
      step(sA1, sA0, sB0, sB1, S2, S1);
      step(sA2, sA1, sB1, sB0, S0, S2);
    }
  }
#endif  // __HIP_DEVICE_COMPILE__
}

// ---------------------------------------------------------------------------
// Fused small-m launch with the weights dequantized straight into MFMA
// B-operand registers.  At m <= 128 one workgroup tile holds every row, so
// each of the 4 waves owns a disjoint set of 32 FN output columns: its weights
// are used by that wave only and need no LDS round trip.  Only the x tile
// goes through LDS (copied by buffer loads, four buffers, three steps ahead).
//
// Within a K-tile of 64, MFMA step s (16 values of k) takes from the lane
// with column c and half h = lane / 32 the weights k = 32 h + 8 s .. + 7, and
// from the x row the same k; over s = 0..3 every k of the tile is used once.
// So a lane's weights for the whole K-tile are block h of its row (Q8_0: 32
// codes = two 16-byte loads, Q4_0: 16 bytes holding k and k + 16 in the low
// and high nibbles) plus its scale, loaded four steps ahead into one of four
// register sets.
// ---------------------------------------------------------------------------
template <int QT, int XT, int YT, int BM, int FN>
__global__ void __launch_bounds__(256)
    mm_breg_kernel(const MMOp *__restrict__ ops, int nops, const int64_t *__restrict__ wg,
                   int groups) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int WAVES = 4;
  constexpr int BN = WAVES * 32 * FN;
  constexpr int FM = BM / 32;
  constexpr int ADMA = BM / (8 * WAVES);
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;
  constexpr int NQ = (QT == EB_Q8_0) ? 2 : 1;  // 16-byte code loads per fragment
  constexpr int ABYTES = BM * kBK * 2;
  constexpr int YSZ = (YT == EB_F32) ? 4 : 2;
  constexpr int NX = ADMA, NW = FN * (NQ + 1);
  constexpr int NWAIT = 2 * NX + 3 * NW;  // at a barrier: all but x tile t+1 may be in flight
  static_assert(ADMA >= 1 && ADMA * 8 * WAVES == BM, "x tile must split into 8-row copies");
  static_assert(NWAIT <= 63, "vmcnt range");

  __shared__ __attribute__((aligned(1024))) uint8_t sA0[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA2[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA3[ABYTES];

  const int g = blockIdx.x;
  const int p = (g % kXcds) * (groups / kXcds) + g / kXcds;
  const int64_t u_begin = wg[p], u_end = wg[p + 1];
  if (u_begin >= u_end) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  int lo = 0, hi = nops - 1;
  while (lo < hi) {
    const int mid = (lo + hi) / 2;
    if (ops[mid].unit_end <= u_begin) lo = mid + 1; else hi = mid;
  }
  int64_t nsteps = 0;
  for (int o = lo;; ++o) {
    const int64_t first = o ? ops[o - 1].unit_end : 0;
    nsteps += (min(ops[o].unit_end, u_end) - max(first, u_begin)) * ops[o].nk;
    if (ops[o].unit_end >= u_end) break;
  }

  // --- x copies (as in mfma_multi_kernel) -------------------------------------
  uint32_t xr_[ADMA], xc_[ADMA];
#pragma unroll
  for (int i = 0; i < ADMA; ++i) {
    const uint32_t r = 8 * (i * WAVES + wave) + (lane >> 3);
    xr_[i] = r;
    xc_[i] = ((lane & 7) ^ swz(r)) << 4;
  }
  struct XState {
    MMPos p;
    const uint8_t *base;
    uint32_t rec;
    uint32_t v[ADMA];
  };
  auto x_enter = [&](XState &s) __attribute__((always_inline)) {
    if (!s.p.valid) {
      s.rec = 0;
      return;
    }
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, s.p, m0, n0, rm, rn);
    const MMOp &o = ops[s.p.op];
    const uint32_t row = (uint32_t)o.k * 2;
    s.base = reinterpret_cast<const uint8_t *>(o.x) + m0 * row;
    s.rec = (uint32_t)rm * row;
#pragma unroll
    for (int i = 0; i < ADMA; ++i) s.v[i] = xr_[i] * row + xc_[i];
  };
  auto x_issue = [&](uint8_t *sA, XState &s) __attribute__((always_inline)) {
    const auto r = ursrc(s.base, s.rec);
#pragma unroll
    for (int i = 0; i < ADMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(sA + (i * WAVES + wave) * 1024), 16,
                                               (int)s.v[i], 0, 0, 0);
    if (mm_step(ops, s.p, u_end)) {
      x_enter(s);
    } else if (s.p.valid) {
      s.base += kBK * 2;
      s.rec -= kBK * 2;
    }
  };

  // --- weights: this wave's 32 FN columns, block h = lane / 32 of each row ---
  const uint32_t wrow0 = (uint32_t)(wave * 32 * FN + (lane & 31));  // tile-local row of fragment 0
  const uint32_t wh = (uint32_t)(lane >> 5);
  struct Raw {
    uint4 q[FN][NQ];
    uint16_t d[FN];
  };
  struct WState {
    MMPos p;
    const uint8_t *qb, *db;
    uint32_t qrec, drec;
    uint32_t qv, dv;  // lane offsets of fragment 0; fragment j adds 32 j rows
    uint32_t qrow32, drow32;
  };
  auto w_enter = [&](WState &s) __attribute__((always_inline)) {
    if (!s.p.valid) {
      s.qrec = s.drec = 0;
      return;
    }
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, s.p, m0, n0, rm, rn);
    const MMOp &o = ops[s.p.op];
    const uint32_t qrow = (uint32_t)(o.k / kQK) * QSB, drow = (uint32_t)o.ds * 2;
    s.qb = o.w + n0 * qrow;
    s.db = o.w + o.d_off + n0 * drow;
    s.qrec = (uint32_t)rn * qrow;
    s.drec = (uint32_t)rn * drow;
    s.qv = wrow0 * qrow + wh * QSB;
    s.dv = wrow0 * drow + wh * 2;
    s.qrow32 = 32 * qrow;
    s.drow32 = 32 * drow;
  };
  auto w_issue = [&](Raw &S, WState &s) __attribute__((always_inline)) {
    const auto qr = ursrc(s.qb, s.qrec);
    const auto dr = ursrc(s.db, s.drec);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int h = 0; h < NQ; ++h) S.q[j][h] = bload(qr, s.qv + j * s.qrow32 + 16 * h);
      S.d[j] = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)(s.dv + j * s.drow32), 0, 0);
    }
    if (mm_step(ops, s.p, u_end)) {
      w_enter(s);
    } else if (s.p.valid) {
      s.qb += 2 * QSB;
      s.qrec -= 2 * QSB;
      s.db += 4;
      s.drec -= 4;
    }
  };

  // --- MFMAs: A fragment i, step s at chunk (4 h + s) ^ swz(row) -------------
  uint32_t abase[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t r = i * 32 + (lane & 31);
    abase[i] = r * (kBK * 2) + (((4u * wh) ^ swz(r)) << 4);
  }
  f32x16_t acc[FM][FN];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  };
  zero_acc();

  auto epilogue = [&](const MMPos &c) __attribute__((always_inline)) {
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, c, m0, n0, rm, rn);
    const MMOp &o = ops[c.op];
    const uint32_t n = (uint32_t)o.n;
    const auto yr = ursrc(o.y, (uint32_t)o.m * n * YSZ);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int cl = wave * 32 * FN + j * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint32_t row0 = (uint32_t)m0 + i * 32 + 4 * (lane >> 5);
        const uint32_t base = cl < rn ? (row0 * n + (uint32_t)n0 + cl) * YSZ : 0x80000000u;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t off = base + (uint32_t)(8 * (r >> 2) + (r & 3)) * n * YSZ;
          const float v = acc[i][j][r];  // copy first: see mfma_multi_kernel
          if constexpr (YT == EB_F32)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), yr, (int)off, 0, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, (__bf16)v), yr,
                                                  (int)off, 0, 0);
        }
      }
    }
  };

  {
    constexpr int Z = ABYTES / 16 / 256;
    static_assert(Z * 256 * 16 == ABYTES, "zero fill must cover the x buffers");
#pragma unroll
    for (int i = 0; i < Z; ++i) {
      const int o = (tid + i * 256) * 16;
      *reinterpret_cast<uint4 *>(sA0 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA1 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA2 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA3 + o) = make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();

  MMPos C;
  C.op = lo;
  C.u = u_begin;
  C.valid = true;
  mm_seek(ops, C, u_end);
  XState X;
  X.p = C;
  x_enter(X);
  WState Wc;
  Wc.p = C;
  w_enter(Wc);

  // prologue: x of steps 0..2, weights of steps 0..3
  Raw S0, S1, S2, S3;
  x_issue(sA0, X);
  x_issue(sA1, X);
  x_issue(sA2, X);
  w_issue(S0, Wc);
  w_issue(S1, Wc);
  w_issue(S2, Wc);
  w_issue(S3, Wc);
  __syncthreads();

  // step t: copy x tile t+3, dequantize weight tile t (set t % 4), then reuse
  // that set for weight tile t+4, run the MFMAs of tile t
  auto step = [&](const uint8_t *A, uint8_t *Anew, Raw &S) __attribute__((always_inline)) {
    x_issue(Anew, X);
    uint4 bq[FN][4];
#pragma unroll
    for (int j = 0; j < FN; ++j)
      dequant_b<QT, XT>(S.q[j], (float)__builtin_bit_cast(_Float16, S.d[j]), bq[j]);
    w_issue(S, Wc);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 af[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(A + (abase[i] ^ (16u * s)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[i], bq[j][s], acc[i][j]);
    }
    if (C.valid && C.kt == C.nk - 1) {
      epilogue(C);
      zero_acc();
      wait_vm_barrier<0>();
    } else {
      wait_vm_barrier<NWAIT>();
    }
    mm_step(ops, C, u_end);
  };
  for (int64_t j = 0; j < nsteps; j += 4) {
    step(sA0, sA3, S0);
    step(sA1, sA0, S1);
    step(sA2, sA1, S2);
    step(sA3, sA2, S3);
  }
#endif  // __HIP_DEVICE_COMPILE__
}

// ---------------------------------------------------------------------------
// Fused small-m launch, weights through LDS as raw codes.  Per K-tile step a
// workgroup copies, with buffer loads that write LDS directly and read whole
// row segments (Q8_0: 16 rows x 64 B per instruction, Q4_0: 32 rows x 32 B),
// the x tile, the packed codes of its BN = 128 * FN weight rows and their two
// scales; each of the 4 waves then reads the codes of its own 32 * FN columns
// from LDS, dequantizes them into MFMA registers (k order as in
// mm_breg_kernel) and runs its 64 x (32 * FN) sub-tile.  Loads keep whole-row
// coalescing; LDS carries 1 B per Q8_0 weight each way instead of 2.
// The weights are the MFMA A operand, so a lane's accumulators hold 4
// consecutive output columns of one row: y goes out in 8-byte (bf16/f16) or
// 16-byte (f32) stores, and a tile's stores stay in flight while the next
// tile starts (the vector-memory counter only waits for the next step's
// copies).  Three stages of every buffer; copies run two steps ahead.
// Code chunk c (16 B) of tile row r sits at chunk c ^ g(r) of the row
// (g(r) = (r >> 2) & 3 for 64-byte Q8_0 rows, (r >> 3) & 1 for 32-byte Q4_0
// rows), so the 16-lane phases of the per-column reads hit distinct banks.
// Each wave copies the scales of its own columns into its own 256-byte slot.
// ---------------------------------------------------------------------------
template <int QT, int XT, int YT, int FN>
__global__ void __launch_bounds__(256)
    mm_ldsw_kernel(const MMOp *__restrict__ ops, int nops, const int64_t *__restrict__ wg,
                   int groups) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int WAVES = 4, BM = 64, BN = WAVES * 32 * FN;
  constexpr int FM = BM / 32;
  constexpr int ADMA = BM / (8 * WAVES);  // x copies per wave
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;
  constexpr int ROWB = 2 * QSB;           // code bytes per row per K-tile
  constexpr int RPI = 1024 / ROWB;        // rows per 1 KB copy
  constexpr int WDMA = BN / RPI / WAVES;  // code copies per wave
  constexpr int RPW = 32 * FN;            // columns (and scale rows) per wave
  constexpr int ABYTES = BM * kBK * 2, WBYTES = BN * ROWB, SBYTES = WAVES * 256;
  constexpr int YSZ = (YT == EB_F32) ? 4 : 2;
  constexpr int NSTEP = ADMA + WDMA + 1;  // vector-memory ops per lane per step
  constexpr int NST = FM * FN * 4;        // packed y stores per lane per tile
  static_assert(ADMA * 8 * WAVES == BM && WDMA * RPI * WAVES == BN, "copies must tile");
  static_assert(RPW <= 64 && NSTEP + NST <= 63, "scale slot / wait count range");

  __shared__ __attribute__((aligned(1024))) uint8_t sA0[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA2[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW0[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW1[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW2[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sS0[SBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sS1[SBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sS2[SBYTES];

  const int g = blockIdx.x;
  const int p = (g % kXcds) * (groups / kXcds) + g / kXcds;
  const int64_t u_begin = wg[p], u_end = wg[p + 1];
  if (u_begin >= u_end) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  int lo = 0, hi = nops - 1;
  while (lo < hi) {
    const int mid = (lo + hi) / 2;
    if (ops[mid].unit_end <= u_begin) lo = mid + 1; else hi = mid;
  }
  int64_t nsteps = 0;
  for (int o = lo;; ++o) {
    const int64_t first = o ? ops[o - 1].unit_end : 0;
    nsteps += (min(ops[o].unit_end, u_end) - max(first, u_begin)) * ops[o].nk;
    if (ops[o].unit_end >= u_end) break;
  }

  auto gsw = [](uint32_t r) -> uint32_t {
    return QT == EB_Q8_0 ? ((r >> 2) & 3) : ((r >> 3) & 1);
  };

  // --- lane parts of the copies (tile-local) ----------------------------------
  uint32_t xr_[ADMA], xc_[ADMA];
#pragma unroll
  for (int i = 0; i < ADMA; ++i) {
    const uint32_t r = 8 * (i * WAVES + wave) + (lane >> 3);
    xr_[i] = r;
    xc_[i] = ((lane & 7) ^ swz(r)) << 4;
  }
  uint32_t wr_[WDMA], wc_[WDMA];
#pragma unroll
  for (int i = 0; i < WDMA; ++i) {
    const uint32_t r = RPI * (i * WAVES + wave) + lane / (ROWB / 16);
    const uint32_t c = lane % (ROWB / 16);
    wr_[i] = r;
    wc_[i] = (c ^ gsw(r)) * 16;  // stored chunk c of row r holds chunk c ^ g(r)
  }
  const uint32_t sr_ = wave * RPW + lane % RPW;  // 4 scale bytes of one row per lane

  // --- the copy cursor: x, codes and scales of one step ---------------------
  struct LState {
    MMPos p;
    const uint8_t *xb, *qb, *db;
    uint32_t xrec, qrec, drec;
    uint32_t xv[ADMA], qv[WDMA < 2 ? 2 : WDMA], dv;  // a 1-element array here ends up in scratch
  };
  auto l_enter = [&](LState &s) __attribute__((always_inline)) {
    if (!s.p.valid) {
      s.xrec = s.qrec = s.drec = 0;
      return;
    }
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, s.p, m0, n0, rm, rn);
    const MMOp &o = ops[s.p.op];
    const uint32_t xrow = (uint32_t)o.k * 2;
    const uint32_t qrow = (uint32_t)(o.k / kQK) * QSB, drow = (uint32_t)o.ds * 2;
    s.xb = reinterpret_cast<const uint8_t *>(o.x) + m0 * xrow;
    s.xrec = (uint32_t)rm * xrow;
    s.qb = o.w + n0 * qrow;
    s.qrec = (uint32_t)rn * qrow;
    s.db = o.w + o.d_off + n0 * drow;
    s.drec = (uint32_t)rn * drow;
#pragma unroll
    for (int i = 0; i < ADMA; ++i) s.xv[i] = xr_[i] * xrow + xc_[i];
#pragma unroll
    for (int i = 0; i < WDMA; ++i) s.qv[i] = wr_[i] * qrow + wc_[i];
    s.dv = sr_ * drow;
  };
  auto l_issue = [&](uint8_t *sA, uint8_t *sW, uint8_t *sS, LState &s) __attribute__((always_inline)) {
    const auto xr = ursrc(s.xb, s.xrec);
    const auto qr = ursrc(s.qb, s.qrec);
    const auto dr = ursrc(s.db, s.drec);
#pragma unroll
    for (int i = 0; i < ADMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(sA + (i * WAVES + wave) * 1024), 16,
                                               (int)s.xv[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < WDMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(qr, (lds_void *)(sW + (i * WAVES + wave) * 1024), 16,
                                               (int)s.qv[i], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(dr, (lds_void *)(sS + wave * 256), 4, (int)s.dv, 0, 0, 0);
    if (mm_step(ops, s.p, u_end)) {
      l_enter(s);
    } else if (s.p.valid) {
      s.xb += kBK * 2;
      s.xrec -= kBK * 2;
      s.qb += ROWB;
      s.qrec -= ROWB;
      s.db += 4;
      s.drec -= 4;
    }
  };

  // --- per-lane reads of its columns' codes and scales --------------------
  const uint32_t wh = (uint32_t)(lane >> 5);
  uint32_t bq_off[FN][QT == EB_Q8_0 ? 2 : 1], bs_off[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const uint32_t c = j * 32 + (lane & 31);  // column within the wave's slice
    const uint32_t r = wave * RPW + c;
    if constexpr (QT == EB_Q8_0) {
      bq_off[j][0] = r * ROWB + (((2 * wh) ^ gsw(r)) << 4);
      bq_off[j][1] = r * ROWB + (((2 * wh + 1) ^ gsw(r)) << 4);
    } else {
      bq_off[j][0] = r * ROWB + ((wh ^ gsw(r)) << 4);
    }
    bs_off[j] = wave * 256 + c * 4 + 2 * wh;
  }
  uint32_t abase[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t r = i * 32 + (lane & 31);
    abase[i] = r * (kBK * 2) + (((4u * wh) ^ swz(r)) << 4);
  }
  f32x16_t acc[FM][FN];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  };
  zero_acc();

  // lane (l, reg r) of sub-tile (i, j) holds y[m0 + 32 i + l % 32][n0 + wave * RPW +
  // 32 j + 8 (r / 4) + 4 (l / 32) + r % 4].  Rows past m fall outside the
  // buffer's range and are dropped; columns past the tile's rn get the
  // out-of-range offset 0x80000000.  Returns false when it used 1-element
  // stores (n not a multiple of 4), which must drain before the next tile.
  auto epilogue = [&](const MMPos &c) __attribute__((always_inline)) -> bool {
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, c, m0, n0, rm, rn);
    const MMOp &o = ops[c.op];
    const uint32_t n = (uint32_t)o.n;
    const auto yr = ursrc(o.y, (uint32_t)o.m * n * YSZ);
    const bool packed = (n & 3) == 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint32_t row = (uint32_t)m0 + i * 32 + (lane & 31);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cl = wave * RPW + j * 32 + 8 * q + 4 * (int)wh;
          const uint32_t base = (row * n + (uint32_t)n0 + cl) * YSZ;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];  // copy first: see mfma_multi_kernel
          if (packed) {
            const uint32_t off = cl < rn ? base : 0x80000000u;
            if constexpr (YT == EB_F32) {
              u32x4_t w;
#pragma unroll
              for (int e = 0; e < 4; ++e) w[e] = __builtin_bit_cast(uint32_t, v[e]);
              __builtin_amdgcn_raw_buffer_store_b128(w, yr, (int)off, 0, 0);
            } else {
              u32x2_t w;
#pragma unroll
              for (int e = 0; e < 2; ++e)
                w[e] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2 * e]) |
                       ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2 * e + 1]) << 16);
              __builtin_amdgcn_raw_buffer_store_b64(w, yr, (int)off, 0, 0);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t off = cl + e < rn ? base + e * YSZ : 0x80000000u;
              if constexpr (YT == EB_F32)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[e]), yr, (int)off, 0, 0);
              else
                __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, (__bf16)v[e]), yr,
                                                      (int)off, 0, 0);
            }
          }
        }
      }
    }
    return packed;
  };

  {
    constexpr int Z = ABYTES / 16 / 256;
    static_assert(Z * 256 * 16 == ABYTES, "zero fill must cover the x buffers");
#pragma unroll
    for (int i = 0; i < Z; ++i) {
      const int o = (tid + i * 256) * 16;
      *reinterpret_cast<uint4 *>(sA0 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA1 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sA2 + o) = make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();

  MMPos C;
  C.op = lo;
  C.u = u_begin;
  C.valid = true;
  mm_seek(ops, C, u_end);
  LState L;
  L.p = C;
  l_enter(L);
  // prologue: steps 0 and 1, wait for step 0
  l_issue(sA0, sW0, sS0, L);
  l_issue(sA1, sW1, sS1, L);
  wait_vm_barrier<NSTEP>();

  // step t: copy step t+2 into the free stage, read this wave's codes of step t,
  // dequantize, MFMAs; at a tile's last K step store y; then wait for the
  // copies of step t+1.  The copies of step t+1 were issued before this step's
  // copies and before any stores of this step or the one before it, so with
  // packed stores pending the wait leaves up to NSTEP + NST newer ops in flight
  // (which may also force the older tile's stores out; waiting longer is safe).
  bool pend = false;
  auto step = [&](const uint8_t *A, const uint8_t *Wt, const uint8_t *St, uint8_t *A2, uint8_t *W2,
                  uint8_t *S2) __attribute__((always_inline)) {
    l_issue(A2, W2, S2, L);
    uint4 bq[FN][4];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      uint4 q[QT == EB_Q8_0 ? 2 : 1];
#pragma unroll
      for (int h = 0; h < (QT == EB_Q8_0 ? 2 : 1); ++h)
        q[h] = *reinterpret_cast<const uint4 *>(Wt + bq_off[j][h]);
      const uint16_t d = *reinterpret_cast<const uint16_t *>(St + bs_off[j]);
      dequant_b<QT, XT>(q, (float)__builtin_bit_cast(_Float16, d), bq[j]);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 af[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(A + (abase[i] ^ (16u * s)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(bq[j][s], af[i], acc[i][j]);
    }
    if (C.valid && C.kt == C.nk - 1) {
      const bool packed = epilogue(C);
      zero_acc();
      if (packed) {
        wait_vm_barrier<NSTEP + NST>();
      } else {
        wait_vm_barrier<0>();
      }
      pend = packed;
    } else {
      if (pend) {
        wait_vm_barrier<NSTEP + NST>();
      } else {
        wait_vm_barrier<NSTEP>();
      }
      pend = false;
    }
    mm_step(ops, C, u_end);
  };
  for (int64_t j = 0; j < nsteps; j += 3) {
    step(sA0, sW0, sS0, sA2, sW2, sS2);
    step(sA1, sW1, sS1, sA0, sW0, sS0);
    step(sA2, sW2, sS2, sA1, sW1, sS1);
  }
  // the copies issued for steps past the end still write LDS: let them land
  // before the workgroup's LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#endif  // __HIP_DEVICE_COMPILE__
}

template <int QT, int XT, int YT>
hipError_t launch_multi_q(int cfg, const MMOp *ops, int nops, const int64_t *wg, int groups,
                          hipStream_t s) {
  switch (cfg) {
    case 0:
      mm_breg_kernel<QT, XT, YT, 64, 2><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      break;
    case 4:
      mm_ldsw_kernel<QT, XT, YT, 2><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      break;
    case 5:
      mm_ldsw_kernel<QT, XT, YT, 1><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      break;
    case 6:
      return launch_lds2(QT, XT, YT, ops, nops, wg, groups, s);
    case 1:
      mm_breg_kernel<QT, XT, YT, 128, 1><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      break;
    case 2:
      mfma_multi_kernel<QT, XT, YT, 64, 128, 2, 2, 3><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      break;
    default:
      mfma_multi_kernel<QT, XT, YT, 256, 256, 2, 4, 2><<<groups, 512, 0, s>>>(ops, nops, wg, groups);
      break;
  }
  return hipGetLastError();
}

template <int QT, int XT>
hipError_t launch_multi_y(int32_t yt, int cfg, const MMOp *ops, int nops, const int64_t *wg,
                          int groups, hipStream_t s) {
  if (yt == EB_F32) return launch_multi_q<QT, XT, EB_F32>(cfg, ops, nops, wg, groups, s);
  return launch_multi_q<QT, XT, EB_BF16>(cfg, ops, nops, wg, groups, s);
}

// {BM, BN, workgroups per CU, k per step}: 0, 1 weights in registers (m <= 64,
// m <= 128); 2, 3 weights dequantized through LDS (64 x 128 kept for
// comparison, 256 x 256 for m > 128); 4, 5 raw codes through LDS; 6 raw codes
// through LDS in 128-wide K steps
constexpr int kMMTiles[7][4] = {{64, 256, 2, 64}, {128, 128, 2, 64}, {64, 128, 2, 64},
                                {256, 256, 1, 64}, {64, 256, 2, 64}, {64, 128, 3, 64},
                                {64, 256, 1, 128}};
constexpr int kMMCfgs = 7;

}  // namespace

int mm_cfg(int64_t max_m) {
  static const int forced = [] {
    const char *e = getenv("EB_MM_CFG");  // tuning: force the fused tile
    return e ? atoi(e) : -1;
  }();
  if (forced >= 0 && forced < kMMCfgs && (max_m <= 64 || forced == 1 || forced == 3)) return forced;
  return max_m <= 64 ? 6 : (max_m <= 128 ? 1 : 3);
}

int mm_bk(int cfg) { return kMMTiles[cfg][3]; }

int64_t mm_tiles(int cfg, int64_t m, int64_t n) {
  const int bm = kMMTiles[cfg][0], bn = kMMTiles[cfg][1];
  return ((m + bm - 1) / bm) * ((n + bn - 1) / bn);
}

int mm_partition(const std::vector<MMOp> &ops, int cfg, std::vector<int64_t> &wg) {
  int64_t steps = 0, units = 0;
  for (const MMOp &o : ops) {
    steps += (o.unit_end - units) * o.nk;
    units = o.unit_end;
  }
  // as many workgroups as fit on the CUs at once, a multiple of 8
  int64_t groups = std::min<int64_t>((int64_t)device_cu_count() * kMMTiles[cfg][2], units);
  groups = std::max<int64_t>(kXcds, (groups + kXcds - 1) / kXcds * kXcds);
  // workgroup p ends at the first unit boundary at or past (p + 1) * steps / groups
  wg.assign(groups + 1, units);
  wg[0] = 0;
  int64_t acc = 0, u = 0;
  size_t oi = 0;
  for (int64_t p = 0; p + 1 < groups; ++p) {
    const int64_t target = (p + 1) * steps / groups;
    while (u < units && acc < target) {
      while (ops[oi].unit_end <= u) ++oi;
      const int64_t take = std::min(ops[oi].unit_end - u,
                                    std::max<int64_t>(1, (target - acc + ops[oi].nk - 1) / ops[oi].nk));
      acc += take * ops[oi].nk;
      u += take;
    }
    wg[p + 1] = u;
  }
  return (int)groups;
}

hipError_t launch_mfma_multi(int32_t type, int32_t xt, int32_t yt, int cfg, const MMOp *dev_ops,
                             int nops, const int64_t *dev_wg, int groups, hipStream_t s) {
  if (nops < 1 || groups < kXcds || groups % kXcds != 0) return hipErrorInvalidValue;
  if (type == EB_Q4_0) {
    if (xt == EB_F16)
      return launch_multi_y<EB_Q4_0, EB_F16>(yt, cfg, dev_ops, nops, dev_wg, groups, s);
    return launch_multi_y<EB_Q4_0, EB_BF16>(yt, cfg, dev_ops, nops, dev_wg, groups, s);
  }
  if (xt == EB_F16) return launch_multi_y<EB_Q8_0, EB_F16>(yt, cfg, dev_ops, nops, dev_wg, groups, s);
  return launch_multi_y<EB_Q8_0, EB_BF16>(yt, cfg, dev_ops, nops, dev_wg, groups, s);
}
}  // namespace eb
