// mfma_lds2.hip -- fused MFMA launch over many independent small-m ops
// (m <= 64) of a stack, in 128-wide K steps (paper section 3.2: operator
// fusion for batch-1 execution; the action-chunk denoising steps of section
// 2.1 / Table 1 run hundreds of such layers per pass).  Built with the MFMA
// accumulators in AGPRs: this kernel's loop keeps them there without copies,
// which leaves the VGPRs for the software pipeline.
#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"
#include "mm_common.h"

namespace eb {
namespace {

// ---------------------------------------------------------------------------
// Fused small-m launch with 128-wide K steps.  Memory cost here follows the
// number of cache lines a load touches more than its bytes, so every load is
// shaped to use whole lines:
//  * codes: a step covers two K-tiles, so a Q8_0 row segment is a full
//    128-byte line (Q4_0: 64 bytes); copied into LDS by 8 (16) rows per
//    1 KB buffer load that writes LDS directly, three stages, two steps ahead;
//  * x: 64 rows x 256 bytes per step, two stages, one step ahead (x is small
//    and stays in L2);
//  * scales: once per group of four steps (16 blocks, 32 bytes of a row),
//    two 16-byte lanes per row, loaded into registers a step ahead and written
//    to one of two LDS stages at the end of the next step.  Steps without a
//    scale load issue the same loads with an empty range (no memory access),
//    so every step has the same number of vector-memory ops in flight.
// One workgroup of WAVES waves per CU (launched with 8); wave w owns the
// 256 / WAVES columns from (256 / WAVES) w of the 64 x 256 tile and
// dequantizes its codes straight into MFMA registers, with
// the k order of mm_breg_kernel applied to each 64-wide half of the step.
// The weights are the MFMA A operand, so y leaves in 4-column packed stores.
// Chunk (16 B) swizzles keep the 16-lane phases of every LDS read on distinct
// banks: x chunk c of row r at c ^ (r & 15); Q8_0 codes at c ^ ((r >> 1) & 7);
// Q4_0 codes at c ^ ((r >> 2) & 3).
// ---------------------------------------------------------------------------
// HL: bfloat16 activations with w_hat as hi/lo bfloat16 pairs (two MFMAs per
// product, w_hat carried to 2^-16); without it w_hat is rounded once to the
// activation type (binary16 holds it to 2^-11, bfloat16 to 2^-8).
template <int QT, int XT, int YT, int WAVES, bool HL>
__global__ void __launch_bounds__(WAVES * 64)
    mm_lds2_kernel(const MMOp *__restrict__ ops, int nops, const int64_t *__restrict__ wg,
                   int groups) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int BM = 64, BN = 256, FN = BN / (32 * WAVES), FM = BM / 32;
  constexpr int T = WAVES * 64;
  static_assert((WAVES == 4 || WAVES == 8) && FN * 32 * WAVES == BN, "4 or 8 waves");
  constexpr int BKS = 2 * kBK;                    // k per step
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;  // code bytes per block
  constexpr int NQ = (QT == EB_Q8_0) ? 2 : 1;     // 16-byte chunks per block
  constexpr int CROW = 4 * QSB;                   // code bytes per row per step
  constexpr int CCH = CROW / 16;                  // code chunks per row per step
  constexpr int XROW = BKS * 2;                   // x bytes per row per step
  constexpr int XBYTES = BM * XROW, WBYTES = BN * CROW, SBYTES = BN * 32;
  constexpr int NX = XBYTES / 1024 / WAVES;       // x copies per lane per step
  constexpr int NW = WBYTES / 1024 / WAVES;       // code copies per lane per step
  constexpr int NS = SBYTES / 16 / T;             // scale loads per lane per step
  constexpr int NST = FM * FN * 4;                // packed y stores per lane per tile
  constexpr int YSZ = (YT == EB_F32) ? 4 : 2;
  static_assert(NX * 1024 * WAVES == XBYTES && NW * 1024 * WAVES == WBYTES, "copies must tile");
  static_assert(NS * 16 * T == SBYTES && NW + NS + NST <= 63, "scale loads / wait count range");
  static_assert(!HL || XT == EB_BF16, "hi/lo pairs are for bfloat16 activations");

  __shared__ __attribute__((aligned(1024))) uint8_t sX0[XBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sX1[XBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW0[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW1[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sW2[WBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sS[2 * SBYTES];

  const int g = blockIdx.x;
  const int p = (g % kXcds) * (groups / kXcds) + g / kXcds;
  const int64_t u_begin = wg[p], u_end = wg[p + 1];
  if (u_begin >= u_end) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const uint32_t wh = (uint32_t)(lane >> 5);

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
    return QT == EB_Q8_0 ? ((r >> 1) & 7) : ((r >> 2) & 3);
  };

  // --- lane parts of the loads (tile-local offsets) ----------------------------
  uint32_t xo_[NX], wo_[NW], so_[NS], sd_[NS];
#pragma unroll
  for (int i = 0; i < NX; ++i) {
    const uint32_t r = 4 * (i * WAVES + wave) + (lane >> 4);
    xo_[i] = r;  // row; chunk part added per op (row stride differs)
  }
  const uint32_t xc_ = (uint32_t)(lane & 15);
#pragma unroll
  for (int i = 0; i < NW; ++i) wo_[i] = (1024 / CROW) * (i * WAVES + wave) + lane / CCH;
  const uint32_t wc_ = (uint32_t)(lane % CCH);
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const uint32_t r = i * (T / 2) + (tid >> 1);
    so_[i] = r;
    sd_[i] = r * 32 + (tid & 1) * 16;  // LDS offset within a scale stage
  }

  // --- x cursor (one step ahead) ----------------------------------------------
  struct XState {
    MMPos p;
    const uint8_t *b;
    uint32_t rec, v[NX];
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
    const uint32_t xrow = (uint32_t)o.k * 2;
    s.b = reinterpret_cast<const uint8_t *>(o.x) + m0 * xrow;
    s.rec = (uint32_t)rm * xrow;
#pragma unroll
    for (int i = 0; i < NX; ++i) s.v[i] = xo_[i] * xrow + ((xc_ ^ (xo_[i] & 15)) << 4);
  };
  // one of the four x copies of a step (the cursor's current step)
  auto x_copy = [&](uint8_t *sX, const __amdgpu_buffer_rsrc_t &r, const XState &s, int i)
      __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(sX + (i * WAVES + wave) * 1024), 16,
                                             (int)s.v[i], 0, 0, 0);
  };
  auto x_advance = [&](XState &s) __attribute__((always_inline)) {
    if (mm_step(ops, s.p, u_end)) {
      x_enter(s);
    } else if (s.p.valid) {
      s.b += XROW;
      s.rec -= XROW;
    }
  };

  // --- codes + scales cursor (two steps ahead) -------------------------------
  struct WState {
    MMPos p;
    const uint8_t *qb, *db;
    uint32_t qrec, drec, qv[NW], dv[NS];
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
    s.qrec = (uint32_t)rn * qrow;
    s.db = o.w + o.d_off + n0 * drow;
    s.drec = (uint32_t)rn * drow;
#pragma unroll
    for (int i = 0; i < NW; ++i) s.qv[i] = wo_[i] * qrow + ((wc_ ^ gsw(wo_[i])) << 4);
#pragma unroll
    for (int i = 0; i < NS; ++i) s.dv[i] = so_[i] * drow + (tid & 1) * 16;
  };
  // returns whether the scale loads were real (the step starts a group)
  auto w_copy = [&](uint8_t *sW, const __amdgpu_buffer_rsrc_t &r, const WState &s, int i)
      __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(sW + (i * WAVES + wave) * 1024), 16,
                                             (int)s.qv[i], 0, 0, 0);
  };
  auto w_advance = [&](WState &s) __attribute__((always_inline)) {
    if (mm_step(ops, s.p, u_end)) {
      w_enter(s);
    } else if (s.p.valid) {
      s.qb += CROW;
      s.qrec -= CROW;
      if ((s.p.kt & 3) == 0) {
        s.db += 32;
        s.drec -= 32;
      }
    }
  };

  // --- per-lane LDS read offsets ---------------------------------------------
  uint32_t bq_off[FN][2][NQ], bs_off[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const uint32_t r = wave * 32 * FN + j * 32 + (lane & 31);
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int h = 0; h < NQ; ++h) {
        const uint32_t c = (2 * q + wh) * NQ + h;  // chunk of block 2q + wh
        bq_off[j][q][h] = r * CROW + ((c ^ gsw(r)) << 4);
      }
    bs_off[j] = r * 32;
  }
  uint32_t abase[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const uint32_t r = i * 32 + (lane & 31);
    abase[i] = r * XROW + (((4u * wh) ^ (r & 15)) << 4);
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

  // lane (l, reg r) of sub-tile (i, j) holds y[m0 + 32 i + l % 32][n0 + 32 FN wave
  // + 32 j + 8 (r / 4) + 4 (l / 32) + r % 4]; rows past the op's m read zero x
  // (x rows past the buffer) and columns past its n are not stored.
  //
  // Fused steps: the residual of EB_EPI_ADD is read with the same packed
  // accesses as the stores; with EB_EPI_GLU the four columns of a packed
  // store are two gate/up pairs, giving two adjacent outputs, so the packed
  // path still issues NST stores per tile.  YT only fixes the output size:
  // 16-bit outputs are bf16 or fp16 by the op's type.
  auto epilogue = [&](const MMPos &c) __attribute__((always_inline)) -> bool {
    int64_t m0, n0;
    int rm, rn;
    mm_tile<BM, BN>(ops, c, m0, n0, rm, rn);
    const MMOp &o = ops[c.op];
    const uint32_t n = (uint32_t)o.n;
    const int yt = o.yt;
    const bool glu = o.f.epi == EB_EPI_GLU, add = o.f.epi == EB_EPI_ADD;
    const uint32_t nout = glu ? n / 2 : n;
    const auto yr = ursrc(o.y, (uint32_t)o.m * nout * YSZ);
    const auto rr = ursrc(add ? o.f.r : o.y, (uint32_t)o.m * n * YSZ);
    const bool packed = (n & 3) == 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint32_t row = (uint32_t)m0 + i * 32 + (lane & 31);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        // the fragment's 16 residuals read before any output is written (an
        // output reads only its own residual; one group after the other,
        // each read would wait behind the previous write)
        float res[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) res[q][e] = 0.f;
        if (add) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int cl = wave * 32 * FN + j * 32 + 8 * q + 4 * (int)wh;
            const uint32_t base = (row * n + (uint32_t)n0 + cl) * YSZ;
            if (packed) {
              const uint32_t off = cl < rn ? base : 0x80000000u;
              if constexpr (YT == EB_F32) {
                const u32x4_t r = __builtin_amdgcn_raw_buffer_load_b128(rr, (int)off, 0, 0);
                // element values: this compiler turns __builtin_bit_cast of a
                // vector element into element 0 of the vector (one dword loaded)
#pragma unroll
                for (int e = 0; e < 4; ++e) res[q][e] = __uint_as_float((uint32_t)r[e]);
              } else {
                const u32x2_t r = __builtin_amdgcn_raw_buffer_load_b64(rr, (int)off, 0, 0);
#pragma unroll
                for (int e = 0; e < 4; ++e) res[q][e] = from_y16((uint16_t)(r[e >> 1] >> (16 * (e & 1))), yt);
              }
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t off = cl + e < rn ? base + e * YSZ : 0x80000000u;
                if constexpr (YT == EB_F32)
                  res[q][e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (int)off, 0, 0));
                else
                  res[q][e] = from_y16(__builtin_amdgcn_raw_buffer_load_b16(rr, (int)off, 0, 0), yt);
              }
            }
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cl = wave * 32 * FN + j * 32 + 8 * q + 4 * (int)wh;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e];  // copy first: see mfma_multi_kernel
          if (glu) {
            const float g0 = silu_mul(v[0], v[1]), g1 = silu_mul(v[2], v[3]);
            const uint32_t gb = (row * nout + ((uint32_t)n0 + cl) / 2) * YSZ;
            if (packed) {
              const uint32_t off = cl < rn ? gb : 0x80000000u;
              if constexpr (YT == EB_F32) {
                u32x2_t w;
                w[0] = __builtin_bit_cast(uint32_t, g0);
                w[1] = __builtin_bit_cast(uint32_t, g1);
                __builtin_amdgcn_raw_buffer_store_b64(w, yr, (int)off, 0, 0);
              } else {
                const uint32_t w = (uint32_t)to_y16(g0, yt) | ((uint32_t)to_y16(g1, yt) << 16);
                __builtin_amdgcn_raw_buffer_store_b32(w, yr, (int)off, 0, 0);
              }
            } else {
#pragma unroll
              for (int e = 0; e < 2; ++e) {
                const uint32_t off = cl + 2 * e < rn ? gb + e * YSZ : 0x80000000u;
                const float g = e ? g1 : g0;
                if constexpr (YT == EB_F32)
                  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, g), yr, (int)off, 0, 0);
                else
                  __builtin_amdgcn_raw_buffer_store_b16(to_y16(g, yt), yr, (int)off, 0, 0);
              }
            }
            continue;
          }
          const uint32_t base = (row * n + (uint32_t)n0 + cl) * YSZ;
          if (packed) {
            const uint32_t off = cl < rn ? base : 0x80000000u;
            if constexpr (YT == EB_F32) {
              if (add) {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] += res[q][e];
              }
              u32x4_t w;
#pragma unroll
              for (int e = 0; e < 4; ++e) w[e] = __builtin_bit_cast(uint32_t, v[e]);
              __builtin_amdgcn_raw_buffer_store_b128(w, yr, (int)off, 0, 0);
            } else {
              if (add) {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] += res[q][e];
              }
              u32x2_t w;
#pragma unroll
              for (int e = 0; e < 2; ++e)
                w[e] = (uint32_t)to_y16(v[2 * e], yt) | ((uint32_t)to_y16(v[2 * e + 1], yt) << 16);
              __builtin_amdgcn_raw_buffer_store_b64(w, yr, (int)off, 0, 0);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t off = cl + e < rn ? base + e * YSZ : 0x80000000u;
              if (add) v[e] += res[q][e];
              if constexpr (YT == EB_F32)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[e]), yr, (int)off, 0, 0);
              else
                __builtin_amdgcn_raw_buffer_store_b16(to_y16(v[e], yt), yr, (int)off, 0, 0);
            }
          }
        }
      }
    }
    return packed;
  };

  {
    constexpr int Z = XBYTES / 16 / T;
    static_assert(Z * T * 16 == XBYTES, "zero fill must cover the x buffers");
#pragma unroll
    for (int i = 0; i < Z; ++i) {
      const int o = (tid + i * T) * 16;
      *reinterpret_cast<uint4 *>(sX0 + o) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(sX1 + o) = make_uint4(0, 0, 0, 0);
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
  WState W;
  W.p = C;
  w_enter(W);

  // prologue: x of step 0, codes and scales of steps 0 and 1; the scales of
  // step 0 (always a group start) go to stage 0 once they have arrived
  uint4 sa[NS], sb[NS];
  auto w_issue = [&](uint8_t *sW, uint4 (&sreg)[NS], WState &s) __attribute__((always_inline)) -> bool {
    const bool grp = s.p.valid && (s.p.kt & 3) == 0;
    const auto qr = ursrc(s.qb, s.qrec);
    const auto dr = ursrc(s.db, grp ? s.drec : 0u);
#pragma unroll
    for (int i = 0; i < NW; ++i) w_copy(sW, qr, s, i);
#pragma unroll
    for (int i = 0; i < NS; ++i) sreg[i] = bload(dr, s.dv[i]);
    w_advance(s);
    return grp;
  };
  {
    const auto xr = ursrc(X.b, X.rec);
#pragma unroll
    for (int i = 0; i < NX; ++i) x_copy(sX0, xr, X, i);
    x_advance(X);
  }
  w_issue(sW0, sa, W);
  bool spend = w_issue(sW1, sb, W);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NW + NS) : "memory");
#pragma unroll
  for (int i = 0; i < NS; ++i) *reinterpret_cast<uint4 *>(sS + sd_[i]) = sa[i];
  wait_vm_barrier<NW + NS>();

  uint32_t gstage = 0;  // LDS scale stage of the current step's group
  // step t: x of step t+1, codes and scales of step t+2; read this step's
  // scales and codes, dequantize, MFMAs; at a tile's last step store y; write
  // the scales loaded in the previous step (group starting at step t+1) to
  // the other stage; wait for step t+1's copies.
  auto step = [&](const uint8_t *Xc, const uint8_t *Wc, uint8_t *Xn, uint8_t *Wn, uint4 (&sprev)[NS],
                  uint4 (&snew)[NS]) __attribute__((always_inline)) {
    // This step's copies (x of step t+1, codes and scales of step t+2) are
    // spread over the compute in small groups: issued all at once, a wave
    // stalls until the CU's memory pipeline has taken most of them.  The
    // fences keep each group in place; between them the scheduler is free.
    const bool snext = W.p.valid && (W.p.kt & 3) == 0;
    const auto xr = ursrc(X.b, X.rec);
    const auto qr = ursrc(W.qb, W.qrec);
    const auto dr = ursrc(W.db, snext ? W.drec : 0u);
    const uint8_t *Sc = sS + gstage * SBYTES + 8 * (C.kt & 3);
    auto fence = []() __attribute__((always_inline)) { __builtin_amdgcn_sched_barrier(0); };
    uint4 cq[2][FN][NQ];
    uint16_t dq[2][FN];
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int h = 0; h < NQ; ++h) cq[q][j][h] = *reinterpret_cast<const uint4 *>(Wc + bq_off[j][q][h]);
        const uint32_t d2 = *reinterpret_cast<const uint32_t *>(Sc + bs_off[j] + 4 * q);
        dq[q][j] = (uint16_t)(d2 >> (16 * wh));
      }
    uint4 bq[2][FN][4];
    uint4 bl[2][FN][HL ? 4 : 1];  // bfloat16: the low parts of the hi/lo pairs
    auto deq = [&](int q, int j) __attribute__((always_inline)) {
      const float d = (float)__builtin_bit_cast(_Float16, dq[q][j]);
      if constexpr (HL)
        dequant_b_hl<QT>(cq[q][j], d, bq[q][j], bl[q][j]);
      else
        dequant_b<QT, XT>(cq[q][j], d, bq[q][j]);
    };
    auto mm = [&](int q, int s) __attribute__((always_inline)) {
      uint4 af[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const uint4 *>(Xc + (abase[i] ^ ((8u * q + s) << 4)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(bq[q][j][s], af[i], acc[i][j]);
      if constexpr (HL) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(bl[q][j][HL ? s : 0], af[i], acc[i][j]);
      }
    };
    // copy c of this step: x copies first, then codes, then scale loads (the
    // order the barrier's wait counts assume)
    auto copy = [&](int c) __attribute__((always_inline)) {
      if (c < NX)
        x_copy(Xn, xr, X, c);
      else if (c < NX + NW)
        w_copy(Wn, qr, W, c - NX);
      else
        snew[c - NX - NW] = bload(dr, W.dv[c - NX - NW]);
    };
    constexpr int NC = NX + NW + NS;
    // compute in six chunks; after chunk k the copies [k NC / 6, (k + 1) NC / 6)
    auto copies_after = [&](int k) __attribute__((always_inline)) {
      fence();
#pragma unroll
      for (int c = k * NC / 6; c < (k + 1) * NC / 6; ++c) copy(c);
      fence();
    };
#pragma unroll
    for (int j = 0; j < FN; ++j) deq(0, j);
    copies_after(0);
    mm(0, 0);
    mm(0, 1);
    copies_after(1);
#pragma unroll
    for (int j = 0; j < FN; ++j) deq(1, j);
    copies_after(2);
    mm(0, 2);
    mm(0, 3);
    copies_after(3);
    mm(1, 0);
    mm(1, 1);
    copies_after(4);
    mm(1, 2);
    mm(1, 3);
    copies_after(5);
    x_advance(X);
    w_advance(W);
    // before the y stores: the wait for sprev then covers only older loads
    if (spend) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
        *reinterpret_cast<uint4 *>(sS + (gstage ^ 1) * SBYTES + sd_[i]) = sprev[i];
    }
    spend = snext;
    bool stored = false;
    if (C.valid && C.kt == C.nk - 1) {
      stored = epilogue(C);
      zero_acc();
      if (!stored) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    if (stored) {
      wait_vm_barrier<NW + NS + NST>();
    } else {
      wait_vm_barrier<NW + NS>();
    }
    mm_step(ops, C, u_end);
    if (C.valid && (C.kt & 3) == 0) gstage ^= 1;
  };
  for (int64_t j = 0; j < nsteps; j += 6) {
    step(sX0, sW0, sX1, sW2, sb, sa);
    step(sX1, sW1, sX0, sW0, sa, sb);
    step(sX0, sW2, sX1, sW1, sb, sa);
    step(sX1, sW0, sX0, sW2, sa, sb);
    step(sX0, sW1, sX1, sW0, sb, sa);
    step(sX1, sW2, sX0, sW1, sa, sb);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#endif  // __HIP_DEVICE_COMPILE__
}

// YT = EB_F32 for fp32 outputs, EB_BF16 for either 16-bit output type.
template <int QT, int XT, int WAVES, bool HL>
hipError_t lds2_y(int32_t yt, const MMOp *ops, int nops, const int64_t *wg, int groups, hipStream_t s) {
  if (yt == EB_F32)
    mm_lds2_kernel<QT, XT, EB_F32, WAVES, HL><<<groups, WAVES * 64, 0, s>>>(ops, nops, wg, groups);
  else
    mm_lds2_kernel<QT, XT, EB_BF16, WAVES, HL><<<groups, WAVES * 64, 0, s>>>(ops, nops, wg, groups);
  return hipGetLastError();
}

template <int QT, int WAVES>
hipError_t lds2_x(int32_t xt, bool hl, int32_t yt, const MMOp *ops, int nops, const int64_t *wg,
                  int groups, hipStream_t s) {
  if (xt == EB_F16) return lds2_y<QT, EB_F16, WAVES, false>(yt, ops, nops, wg, groups, s);
  if (hl) return lds2_y<QT, EB_BF16, WAVES, true>(yt, ops, nops, wg, groups, s);
  return lds2_y<QT, EB_BF16, WAVES, false>(yt, ops, nops, wg, groups, s);
}

template <int WAVES>
hipError_t lds2_q(int32_t type, int32_t xt, bool hl, int32_t yt, const MMOp *ops, int nops,
                  const int64_t *wg, int groups, hipStream_t s) {
  if (type == EB_Q4_0) return lds2_x<EB_Q4_0, WAVES>(xt, hl, yt, ops, nops, wg, groups, s);
  return lds2_x<EB_Q8_0, WAVES>(xt, hl, yt, ops, nops, wg, groups, s);
}

}  // namespace

hipError_t launch_lds2(int32_t type, int32_t xt, bool hl, int32_t yt, const MMOp *ops, int nops,
                       const int64_t *wg, int groups, hipStream_t s) {
  // 8 waves: two per SIMD, so one wave's LDS and memory waits overlap the
  // other's dequantization and MFMAs (4 waves measured 6% slower)
  return lds2_q<8>(type, xt, hl, yt, ops, nops, wg, groups, s);
}

}  // namespace eb
