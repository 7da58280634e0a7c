// mfma_tile.h -- the tile kernel of the matrix-core path and its launch
// templates.  Included only by the per-format translation units
// (mfma_<format>_<activation>.hip), which instantiate mfma_tile_launch and
// mfma_tile_launch_grouped for one weight format and activation type each, so
// the kernel variants compile in parallel; mfma.hip holds the planning, the
// split-K reductions and the dispatch to these instantiations.
//
// The matrix-core path of the quantized linear layer for m > 4 activation
// rows: prefill of image/text tokens, action-chunk denoising and video-latent
// tokens (paper section 2.1 / Table 1 model families; section 3.2
// "operator fusion, backend-specific dispatch").
//
// y[m][n] = sum_k x[m][k] * w_hat[n][k], w_hat = code * d16 (Q6_S: (u - 32)
// d16 sc_j) rounded once to the activation type (bfloat16 or binary16), or,
// for bfloat16 activations on the small tiles (m <= 128; Q8_0 and Q4_0),
// carried as a hi/lo pair of bfloat16 values; fp32 accumulation.
//
// A workgroup of WM x WN waves computes a BM x BN tile of y; each wave owns a
// (BM/WM) x (BN/WN) sub-tile of fp32 accumulators.  Per K-tile of 64:
//   * global -> LDS: the x tile is copied by buffer loads that write LDS
//     directly (no register staging), into one of three buffers;
//   * global -> registers: the packed weight tile (16-byte code loads plus
//     binary16 scales) into one of three register sets;
//   * registers -> LDS: weights dequantized (code * d16 exact in fp32, one
//     round-to-nearest-even to 16 bits) into one of two buffers -- fused into
//     the tile load, no dequantized weight ever reaches HBM;
//   * LDS -> MFMA: v_mfma_f32_32x32x16_{bf16,f16}, A = x rows, B = w_hat rows.
// Each K-tile step issues the x copy of tile t+2 and the weight loads of tile
// t+3, runs the MFMAs of tile t with the dequantization of tile t+1
// interleaved, and waits only for x tile t+1 before its barrier, so every load
// has about two steps of MFMA work to land.
//
// Problems with too few tiles to fill the GPU split k over workgroups; each
// split writes an fp32 partial tile and a second kernel sums them in order.
//
// Tiles are ordered for the 8 XCDs of MI355X (workgroups are dispatched to
// XCDs round-robin, each XCD has its own L2): each XCD gets a contiguous range
// of tiles, N-tile fastest, so the workgroups sharing an L2 mostly share one
// block of x rows.
#ifndef EB_MFMA_TILE_H
#define EB_MFMA_TILE_H

#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"

namespace eb {
namespace {

// A 1 KiB-aligned LDS array of its own (one per BYTES, ID), allocated only in
// kernels that call this.
template <int BYTES, int ID>
__device__ inline uint8_t *lds_array() {
  __shared__ __attribute__((aligned(1024))) uint8_t a[BYTES];
  return a;
}

// G: grouped launch over several independent ops -- workgroup b runs tile
// gorder[b].y of op gorder[b].x (entries with a negative op do nothing), with
// the op's operands from gops; the scalar arguments are then unused.
// HL (bfloat16 activations, small tiles): w_hat enters the matrix cores as a
// hi/lo pair of bfloat16 tiles (split2_bf16), two MFMAs per product, so the
// product carries w_hat to 2^-16 instead of the 2^-8 of one bfloat16 rounding.
template <int QT, int XT, int BM, int BN, int WM, int WN, bool G = false, bool HL = false>
__global__ void __launch_bounds__(WM *WN * 64)
    mfma_kernel(const uint8_t *__restrict__ wdata_, int64_t n_, int64_t k_, int64_t d_off_,
                int64_t ds_, int64_t sc_off_, const uint16_t *__restrict__ x_, int64_t m_, void *__restrict__ y_,
                int yt_, Fuse f_, int kts_, float *__restrict__ ws, int64_t ws_stride,
                const GOp *__restrict__ gops, const int2 *__restrict__ gorder) {
  const uint8_t *wdata = wdata_;
  const uint16_t *x = x_;
  void *y = y_;
  int64_t n = n_, k = k_, d_off = d_off_, ds = ds_, sc_off = sc_off_, m = m_;
  int yt = yt_, kts = kts_;
  Fuse f = f_;
  int64_t gtile = 0;
  if constexpr (G) {
    const int2 e = gorder[blockIdx.x];
    if (e.x < 0) return;
    const GOp &o = gops[e.x];
    wdata = o.w;
    x = o.x;
    y = o.y;
    n = o.n;
    k = o.k;
    d_off = o.d_off;
    ds = o.ds;
    sc_off = o.sc_off;
    m = o.m;
    yt = o.yt;
    f = o.f;
    kts = (int)((k + kBK - 1) / kBK);
    gtile = e.y;
  }
  constexpr int T = WM * WN * 64;
  constexpr int WAVES = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;        // wave sub-tile
  constexpr int FM = TM / 32, FN = TN / 32;        // 32x32 fragments per wave
  constexpr int ADMA = BM / (8 * WAVES);           // x copies per wave per K-tile (8 rows each)
  constexpr int WCPR = WTile<QT>::kChunksPerRow;
  constexpr int WCH = BN * WCPR;                   // weight chunks per K-tile
  constexpr int BCH = (WCH + T - 1) / T;           // per thread (the last may be partial)
  constexpr int KSTEPS = kBK / 16;
  constexpr bool Q6 = QT == EB_Q6_S;
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : (Q6 ? 24 : 16);  // code bytes per 32 weights
  constexpr int NV = Deq<QT>::kVecs;               // 16-byte vectors per dequantized chunk
  constexpr int ABYTES = BM * kBK * 2, BBYTES = BN * kBK * 2;
  static_assert(!HL || XT == EB_BF16, "hi/lo weight tiles are for bfloat16 activations");
  static_assert(!HL || !Q6, "Q6_S takes this kernel only without hi/lo tiles (m > 128)");
  constexpr int BW = (HL ? 4 : 2) * BBYTES;         // the two weight buffers (hi and lo parts)
  constexpr int NRD = FM + FN * (HL ? 2 : 1);       // LDS fragment reads per k-step
  constexpr int NMF = FM * FN * (HL ? 2 : 1);       // MFMAs per k-step
  // vector-memory operations one thread issues per K-tile
  constexpr int NX = ADMA, NW = (Q6 ? 4 : 2) * BCH;  // Q6_S: codes, top bits, d16, sub-scales
  static_assert(ADMA >= 1 && ADMA * 8 * WAVES == BM, "x tile must split into 8-row copies");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave sub-tile must be whole fragments");
  static_assert(2 * NW + NX <= 63, "vmcnt range");
  // x buffers: three when they fit the 160 KiB of LDS beside the two weight
  // buffers (x tile t + 2 is copied during step t), else two (x tile t + 1).
  // With hi/lo weight tiles, three only while two workgroups still fit a CU.
  constexpr int NA = HL ? ((2 * (3 * ABYTES + BW) <= 160 * 1024) ? 3 : 2)
                        : ((3 * ABYTES + BW <= 160 * 1024) ? 3 : 2);
  static_assert(NA * ABYTES + BW <= 160 * 1024, "tile does not fit the LDS");

  // NA x buffers (tile kt in use, kt+1 landing, kt+2 being copied; or tile kt
  // in use, kt+1 being copied) and two weight buffers.  Separate objects, so the compiler can tell the
  // asynchronous copies into one x buffer from the reads of another.  Both
  // tiles use unpadded 128-byte rows with 16-byte chunk c of row r stored at
  // position c ^ swz(r).
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[ABYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sA1[ABYTES];
  // weight buffer i: the (hi) tile, then with HL the lo tile at + BBYTES
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[HL ? 2 * BBYTES : BBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB1[HL ? 2 * BBYTES : BBYTES];
  uint8_t *sA2 = nullptr;
  if constexpr (NA == 3) sA2 = lds_array<ABYTES, 2>();

  // Workgroup -> (K split, output tile).  Split s covers K-tiles
  // [s kts, (s + 1) kts) and, when there are several splits (ws != null),
  // writes its fp32 partial tile to ws + s ws_stride; a second kernel sums them.
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int64_t tiles = tiles_m * tiles_n;
  const int split = G ? 0 : (int)(blockIdx.x / tiles);
  const int64_t bid = G ? 0 : blockIdx.x % tiles;
  // XCD-aware tile order (a grouped launch's table is already in that order)
  int64_t t = G ? gtile : bid;
  if (!G && tiles % kXcds == 0) t = (bid % kXcds) * (tiles / kXcds) + bid / kXcds;
  const int64_t tm = t / tiles_n, tn = t % tiles_n;
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int64_t nb = k / kQK;
  const int rows_m = (int)min((int64_t)BM, m - m0), rows_n = (int)min((int64_t)BN, n - n0);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // Per-workgroup bases, starting at this split's first K-tile; the byte
  // counts shrink with them, so every range check still ends at the end of the
  // tile's rows.  The host guarantees that they fit in 32 bits.
  const int kt0 = split * kts;
  const int nk = (int)min((int64_t)kts, (k + kBK - 1) / kBK - kt0);
  const uint8_t *const xbase = reinterpret_cast<const uint8_t *>(x) + m0 * k * 2 + kt0 * (kBK * 2);
  const uint8_t *const qbase = wdata + n0 * nb * QSB + kt0 * (2 * QSB);
  // scales: Q8_0 / Q4_0 two binary16 scales per row per K-tile; Q6_S one d16
  // per four K-tiles (found by K-tile index, not by a linear advance) and
  // four int8 sub-scales per row per K-tile in the sub-scale plane
  const uint8_t *const dbase = wdata + d_off + n0 * ds * 2 + (Q6 ? 0 : kt0 * 4);
  const int64_t srow = k / 16;
  const uint8_t *const sbase = wdata + sc_off + n0 * srow + kt0 * 4;
  const uint32_t xrec = (uint32_t)(rows_m * k * 2 - kt0 * (kBK * 2));
  const uint32_t qrec = (uint32_t)(rows_n * nb * QSB - kt0 * (2 * QSB));
  const uint32_t drec = (uint32_t)(rows_n * ds * 2 - (Q6 ? 0 : kt0 * 4));
  const uint32_t srec = Q6 ? (uint32_t)(rows_n * srow - kt0 * 4) : 0u;

  // x copy: wave `wave`, copy i moves tile rows 8 (i WAVES + wave) .. +7; lane
  // j fills LDS chunk position j % 8 of row j / 8, i.e. logical chunk
  // (j % 8) ^ swz(row).  Rows past m fall past xrec and read zeros.
  uint32_t xv[ADMA];
#pragma unroll
  for (int i = 0; i < ADMA; ++i) {
    const uint32_t r = 8 * (i * WAVES + wave) + (lane >> 3);
    xv[i] = (uint32_t)(r * k * 2) + (((lane & 7) ^ swz(r)) << 4);
  }
  // Weight chunks: rows past n fall past qrec/drec and read zeros; chunk
  // indices past the tile (only when T does not divide it) are moved past the
  // buffers too and their stores are skipped.  Chunk c of a row covers logical
  // 16-byte positions NV c .. NV c + NV - 1; since NV c is a multiple of NV the
  // stored position of part q is (NV c ^ swz(r)) ^ q, so wl ^ (16 q).  A Q6_S
  // chunk c (bytes 24 c .. 24 c + 23 of the row's 48-byte unit) is read as its
  // 16 code bytes and its 8 top-bit bytes (8-byte aligned loads), with its two
  // sub-scales.
  uint32_t qo[BCH], dof[BCH], wl[BCH], so[Q6 ? BCH : 1];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int idx = min(tid + i * T, WCH), r = idx / WCPR, c = idx % WCPR;
    const int blk = (QT == EB_Q8_0) ? (c >> 1) : c;
    if constexpr (Q6) {
      qo[i] = (uint32_t)(r * nb * QSB + 24 * c);
      dof[i] = (uint32_t)(r * ds * 2);
      so[i] = (uint32_t)(r * srow + 2 * c);
    } else {
      qo[i] = (uint32_t)((r * nb + blk) * QSB + ((QT == EB_Q8_0) ? (c & 1) * 16 : 0));
      dof[i] = (uint32_t)((r * ds + blk) * 2);
    }
    wl[i] = (uint32_t)(r * (kBK * 2) + (((NV * c) ^ swz(r)) << 4));
  }

  auto load_x = [&](uint8_t *sA, int kt) __attribute__((always_inline)) {
    const uint32_t adv = (uint32_t)kt * (kBK * 2);
    const auto xr = rsrc(xbase + adv, xrec - adv);
#pragma unroll
    for (int i = 0; i < ADMA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          xr, (lds_void *)(sA + (i * WAVES + wave) * 1024), 16, (int)xv[i], 0, 0, 0);
  };

  // Raw weight registers of one K-tile.  The K-tail block of an odd block count
  // reads a zero scale from the scale-plane padding, so its weights are zeros.
  struct Raw {
    uint4 b[BCH];
    uint2 h[Q6 ? BCH : 1];      // Q6_S: the chunk's 8 top-bit bytes
    uint16_t d[BCH];
    uint16_t sc[Q6 ? BCH : 1];  // Q6_S: the chunk's two int8 sub-scales
  };
  Raw S0, S1, S2;
  auto load_w = [&](Raw &S, int kt) __attribute__((always_inline)) {
    const uint32_t qadv = (uint32_t)kt * (2 * QSB);
    const uint32_t dadv = Q6 ? (uint32_t)((kt0 + kt) >> 2) * 2 : (uint32_t)kt * 4;
    const auto qr = rsrc(qbase + qadv, qrec - qadv);
    const auto dr = rsrc(dbase + dadv, drec - dadv);
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      S.b[i] = bload(qr, qo[i]);
      if constexpr (Q6) {
        const auto t = __builtin_amdgcn_raw_buffer_load_b64(qr, (int)qo[i] + 16, 0, 0);
        S.h[i] = make_uint2(t[0], t[1]);
      }
      S.d[i] = __builtin_amdgcn_raw_buffer_load_b16(dr, (int)dof[i], 0, 0);
    }
    if constexpr (Q6) {
      const auto sr = rsrc(sbase + (uint32_t)kt * 4, srec - (uint32_t)kt * 4);
#pragma unroll
      for (int i = 0; i < BCH; ++i) S.sc[i] = __builtin_amdgcn_raw_buffer_load_b16(sr, (int)so[i], 0, 0);
    }
  };
  auto store_w = [&](const Raw &S, uint8_t *sB, int i) __attribute__((always_inline)) {
    if (WCH % T != 0 && i == BCH - 1 && tid + i * T >= WCH) return;
    uint4 v[NV];
    const float d = (float)__builtin_bit_cast(_Float16, S.d[i]);
    if constexpr (Q6) {
      dequant_chunk_q6<XT>(S.b[i], S.h[i], S.sc[i], d, v);
    } else if constexpr (HL) {
      uint4 vl[NV];
      dequant_chunk_hl<QT>(S.b[i], d, v, vl);
#pragma unroll
      for (int q = 0; q < NV; ++q) *reinterpret_cast<uint4 *>(sB + BBYTES + (wl[i] ^ (16u * q))) = vl[q];
    } else {
      dequant_chunk<QT, XT>(S.b[i], d, v);
    }
#pragma unroll
    for (int q = 0; q < NV; ++q) *reinterpret_cast<uint4 *>(sB + (wl[i] ^ (16u * q))) = v[q];
  };

  // Fragment addresses: lane reads row (lane & 31) of a fragment, logical
  // chunk 2 ks + lane / 32, stored at (2 ks + lane / 32) ^ swz(row).  Adding
  // 32 to a row flips bit 2 of swz (adding 4 to the 3-bit row / 8 term), so
  // fragment i of k-step ks sits at
  //   (a0 ^ 32 (ks ^ 2 (i & 1))) + 4096 i,
  // a0 = this lane's address in fragment 0 of k-step 0: four lane addresses
  // per operand serve every fragment of every k-step, the rest is an
  // immediate offset.
  uint32_t aq[4], bq[4];
  {
    const uint32_t ra = wm * TM + (lane & 31), rb = wn * TN + (lane & 31);
    const uint32_t a0 = ra * (kBK * 2) + ((((uint32_t)lane >> 5) ^ swz(ra)) << 4);
    const uint32_t b0 = rb * (kBK * 2) + ((((uint32_t)lane >> 5) ^ swz(rb)) << 4);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      aq[q] = a0 ^ (32u * q);
      bq[q] = b0 ^ (32u * q);
    }
  }

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto read_frags = [&](const uint8_t *sA, const uint8_t *sB, int ks, uint4 (&af)[FM],
                        uint4 (&bfr)[FN], uint4 (&bfl)[HL ? FN : 1]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
      af[i] = *reinterpret_cast<const uint4 *>(sA + aq[ks ^ (2 * (i & 1))] + 4096 * i);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      bfr[j] = *reinterpret_cast<const uint4 *>(sB + bq[ks ^ (2 * (j & 1))] + 4096 * j);
    if constexpr (HL) {
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfl[j] = *reinterpret_cast<const uint4 *>(sB + BBYTES + bq[ks ^ (2 * (j & 1))] + 4096 * j);
    }
  };

  // MFMAs of the tile in (sA, sB); the dequantizing stores of the next tile
  // (raw set `nxt`, already in registers) into sBn are spread over the k-steps
  // so the VALU work overlaps the matrix cores.  The fragments of k-step ks + 1
  // are read while the MFMAs of k-step ks run (two register sets), and the
  // scheduling groups at the end keep that order: each LDS read then has a
  // whole k-step of MFMA work to land instead of stalling the chain.
  auto compute = [&](const uint8_t *sA, const uint8_t *sB, const Raw &nxt, uint8_t *sBn,
                     bool more) __attribute__((always_inline)) {
    uint4 af[2][FM], bfr[2][FN], bfl[2][HL ? FN : 1];
    read_frags(sA, sB, 0, af[0], bfr[0], bfl[0]);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS)
        read_frags(sA, sB, ks + 1, af[(ks + 1) & 1], bfr[(ks + 1) & 1], bfl[(ks + 1) & 1]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[ks & 1][i], bfr[ks & 1][j], acc[i][j]);
      if constexpr (HL) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = mfma32<XT>(af[ks & 1][i], bfl[ks & 1][HL ? j : 0], acc[i][j]);
      }
      if (more) {
        constexpr int per = (BCH + KSTEPS - 1) / KSTEPS;
#pragma unroll
        for (int i = ks * per; i < ks * per + per && i < BCH; ++i) store_w(nxt, sBn, i);
      }
    }
    // reads of k-step 0, the step's weight loads, then per k-step the reads
    // of the next k-step ahead of this k-step's MFMAs.  For Q4_0 the
    // dequantizing VALU work (about 80 instructions per 32-weight chunk) is
    // spread evenly between the MFMAs instead of in bursts (measured: 2.5%
    // faster on the video projections; for Q8_0 the same spreading was 1-4%
    // slower, so its VALU work is left to the compiler).
    constexpr int kVpm = (BCH * (HL ? 160 : (Q6 ? 100 : 80)) + KSTEPS * NMF - 1) / (KSTEPS * NMF);
    __builtin_amdgcn_sched_group_barrier(0x100, NRD, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, NW, 0);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) __builtin_amdgcn_sched_group_barrier(0x100, NRD, 0);
#pragma unroll
      for (int j = 0; j < NMF; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (QT != EB_Q8_0) __builtin_amdgcn_sched_group_barrier(0x002, kVpm, 0);
      }
    }
  };

  // Rows of the x buffers that no copy fills (past m) keep these zeros.
  {
    constexpr int Z = NA * ABYTES / 16 / T;
    static_assert(Z * T * 16 == NA * ABYTES, "zero fill must cover the x buffers");
#pragma unroll
    for (int i = 0; i < Z; ++i) {
      const int o = (tid + i * T) * 16;
      uint8_t *dst = o < ABYTES ? sA0 + o : (NA == 2 || o < 2 * ABYTES ? sA1 + (o - ABYTES) : sA2 + (o - 2 * ABYTES));
      *reinterpret_cast<uint4 *>(dst) = make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();

  // Pipeline: entering the step of tile t, x tile t is in LDS, x tile t+1 is
  // being copied (NA = 3), the weights of tile t+1 are in registers (or
  // arriving) and those of tile t+2 are in flight.  The step issues x tile
  // t + NA - 1 and weight tile t+3, runs the MFMAs of tile t while
  // dequantizing weight tile t+1 into the other weight buffer, then waits only
  // for x tile t+1 before the barrier: weight loads have about two steps to
  // land, x copies NA - 1.
  load_x(sA0, 0);
  load_w(S0, 0);
  if (NA == 3 && nk > 1) load_x(sA1, 1);
  if (nk > 1) load_w(S1, 1);
  if (nk > 2) load_w(S2, 2);
#pragma unroll
  for (int i = 0; i < BCH; ++i) store_w(S0, sB0, i);
  __syncthreads();

  // In the main loop every load is in range, so the steps issue them
  // unconditionally and the compiler's own wait counts stay exact across the
  // loop; the last (up to 8) tiles run through guarded copies of the steps.
  auto step = [&](int t, const uint8_t *A, uint8_t *A2, const uint8_t *B, uint8_t *Bn,
                  const Raw &deq, Raw &ld, bool guarded) __attribute__((always_inline)) {
    if (guarded && t >= nk) return;
    if (!guarded || t + NA - 1 < nk) load_x(A2, t + NA - 1);
    // the x copies stay ahead of the weight loads: the wait below counts on
    // the copy of tile t + 1 being older than the last 2 NW + NX operations
    // (NA = 3: weights t + 2, x t + 2, weights t + 3), or NW (NA = 2: weights
    // t + 3)
    __builtin_amdgcn_sched_barrier(0);
    if (!guarded || t + 3 < nk) load_w(ld, t + 3);
    compute(A, B, deq, Bn, !guarded || t + 1 < nk);
    if (!guarded || t + 3 < nk)
      wait_vm_barrier<NA == 3 ? 2 * NW + NX : NW>();
    else
      wait_vm_barrier<0>();
  };
  int kt = 0;
  if constexpr (NA == 3) {
    for (; kt + 8 < nk; kt += 6) {
      step(kt + 0, sA0, sA2, sB0, sB1, S1, S0, false);
      step(kt + 1, sA1, sA0, sB1, sB0, S2, S1, false);
      step(kt + 2, sA2, sA1, sB0, sB1, S0, S2, false);
      step(kt + 3, sA0, sA2, sB1, sB0, S1, S0, false);
      step(kt + 4, sA1, sA0, sB0, sB1, S2, S1, false);
      step(kt + 5, sA2, sA1, sB1, sB0, S0, S2, false);
    }
    for (; kt < nk; kt += 6) {
      step(kt + 0, sA0, sA2, sB0, sB1, S1, S0, true);
      step(kt + 1, sA1, sA0, sB1, sB0, S2, S1, true);
      step(kt + 2, sA2, sA1, sB0, sB1, S0, S2, true);
      step(kt + 3, sA0, sA2, sB1, sB0, S1, S0, true);
      step(kt + 4, sA1, sA0, sB0, sB1, S2, S1, true);
      step(kt + 5, sA2, sA1, sB1, sB0, S0, S2, true);
    }
  } else {
    for (; kt + 8 < nk; kt += 6) {
      step(kt + 0, sA0, sA1, sB0, sB1, S1, S0, false);
      step(kt + 1, sA1, sA0, sB1, sB0, S2, S1, false);
      step(kt + 2, sA0, sA1, sB0, sB1, S0, S2, false);
      step(kt + 3, sA1, sA0, sB1, sB0, S1, S0, false);
      step(kt + 4, sA0, sA1, sB0, sB1, S2, S1, false);
      step(kt + 5, sA1, sA0, sB1, sB0, S0, S2, false);
    }
    for (; kt < nk; kt += 6) {
      step(kt + 0, sA0, sA1, sB0, sB1, S1, S0, true);
      step(kt + 1, sA1, sA0, sB1, sB0, S2, S1, true);
      step(kt + 2, sA0, sA1, sB0, sB1, S0, S2, true);
      step(kt + 3, sA1, sA0, sB1, sB0, S1, S0, true);
      step(kt + 4, sA0, sA1, sB0, sB1, S2, S1, true);
      step(kt + 5, sA1, sA0, sB1, sB0, S0, S2, true);
    }
  }

  // epilogue: lane holds column (lane & 31), rows 8*(r/4) + 4*(lane/32) + r%4;
  // the gate/up pair of columns 2c, 2c + 1 sits in lanes l, l ^ 1 (n is even,
  // so both or neither are inside the tile)
  if (!ws && f.epi == EB_EPI_GLU) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int cl = wn * TN + j * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float g = acc[i][j][r];
          const float u = __builtin_bit_cast(
              float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, g), 0xB1, 0xF, 0xF, true));
          const int rl = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (cl >= rows_n || rl >= rows_m || (cl & 1)) continue;
          store_y(y, (m0 + rl) * (n / 2) + (n0 + cl) / 2, silu_mul(g, u), yt);
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int cl = wn * TN + j * 32 + (lane & 31);
      // the fragment's 16 residuals read together (where the registers allow:
      // not with 256 accumulators per lane)
      if (FM * FN <= 8 && !ws && f.epi == EB_EPI_ADD) {
        uint32_t rel[16];
        bool ok[16];
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          rel[r] = (uint32_t)rl * (uint32_t)n + (uint32_t)cl;
          ok[r] = cl < rows_n && rl < rows_m;
          v[r] = acc[i][j][r];
        }
        // elements m0 n + n0 + rel, within the tile's rows_m rows of n
        if (put_y_add(y, f.r, m0 * n + n0, (int64_t)rows_m * n, rel, ok, v, yt)) continue;
      }
      if (cl >= rows_n) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wm * TM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (rl >= rows_m) continue;
        const int64_t o = (m0 + rl) * n + n0 + cl;
        if (ws)
          ws[split * ws_stride + o] = acc[i][j][r];
        else
          put_y(y, o, acc[i][j][r], yt, f);
      }
    }
}

template <int QT, int XT, int BM, int BN, int WM, int WN, bool HL = false>
hipError_t launch_t(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, int splits, int kts, float *ws, int64_t ws_stride,
                    hipStream_t s) {
  const Layout L = layout_of(QT, n, k);
  const int64_t tiles = ((m + BM - 1) / BM) * ((n + BN - 1) / BN);
  if (tiles * splits > 0x7fffffff) return hipErrorInvalidValue;
  if (!mfma_fits_offsets(QT, n, k, BM, BN)) return hipErrorInvalidValue;
  mfma_kernel<QT, XT, BM, BN, WM, WN, false, HL><<<(unsigned)(tiles * splits), WM * WN * 64, 0, s>>>(
      (const uint8_t *)wdata, n, k, L.d_off, L.ds, L.sc_off, (const uint16_t *)x, m, y, yt, f, kts,
      splits > 1 ? ws : nullptr, ws_stride, nullptr, nullptr);
  return hipGetLastError();
}

template <int QT, int XT, int BM, int BN, int WM, int WN>
hipError_t launch_g(const GOp *ops, const int2 *order, int64_t entries, hipStream_t s) {
  if (entries <= 0 || entries > 0x7fffffff) return hipErrorInvalidValue;
  mfma_kernel<QT, XT, BM, BN, WM, WN, true><<<(unsigned)entries, WM * WN * 64, 0, s>>>(
      nullptr, 0, 0, 0, 0, 0, nullptr, 0, nullptr, 0, Fuse{}, 0, nullptr, 0, ops, order);
  return hipGetLastError();
}

}  // namespace

template <int QT, int XT>
hipError_t mfma_tile_launch(int cfg, bool hl, const void *wdata, int64_t n, int64_t k, const void *x,
                            int64_t m, void *y, int32_t yt, const Fuse &f, int sp, int kts,
                            float *ws, int64_t st, hipStream_t s) {
  if constexpr (XT == EB_BF16 && QT != EB_Q6_S) {
    if (hl) {  // the configurations with hi/lo weight tiles
      if (cfg == 0) return launch_t<QT, XT, 64, 128, 2, 2, true>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
      if (cfg == 1) return launch_t<QT, XT, 128, 128, 2, 2, true>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
      return hipErrorInvalidValue;
    }
  }
  if (hl) return hipErrorInvalidValue;
  switch (cfg) {
    case 0: return launch_t<QT, XT, 64, 128, 2, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 1: return launch_t<QT, XT, 128, 128, 2, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 2: return launch_t<QT, XT, 128, 256, 2, 4>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 3: return launch_t<QT, XT, 256, 128, 4, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 4: return launch_t<QT, XT, 256, 192, 4, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 5: return launch_t<QT, XT, 256, 256, 4, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 6: return launch_t<QT, XT, 256, 256, 2, 4>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 7: return launch_t<QT, XT, 256, 256, 2, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    case 8: return launch_t<QT, XT, 512, 128, 4, 2>(wdata, n, k, x, m, y, yt, f, sp, kts, ws, st, s);
    default: return hipErrorInvalidValue;
  }
}

template <int QT, int XT>
hipError_t mfma_tile_launch_grouped(int cfg, const GOp *ops, const int2 *order, int64_t entries,
                                    hipStream_t s) {
  switch (cfg) {
    case 1: return launch_g<QT, XT, 128, 128, 2, 2>(ops, order, entries, s);
    case 2: return launch_g<QT, XT, 128, 256, 2, 4>(ops, order, entries, s);
    case 4: return launch_g<QT, XT, 256, 192, 4, 2>(ops, order, entries, s);
    case 6: return launch_g<QT, XT, 256, 256, 2, 4>(ops, order, entries, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace eb

#endif  // EB_MFMA_TILE_H
