// mfma_multi.hip -- fused MFMA launch over many independent small-m ops of
// a stack (paper section 3.2: operator fusion and graph replay for batch-1
// execution; the action-chunk denoising steps of section 2.1 / Table 1 run
// hundreds of such layers per pass): the host side (tile configurations,
// the split of the ops' tiles over workgroups, dispatch) and the kernel for
// 64 < m <= 128.  The kernel for m <= 64 is in mfma_lds2.hip.  Built with the
// MFMA accumulators in VGPRs: this kernel's persistent loop otherwise moves
// them between register files on every trip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <vector>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"
#include "mm_common.h"

namespace eb {
namespace {

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
template <int QT, int XT, int YT, int BM, int FN, bool HL>
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
  // HL: bfloat16 activations with w_hat as hi/lo bfloat16 pairs (two MFMAs
  // per product, w_hat carried to 2^-16); without it w_hat is rounded once to
  // the activation type
  static_assert(!HL || XT == EB_BF16, "hi/lo pairs are for bfloat16 activations");

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

  // Fused steps: EB_EPI_ADD reads the residual at the store's offset; with
  // EB_EPI_GLU the gate/up columns 2c, 2c + 1 sit in lanes l, l ^ 1 and the
  // even lane stores silu(gate) * up into column c of n / 2.  YT only fixes
  // the output size (16-bit outputs are bf16 or fp16 by the op's type).
  auto epilogue = [&](const MMPos &c) __attribute__((always_inline)) {
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
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int cl = wave * 32 * FN + j * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint32_t row0 = (uint32_t)m0 + i * 32 + 4 * (lane >> 5);
        const uint32_t col = glu ? ((uint32_t)n0 + cl) / 2 : (uint32_t)n0 + cl;
        const bool keep = cl < rn && (!glu || (cl & 1) == 0);
        const uint32_t base = keep ? (row0 * nout + col) * YSZ : 0x80000000u;
        // the 16 residuals read before any output is written (an output
        // reads only its own residual; element by element, each read would
        // wait behind the previous write)
        float res[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) res[r] = 0.f;
        if (add) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const uint32_t off = base + (uint32_t)(8 * (r >> 2) + (r & 3)) * nout * YSZ;
            if constexpr (YT == EB_F32)
              res[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (int)off, 0, 0));
            else
              res[r] = from_y16(__builtin_amdgcn_raw_buffer_load_b16(rr, (int)off, 0, 0), yt);
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t off = base + (uint32_t)(8 * (r >> 2) + (r & 3)) * nout * YSZ;
          float v = acc[i][j][r];  // copy first: see mfma_multi_kernel
          if (glu) {
            const float u = __builtin_bit_cast(
                float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
            v = silu_mul(v, u);
          } else if (add) {
            v += res[r];
          }
          if constexpr (YT == EB_F32)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), yr, (int)off, 0, 0);
          else
            __builtin_amdgcn_raw_buffer_store_b16(to_y16(v, yt), yr, (int)off, 0, 0);
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
    uint4 bl[FN][HL ? 4 : 1];  // bfloat16: the low parts of the hi/lo pairs
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const float d = (float)__builtin_bit_cast(_Float16, S.d[j]);
      if constexpr (HL)
        dequant_b_hl<QT>(S.q[j], d, bq[j], bl[j]);
      else
        dequant_b<QT, XT>(S.q[j], d, bq[j]);
    }
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
      if constexpr (HL) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) acc[i][j] = mfma32<XT>(af[i], bl[j][HL ? s : 0], acc[i][j]);
      }
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

template <int QT, int XT, int YT>
hipError_t launch_multi_q(int cfg, bool hl, const MMOp *ops, int nops, const int64_t *wg, int groups,
                          hipStream_t s) {
  if (cfg == 0) return launch_lds2(QT, XT, hl, YT, ops, nops, wg, groups, s);
  if constexpr (XT == EB_BF16) {
    if (hl) {
      mm_breg_kernel<QT, XT, YT, 128, 1, true><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
      return hipGetLastError();
    }
  }
  mm_breg_kernel<QT, XT, YT, 128, 1, false><<<groups, 256, 0, s>>>(ops, nops, wg, groups);
  return hipGetLastError();
}

template <int QT, int XT>
hipError_t launch_multi_y(int32_t yt, int cfg, bool hl, const MMOp *ops, int nops, const int64_t *wg,
                          int groups, hipStream_t s) {
  if (yt == EB_F32) return launch_multi_q<QT, XT, EB_F32>(cfg, hl, ops, nops, wg, groups, s);
  return launch_multi_q<QT, XT, EB_BF16>(cfg, hl, ops, nops, wg, groups, s);
}

// {BM, BN, workgroups per CU, k per step}: 0 the 128-wide-step kernel with
// raw codes through LDS (mfma_lds2.hip, m <= 64), 1 weights loaded straight
// into registers (mm_breg_kernel, any m; used for 64 < m <= 128)
constexpr int kMMTiles[2][4] = {{64, 256, 1, 128}, {128, 128, 2, 64}};
constexpr int kMMCfgs = 2;

}  // namespace

int mm_cfg(int64_t max_m) {
  static const int forced = [] {
    const char *e = getenv("EB_MM_CFG");  // tuning: force the fused tile
    return e ? atoi(e) : -1;
  }();
  if (forced >= 0 && forced < kMMCfgs && (max_m <= 64 || forced == 1)) return forced;
  return max_m <= 64 ? 0 : 1;
}

int mm_bk(int cfg) { return kMMTiles[cfg][3]; }

int64_t mm_tiles(int cfg, int64_t m, int64_t n) {
  const int bm = kMMTiles[cfg][0], bn = kMMTiles[cfg][1];
  return ((m + bm - 1) / bm) * ((n + bn - 1) / bn);
}

int mm_partition(const std::vector<MMOp> &ops, int cfg, std::vector<int64_t> &wg,
                 int max_groups) {
  int64_t steps = 0, units = 0;
  for (const MMOp &o : ops) {
    steps += (o.unit_end - units) * o.nk;
    units = o.unit_end;
  }
  // as many workgroups as fit on the CUs at once, a multiple of 8
  int64_t groups = std::min<int64_t>((int64_t)device_cu_count() * kMMTiles[cfg][2], units);
  if (max_groups > 0) groups = std::min<int64_t>(groups, max_groups);
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

hipError_t launch_mfma_multi(int32_t type, int32_t xt, bool hl, int32_t yt, int cfg,
                             const MMOp *dev_ops, int nops, const int64_t *dev_wg, int groups,
                             hipStream_t s) {
  if (nops < 1 || groups < kXcds || groups % kXcds != 0) return hipErrorInvalidValue;
  hl = hl && xt == EB_BF16;
  if (type == EB_Q4_0) {
    if (xt == EB_F16)
      return launch_multi_y<EB_Q4_0, EB_F16>(yt, cfg, false, dev_ops, nops, dev_wg, groups, s);
    return launch_multi_y<EB_Q4_0, EB_BF16>(yt, cfg, hl, dev_ops, nops, dev_wg, groups, s);
  }
  if (xt == EB_F16)
    return launch_multi_y<EB_Q8_0, EB_F16>(yt, cfg, false, dev_ops, nops, dev_wg, groups, s);
  return launch_multi_y<EB_Q8_0, EB_BF16>(yt, cfg, hl, dev_ops, nops, dev_wg, groups, s);
}
}  // namespace eb
