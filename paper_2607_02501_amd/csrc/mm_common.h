// mm_common.h -- device helpers shared by the fused small-m kernels: the
// cursor over a workgroup's stream of units and K steps, and the dequantizer
// that turns one block of a lane's weights into MFMA operand registers.
#ifndef EB_MM_COMMON_H
#define EB_MM_COMMON_H

#include <hip/hip_runtime.h>

#include <algorithm>

#include "eb_internal.h"
#include "mfma_common.h"

namespace eb {
namespace {

// Position in a workgroup's stream of units: the unit, its op and K-tile.
struct MMPos {
  int op;
  int64_t u;
  int kt, nk;
  int64_t op_end;
  bool valid;
};

// Moves to the first step of unit p.u (p.op must not be past its op).
__host__ __device__ inline void mm_seek(const MMOp *__restrict__ ops, MMPos &p, int64_t u_end) {
  p.kt = 0;
  if (p.u >= u_end) {
    p.valid = false;
    return;
  }
  while (p.u >= ops[p.op].unit_end) ++p.op;
  p.nk = ops[p.op].nk;
  p.op_end = ops[p.op].unit_end;
}

// Advances one step; returns true when a new unit starts (p.valid tells
// whether there is one).
__host__ __device__ inline bool mm_step(const MMOp *__restrict__ ops, MMPos &p, int64_t u_end) {
  if (!p.valid) return false;
  if (++p.kt < p.nk) return false;
  ++p.u;
  mm_seek(ops, p, u_end);
  return true;
}

// Tile (m0, n0) and valid extent of unit p.u of op p.op.
template <int BM, int BN>
__host__ __device__ inline void mm_tile(const MMOp *__restrict__ ops, const MMPos &p, int64_t &m0,
                               int64_t &n0, int &rows_m, int &rows_n) {
  const MMOp &o = ops[p.op];
  const int64_t first = p.op ? ops[p.op - 1].unit_end : 0;
  const uint32_t uin = (uint32_t)(p.u - first), tiles_n = (uint32_t)o.tiles_n;
  const uint32_t tm = uin / tiles_n, tn = uin - tm * tiles_n;
  m0 = (int64_t)tm * BM;
  n0 = (int64_t)tn * BN;
  rows_m = (int)std::min((int64_t)BM, (int64_t)o.m - m0);
  rows_n = (int)std::min((int64_t)BN, (int64_t)o.n - n0);
}

// Dequantizes block h of a lane's weight row (Q8_0: 32 codes in two 16-byte
// chunks; Q4_0: 16 bytes holding k and k + 16 in the low and high nibbles)
// with scale d into four MFMA operand registers: b[s] holds the weights
// k = 8 s .. 8 s + 7 of the block (section 2.2: w = d * code, rounded once).
template <int QT, int XT>
__device__ inline void dequant_b(const uint4 (&q)[QT == EB_Q8_0 ? 2 : 1], float d, uint4 (&b)[4]) {
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  if constexpr (QT == EB_Q8_0) {
    const float c = -1152.0f * d;
    const uint32_t w[8] = {q[0].x, q[0].y, q[0].z, q[0].w, q[1].x, q[1].y, q[1].z, q[1].w};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t u0 = w[2 * s] ^ 0x80808080u, u1 = w[2 * s + 1] ^ 0x80808080u;
      b[s] = make_uint4(deq_pair<XT>(under_1024(u0, kSelLo), d, c),
                        deq_pair<XT>(under_1024(u0, kSelHi), d, c),
                        deq_pair<XT>(under_1024(u1, kSelLo), d, c),
                        deq_pair<XT>(under_1024(u1, kSelHi), d, c));
    }
  } else {
    const float c = -1032.0f * d;
    const uint32_t w[4] = {q[0].x, q[0].y, q[0].z, q[0].w};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      // s = 0, 1: low nibbles of bytes 0..7, 8..15; s = 2, 3: high nibbles
      const uint32_t sh = s < 2 ? 0 : 4;
      const uint32_t l0 = (w[2 * (s & 1)] >> sh) & 0x0f0f0f0fu;
      const uint32_t l1 = (w[2 * (s & 1) + 1] >> sh) & 0x0f0f0f0fu;
      b[s] = make_uint4(deq_pair<XT>(under_1024(l0, kSelLo), d, c),
                        deq_pair<XT>(under_1024(l0, kSelHi), d, c),
                        deq_pair<XT>(under_1024(l1, kSelLo), d, c),
                        deq_pair<XT>(under_1024(l1, kSelHi), d, c));
    }
  }
}

// dequant_b for bfloat16 activations as hi/lo pairs (split2_bf16 in
// mfma_common.h): bh[s] the bfloat16 roundings, bl[s] those of the remainders.
template <int QT>
__device__ inline void dequant_b_hl(const uint4 (&q)[QT == EB_Q8_0 ? 2 : 1], float d, uint4 (&bh)[4],
                                    uint4 (&bl)[4]) {
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  uint32_t h[16], l[16];
  if constexpr (QT == EB_Q8_0) {
    const float c = -1152.0f * d;
    const uint32_t w[8] = {q[0].x, q[0].y, q[0].z, q[0].w, q[1].x, q[1].y, q[1].z, q[1].w};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t u0 = w[2 * s] ^ 0x80808080u, u1 = w[2 * s + 1] ^ 0x80808080u;
      deq_pair_hl(under_1024(u0, kSelLo), d, c, h[4 * s], l[4 * s]);
      deq_pair_hl(under_1024(u0, kSelHi), d, c, h[4 * s + 1], l[4 * s + 1]);
      deq_pair_hl(under_1024(u1, kSelLo), d, c, h[4 * s + 2], l[4 * s + 2]);
      deq_pair_hl(under_1024(u1, kSelHi), d, c, h[4 * s + 3], l[4 * s + 3]);
    }
  } else {
    const float c = -1032.0f * d;
    const uint32_t w[4] = {q[0].x, q[0].y, q[0].z, q[0].w};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t sh = s < 2 ? 0 : 4;
      const uint32_t l0 = (w[2 * (s & 1)] >> sh) & 0x0f0f0f0fu;
      const uint32_t l1 = (w[2 * (s & 1) + 1] >> sh) & 0x0f0f0f0fu;
      deq_pair_hl(under_1024(l0, kSelLo), d, c, h[4 * s], l[4 * s]);
      deq_pair_hl(under_1024(l0, kSelHi), d, c, h[4 * s + 1], l[4 * s + 1]);
      deq_pair_hl(under_1024(l1, kSelLo), d, c, h[4 * s + 2], l[4 * s + 2]);
      deq_pair_hl(under_1024(l1, kSelHi), d, c, h[4 * s + 3], l[4 * s + 3]);
    }
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    bh[s] = make_uint4(h[4 * s], h[4 * s + 1], h[4 * s + 2], h[4 * s + 3]);
    bl[s] = make_uint4(l[4 * s], l[4 * s + 1], l[4 * s + 2], l[4 * s + 3]);
  }
}

}  // namespace
}  // namespace eb

#endif  // EB_MM_COMMON_H
