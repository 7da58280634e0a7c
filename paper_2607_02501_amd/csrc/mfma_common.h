// mfma_common.h -- device helpers shared by the single-op and fused MFMA
// kernels: 16-bit packing, the 32x32x16 MFMA, dequantization of code chunks,
// raw buffer descriptors, the x-tile swizzle and the partial-drain barrier.
#ifndef EB_MFMA_COMMON_H
#define EB_MFMA_COMMON_H

#include <hip/hip_runtime.h>

#include "eb_internal.h"

namespace eb {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kBK = 64;        // K elements per tile (2 blocks)
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
  // weight chunks per row per K-tile: Q8_0 four 16-byte half-blocks, Q4_0 two
  // 16-byte blocks, Q6_S two 24-byte code chunks (one 48-byte unit of 64 weights)
  static constexpr int kChunksPerRow = (QT == EB_Q8_0) ? 4 : 2;
  static constexpr int kElemsPerChunk = (QT == EB_Q8_0) ? 16 : 32;
};

// Dequantize one 16-byte chunk of codes into 16-byte vectors of 16-bit
// weights, in k order: Q8_0 16 codes -> 2 vectors, Q4_0 one block -> 4.
// Each code c in 0..255 (Q8_0: q + 128) or 0..15 (Q4_0 nibble) is placed
// under the binary16 exponent of 1024 by one byte permute per two codes,
// giving the binary16 value 1024 + c exactly; then
//   fma(1024 + c, d, -(1024 + z) d) = (c - z) d,   z = 128 (Q8_0) or 8 (Q4_0),
// is exact (1152 d and 1032 d need at most 19 significant bits), and the one
// rounding to the 16-bit activation type is round-to-nearest-even.
template <int QT>
struct Deq {
  static constexpr int kVecs = (QT == EB_Q8_0) ? 2 : 4;
};


// two codes in bytes b0, b1 of v -> 16-bit halves 0x64bb of the result
__device__ inline uint32_t under_1024(uint32_t v, uint32_t sel) {
  return __builtin_amdgcn_perm(0x64646464u, v, sel);
}

template <int XT>
__device__ inline uint32_t deq_pair(uint32_t h2, float d, float c) {
  const _Float16 a = __builtin_bit_cast(_Float16, (uint16_t)(h2 & 0xffffu));
  const _Float16 b = __builtin_bit_cast(_Float16, (uint16_t)(h2 >> 16));
  return pack2<XT>(__builtin_fmaf((float)a, d, c), __builtin_fmaf((float)b, d, c));
}

// bfloat16 activations: w_hat = (c - z) d is exact in fp32 but needs up to 19
// significant bits, while bfloat16 keeps 8 (one rounding costs up to 2^-8 of
// |w_hat|, which a one-hot x exposes whole).  A hi/lo pair keeps 16:
// hi = bf16_RNE(w), lo = bf16_RNE(w - hi) (w - hi is exact in fp32), so
// |w - hi - lo| <= 2^-16 |w| and x hi + x lo, each product exact in fp32 and
// accumulated by the matrix cores, carries w_hat to within 2^-16.
__device__ inline void split2_bf16(float a, float b, uint32_t &hi, uint32_t &lo) {
  hi = pack2<EB_BF16>(a, b);
  const float ha = __uint_as_float(hi << 16), hb = __uint_as_float(hi & 0xffff0000u);
  lo = pack2<EB_BF16>(a - ha, b - hb);
}

// two codes (binary16 1024 + c halves of h2) -> hi and lo bfloat16 pairs of (c - z) d
__device__ inline void deq_pair_hl(uint32_t h2, float d, float c, uint32_t &hi, uint32_t &lo) {
  const _Float16 a = __builtin_bit_cast(_Float16, (uint16_t)(h2 & 0xffffu));
  const _Float16 b = __builtin_bit_cast(_Float16, (uint16_t)(h2 >> 16));
  split2_bf16(__builtin_fmaf((float)a, d, c), __builtin_fmaf((float)b, d, c), hi, lo);
}

template <int QT, int XT>
__device__ inline void dequant_chunk(const uint4 q, float d, uint4 (&v)[Deq<QT>::kVecs]) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  // byte selectors: {S1.b0, 0x64, S1.b1, 0x64} and {S1.b2, 0x64, S1.b3, 0x64}
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  if constexpr (QT == EB_Q8_0) {
    const float c = -1152.0f * d;
    uint32_t o[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t u = w[j] ^ 0x80808080u;
      o[2 * j] = deq_pair<XT>(under_1024(u, kSelLo), d, c);
      o[2 * j + 1] = deq_pair<XT>(under_1024(u, kSelHi), d, c);
    }
    v[0] = make_uint4(o[0], o[1], o[2], o[3]);
    v[1] = make_uint4(o[4], o[5], o[6], o[7]);
  } else {
    const float c = -1032.0f * d;
    uint32_t lo[8], hi[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t l = w[j] & 0x0f0f0f0fu, h = (w[j] >> 4) & 0x0f0f0f0fu;
      lo[2 * j] = deq_pair<XT>(under_1024(l, kSelLo), d, c);
      lo[2 * j + 1] = deq_pair<XT>(under_1024(l, kSelHi), d, c);
      hi[2 * j] = deq_pair<XT>(under_1024(h, kSelLo), d, c);
      hi[2 * j + 1] = deq_pair<XT>(under_1024(h, kSelHi), d, c);
    }
    v[0] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    v[1] = make_uint4(lo[4], lo[5], lo[6], lo[7]);
    v[2] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    v[3] = make_uint4(hi[4], hi[5], hi[6], hi[7]);
  }
}

// Q6_S: one 24-byte chunk of 32 weights -> 4 vectors, in k order.  The
// chunk's 16 low-nibble bytes L (byte t: weight t in bits 0..3, weight t + 16
// in bits 4..7) and 8 top-bit bytes H (byte t: the top bits of weights t,
// t + 8, t + 16, t + 24 at bits 0, 2, 4, 6) are merged into bytes u = 0..63,
// four per word, placed under binary16 1024 by one byte permute per two
// codes, and
//   fma(1024 + u, e, -1056 e) = (u - 32) e,   e = d16 sc_j
// is exact (e has at most 18 significant bits, 1056 e and the result at most
// 24); one rounding to the 16-bit activation type.  Weights 0..15 of the
// chunk use sub-scale sc0, 16..31 sc1.
template <int XT>
__device__ inline void dequant_chunk_q6(const uint4 l16, const uint2 h8, uint32_t sc2, float d,
                                        uint4 (&v)[4]) {
  const uint32_t L[4] = {l16.x, l16.y, l16.z, l16.w};
  const uint32_t H[2] = {h8.x, h8.y};
  const float e0 = d * (float)(int8_t)(sc2 & 0xffu), e1 = d * (float)(int8_t)((sc2 >> 8) & 0xffu);
  const float c0 = -1056.0f * e0, c1 = -1056.0f * e1;
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  uint32_t lo[8], hi[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    // word j: weights 4j .. 4j + 3 (low nibbles) and 4j + 16 .. (high), their
    // top bits in top-bit word j & 1 at shift 2 (j >> 1) and 2 (j >> 1) + 4
    const uint32_t t = H[j & 1] >> (2 * (j >> 1));
    const uint32_t ul = (L[j] & 0x0f0f0f0fu) | ((t & 0x03030303u) << 4);
    const uint32_t uh = ((L[j] >> 4) & 0x0f0f0f0fu) | ((t & 0x30303030u));
    lo[2 * j] = deq_pair<XT>(under_1024(ul, kSelLo), e0, c0);
    lo[2 * j + 1] = deq_pair<XT>(under_1024(ul, kSelHi), e0, c0);
    hi[2 * j] = deq_pair<XT>(under_1024(uh, kSelLo), e1, c1);
    hi[2 * j + 1] = deq_pair<XT>(under_1024(uh, kSelHi), e1, c1);
  }
  v[0] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
  v[1] = make_uint4(lo[4], lo[5], lo[6], lo[7]);
  v[2] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  v[3] = make_uint4(hi[4], hi[5], hi[6], hi[7]);
}

// dequant_chunk for bfloat16 activations, as hi/lo pairs (split2_bf16):
// vh holds the bfloat16 roundings, vl the roundings of the remainders.
template <int QT>
__device__ inline void dequant_chunk_hl(const uint4 q, float d, uint4 (&vh)[Deq<QT>::kVecs],
                                        uint4 (&vl)[Deq<QT>::kVecs]) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  constexpr uint32_t kSelLo = 0x04010400u, kSelHi = 0x04030402u;
  if constexpr (QT == EB_Q8_0) {
    const float c = -1152.0f * d;
    uint32_t h[8], l[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t u = w[j] ^ 0x80808080u;
      deq_pair_hl(under_1024(u, kSelLo), d, c, h[2 * j], l[2 * j]);
      deq_pair_hl(under_1024(u, kSelHi), d, c, h[2 * j + 1], l[2 * j + 1]);
    }
    vh[0] = make_uint4(h[0], h[1], h[2], h[3]);
    vh[1] = make_uint4(h[4], h[5], h[6], h[7]);
    vl[0] = make_uint4(l[0], l[1], l[2], l[3]);
    vl[1] = make_uint4(l[4], l[5], l[6], l[7]);
  } else {
    const float c = -1032.0f * d;
    uint32_t h[16], l[16];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo4 = w[j] & 0x0f0f0f0fu, hi4 = (w[j] >> 4) & 0x0f0f0f0fu;
      deq_pair_hl(under_1024(lo4, kSelLo), d, c, h[2 * j], l[2 * j]);
      deq_pair_hl(under_1024(lo4, kSelHi), d, c, h[2 * j + 1], l[2 * j + 1]);
      deq_pair_hl(under_1024(hi4, kSelLo), d, c, h[8 + 2 * j], l[8 + 2 * j]);
      deq_pair_hl(under_1024(hi4, kSelHi), d, c, h[8 + 2 * j + 1], l[8 + 2 * j + 1]);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      vh[v] = make_uint4(h[4 * v], h[4 * v + 1], h[4 * v + 2], h[4 * v + 3]);
      vl[v] = make_uint4(l[4 * v], l[4 * v + 1], l[4 * v + 2], l[4 * v + 3]);
    }
  }
}

// Raw buffer descriptor over [base, base + bytes): every lane whose offset is
// at or past `bytes` reads zeros, which is how the kernel handles rows past m
// or n without branches.  The descriptor is rebuilt per K-tile (scalar work),
// so the hardware range check always covers the whole access.
__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// The same for a base and size that are uniform across the wave but that the
// compiler cannot prove uniform (cursor state carried through loops): without
// the read-first-lane it keeps them in vector registers and wraps every load
// in a loop over distinct descriptor values.
__device__ inline __amdgpu_buffer_rsrc_t ursrc(const void *base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return rsrc(reinterpret_cast<const void *>(((uint64_t)hi << 32) | lo),
              __builtin_amdgcn_readfirstlane(bytes));
}

__device__ inline uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

typedef __attribute__((address_space(3))) void lds_void;

// Position of 16-byte chunk c of row r in the unpadded x tile (128-byte rows):
// c ^ swz(r).  Any 16 consecutive rows read at one chunk index hit 16 distinct
// 16-byte bank groups, and any 8 consecutive rows 8 distinct ones.
__device__ inline uint32_t swz(uint32_t r) { return (r ^ (r >> 3)) & 7; }

// Wait until at most N vector-memory operations of this wave are outstanding
// and its LDS writes are done, then barrier.  Unlike __syncthreads this does
// not drain every load, so loads issued for later K-tiles stay in flight.  The
// "memory" clobber keeps IR passes, and the scheduling barriers the machine
// scheduler, from moving memory accesses across it.
template <int N>
__device__ inline void wait_vm_barrier() {
  // sched_barrier(0): the machine scheduler moves nothing across this point
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
  __builtin_amdgcn_sched_barrier(0);
}

}  // namespace
}  // namespace eb

#endif  // EB_MFMA_COMMON_H
