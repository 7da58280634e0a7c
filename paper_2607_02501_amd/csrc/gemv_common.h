// gemv_common.h -- helpers shared by the GEMV kernels (m <= 8): dot products of
// 16-bit pairs, the in-register decode of small integer codes through binary16 /
// bfloat16 magic numbers, cross-lane reductions of a wave's row sums, and raw
// buffer descriptors for the streamed weight loads.
#pragma once

#include <hip/hip_runtime.h>

#include "eb_internal.h"

namespace eb {
namespace {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf162_t __attribute__((ext_vector_type(2)));

__device__ inline float dot2h(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c,
                                false);
}
__device__ inline float dot2bf(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf162_t, a),
                                         __builtin_bit_cast(bf162_t, b), c, false);
}

// (a & mask) | magic should be one v_and_or_b32, but gfx9 VOP3 encodings take
// no literal and read at most one scalar operand, so with two constants the
// compiler splits it into v_and + v_or.  vconst() hands the compiler the magic
// constant as an opaque VGPR value (an identity DPP move), leaving the mask as
// the single scalar operand; this halves the decode cost of 4-bit codes.
__device__ inline uint32_t vconst(uint32_t c) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)c, 0xE4, 0xF, 0xF, false);  // quad_perm [0,1,2,3]
}
__device__ inline uint32_t and_or(uint32_t a, uint32_t mask, uint32_t magic) {
  return (a & mask) | magic;
}

// two binary16 values 1024 + v (or 1024 + 16 v) -> v - z exactly (one v_pk_add_f16)
__device__ inline uint32_t sub_h2(uint32_t h2, _Float16 z) {
  const half2_t r = __builtin_bit_cast(half2_t, h2) - half2_t{z, z};
  return __builtin_bit_cast(uint32_t, r);
}

template <int XT>
__device__ inline double x_to_f64(uint32_t h) {
  if (XT == EB_F16) return (double)__builtin_bit_cast(_Float16, (uint16_t)h);
  return (double)__builtin_bit_cast(float, h << 16);
}

template <int XT>
__device__ inline uint32_t pack_x16(float a, float b) {
  if (XT == EB_F16)
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) |
           ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)b) << 16);
}

template <int CTRL>
__device__ inline float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

__device__ inline float red8(float v) {  // sum over aligned groups of 8 lanes
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  return v;
}
__device__ inline float red16(float v) {  // sum over 16-lane rows
  v = red8(v);
  return v + dpp<0x140>(v);  // row_mirror
}
// lanes 0..31 get a[l] + a[l+32]; lanes 32..63 get b[l-32] + b[l]
__device__ inline float swap32(float a, float b) {
  auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, a),
                                            __builtin_bit_cast(unsigned, b), false, false);
  return __builtin_bit_cast(float, (unsigned)p[0]) + __builtin_bit_cast(float, (unsigned)p[1]);
}
// even 16-lane rows get a + a(partner row); odd rows get b + b(partner row)
__device__ inline float swap16(float a, float b) {
  auto p = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, a),
                                            __builtin_bit_cast(unsigned, b), false, false);
  return __builtin_bit_cast(float, (unsigned)p[0]) + __builtin_bit_cast(float, (unsigned)p[1]);
}
// lower 8 lanes of each row get a + a(l^8); upper 8 get b + b(l^8)
__device__ inline float half8(float a, float b, int lane) {
  const bool lo = (lane & 8) == 0;
  const float keep = lo ? a : b, send = lo ? b : a;
  return keep + dpp<0x128>(send);  // row_ror:8
}

// The row whose total reduce_rows<R> returns in `lane`.
template <int R>
__device__ inline int reduce_row(int lane) {
  if constexpr (R == 8) return ((lane >> 3) & 1) + 2 * ((lane >> 4) & 1) + 4 * (lane >> 5);
  if constexpr (R == 4) return ((lane >> 4) & 1) + 2 * (lane >> 5);
  if constexpr (R == 2) return lane >> 5;
  return 0;
}

// Reduce v[0..R) over the 64 lanes.  Returns the total of row `row` (a
// function of the lane, reduce_row<R>) in every lane; `writer` marks one lane
// per row.
template <int R>
__device__ inline float reduce_rows(const float (&v)[R], int lane, int &row, bool &writer) {
  if constexpr (R == 8) {
    float a0 = swap32(v[0], v[4]), a1 = swap32(v[1], v[5]), a2 = swap32(v[2], v[6]),
          a3 = swap32(v[3], v[7]);
    float b0 = swap16(a0, a2), b1 = swap16(a1, a3);
    float c = red8(half8(b0, b1, lane));
    row = reduce_row<R>(lane);
    writer = (lane & 7) == 0;
    return c;
  } else if constexpr (R == 4) {
    float a0 = swap32(v[0], v[2]), a1 = swap32(v[1], v[3]);
    float b = red16(swap16(a0, a1));
    row = reduce_row<R>(lane);
    writer = (lane & 15) == 0;
    return b;
  } else if constexpr (R == 2) {
    float a = red16(swap32(v[0], v[1]));
    a = swap16(a, a);
    row = reduce_row<R>(lane);
    writer = (lane & 31) == 0;
    return a;
  } else {
    // the association of R == 2 for its first row (lanes l and l + 32, then
    // 16-lane rows, then the two halves), so one- and two-row launches give
    // the same bits for a row
    float a = red16(swap32(v[0], v[0]));
    a = swap16(a, a);
    row = reduce_row<R>(lane);
    writer = lane == 0;
    return a;
  }
}

// Cache-policy bits of a buffer load: NT (non-temporal).  Weights are read
// exactly once per call, so they are streamed past the caches; on MI355X this
// raises the sustained HBM read rate by about 13% over ordinary loads.
constexpr int kNT = 2;

// Raw buffer descriptor over [base, base + bytes): the address of every load
// is then a scalar base plus a per-lane constant offset, with no per-lane
// 64-bit pointer arithmetic in the loop.  Word 3 (0x00020000) selects a raw
// 32-bit buffer with no format conversion.
__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}

}  // namespace
}  // namespace eb
