// epilogue.h -- device helpers for the steps fused after a projection's
// product (paper section 3.2, operator fusion): the output conversion, the
// residual addition and the SiLU-gated product of a gate/up row pair.
//
// Gate/up convention: rows 2j and 2j + 1 of the weights are the gate and up
// rows of feature j; the output of feature j goes to column j of a row of
// n / 2 outputs.  Every kernel holds the two rows of a pair either in one
// lane or in two lanes it can exchange values between.
#ifndef EB_EPILOGUE_H
#define EB_EPILOGUE_H

#include <hip/hip_runtime.h>

#include "eb_internal.h"

namespace eb {
namespace {

// silu(g) * u with silu(t) = t / (1 + e^-t); saturates to g * u for large g
// and to -0 * u for very negative g (e^-g overflows to infinity).
__device__ inline float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

__device__ inline uint16_t to_y16(float v, int yt) {
  return yt == EB_F16 ? __builtin_bit_cast(uint16_t, (_Float16)v)
                      : __builtin_bit_cast(uint16_t, (__bf16)v);
}

__device__ inline float from_y16(uint16_t h, int yt) {
  return yt == EB_F16 ? (float)__builtin_bit_cast(_Float16, h)
                      : __builtin_bit_cast(float, (uint32_t)h << 16);
}

__device__ inline float load_y(const void *p, int64_t i, int yt) {
  return yt == EB_F32 ? reinterpret_cast<const float *>(p)[i]
                      : from_y16(reinterpret_cast<const uint16_t *>(p)[i], yt);
}

__device__ inline void store_y(void *p, int64_t i, float v, int yt) {
  if (yt == EB_F32)
    reinterpret_cast<float *>(p)[i] = v;
  else
    reinterpret_cast<uint16_t *>(p)[i] = to_y16(v, yt);
}

// Output element i of a plain or residual-adding op.
__device__ inline void put_y(void *y, int64_t i, float v, int yt, const Fuse &f) {
  if (f.epi == EB_EPI_ADD) v += load_y(f.r, i, yt);
  store_y(y, i, v, yt);
}

// N outputs of a residual-adding op: y[e] = v[t] + res[e] for the elements
// e = base + rel[t] where ok[t] (rel[t] < span), with put_y's arithmetic.
// All N residuals are read before any output is written.  Each output reads
// only its own element of the residual (which is y itself or does not
// overlap it), so this order is safe; element by element, as put_y does,
// each read waits behind the previous write for a full memory round trip.
// Buffer accesses with offsets past the range for the elements not kept (they
// read zero and store nothing) keep the code free of per-element branches,
// whose merged paths would make the compiler wait before every store.
// base and span must be the same in every lane of the wave (the buffer
// descriptors are scalar; a per-lane base would make the compiler loop over
// the lanes for every access).  Returns false (nothing done) when span
// elements of 4 bytes do not fit the 31-bit offsets; the caller then stores
// element by element.
template <int N>
__device__ inline bool put_y_add(void *y, const void *res, int64_t base, int64_t span,
                                 const uint32_t (&rel)[N], const bool (&ok)[N], const float (&v)[N],
                                 int yt) {
  auto uni = [](int64_t a) __attribute__((always_inline)) {
    const uint64_t u = (uint64_t)a;
    return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(u >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)u));
  };
  base = uni(base);
  span = uni(span);
  if (span > (int64_t)(0x7fffffff / 4)) return false;
  constexpr uint32_t kPast = 0x80000000u;
  const int ysz = yt == EB_F32 ? 4 : 2;
  const auto yr = __builtin_amdgcn_make_buffer_rsrc(static_cast<char *>(y) + base * ysz, (short)0,
                                                    (int)(span * ysz), 0x00020000);
  const auto rr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char *>(static_cast<const char *>(res)) + base * ysz, (short)0, (int)(span * ysz),
      0x00020000);
  uint32_t off[N];
#pragma unroll
  for (int t = 0; t < N; ++t) off[t] = ok[t] ? rel[t] * (uint32_t)ysz : kPast;
  if (yt == EB_F32) {
    float r[N];
#pragma unroll
    for (int t = 0; t < N; ++t)
      r[t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (int)off[t], 0, 0));
#pragma unroll
    for (int t = 0; t < N; ++t)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v[t] + r[t]), yr, (int)off[t], 0, 0);
  } else {
    uint16_t h[N];
#pragma unroll
    for (int t = 0; t < N; ++t) h[t] = __builtin_amdgcn_raw_buffer_load_b16(rr, (int)off[t], 0, 0);
#pragma unroll
    for (int t = 0; t < N; ++t)
      __builtin_amdgcn_raw_buffer_store_b16(to_y16(v[t] + from_y16(h[t], yt), yt), yr, (int)off[t], 0, 0);
  }
  return true;
}

}  // namespace
}  // namespace eb

#endif  // EB_EPILOGUE_H
