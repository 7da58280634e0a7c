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

}  // namespace
}  // namespace eb

#endif  // EB_EPILOGUE_H
