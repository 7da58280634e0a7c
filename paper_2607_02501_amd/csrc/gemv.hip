// gemv.hip -- bandwidth-bound path of the quantized linear layer for m <= 8
// activation rows (batch-1 decode: paper section 3.1, "latency-first
// closed-loop control" runs effectively at batch 1; section 3.2 asks for
// fused, backend-specific kernels for it).
//
// y[m][n] = sum_b d16[n][b] * sum_{j in block b} x[m][32b + j] * code[n][32b + j]
//
// Work decomposition (wave64):
//   * a wave owns 4 weight rows at a time; 16 lanes per row, lane c of a row
//     walks the row's 16-byte "units" u = c, c + 16, ... (a unit is one Q4_0
//     block = 32 weights, or half a Q8_0 block = 16 weights), so each load
//     instruction reads 4 contiguous 256-byte runs of packed codes;
//   * RS such 4-row sets are in flight per wave;
//   * the activations x[m][k] are staged once per workgroup into LDS, already
//     permuted into the pair order the code decoder produces, together with a
//     per-unit offset (see below);
//   * the 16 partial sums of a row are added with four DPP steps.
//
// In-register dequantization.  A 4-bit code n (stored value c + 8) OR-ed into
// the mantissa of binary16 1024.0 reads as 1024 + n; OR-ed one nibble higher
// it reads 1024 + 16 n.  For int8 codes q, (q ^ 0x80) = q + 128 is placed the
// same way.  With binary16 activations one packed binary16 add per pair then
// subtracts 1032, 1152 (or 1152) exactly, leaving the signed codes c (16 c), and
// v_dot2_f32_f16 multiplies exact pairs: the fp32 sum only ever holds
// products c x, so its rounding error is relative to sum |x||c|.  For bfloat16
// activations the magic constant is bfloat16 128.0 (4-bit codes) or the codes
// are converted to fp32 (8-bit codes), and the constant part (e.g. 136 * sum x)
// is removed once per unit with an offset precomputed from x in binary64 when
// x is staged.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

#include "eb_internal.h"
#include "epilogue.h"
#include "gemv_common.h"

namespace eb {
namespace {

constexpr int kLanesPerRow = 16;
constexpr int kRowsPerSet = 64 / kLanesPerRow;  // 4
constexpr int kWaves = 4;                        // waves per workgroup
constexpr int kM1MaxSlots = 8;                   // m == 1 kernel: up to 8 units per lane

template <int QT>
struct Unit {
  static constexpr int kElems = (QT == EB_Q4_0) ? 32 : 16;  // weights per 16-byte unit
  static constexpr int kChunks = kElems * 2 / 16;            // 16-byte x chunks per unit
};

__device__ inline float dpp_row_sum(float v) {
  // quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_ror:4, row_ror:8
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x124, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xF, 0xF, true));
  return v;
}

__device__ inline uint4 load_nt(const uint4 *p) {
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
  const u4 t = __builtin_nontemporal_load(reinterpret_cast<const u4 *>(p));
  return make_uint4(t[0], t[1], t[2], t[3]);
}

// Sum over one unit of code_j * x_j (bfloat16 x: of (stored code value with
// the magic offset) * x_j, minus the precomputed offset `off`; binary16 x
// needs no offset and ignores it).
template <int QT, int XT>
__device__ inline float unit_dot(const uint4 q, const uint4 *xc, float off);

// Q4_0, binary16 x.  x chunk i = pairs (x4i,x4i+2) (x4i+1,x4i+3) (x16+4i,x16+4i+2) (x16+4i+1,x16+4i+3)
template <>
__device__ inline float unit_dot<EB_Q4_0, EB_F16>(const uint4 q, const uint4 *xc, float off) {
  (void)off;
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  const uint32_t mlo = 0x000F000Fu, mhi = 0x00F000F0u, magic = vconst(0x64006400u);
  float lo = 0.f, hi = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t v = w[i], v8 = w[i] >> 8;
    // low nibbles read 1024 + n = c + 1032, high nibbles 1024 + 16 n = 16 c + 1152
    lo = dot2h(sub_h2(and_or(v, mlo, magic), (_Float16)1032.0f), xc[i].x, lo);
    lo = dot2h(sub_h2(and_or(v8, mlo, magic), (_Float16)1032.0f), xc[i].y, lo);
    hi = dot2h(sub_h2(and_or(v, mhi, magic), (_Float16)1152.0f), xc[i].z, hi);
    hi = dot2h(sub_h2(and_or(v8, mhi, magic), (_Float16)1152.0f), xc[i].w, hi);
  }
  return __builtin_fmaf(hi, 0.0625f, lo);  // hi holds 16 c x
}

// Q4_0, bfloat16 x: bfloat16 128.0 | nibble = 128 + n = c + 136.
template <>
__device__ inline float unit_dot<EB_Q4_0, EB_BF16>(const uint4 q, const uint4 *xc, float off) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  const uint32_t mlo = 0x000F000Fu, magic = vconst(0x43004300u);
  float a = 0.f, b = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t v = w[i];
    a = dot2bf(and_or(v, mlo, magic), xc[i].x, a);
    a = dot2bf(and_or(v >> 8, mlo, magic), xc[i].y, a);
    b = dot2bf(and_or(v >> 4, mlo, magic), xc[i].z, b);
    b = dot2bf(and_or(v >> 12, mlo, magic), xc[i].w, b);
  }
  return (a + b) - off;
}

// Q8_0 half block, binary16 x: (q ^ 0x80) placed under 0x64 reads 1024 + q + 128.
template <>
__device__ inline float unit_dot<EB_Q8_0, EB_F16>(const uint4 q, const uint4 *xc, float off) {
  (void)off;
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  const uint32_t xs[8] = {xc[0].x, xc[0].y, xc[0].z, xc[0].w, xc[1].x, xc[1].y, xc[1].z, xc[1].w};
  float a = 0.f, b = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t u = w[i] ^ 0x80808080u;
    a = dot2h(sub_h2(__builtin_amdgcn_perm(0x64646464u, u, 0x04020400u), (_Float16)1152.0f), xs[2 * i], a);
    b = dot2h(sub_h2(__builtin_amdgcn_perm(0x64646464u, u, 0x04030401u), (_Float16)1152.0f), xs[2 * i + 1], b);
  }
  return a + b;
}

// Q8_0 half block, bfloat16 x (natural order): codes via fp32 byte conversion.
template <>
__device__ inline float unit_dot<EB_Q8_0, EB_BF16>(const uint4 q, const uint4 *xc, float off) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  const uint32_t xs[8] = {xc[0].x, xc[0].y, xc[0].z, xc[0].w, xc[1].x, xc[1].y, xc[1].z, xc[1].w};
  float a = 0.f, b = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t u = w[i] ^ 0x80808080u;
    const uint32_t x01 = xs[2 * i], x23 = xs[2 * i + 1];
    a = __builtin_fmaf((float)(u & 0xffu), __builtin_bit_cast(float, x01 << 16), a);
    b = __builtin_fmaf((float)((u >> 8) & 0xffu), __builtin_bit_cast(float, x01 & 0xffff0000u), b);
    a = __builtin_fmaf((float)((u >> 16) & 0xffu), __builtin_bit_cast(float, x23 << 16), a);
    b = __builtin_fmaf((float)(u >> 24), __builtin_bit_cast(float, x23 & 0xffff0000u), b);
  }
  return (a + b) - off;
}

// Per-row factors of the RMS-normalisation prologue, r_i = 1 / sqrt(eps +
// mean_j h[i][j]^2) for the m <= MT rows of the fp32 residual stream h, in
// every thread of the workgroup.  Each thread sums the squares of a strided
// part of every row in fp32; the 64 lanes of a wave, then the waves (through
// `red`, (waves per workgroup) * MT floats of LDS), are added in a fixed order.  Ends with a
// barrier after which `red` may be reused.
template <int MT>
__device__ inline void norm_factors(const float *__restrict__ h, int m, int64_t k, float eps,
                                    float *red, float (&rs)[MT]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) {
    float ss = 0.f;
    if (mm < m) {
      const float4 *row = reinterpret_cast<const float4 *>(h + (int64_t)mm * k);
      for (int64_t i = threadIdx.x; i < k / 4; i += blockDim.x) {
        const float4 v = row[i];
        ss = __builtin_fmaf(v.x, v.x, ss);
        ss = __builtin_fmaf(v.y, v.y, ss);
        ss = __builtin_fmaf(v.z, v.z, ss);
        ss = __builtin_fmaf(v.w, v.w, ss);
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
    if (lane == 0) red[wave * MT + mm] = ss;
  }
  __syncthreads();
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) {
    float ss = 0.f;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) ss += red[w * MT + mm];
    rs[mm] = 1.0f / __builtin_sqrtf(ss / (float)k + eps);
  }
  __syncthreads();
}

// Stage x[m][k] (m <= MT rows; missing rows are zero) into LDS in the pair
// order of unit_dot<QT, XT>, plus one offset per (row, unit).  With the
// normalisation prologue (norm) x is the fp32 residual stream and
// the staged activations are round_XT(h * gamma * rs[row]).
template <int QT, int XT, int MT>
__device__ __attribute__((always_inline)) inline void stage_x(
    const void *__restrict__ xv, int m, int64_t k, int64_t ku, uint4 *xs, float *xoff,
    int64_t pitch, bool norm, const float *__restrict__ gamma, const float (&rs)[MT]) {
  constexpr int E = Unit<QT>::kElems;
  constexpr int CH = Unit<QT>::kChunks;
  for (int64_t idx = threadIdx.x; idx < (int64_t)MT * ku; idx += blockDim.x) {
    const int mm = (int)(idx / ku);
    const int64_t u = idx % ku;
    uint32_t r[E / 2];  // raw dwords: r[j] = (h[2j], h[2j+1])
    if (mm < m && norm) {
      const float4 *src = reinterpret_cast<const float4 *>(static_cast<const float *>(xv) +
                                                           (int64_t)mm * k + u * E);
      const float4 *gs = reinterpret_cast<const float4 *>(gamma + u * E);
      float f = 0.f;
#pragma unroll
      for (int i = 0; i < MT; ++i)
        if (i == mm) f = rs[i];
#pragma unroll
      for (int c = 0; c < E / 4; ++c) {
        const float4 v = src[c], g = gs[c];
        r[2 * c] = pack_x16<XT>(v.x * g.x * f, v.y * g.y * f);
        r[2 * c + 1] = pack_x16<XT>(v.z * g.z * f, v.w * g.w * f);
      }
    } else if (mm < m) {
      const uint4 *src = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(xv) +
                                                         (int64_t)mm * k + u * E);
#pragma unroll
      for (int c = 0; c < E / 8; ++c) {
        uint4 t = src[c];
        r[4 * c] = t.x;
        r[4 * c + 1] = t.y;
        r[4 * c + 2] = t.z;
        r[4 * c + 3] = t.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < E / 2; ++j) r[j] = 0;
    }
    double s_lo = 0.0, s_hi = 0.0;
#pragma unroll
    for (int j = 0; j < E / 2; ++j) {
      double v = x_to_f64<XT>(r[j] & 0xffffu) + x_to_f64<XT>(r[j] >> 16);
      if (2 * j < 16)
        s_lo += v;
      else
        s_hi += v;
    }
    uint4 out[CH];
    double off;
    if (QT == EB_Q4_0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t a = r[2 * i], b = r[2 * i + 1], c = r[8 + 2 * i], d = r[8 + 2 * i + 1];
        out[i] = make_uint4((a & 0xffffu) | (b << 16), (a >> 16) | (b & 0xffff0000u),
                            (c & 0xffffu) | (d << 16), (c >> 16) | (d & 0xffff0000u));
      }
      off = (XT == EB_F16) ? 0.0 : 136.0 * (s_lo + s_hi);
    } else {
      if (XT == EB_F16) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint32_t a = r[4 * c], b = r[4 * c + 1], e = r[4 * c + 2], f = r[4 * c + 3];
          out[c] = make_uint4((a & 0xffffu) | (b << 16), (a >> 16) | (b & 0xffff0000u),
                              (e & 0xffffu) | (f << 16), (e >> 16) | (f & 0xffff0000u));
        }
        off = 0.0;
      } else {
#pragma unroll
        for (int c = 0; c < 2; ++c) out[c] = make_uint4(r[4 * c], r[4 * c + 1], r[4 * c + 2], r[4 * c + 3]);
        off = 128.0 * s_lo;
      }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) xs[((int64_t)mm * CH + c) * pitch + u] = out[c];
    xoff[(int64_t)mm * pitch + u] = (float)off;
  }
}

// m == 1, binary16 activations: stage the row into LDS for m1_rows in one
// pass.  One thread per 16-byte chunk of the staged row: chunk (unit u, part
// i) holds the pairs (a0,a2) (a1,a3) (b0,b2) (b1,b3) of a = x[e0 .. e0+3],
// b = x[e1 .. e1+3] (Q4_0: e0 = 32 u + 4 i, e1 = e0 + 16; Q8_0: e0 = 16 u +
// 8 i, e1 = e0 + 4), stored at xs[i * P + u].  With the normalisation
// prologue the thread's h values stay in registers between the sum of
// squares and the normalisation, so h is read from memory once; the sum is
// reduced over the wave by exchanges and over the waves in order through
// `red` (one float per wave, not aliasing xs).
//
// Two phases: x1_issue loads the thread's first chunk (h and gamma), or the
// raw binary16 values of its first two, into registers, and x1_finish stages
// them with the rest.  The
// caller issues its first weight loads in between: vector-memory loads
// complete in issue order, so waiting for activations loaded after the
// weights would wait for all of those weights, and no decoding could begin
// before the workgroup barrier that ends the staging.
struct X1Regs {
  // normalisation prologue: h[e0..e0+3], h[e1..e1+3] and gamma there, for
  // the thread's first chunk; otherwise the raw 8-byte halves of its first
  // two chunks (a = {chunk 0 at e0, chunk 1 at e0}, b likewise at e1)
  uint4 a, b, ga, gb;
};

template <int QT>
__device__ __attribute__((always_inline)) inline void x1_chunk(int c, int &u, int &i, int &e0, int &e1) {
  constexpr int CH = Unit<QT>::kChunks;
  u = c / CH;
  i = c - u * CH;
  e0 = (QT == EB_Q4_0) ? u * 32 + 4 * i : u * 16 + 8 * i;
  e1 = e0 + ((QT == EB_Q4_0) ? 16 : 4);
}

template <int QT>
__device__ __attribute__((always_inline)) inline void x1_issue(const void *__restrict__ xv, int ku, bool norm,
                                                               const float *__restrict__ gamma, X1Regs &R) {
  constexpr int CH = Unit<QT>::kChunks;
  const int nch = ku * CH, T = (int)blockDim.x, tid = (int)threadIdx.x;
  int u, i, e0, e1;
  if (norm) {
    if (tid < nch) {
      x1_chunk<QT>(tid, u, i, e0, e1);
      const float *h = static_cast<const float *>(xv);
      R.a = *reinterpret_cast<const uint4 *>(h + e0);
      R.b = *reinterpret_cast<const uint4 *>(h + e1);
      R.ga = *reinterpret_cast<const uint4 *>(gamma + e0);
      R.gb = *reinterpret_cast<const uint4 *>(gamma + e1);
    }
  } else {
    const uint16_t *x = static_cast<const uint16_t *>(xv);
    if (tid < nch) {
      x1_chunk<QT>(tid, u, i, e0, e1);
      const uint2 ra = *reinterpret_cast<const uint2 *>(x + e0), rb = *reinterpret_cast<const uint2 *>(x + e1);
      R.a.x = ra.x, R.a.y = ra.y, R.b.x = rb.x, R.b.y = rb.y;
    }
    if (tid + T < nch) {
      x1_chunk<QT>(tid + T, u, i, e0, e1);
      const uint2 ra = *reinterpret_cast<const uint2 *>(x + e0), rb = *reinterpret_cast<const uint2 *>(x + e1);
      R.a.z = ra.x, R.a.w = ra.y, R.b.z = rb.x, R.b.w = rb.y;
    }
  }
}

template <int QT>
__device__ __attribute__((always_inline)) inline void x1_finish(
    const void *__restrict__ xv, int64_t k, int ku, uint4 *xs, int P, bool norm,
    const float *__restrict__ gamma, float eps, float *red, const X1Regs &R) {
  constexpr int CH = Unit<QT>::kChunks;
  const int nch = ku * CH, T = (int)blockDim.x, tid = (int)threadIdx.x;
  auto f4 = [](uint4 v) __attribute__((always_inline)) {
    return make_float4(__builtin_bit_cast(float, v.x), __builtin_bit_cast(float, v.y),
                       __builtin_bit_cast(float, v.z), __builtin_bit_cast(float, v.w));
  };
  auto put = [&](int u, int i, float4 a, float4 b) __attribute__((always_inline)) {
    xs[i * P + u] = make_uint4(pack_x16<EB_F16>(a.x, a.z), pack_x16<EB_F16>(a.y, a.w),
                               pack_x16<EB_F16>(b.x, b.z), pack_x16<EB_F16>(b.y, b.w));
  };
  // (a0 a1)(a2 a3) -> (a0 a2)(a1 a3)
  auto put_raw = [&](int u, int i, uint2 a, uint2 b) __attribute__((always_inline)) {
    xs[i * P + u] = make_uint4((a.x & 0xffffu) | (a.y << 16), (a.x >> 16) | (a.y & 0xffff0000u),
                               (b.x & 0xffffu) | (b.y << 16), (b.x >> 16) | (b.y & 0xffff0000u));
  };
  if (!norm) {
    const uint16_t *x = static_cast<const uint16_t *>(xv);
    int u, i, e0, e1;
    if (tid < nch) {
      x1_chunk<QT>(tid, u, i, e0, e1);
      put_raw(u, i, make_uint2(R.a.x, R.a.y), make_uint2(R.b.x, R.b.y));
    }
    if (tid + T < nch) {
      x1_chunk<QT>(tid + T, u, i, e0, e1);
      put_raw(u, i, make_uint2(R.a.z, R.a.w), make_uint2(R.b.z, R.b.w));
    }
    for (int c = tid + 2 * T; c < nch; c += T) {
      int u, i, e0, e1;
      x1_chunk<QT>(c, u, i, e0, e1);
      put_raw(u, i, *reinterpret_cast<const uint2 *>(x + e0), *reinterpret_cast<const uint2 *>(x + e1));
    }
    return;
  }
  const float *h = static_cast<const float *>(xv);
  float ss = 0.f;
  auto sq = [](float acc, float4 v) __attribute__((always_inline)) {
    acc = __builtin_fmaf(v.x, v.x, acc);
    acc = __builtin_fmaf(v.y, v.y, acc);
    acc = __builtin_fmaf(v.z, v.z, acc);
    return __builtin_fmaf(v.w, v.w, acc);
  };
  if (tid < nch) ss = sq(sq(ss, f4(R.a)), f4(R.b));
  for (int c = tid + T; c < nch; c += T) {
    int u, i, e0, e1;
    x1_chunk<QT>(c, u, i, e0, e1);
    ss = sq(sq(ss, *reinterpret_cast<const float4 *>(h + e0)), *reinterpret_cast<const float4 *>(h + e1));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (T >> 6); ++w) tot += red[w];
  const float r = 1.0f / __builtin_sqrtf(tot / (float)k + eps);
  auto normed = [&](float4 v, float4 gg) __attribute__((always_inline)) {
    return make_float4(v.x * gg.x * r, v.y * gg.y * r, v.z * gg.z * r, v.w * gg.w * r);
  };
  if (tid < nch) {
    int u, i, e0, e1;
    x1_chunk<QT>(tid, u, i, e0, e1);
    put(u, i, normed(f4(R.a), f4(R.ga)), normed(f4(R.b), f4(R.gb)));
  }
  for (int c = tid + T; c < nch; c += T) {
    int u, i, e0, e1;
    x1_chunk<QT>(c, u, i, e0, e1);
    put(u, i, normed(*reinterpret_cast<const float4 *>(h + e0), *reinterpret_cast<const float4 *>(gamma + e0)),
        normed(*reinterpret_cast<const float4 *>(h + e1), *reinterpret_cast<const float4 *>(gamma + e1)));
  }
}

template <int QT, int XT, int MT, int RS>
__global__ void __launch_bounds__(64 * kWaves)
    gemv_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off, int64_t ds,
                const void *__restrict__ x, int m, void *__restrict__ y, int yt, Fuse f) {
  constexpr int CH = Unit<QT>::kChunks;
  const int64_t ku = k / Unit<QT>::kElems;
  extern __shared__ uint4 smem[];
  uint4 *xs = smem;
  float *xoff = reinterpret_cast<float *>(smem + (int64_t)MT * CH * ku);

  float rs[MT];
  const bool norm = f.pro == EB_PRO_RMSNORM;
  if (norm) norm_factors<MT>(static_cast<const float *>(x), m, k, f.eps, reinterpret_cast<float *>(xs), rs);
  stage_x<QT, XT, MT>(x, m, k, ku, xs, xoff, ku, norm, f.gamma, rs);
  __syncthreads();

  const uint4 *__restrict__ qs = reinterpret_cast<const uint4 *>(wdata);
  const uint16_t *__restrict__ dplane = reinterpret_cast<const uint16_t *>(wdata + d_off);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rsub = lane / kLanesPerRow;
  const int c = lane % kLanesPerRow;
  constexpr int kRowsPerItem = kRowsPerSet * RS;
  const int64_t items = (n + kRowsPerItem - 1) / kRowsPerItem;

  for (int64_t it = (int64_t)blockIdx.x * kWaves + wave; it < items;
       it += (int64_t)gridDim.x * kWaves) {
    int64_t rows[RS];
#pragma unroll
    for (int s = 0; s < RS; ++s) {
      const int64_t r = it * kRowsPerItem + s * kRowsPerSet + rsub;
      rows[s] = r < n ? r : n - 1;  // clamp the tail; its results are not stored
    }
    float acc[RS][MT];
#pragma unroll
    for (int s = 0; s < RS; ++s)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) acc[s][mm] = 0.f;

#pragma unroll 2
    for (int64_t u = c; u < ku; u += kLanesPerRow) {
      const int64_t b = (QT == EB_Q4_0) ? u : (u >> 1);
      uint4 q[RS];
      float d[RS];
#pragma unroll
      for (int s = 0; s < RS; ++s) {
        q[s] = load_nt(qs + rows[s] * ku + u);
        d[s] = (float)__builtin_bit_cast(_Float16, __builtin_nontemporal_load(dplane + rows[s] * ds + b));
      }
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        uint4 xc[CH];
#pragma unroll
        for (int ch = 0; ch < CH; ++ch) xc[ch] = xs[((int64_t)mm * CH + ch) * ku + u];
        const float off = xoff[(int64_t)mm * ku + u];
#pragma unroll
        for (int s = 0; s < RS; ++s)
          acc[s][mm] = __builtin_fmaf(d[s], unit_dot<QT, XT>(q[s], xc, off), acc[s][mm]);
      }
    }

#pragma unroll
    for (int s = 0; s < RS; ++s)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) acc[s][mm] = dpp_row_sum(acc[s][mm]);

    if (f.epi == EB_EPI_GLU) {
      // rows r (even rsub: gate) and r + 1 (odd rsub: up) sit 16 lanes apart
#pragma unroll
      for (int s = 0; s < RS; ++s)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm) {
          const float up = __shfl_xor(acc[s][mm], 16);
          const int64_t r = it * kRowsPerItem + s * kRowsPerSet + rsub;
          if (c == 0 && (rsub & 1) == 0 && r < n && mm < m)
            store_y(y, (int64_t)mm * (n / 2) + r / 2, silu_mul(acc[s][mm], up), yt);
        }
    } else if (c == 0) {
#pragma unroll
      for (int s = 0; s < RS; ++s) {
        const int64_t r = it * kRowsPerItem + s * kRowsPerSet + rsub;
        if (f.epi == EB_EPI_ADD) {  // the row's residuals read together
          // offsets from the item's first row (the same in every lane)
          const int64_t b0 = it * kRowsPerItem;
          uint32_t rel[MT];
          bool ok[MT];
#pragma unroll
          for (int mm = 0; mm < MT; ++mm) {
            rel[mm] = (uint32_t)mm * (uint32_t)n + (uint32_t)(r - b0);
            ok[mm] = mm < m && r < n;
          }
          if (put_y_add(y, f.r, b0, (int64_t)(m - 1) * n + kRowsPerItem, rel, ok, acc[s], yt)) continue;
        }
        if (r >= n) continue;
#pragma unroll
        for (int mm = 0; mm < MT; ++mm) {
          if (mm >= m) continue;
          put_y(y, (int64_t)mm * n + r, acc[s][mm], yt, f);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// m == 1: one wave per weight row across the whole of k.  Lane l owns units
// l, l + 64, ... of every row, so each load instruction reads 1 KiB of
// contiguous packed codes; the lane's x fragments (already in pair order) stay
// in VGPRs for the whole launch.  R rows are in flight per wave; their 64-lane
// partial sums are reduced together by halving exchanges (v_permlane32_swap,
// v_permlane16_swap, then DPP inside 16-lane rows), R values in O(R + log 64)
// instructions.
// ---------------------------------------------------------------------------

// Items in flight per wave for a group of `items` items: the largest divisor
// of it up to `cap` (so that an item's register set is a compile-time
// function of its index).  Lone launches cap it at 4: measured on the decode
// chain's projections (1, 2, 4 and 6 items per group), 0.993 ms per pass
// against 1.003 (cap 3), 1.002 (cap 2) and 1.017 (no cap; the 6-item down
// projection 11% slower, and still 6% slower with the first group split
// around the staging of x).  The fused multi-matrix kernel, whose workgroups
// run many groups each, does not cap it (2% faster on its 6-slot matrices).
constexpr int kM1Ring = 4;
__host__ __device__ constexpr int m1_ring(int items, int cap) {
  int d = items < cap ? items : cap;
  while (items % d) --d;
  return d;
}

// Rows g*R .. g*R+R-1 for the wave's groups g in [gbase, g_end) of one
// matrix, m == 1: gbase + vb, + gstride, ... in the whole rounds of gstride
// groups, and gbase + (whole rounds) gstride + vw in the last, partial one
// (vb and vw number the gstride waves; callers that pass vb == vw walk
// gbase + vb + i gstride).  Called by every thread of the workgroup (it stages
// x into LDS and synchronises once); waves without a group only help with the
// staging.  PRE (residual-adding ops with fp32 output, EB_EPI_ADD): the
// residual of each lane's row is loaded before the group's weights, so the
// epilogue does not wait a memory round trip for it after the reduction.
// SPLIT (lone launches): with 3 or more items in flight, half of the first
// group's items are requested before x is staged, the rest right after it.
template <int QT, int XT, int NS, int R, int RING, bool PRE = false, bool SPLIT = false>
__device__ __attribute__((always_inline)) inline void m1_rows(const uint8_t *__restrict__ wdata, int64_t n, int64_t k,
                               int64_t d_off, int64_t ds, const void *__restrict__ x,
                               void *__restrict__ y, int yt, const Fuse &f, int64_t gbase, int64_t vb,
                               int64_t vw, int64_t g_end, int64_t gstride, uint4 *smem) {
  // The wave's groups: gbase + vb + i gstride in the whole rounds i < full,
  // then, in the last, partial round, gbase + full gstride + vw (a numbering
  // that spreads that round's groups over the compute units; past the end:
  // g_end, a dead group).
  const int64_t full = (g_end - gbase) / gstride, rem = g_end - gbase - full * gstride;
  const int64_t cnt = full + (vw < rem ? 1 : 0);
  auto grp = [&](int64_t i) __attribute__((always_inline)) {
    return i < full ? gbase + vb + i * gstride : (i == full && vw < rem ? gbase + full * gstride + vw : g_end);
  };
  int64_t g = grp(0), gnext = g_end;
  constexpr int CH = Unit<QT>::kChunks;
  // LDS: CH chunk rows of P entries; entry 64 * NS of every row is zero and
  // stands in for units past the end of the row.  P is a compile-time
  // constant so every x read is one base register plus an immediate offset.
  constexpr int P = 64 * NS + 1;
  const int ku = (int)(k / Unit<QT>::kElems);  // 64 * (NS - 1) < ku <= 64 * NS
  uint4 *xs = smem;
  float *xoff = reinterpret_cast<float *>(smem + CH * P);
  const int lane = threadIdx.x & 63;
  const uint32_t qs_row = (uint32_t)ku * 16u, d_row = (uint32_t)(ds * 2);
  const uint8_t *__restrict__ dbase = wdata + d_off;

  // Per-lane offsets of the lane's unit u = lane + 64 s in slot s.  Only the
  // last slot can pass the end of the row (ku > 64 (NS - 1)): its units are
  // clamped to the row's last unit and read the zero x entry, so they add
  // exactly 0.  The other slots are the lane's base offset plus a constant
  // (a scalar or immediate operand, not a register per slot).
  const int ul = lane + 64 * (NS - 1), ulc = min(ul, ku - 1);
  const uint32_t qlast = (uint32_t)ulc * 16u;
  const uint32_t dlast = (uint32_t)((QT == EB_Q4_0) ? ulc : (ulc >> 1)) * 2u;
  const uint32_t xlast = ul < ku ? (uint32_t)ul : 64u * NS;
  const uint32_t qbase = (uint32_t)lane * 16u;
  const uint32_t dbase_l = (uint32_t)((QT == EB_Q4_0) ? lane : (lane >> 1)) * 2u;
  // slot s < NS - 1: code bytes at qbase + 1024 s, scale at dbase_l + dstep s
  constexpr uint32_t dstep = (QT == EB_Q4_0) ? 128u : 64u;

  // A ring of D register sets for the NS R items of a group (item i = slot
  // s of row r, i = s R + r: the lane's 16 code bytes and their scale).
  // Item i lives in set i % D; right after it has been used, its set is
  // reloaded with item i + D, of this group or of the wave's next one.  A
  // wave thus keeps D items (D KiB) of reads in flight without pauses while
  // it decodes.  (Measured on the 32-layer decode chain: with two groups'
  // items in flight instead of one, 1.16 against 1.02 ms per pass; with more
  // reads queued, an item completes only when nearly all of them have
  // arrived, and the decoding no longer overlaps the loads.)
  constexpr int I = NS * R, D = m1_ring(I, RING);
  struct Item {
    uint4 q;
    uint16_t dh;
  };
  Item ring[D];
  // A group past g_end gets zero-sized buffer ranges: its loads return zeros
  // without a memory access.  Every load is therefore issued on every path:
  // a load issued on only some paths makes the compiler's counter wait for
  // an earlier load a wait for everything.
  // Buffer ranges of the R rows of group grp:
  struct GRes {
    __amdgpu_buffer_rsrc_t q[R], d[R];
  };
  auto group_res = [&](int64_t grp, GRes &G) __attribute__((always_inline)) {
    const bool live = grp < g_end;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      int64_t row = grp * R + r;
      row = row < n ? row : n - 1;  // tail rows are computed but not stored
      G.q[r] = rsrc(wdata + row * qs_row, live ? qs_row : 0u);
      G.d[r] = rsrc(dbase + row * d_row, live ? d_row : 0u);
    }
  };
  auto load_item = [&](Item &it, const GRes &G, int i) __attribute__((always_inline)) {
    const int s = i / R, r = i % R;
    const bool last = s == NS - 1;
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(G.q[r], (int)(last ? qlast : qbase),
                                                         last ? 0 : 1024 * s, kNT);
    it.q = make_uint4(v[0], v[1], v[2], v[3]);
    it.dh = __builtin_amdgcn_raw_buffer_load_b16(G.d[r], (int)(last ? dlast : dbase_l),
                                                 last ? 0 : (int)dstep * s, kNT);
  };
  // Binary16 activations: their loads are issued first, then the weight
  // loads of the first group, which stay in flight while x is staged
  // (and, with the prologue, normalised); waiting for the activations does
  // not wait for the weights (loads complete in issue order).
  const bool norm = f.pro == EB_PRO_RMSNORM;
  X1Regs xr;
  if constexpr (XT == EB_F16) x1_issue<QT>(x, ku, norm, f.gamma, xr);
  __builtin_amdgcn_sched_barrier(0);
  // PRE: the fp32 residual of the row this lane's reduction ends in, for
  // group grp (a group past g_end reads zero without a memory access).  The
  // first group's is loaded before its weights, the next group's right after
  // this group's output: either way it is older than every load issued while
  // its group is decoded, so waiting for it never waits for those.
  const uint32_t res_off = 4u * (uint32_t)reduce_row<R>(lane);
  auto res_load = [&](int64_t grp) __attribute__((always_inline)) -> float {
    const bool live = grp < g_end;
    const int64_t r0 = live ? grp * R : 0;
    const uint32_t bytes = live ? 4u * (uint32_t)min((int64_t)R, n - r0) : 0u;
    const auto rs = rsrc(static_cast<const float *>(f.r) + r0, bytes);
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (int)res_off, 0, 0));
  };
  float res_cur = 0.f;
  if constexpr (PRE) {
    res_cur = res_load(g);
    __builtin_amdgcn_sched_barrier(0);
  }
  // The first group's items, kept in item order (left to the scheduler, the
  // scales would follow all the codes and the first item's wait would be a
  // wait for all of them).  With SPLIT only the first E go before the
  // staging: the activations are read while every wave's first weights
  // stream in, and the fewer those are, the sooner the staging ends
  // (measured on the decode chain: the gate/up launch's staging 2.0 instead
  // of 3.2 us, the launch 1.4-3.5% and the 3-item down projection 2-3%
  // shorter; with 2 items the QKV projection was 2% slower, so it keeps
  // both).
  constexpr int E = SPLIT && D >= 3 ? D / 2 : D;
  GRes G0;
  group_res(g, G0);
#pragma unroll
  for (int i = 0; i < E; ++i) {
    load_item(ring[i], G0, i);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (XT == EB_F16) {
    x1_finish<QT>(x, k, ku, xs, P, norm, f.gamma, f.eps, xoff, xr);
  } else {
    float rs[1] = {0.f};
    if (norm) norm_factors<1>(static_cast<const float *>(x), 1, k, f.eps, reinterpret_cast<float *>(xs), rs);
    stage_x<QT, XT, 1>(x, 1, k, ku, xs, xoff, P, norm, f.gamma, rs);
  }
  if (threadIdx.x < CH) xs[threadIdx.x * P + 64 * NS] = make_uint4(0, 0, 0, 0);
  if (XT != EB_F16 && threadIdx.x == 0) xoff[64 * NS] = 0.f;
  __syncthreads();
#pragma unroll
  for (int i = E; i < D; ++i) {
    __builtin_amdgcn_sched_barrier(0);
    load_item(ring[i], G0, i);
  }
  __builtin_amdgcn_sched_barrier(0);

  // one group (g < g_end)
  auto step = [&]() __attribute__((always_inline)) {
    GRes Gc, Gn;
    if constexpr (D < I) group_res(g, Gc);
    group_res(gnext, Gn);
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint32_t xi = s == NS - 1 ? xlast : (uint32_t)lane + 64u * s;
      const uint4 *xp = xs + xi;
      uint4 xf[CH];
#pragma unroll
      for (int c = 0; c < CH; ++c) xf[c] = xp[c * P];
      const float xo = XT == EB_F16 ? 0.f : xoff[xi];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = s * R + r;
        Item &it = ring[i % D];
        acc[r] = __builtin_fmaf((float)__builtin_bit_cast(_Float16, it.dh), unit_dot<QT, XT>(it.q, xf, xo),
                                acc[r]);
        __builtin_amdgcn_sched_barrier(0);
        if (i + D < I)
          load_item(it, Gc, i + D);
        else
          load_item(it, Gn, i + D - I);
      }
    }
    int rr;
    bool writer;
    const float tot = reduce_rows<R>(acc, lane, rr, writer);
    const int64_t row = g * R + rr;
    // (without PRE, the add epilogue's wait for its residual also waits for
    // the reloads just issued)
    if constexpr (PRE) {
      // put_y's arithmetic: the fp32 sum, then the fp32 store
      if (writer && row < n) store_y(y, row, tot + res_cur, EB_F32);
      res_cur = res_load(gnext);
    } else if constexpr (R >= 2) {
      if (f.epi == EB_EPI_GLU) {
        // the up row (odd) of a pair is held R/2 ... lanes away: 8 (R = 8),
        // 16 (R = 4) or 32 (R = 2) lanes, see reduce_rows
        const float up = __shfl_xor(tot, R == 8 ? 8 : (R == 4 ? 16 : 32));
        if (writer && (rr & 1) == 0 && row < n) store_y(y, row / 2, silu_mul(tot, up), yt);
      } else if (writer && row < n) {
        put_y(y, row, tot, yt, f);
      }
    } else {
      if (writer && row < n) put_y(y, row, tot, yt, f);
    }
  };
  for (int64_t i = 0; i < cnt; ++i) {
    g = grp(i);
    gnext = grp(i + 1);
    step();
  }
}

// One matrix per launch.  WPE: minimum waves per SIMD the register allocation
// must allow; memory latency is hidden by other waves rather than by deep
// per-wave prefetch.  WG waves per workgroup: a lone launch has few row
// groups per wave, so the per-workgroup staging of x (and the normalisation
// prologue's reduction over the whole row) is a large part of it; with 16
// waves per workgroup and one workgroup per CU it is done once per CU instead
// of four times, and the 256 workgroups re-read the shared activations from
// the L2 a quarter as often.
template <int QT, int XT, int NS, int R, int WPE, int WG, bool PRE>
__global__ void __launch_bounds__(64 * WG) __attribute__((amdgpu_waves_per_eu(WPE)))
    gemv_m1_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off,
                   int64_t ds, const void *__restrict__ x, void *__restrict__ y, int yt, Fuse f) {
  extern __shared__ uint4 smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  // Group numbering: the whole rounds block-major (a compute unit's waves
  // take neighbouring rows), the last, partial round wave-major, so that its
  // groups spread over every compute unit instead of filling the first ones
  // (the decode layer's 11008 gate/up pairs over 4096 waves: 43-44 groups per
  // CU instead of 48 on 176 CUs and 32 on the rest).
  m1_rows<QT, XT, NS, R, kM1Ring, PRE, true>(wdata, n, k, d_off, ds, x, y, yt, f, 0,
                                  (int64_t)blockIdx.x * WG + wave, (int64_t)wave * gridDim.x + blockIdx.x,
                                  (n + R - 1) / R, (int64_t)gridDim.x * WG, smem);
}

// Rows per wave for the fused multi-matrix kernel, by slot count (no spills
// at 4 waves per SIMD).
// (A row gets the same bits whatever the rows per wave: reduce_rows adds a
// one-row wave's sums in the two-row order, so a fused stack and single calls,
// one row per wave outside the gate/up pairs, agree bitwise.)
__host__ __device__ constexpr int m1_multi_rows(int ns) { return ns <= 4 ? 2 : 1; }

// Several independent matrices (m == 1, same formats, same slot count NS) in
// one persistent launch, so the matrices of a stack overlap instead of each
// paying a launch, an x staging and a ramp-up.  The launch's work, rows
// weighted by their length (units), is cut into gridDim.x equal shares:
// workgroup b takes units [b U / G, (b+1) U / G) of the concatenated matrices,
// converted to row boundaries rounded down to whole R-row groups (both
// neighbours round the same boundary the same way, so every row is computed
// exactly once), and stages each matrix's x once for the part it covers.
template <int QT, int XT, int NS>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(NS <= 2 ? 4 : 3)))
    gemv_m1_multi_kernel(const M1Op *__restrict__ ops, int nops, int64_t units) {
  constexpr int R = m1_multi_rows(NS);
  extern __shared__ uint4 smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t G = gridDim.x;
  const int64_t u0 = units * (int64_t)blockIdx.x / G, u1 = units * ((int64_t)blockIdx.x + 1) / G;
  // first matrix whose units reach past u0 (binary search; unit_begin ascends)
  int lo = 0, hi = nops - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (ops[mid].unit_begin <= u0) lo = mid; else hi = mid - 1;
  }
  for (int op = lo; op < nops && ops[op].unit_begin < u1; ++op) {
    const M1Op o = ops[op];
    // row boundary of unit u inside this matrix, rounded down to a whole group
    auto row_at = [&](int64_t u) {
      int64_t r = (u - o.unit_begin) / o.ku;
      r = r < 0 ? 0 : (r > o.n ? o.n : r);
      return r == o.n ? r : r / R * R;
    };
    const int64_t r0 = row_at(u0), r1 = row_at(u1);
    if (r0 >= r1) continue;  // uniform across the workgroup
    m1_rows<QT, XT, NS, R, NS * R>(o.w, o.n, o.k, o.d_off, o.ds, o.x, o.y, o.yt, o.f, r0 / R, wave, wave,
                              (r1 + R - 1) / R, kWaves, smem);
    __syncthreads();  // the next matrix restages LDS
  }
}

// ---------------------------------------------------------------------------
template <int QT, int XT, int NS, int R, int WPE, int WG, bool PRE = false>
hipError_t launch_m1_t(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                       const Fuse &f, hipStream_t s, int wg_per_cu) {
  const Layout L = layout_of(QT, n, k);
  const size_t lds = (size_t)(64 * NS + 1) * (Unit<QT>::kChunks * 16 + 4);
  const int64_t groups = (n + R - 1) / R;
  int64_t grid = (groups + WG - 1) / WG;
  const int64_t cap = (int64_t)device_cu_count() * wg_per_cu;
  if (grid > cap) grid = cap;
  gemv_m1_kernel<QT, XT, NS, R, WPE, WG, PRE><<<(unsigned)grid, 64 * WG, lds, s>>>(
      (const uint8_t *)wdata, n, k, L.d_off, L.ds, x, y, yt, f);
  return hipGetLastError();
}

// Launch shape of the m == 1 kernel: rows per wave (R), minimum waves per
// SIMD (WPE), workgroups per CU and waves per workgroup.  The defaults are
// per slot count; the environment variable EB_GEMV_M1="R,WPE,WGPERCU,WAVES"
// overrides them (tuning; WAVES 4 or 16).
struct M1Shape {
  int r, wpe, wg, waves;
};

M1Shape m1_shape(int64_t ns) {
  static const char *env = getenv("EB_GEMV_M1");
  if (env) {
    M1Shape v{0, 0, 0, 0};
    if (sscanf(env, "%d,%d,%d,%d", &v.r, &v.wpe, &v.wg, &v.waves) == 4 && v.r > 0 && v.wpe > 0 &&
        v.wg > 0 && (v.waves == 4 || v.waves == 16))
      return v;
  }
  return {1, 4, 1, 16};
}

template <int QT, int XT, int NS>
hipError_t launch_m1_ns(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                        const Fuse &f, hipStream_t s) {
  // one row per wave by default (a 4096-row matrix then fills all 256 CUs
  // with 16-wave workgroups), two for the gate/up product, which needs both
  // rows of a pair in one wave
  M1Shape v = m1_shape(NS);
  if (f.epi == EB_EPI_GLU && v.r < 2) v.r = 2;
  // residual-adding ops with fp32 output (the decoder layer's O and down
  // projections on the residual stream) in the default shape preload their
  // residuals
  if (f.epi == EB_EPI_ADD && yt == EB_F32 && v.r == 1 && v.wpe == 4 && v.waves == 16)
    return launch_m1_t<QT, XT, NS, 1, 4, 16, true>(wdata, n, k, x, y, yt, f, s, v.wg);
#define EB_M1(R_, W_, G_)                                                                  \
  if (v.r == R_ && v.wpe == W_ && v.waves == G_)                                          \
    return launch_m1_t<QT, XT, NS, R_, W_, G_>(wdata, n, k, x, y, yt, f, s, v.wg);
  EB_M1(1, 4, 16) EB_M1(2, 4, 16) EB_M1(1, 4, 4) EB_M1(2, 4, 4) EB_M1(4, 4, 4) EB_M1(2, 2, 4)
#undef EB_M1
  return hipErrorInvalidValue;
}

template <int QT, int XT>
hipError_t launch_m1(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                     const Fuse &f, hipStream_t s) {
  const int64_t ns = (k / Unit<QT>::kElems + 63) / 64;
  switch (ns) {
    case 1: return launch_m1_ns<QT, XT, 1>(wdata, n, k, x, y, yt, f, s);
    case 2: return launch_m1_ns<QT, XT, 2>(wdata, n, k, x, y, yt, f, s);
    case 3: return launch_m1_ns<QT, XT, 3>(wdata, n, k, x, y, yt, f, s);
    case 4: return launch_m1_ns<QT, XT, 4>(wdata, n, k, x, y, yt, f, s);
    case 5: return launch_m1_ns<QT, XT, 5>(wdata, n, k, x, y, yt, f, s);
    case 6: return launch_m1_ns<QT, XT, 6>(wdata, n, k, x, y, yt, f, s);
    case 7: return launch_m1_ns<QT, XT, 7>(wdata, n, k, x, y, yt, f, s);
    default: return launch_m1_ns<QT, XT, 8>(wdata, n, k, x, y, yt, f, s);
  }
}

template <int QT, int XT, int MT, int RS>
hipError_t launch_t(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(QT, n, k);
  const int64_t ku = k / Unit<QT>::kElems;
  const size_t lds = (size_t)MT * ku * (Unit<QT>::kChunks * 16 + 4);
  const int64_t items = (n + kRowsPerSet * RS - 1) / (kRowsPerSet * RS);
  int64_t grid = (items + kWaves - 1) / kWaves;
  const int64_t cap = (int64_t)device_cu_count() * 8;
  if (grid > cap) grid = cap;
  auto kern = gemv_kernel<QT, XT, MT, RS>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<(unsigned)grid, 64 * kWaves, lds, s>>>((const uint8_t *)wdata, n, k, L.d_off, L.ds, x,
                                                (int)m, y, yt, f);
  return hipGetLastError();
}

template <int QT, int XT>
hipError_t launch_m(const void *wdata, int64_t n, int64_t k, const void *x, int64_t m, void *y,
                    int32_t yt, const Fuse &f, hipStream_t s) {
  const int64_t ns = (k / Unit<QT>::kElems + 63) / 64;
  // the gate/up epilogue needs both rows of a pair in one wave (R >= 2)
  // the gate/up epilogue takes two rows per wave, which fit without spilling
  // up to 4 slots
  const bool m1_ok = ns <= kM1MaxSlots && (f.epi != EB_EPI_GLU || ns <= 4);
  if (m <= 1 && m1_ok) return launch_m1<QT, XT>(wdata, n, k, x, y, yt, f, s);
  if (m <= 1) return launch_t<QT, XT, 1, 2>(wdata, n, k, x, m, y, yt, f, s);
  if (m <= 2) return launch_t<QT, XT, 2, 2>(wdata, n, k, x, m, y, yt, f, s);
  if (m <= 4) return launch_t<QT, XT, 4, 1>(wdata, n, k, x, m, y, yt, f, s);
  return launch_t<QT, XT, 8, 1>(wdata, n, k, x, m, y, yt, f, s);
}

template <int QT, int XT, int NS>
hipError_t launch_multi_t(const M1Op *ops, int nops, int64_t units, int64_t rows,
                          hipStream_t s) {
  const size_t lds = (size_t)(64 * NS + 1) * (Unit<QT>::kChunks * 16 + 4);
  int64_t grid = (int64_t)device_cu_count() * 4;
  const int64_t groups = rows / (kWaves * m1_multi_rows(NS));  // keep every wave busy
  if (grid > groups) grid = groups > 0 ? groups : 1;
  gemv_m1_multi_kernel<QT, XT, NS><<<(unsigned)grid, 64 * kWaves, lds, s>>>(ops, nops, units);
  return hipGetLastError();
}

template <int QT, int XT>
hipError_t launch_multi_q(const M1Op *ops, int nops, int64_t items, int64_t rows, int ns,
                          hipStream_t s) {
  switch (ns) {
    case 1: return launch_multi_t<QT, XT, 1>(ops, nops, items, rows, s);
    case 2: return launch_multi_t<QT, XT, 2>(ops, nops, items, rows, s);
    case 3: return launch_multi_t<QT, XT, 3>(ops, nops, items, rows, s);
    case 4: return launch_multi_t<QT, XT, 4>(ops, nops, items, rows, s);
    case 5: return launch_multi_t<QT, XT, 5>(ops, nops, items, rows, s);
    case 6: return launch_multi_t<QT, XT, 6>(ops, nops, items, rows, s);
    case 7: return launch_multi_t<QT, XT, 7>(ops, nops, items, rows, s);
    case 8: return launch_multi_t<QT, XT, 8>(ops, nops, items, rows, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool m1_fusable(int32_t type, int64_t m, int64_t k, int32_t epi) {
  if (type == EB_Q6_S) return m == 1 && q6_m1_fusable(k, epi);
  const int64_t e = (type == EB_Q4_0) ? Unit<EB_Q4_0>::kElems : Unit<EB_Q8_0>::kElems;
  const int64_t ns = (k / e + 63) / 64;
  return m == 1 && ns <= kM1MaxSlots && (epi != EB_EPI_GLU || m1_multi_rows((int)ns) >= 2);
}

int m1_slots(int32_t type, int64_t k) {
  if (type == EB_Q6_S) return q6_m1_slots(k);
  const int64_t e = (type == EB_Q4_0) ? Unit<EB_Q4_0>::kElems : Unit<EB_Q8_0>::kElems;
  return (int)((k / e + 63) / 64);
}

int64_t m1_fill(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x, void *y,
                int32_t yt, const Fuse &f, int64_t unit_begin, M1Op *o) {
  if (type == EB_Q6_S) return q6_m1_fill(wdata, n, k, x, y, yt, f, unit_begin, o);
  const int64_t e = (type == EB_Q4_0) ? Unit<EB_Q4_0>::kElems : Unit<EB_Q8_0>::kElems;
  const Layout L = layout_of(type, n, k);
  o->w = (const uint8_t *)wdata;
  o->x = x;
  o->y = y;
  o->f = f;
  o->n = n;
  o->d_off = L.d_off;
  o->ds = L.ds;
  o->unit_begin = unit_begin;
  o->k = (int32_t)k;
  o->ku = (int32_t)(k / e);
  o->sc_off = 0;
  o->yt = yt;
  return n * (k / e);
}

hipError_t launch_gemv_m1_multi(int32_t type, int32_t xt, int ns, const M1Op *dev_ops, int nops,
                                int64_t units, int64_t rows, hipStream_t s) {
  if (type == EB_Q6_S) return launch_gemv_q6_multi(xt, ns, dev_ops, nops, units, rows, s);
  if (type == EB_Q4_0) {
    if (xt == EB_F16) return launch_multi_q<EB_Q4_0, EB_F16>(dev_ops, nops, units, rows, ns, s);
    return launch_multi_q<EB_Q4_0, EB_BF16>(dev_ops, nops, units, rows, ns, s);
  }
  if (xt == EB_F16) return launch_multi_q<EB_Q8_0, EB_F16>(dev_ops, nops, units, rows, ns, s);
  return launch_multi_q<EB_Q8_0, EB_BF16>(dev_ops, nops, units, rows, ns, s);
}

hipError_t launch_gemv(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                       int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  if (type == EB_Q6_S) return launch_gemv_q6(wdata, n, k, x, xt, m, y, yt, f, s);
  if (type == EB_Q4_0) {
    if (xt == EB_F16) return launch_m<EB_Q4_0, EB_F16>(wdata, n, k, x, m, y, yt, f, s);
    return launch_m<EB_Q4_0, EB_BF16>(wdata, n, k, x, m, y, yt, f, s);
  }
  if (xt == EB_F16) return launch_m<EB_Q8_0, EB_F16>(wdata, n, k, x, m, y, yt, f, s);
  return launch_m<EB_Q8_0, EB_BF16>(wdata, n, k, x, m, y, yt, f, s);
}

}  // namespace eb
