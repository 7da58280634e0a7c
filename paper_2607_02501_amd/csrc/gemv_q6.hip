// gemv_q6.hip -- batch-1 / few-row (m <= 8) linear layers on Q6_S weights:
// the bandwidth-bound decode case of the 6-bit configuration (paper section
// 4, Table 3; section 3.2, latency-first batch-1 execution).
//
// m == 1 (the decode step): a 64-weight unit is two consecutive 24-byte code
// chunks, 48 bytes at offset 48 u of the row, the four sub-block scales of
// those chunks (one 4-byte word) and their super-block's d16.  Lane l of a
// wave owns units l, l + 64, ... of the wave's rows.  A wave reads the 3 KiB
// of codes of 64 units with three fully coalesced 16-byte loads per lane (1
// KiB contiguous per instruction; a lane's own 48 bytes, read directly, would
// make each instruction touch 3 KiB in 16-byte pieces, which measured 25%
// slower) and hands each lane its unit through a wave-private 3 KiB LDS
// buffer.  The codes are decoded in
// registers into binary16 pairs (low nibble and the two top bits placed into
// the mantissa of 1024, or one nibble higher into 1024 + 16 u; one packed
// subtraction leaves u - 32 or 16 (u - 32) exactly) and multiplied with
// v_dot2_f32_f16 against x, staged once per workgroup into LDS in the
// decoder's pair order; each 16-weight sub-block sum is then scaled by
// e_j = d16 sc_j (exact in fp32).  bfloat16 x takes bfloat16 128 as the magic
// value (128 + u = c + 160) and removes 160 * (sum of the sub-block's x),
// precomputed in binary64 at staging.  One launch per matrix, or one
// persistent launch for a run of independent matrices.
//
// m = 2 .. 8: a wave owns a pair of weight rows (so a gate/up pair's product
// is formed in the wave) and its lanes walk the rows' 24-byte code chunks (32
// weights each) in lane order: one wave load covers 64 consecutive chunks of a
// row, 1536 contiguous bytes, read as three 8-byte loads per lane.  A chunk
// decodes to u = low nibble | top bits << 4, and the lane accumulates
// (u - 32) x in fp32 per 16-weight sub-block (every product exact: 6-bit code
// times 16-bit activation), then e_j times that sum (e_j = d16 sc_j, exact in
// fp32) into its row sum; the wave's lanes are added by a butterfly.  x (all
// m rows, normalised first when the op has the RMS-normalisation prologue)
// is staged in LDS as 16-bit values by the whole workgroup.
#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"
#include "gemv_common.h"

namespace eb {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;

__device__ inline float x_to_f32(uint16_t v, int xt) {
  return xt == EB_F16 ? (float)__builtin_bit_cast(_Float16, v) : __uint_as_float((uint32_t)v << 16);
}

__device__ inline uint16_t f32_to_x(float v, int xt) {
  return xt == EB_F16 ? __builtin_bit_cast(uint16_t, (_Float16)v) : __builtin_bit_cast(uint16_t, (__bf16)v);
}

// Stage the MT rows of x (rows past m as zeros) into xs[MT][k] as 16-bit
// values of type xt; with the prologue, x is the fp32 stream h and each row is
// normalised: r = 1 / sqrt(sum h^2 / k + eps) (each thread's columns
// j = t, t + 512, ... summed in order, then the 64 lanes of a wave, then the
// waves in order), x_hat = round(h g r).
template <int MT>
__device__ void stage_q6(const void *x, int64_t m, int64_t k, int xt, const Fuse &f, uint16_t *xs,
                         float *red) {
  const int t = threadIdx.x;
  if (f.pro == EB_PRO_RMSNORM) {
    const float *h = static_cast<const float *>(x);
    for (int mm = 0; mm < MT; ++mm) {
      if (mm >= m) {
        for (int64_t j = t; j < k; j += kThreads) xs[mm * k + j] = 0;
        continue;
      }
      float ss = 0.f;
      for (int64_t j = t; j < k; j += kThreads) {
        const float v = h[mm * k + j];
        ss = __builtin_fmaf(v, v, ss);
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
      __syncthreads();  // red is reused row after row
      if ((t & 63) == 0) red[t >> 6] = ss;
      __syncthreads();
      float tot = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) tot += red[w];
      const float r = 1.0f / __builtin_sqrtf(tot / (float)k + f.eps);
      for (int64_t j = t; j < k; j += kThreads) xs[mm * k + j] = f32_to_x(h[mm * k + j] * f.gamma[j] * r, xt);
    }
  } else {
    // 16-byte pieces (k is a multiple of 256, so a row is a whole number of them)
    const uint4 *src = static_cast<const uint4 *>(x);
    uint4 *dst = reinterpret_cast<uint4 *>(xs);
    const int64_t per_row = k / 8;
    for (int64_t i = t; i < MT * per_row; i += kThreads)
      dst[i] = (i / per_row < m) ? src[i] : make_uint4(0, 0, 0, 0);
  }
  __syncthreads();
}

// u codes of a chunk, 4 per word: word w holds weights 4w .. 4w + 3.
__device__ inline void decode_chunk(const uint2 a, const uint2 b, const uint2 c, uint32_t u[8]) {
  const uint32_t L0 = a.x, L1 = a.y, L2 = b.x, L3 = b.y, H0 = c.x, H1 = c.y;
  constexpr uint32_t N = 0x0f0f0f0fu, T = 0x03030303u;
  u[0] = (L0 & N) | ((H0 & T) << 4);
  u[1] = (L1 & N) | ((H1 & T) << 4);
  u[2] = (L2 & N) | (((H0 >> 2) & T) << 4);
  u[3] = (L3 & N) | (((H1 >> 2) & T) << 4);
  u[4] = ((L0 >> 4) & N) | (((H0 >> 4) & T) << 4);
  u[5] = ((L1 >> 4) & N) | (((H1 >> 4) & T) << 4);
  u[6] = ((L2 >> 4) & N) | (((H0 >> 6) & T) << 4);
  u[7] = ((L3 >> 4) & N) | (((H1 >> 6) & T) << 4);
}

// sum over 4 weights of word w: (u - 32) x, x from 4 consecutive 16-bit values
// (each byte to float is one v_cvt_f32_ubyte; u - 32 and the product are exact)
__device__ inline float dot4(uint32_t w, uint2 xv, int xt, float acc) {
  const float x0 = x_to_f32((uint16_t)(xv.x & 0xffffu), xt), x1 = x_to_f32((uint16_t)(xv.x >> 16), xt);
  const float x2 = x_to_f32((uint16_t)(xv.y & 0xffffu), xt), x3 = x_to_f32((uint16_t)(xv.y >> 16), xt);
  acc = __builtin_fmaf((float)((w >> 0) & 0xffu) - 32.0f, x0, acc);
  acc = __builtin_fmaf((float)((w >> 8) & 0xffu) - 32.0f, x1, acc);
  acc = __builtin_fmaf((float)((w >> 16) & 0xffu) - 32.0f, x2, acc);
  acc = __builtin_fmaf((float)((w >> 24) & 0xffu) - 32.0f, x3, acc);
  return acc;
}

template <int MT>
__global__ void __launch_bounds__(kThreads)
    gemv_q6_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t sc_off,
                   int64_t d_off, int64_t ds, const void *__restrict__ x, int64_t m, int xt,
                   void *__restrict__ y, int yt, Fuse f) {
  extern __shared__ uint16_t xs[];  // [MT][k]
  __shared__ float red[kWaves];
  stage_q6<MT>(x, m, k, xt, f, xs, red);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t pair = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t r0 = 2 * pair;
  if (r0 >= n) return;
  const bool two = r0 + 1 < n;
  const int64_t nc = k / kQK;              // chunks per row
  const int64_t qrow = nc * 24, srow = k / 16;
  float acc[2][MT];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) acc[rr][mm] = 0.f;

  for (int64_t c = lane; c < nc; c += 64) {
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      if (rr == 1 && !two) break;
      const int64_t row = r0 + rr;
      const uint2 *q = reinterpret_cast<const uint2 *>(wdata + row * qrow + c * 24);
      const uint2 a = q[0], b = q[1], h = q[2];
      const uint16_t sc2 = *reinterpret_cast<const uint16_t *>(wdata + sc_off + row * srow + 2 * c);
      const uint16_t d16 = *reinterpret_cast<const uint16_t *>(wdata + d_off + (row * ds + c / 8) * 2);
      const float d = (float)__builtin_bit_cast(_Float16, d16);
      const float e0 = d * (float)(int8_t)(sc2 & 0xff), e1 = d * (float)(int8_t)(sc2 >> 8);  // exact
      uint32_t u[8];
      decode_chunk(a, b, h, u);
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        const uint4 *xv = reinterpret_cast<const uint4 *>(xs + mm * k + c * 32);
        const uint4 x0 = xv[0], x1 = xv[1], x2 = xv[2], x3 = xv[3];
        // weights 0..15 (sub-block 2c), then 16..31 (sub-block 2c + 1)
        float s0 = 0.f, s1 = 0.f;
        s0 = dot4(u[0], make_uint2(x0.x, x0.y), xt, s0);
        s0 = dot4(u[1], make_uint2(x0.z, x0.w), xt, s0);
        s0 = dot4(u[2], make_uint2(x1.x, x1.y), xt, s0);
        s0 = dot4(u[3], make_uint2(x1.z, x1.w), xt, s0);
        s1 = dot4(u[4], make_uint2(x2.x, x2.y), xt, s1);
        s1 = dot4(u[5], make_uint2(x2.z, x2.w), xt, s1);
        s1 = dot4(u[6], make_uint2(x3.x, x3.y), xt, s1);
        s1 = dot4(u[7], make_uint2(x3.z, x3.w), xt, s1);
        acc[rr][mm] = __builtin_fmaf(e0, s0, acc[rr][mm]);
        acc[rr][mm] = __builtin_fmaf(e1, s1, acc[rr][mm]);
      }
    }
  }
#pragma unroll
  for (int rr = 0; rr < 2; ++rr)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm)
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) acc[rr][mm] += __shfl_xor(acc[rr][mm], o);
  if (lane != 0) return;
  if (f.epi == EB_EPI_ADD) {  // the residuals read together
    uint32_t rel[2 * MT];
    bool ok[2 * MT];
    float v[2 * MT];
#pragma unroll
    for (int mm = 0; mm < MT; ++mm)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        rel[2 * mm + t] = (uint32_t)mm * (uint32_t)n + t;
        ok[2 * mm + t] = mm < m && (t == 0 || two);
        v[2 * mm + t] = acc[t][mm];
      }
    if (put_y_add(y, f.r, r0, (int64_t)(m - 1) * n + 2, rel, ok, v, yt)) return;
  }
  for (int mm = 0; mm < MT && mm < m; ++mm) {
    if (f.epi == EB_EPI_GLU) {  // n even: rows r0, r0 + 1 are a gate/up pair
      store_y(y, (int64_t)mm * (n / 2) + pair, silu_mul(acc[0][mm], acc[1][mm]), yt);
      continue;
    }
    put_y(y, (int64_t)mm * n + r0, acc[0][mm], yt, f);
    if (two) put_y(y, (int64_t)mm * n + r0 + 1, acc[1][mm], yt, f);
  }
}

// ---------------------------------------------------------------------------
// m == 1
// ---------------------------------------------------------------------------

constexpr int kU6 = 64;         // weights per unit (two code chunks)
constexpr int kU6Bytes = 48;    // code bytes per unit
constexpr int kU6Parts = 8;     // 16-byte x parts per unit (4 per chunk)
constexpr int kQ6M1MaxSlots = 4;  // units per lane: k <= 64 * 64 * 4

// Rows per wave of the fused launch by slot count (no spills at 4 waves per
// SIMD); the one-matrix launch adds its rows in the same order, so both agree
// bitwise (reduce_rows gives a row the same association for every R).
__host__ __device__ constexpr int q6_multi_rows(int ns) { return ns <= 2 ? 2 : 1; }

// Sub-block sums of one 32-weight chunk: sa over weights 0..15, sb over
// 16..31.  L: the 16 low-nibble bytes (byte t: weight t in bits 0..3, weight
// t + 16 in bits 4..7); H: the 8 top-bit bytes (byte t: top bits of weights
// t, t + 8, t + 16, t + 24 at bit 0, 2, 4, 6).  Word i of L covers weights
// 4i .. 4i + 3 and 4i + 16 .. 4i + 19, whose top bits sit in top-bit word
// i & 1 at shift 2 (i >> 1) and 2 (i >> 1) + 4.  x part i holds the x pairs
// (4i, 4i+2) (4i+1, 4i+3) (4i+16, 4i+18) (4i+17, 4i+19).
template <int XT>
__device__ inline void chunk_dot6(const uint32_t (&L)[4], uint32_t H0, uint32_t H1, const uint4 *xf,
                                  float offa, float offb, float &sa, float &sb) {
  float lo = 0.f, hi = 0.f;
  if constexpr (XT == EB_F16) {
    const uint32_t magic = vconst(0x64006400u);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t h = (i & 1) ? H1 : H0;
      // top bits of the even / odd bytes' weights moved to bits 4..5 (and,
      // for the weights 16 further on, 8..9) of the 16-bit lanes
      const uint32_t te = (i < 2) ? h << 4 : h << 2, to = (i < 2) ? h >> 4 : h >> 6;
      const uint32_t v = L[i], v8 = L[i] >> 8;
      // 1024 + u - 1056 = u - 32;  1024 + 16 u - 1536 = 16 (u - 32)
      lo = dot2h(sub_h2(and_or(te, 0x00300030u, and_or(v, 0x000F000Fu, magic)), (_Float16)1056.0f),
                 xf[i].x, lo);
      lo = dot2h(sub_h2(and_or(to, 0x00300030u, and_or(v8, 0x000F000Fu, magic)), (_Float16)1056.0f),
                 xf[i].y, lo);
      hi = dot2h(sub_h2(and_or(te, 0x03000300u, and_or(v, 0x00F000F0u, magic)), (_Float16)1536.0f),
                 xf[i].z, hi);
      hi = dot2h(sub_h2(and_or(to, 0x03000300u, and_or(v8, 0x00F000F0u, magic)), (_Float16)1536.0f),
                 xf[i].w, hi);
    }
    (void)offa;
    (void)offb;
    sa = lo;
    sb = hi * 0.0625f;  // exact
  } else {
    const uint32_t magic = vconst(0x43004300u);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t h = (i & 1) ? H1 : H0;
      const int s = 2 * (i >> 1);
      const uint32_t v = L[i];
      // every code at bits 0..5: bfloat16 128 + u
      lo = dot2bf(and_or(h << (4 - s), 0x00300030u, and_or(v, 0x000F000Fu, magic)), xf[i].x, lo);
      lo = dot2bf(and_or(h >> (4 + s), 0x00300030u, and_or(v >> 8, 0x000F000Fu, magic)), xf[i].y, lo);
      hi = dot2bf(and_or(h >> s, 0x00300030u, and_or(v >> 4, 0x000F000Fu, magic)), xf[i].z, hi);
      hi = dot2bf(and_or(h >> (8 + s), 0x00300030u, and_or(v >> 12, 0x000F000Fu, magic)), xf[i].w, hi);
    }
    sa = lo - offa;
    sb = hi - offb;
  }
}

// Stage x (one row) into LDS for q6_rows: part p of unit u at xs[p * P + u]
// (p = 4 h + i: chunk h of the unit, word i), and with bfloat16 x the four
// sub-block offsets 160 * sum x of unit u at xoff[4 u .. 4 u + 3].  One thread
// per part; with the normalisation prologue x is the fp32 stream h, the
// thread's first part's h values stay in registers between the sum of squares
// and the normalisation, and the sum is reduced over the wave by exchanges and
// over the waves in order through `red` (one float per wave).
//
// Two phases: x6_issue loads the thread's first part (h and gamma), or the
// raw 16-bit values of its first two, into registers, and x6_finish stages
// them with the rest.  The caller issues its first weight loads in between:
// vector-memory loads complete in issue order, so waiting for activations
// loaded after the weights would wait for all of those weights.
struct X6Regs {
  // normalisation prologue: h[e0..e0+3], h[e0+16..e0+19] and gamma there,
  // for the thread's first part; otherwise the raw 8-byte halves of its first
  // two parts (a = {part 0 at e0, part 1 at e0}, b likewise at e0 + 16)
  uint4 a, b, ga, gb;
};

__device__ __attribute__((always_inline)) inline void x6_part(int c, int &u, int &p, int &e0) {
  u = c >> 3;
  p = c & 7;
  e0 = u * kU6 + (p >> 2) * 32 + 4 * (p & 3);  // e1 = e0 + 16
}

__device__ __attribute__((always_inline)) inline void x6_issue(const void *__restrict__ xv, int ku, bool norm,
                                                               const float *__restrict__ gamma, X6Regs &R) {
  const int nch = ku * kU6Parts, T = (int)blockDim.x, tid = (int)threadIdx.x;
  int u, p, e0;
  if (norm) {
    if (tid < nch) {
      x6_part(tid, u, p, e0);
      const float *h = static_cast<const float *>(xv);
      R.a = *reinterpret_cast<const uint4 *>(h + e0);
      R.b = *reinterpret_cast<const uint4 *>(h + e0 + 16);
      R.ga = *reinterpret_cast<const uint4 *>(gamma + e0);
      R.gb = *reinterpret_cast<const uint4 *>(gamma + e0 + 16);
    }
  } else {
    const uint16_t *x = static_cast<const uint16_t *>(xv);
    if (tid < nch) {
      x6_part(tid, u, p, e0);
      const uint2 ra = *reinterpret_cast<const uint2 *>(x + e0), rb = *reinterpret_cast<const uint2 *>(x + e0 + 16);
      R.a.x = ra.x, R.a.y = ra.y, R.b.x = rb.x, R.b.y = rb.y;
    }
    if (tid + T < nch) {
      x6_part(tid + T, u, p, e0);
      const uint2 ra = *reinterpret_cast<const uint2 *>(x + e0), rb = *reinterpret_cast<const uint2 *>(x + e0 + 16);
      R.a.z = ra.x, R.a.w = ra.y, R.b.z = rb.x, R.b.w = rb.y;
    }
  }
}

template <int XT>
__device__ __attribute__((always_inline)) inline void x6_finish(
    const void *__restrict__ xv, int64_t k, int ku, uint4 *xs, float *xoff, int P, bool norm,
    const float *__restrict__ gamma, float eps, float *red, const X6Regs &R) {
  const int nch = ku * kU6Parts, T = (int)blockDim.x, tid = (int)threadIdx.x;
  // pairs (a0,a2) (a1,a3) (b0,b2) (b1,b3), and the offsets' partial sums
  auto put = [&](int c, int u, int p, const uint32_t (&ra)[2], const uint32_t (&rb)[2])
      __attribute__((always_inline)) {
    xs[p * P + u] = make_uint4((ra[0] & 0xffffu) | (ra[1] << 16), (ra[0] >> 16) | (ra[1] & 0xffff0000u),
                               (rb[0] & 0xffffu) | (rb[1] << 16), (rb[0] >> 16) | (rb[1] & 0xffff0000u));
    if constexpr (XT == EB_BF16) {
      double sa = 0.0, sb = 0.0;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        sa += x_to_f64<XT>(ra[j] & 0xffffu) + x_to_f64<XT>(ra[j] >> 16);
        sb += x_to_f64<XT>(rb[j] & 0xffffu) + x_to_f64<XT>(rb[j] >> 16);
      }
      // the four parts of a chunk are four consecutive lanes
      sa += __shfl_xor(sa, 1);
      sb += __shfl_xor(sb, 1);
      sa += __shfl_xor(sa, 2);
      sb += __shfl_xor(sb, 2);
      if ((c & 3) == 0) {
        xoff[4 * u + 2 * (p >> 2)] = (float)(160.0 * sa);
        xoff[4 * u + 2 * (p >> 2) + 1] = (float)(160.0 * sb);
      }
    }
  };
  auto f4 = [](uint4 v) __attribute__((always_inline)) {
    return make_float4(__builtin_bit_cast(float, v.x), __builtin_bit_cast(float, v.y),
                       __builtin_bit_cast(float, v.z), __builtin_bit_cast(float, v.w));
  };
  // The offsets' exchanges stay within the four consecutive lanes of a
  // chunk's parts, which are all in or all out of each phase below (nch is a
  // multiple of 8, T of 64).
  if (!norm) {
    const uint16_t *x = static_cast<const uint16_t *>(xv);
    int u, p, e0;
    if (tid < nch) {
      x6_part(tid, u, p, e0);
      const uint32_t ra[2] = {R.a.x, R.a.y}, rb[2] = {R.b.x, R.b.y};
      put(tid, u, p, ra, rb);
    }
    if (tid + T < nch) {
      x6_part(tid + T, u, p, e0);
      const uint32_t ra[2] = {R.a.z, R.a.w}, rb[2] = {R.b.z, R.b.w};
      put(tid + T, u, p, ra, rb);
    }
    for (int c = tid + 2 * T; c < nch; c += T) {
      x6_part(c, u, p, e0);
      const uint2 a = *reinterpret_cast<const uint2 *>(x + e0);
      const uint2 b = *reinterpret_cast<const uint2 *>(x + e0 + 16);
      const uint32_t ra[2] = {a.x, a.y}, rb[2] = {b.x, b.y};
      put(c, u, p, ra, rb);
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
    int u, p, e0;
    x6_part(c, u, p, e0);
    ss = sq(sq(ss, *reinterpret_cast<const float4 *>(h + e0)), *reinterpret_cast<const float4 *>(h + e0 + 16));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (T >> 6); ++w) tot += red[w];
  const float r = 1.0f / __builtin_sqrtf(tot / (float)k + eps);
  auto normed = [&](float4 v, float4 gg, uint32_t (&o)[2]) __attribute__((always_inline)) {
    o[0] = pack_x16<XT>(v.x * gg.x * r, v.y * gg.y * r);
    o[1] = pack_x16<XT>(v.z * gg.z * r, v.w * gg.w * r);
  };
  if (tid < nch) {
    int u, p, e0;
    x6_part(tid, u, p, e0);
    uint32_t ra[2], rb[2];
    normed(f4(R.a), f4(R.ga), ra);
    normed(f4(R.b), f4(R.gb), rb);
    put(tid, u, p, ra, rb);
  }
  for (int c = tid + T; c < nch; c += T) {
    int u, p, e0;
    x6_part(c, u, p, e0);
    uint32_t ra[2], rb[2];
    normed(*reinterpret_cast<const float4 *>(h + e0), *reinterpret_cast<const float4 *>(gamma + e0), ra);
    normed(*reinterpret_cast<const float4 *>(h + e0 + 16), *reinterpret_cast<const float4 *>(gamma + e0 + 16), rb);
    put(c, u, p, ra, rb);
  }
}

// LDS of q6_rows: 8 x part rows of P entries, the bfloat16 offsets (4 P
// floats), a 3 KiB code buffer per wave and one float per wave for the
// normalisation's reduction.
constexpr int kU6WaveBuf = 64 * kU6Bytes / 16;  // uint4 entries per wave
__host__ __device__ constexpr size_t q6_m1_lds(int ns, int waves) {
  return (size_t)kU6Parts * (64 * ns + 1) * 16 + (size_t)4 * (64 * ns + 1) * 4 +
         (size_t)waves * kU6WaveBuf * 16 + (size_t)waves * 4;
}

// Rows g*R .. g*R+R-1 for the wave's groups g in [gbase, g_end) of one
// matrix, m == 1: gbase + vb, + gstride, ... in the whole rounds of gstride
// groups, and gbase + (whole rounds) gstride + vw in the last, partial one
// (vb and vw number the gstride waves; callers that pass vb == vw walk
// gbase + vb + i gstride).  Called by every thread of the workgroup (it stages
// x into LDS and synchronises once); waves without a group only help with the
// staging.
// Items in flight per wave for a group of `items` items: the largest divisor
// of it up to `cap`.
__host__ __device__ constexpr int q6_ring(int items, int cap) {
  int d = items < cap ? items : cap;
  while (items % d) --d;
  return d;
}
constexpr int kQ6Ring = 1;

// PRE (residual-adding ops with fp32 output): each lane's row residual is
// loaded before the group's weights, as in m1_rows.
template <int XT, int NS, int R, int RING, bool PRE = false>
__device__ __attribute__((always_inline)) inline void q6_rows(
    const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t sc_off, int64_t d_off,
    int64_t ds, const void *__restrict__ x, void *__restrict__ y, int yt, const Fuse &f, int64_t gbase,
    int64_t vb, int64_t vw, int64_t g_end, int64_t gstride, uint4 *smem) {
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
  // entry 64 * NS of every part row (and its offsets) is zero and stands in
  // for units past the end of the row
  constexpr int P = 64 * NS + 1;
  const int ku = (int)(k / kU6);  // 64 * (NS - 1) < ku <= 64 * NS
  uint4 *xs = smem;
  float *xoff = reinterpret_cast<float *>(smem + kU6Parts * P);
  uint4 *cbuf = reinterpret_cast<uint4 *>(xoff + 4 * P);  // [waves][192]
  float *red = reinterpret_cast<float *>(cbuf + (blockDim.x >> 6) * kU6WaveBuf);
  const int lane = threadIdx.x & 63;
  uint4 *wbuf = cbuf + (threadIdx.x >> 6) * kU6WaveBuf;
  const uint32_t q_row = (uint32_t)ku * kU6Bytes, s_row = (uint32_t)(k / 16), d_row = (uint32_t)(ds * 2);
  const uint8_t *__restrict__ sbase = wdata + sc_off;
  const uint8_t *__restrict__ dbase = wdata + d_off;

  // Per-lane byte offsets inside a row: the lane's 16-byte pieces of slot
  // s's 3 KiB of codes at 3072 s + 16 lane (+ 1024, + 2048; loads past the
  // row's end return zeros), and its unit's scales.  Only the last slot can
  // pass the end of the row (ku > 64 (NS - 1)): its units read the row's
  // last unit's scales and meet zero x.  The other slots' offsets are the
  // lane's base plus a constant.
  const int ul = lane + 64 * (NS - 1), ulc = min(ul, ku - 1);
  const uint32_t slast = (uint32_t)ulc * 4u, dlast = (uint32_t)(ulc >> 2) * 2u;
  const uint32_t xlast = ul < ku ? (uint32_t)ul : 64u * NS;
  const uint32_t qbase = 16u * lane, sbase_l = 4u * lane, dbase_l = (uint32_t)(lane >> 2) * 2u;

  // A ring of D register sets for the NS R items of a group (item i = slot
  // s of row r, i = s R + r: 48 code bytes, 4 sub-scales and the super-block
  // scale of the lane's unit; 3 KiB per wave).  Item i lives in set i % D;
  // right after it has been used, its set is reloaded with item i + D, of
  // this group or of the wave's next one, so a wave keeps D items of reads in
  // flight without pauses while it decodes.  A group past g_end gets
  // zero-sized buffer ranges (its loads return zeros without a memory
  // access), so every load is issued on every path: a load issued on only
  // some paths makes the compiler's counter wait for an earlier load a wait
  // for everything.
  constexpr int I = NS * R, D = q6_ring(I, RING);
  struct Item {
    uint4 a, b, c;
    uint32_t sc;
    uint16_t dh;
  };
  Item ring[D];
  struct GRes {
    __amdgpu_buffer_rsrc_t q[R], s[R], d[R];
  };
  auto group_res = [&](int64_t grp, GRes &G) __attribute__((always_inline)) {
    const bool live = grp < g_end;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      int64_t row = grp * R + r;
      row = row < n ? row : n - 1;  // tail rows are computed but not stored
      G.q[r] = rsrc(wdata + row * q_row, live ? q_row : 0u);
      G.s[r] = rsrc(sbase + row * s_row, live ? s_row : 0u);
      G.d[r] = rsrc(dbase + row * d_row, live ? d_row : 0u);
    }
  };
  auto load_item = [&](Item &it, const GRes &G, int i) __attribute__((always_inline)) {
    const int s = i / R, r = i % R;
    const bool last = s == NS - 1;
    const auto va = __builtin_amdgcn_raw_buffer_load_b128(G.q[r], (int)qbase, 3072 * s, kNT);
    const auto vb = __builtin_amdgcn_raw_buffer_load_b128(G.q[r], (int)qbase, 3072 * s + 1024, kNT);
    const auto vc = __builtin_amdgcn_raw_buffer_load_b128(G.q[r], (int)qbase, 3072 * s + 2048, kNT);
    it.a = make_uint4(va[0], va[1], va[2], va[3]);
    it.b = make_uint4(vb[0], vb[1], vb[2], vb[3]);
    it.c = make_uint4(vc[0], vc[1], vc[2], vc[3]);
    it.sc = __builtin_amdgcn_raw_buffer_load_b32(G.s[r], (int)(last ? slast : sbase_l), last ? 0 : 256 * s, kNT);
    it.dh = __builtin_amdgcn_raw_buffer_load_b16(G.d[r], (int)(last ? dlast : dbase_l), last ? 0 : 32 * s, kNT);
  };
  // x's loads first, then the first group's weights, which stay in flight
  // while x is staged (and, with the prologue, normalised)
  const bool norm = f.pro == EB_PRO_RMSNORM;
  X6Regs xr;
  x6_issue(x, ku, norm, f.gamma, xr);
  __builtin_amdgcn_sched_barrier(0);
  // PRE: the first group's residual before its weights, each next group's
  // right after this group's output (older than every load issued while its
  // group is decoded); a group past g_end reads zero without a memory access
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
  {
    // in the order step consumes them, kept in that order (left to the
    // scheduler, the scales would follow all the codes and the first item's
    // wait would be a wait for the whole group)
    GRes G;
    group_res(g, G);
#pragma unroll
    for (int i = 0; i < D; ++i) {
      load_item(ring[i], G, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  x6_finish<XT>(x, k, ku, xs, xoff, P, norm, f.gamma, f.eps, red, xr);
  if (threadIdx.x < kU6Parts) xs[threadIdx.x * P + 64 * NS] = make_uint4(0, 0, 0, 0);
  if (threadIdx.x < 4) xoff[4 * 64 * NS + threadIdx.x] = 0.f;
  __syncthreads();

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
      uint4 xf[kU6Parts];
#pragma unroll
      for (int p = 0; p < kU6Parts; ++p) xf[p] = xs[p * P + xi];
      float4 xo = make_float4(0.f, 0.f, 0.f, 0.f);
      if constexpr (XT == EB_BF16) xo = reinterpret_cast<const float4 *>(xoff)[xi];
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = s * R + r;
        Item &it = ring[i % D];
        const float d = (float)__builtin_bit_cast(_Float16, it.dh);
        const uint32_t sc = it.sc;
        // pieces l, l + 64, l + 128 of the wave's 3 KiB in, the lane's own
        // unit (pieces 3 l .. 3 l + 2) out; a wave's LDS operations complete
        // in order, so the reads see the writes and the next writes follow
        // the reads
        wbuf[lane] = it.a;
        wbuf[lane + 64] = it.b;
        wbuf[lane + 128] = it.c;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const uint4 qa = wbuf[3 * lane], qb = wbuf[3 * lane + 1], qc = wbuf[3 * lane + 2];
        __builtin_amdgcn_wave_barrier();
        const uint32_t L0[4] = {qa.x, qa.y, qa.z, qa.w}, L1[4] = {qb.z, qb.w, qc.x, qc.y};
        float s0, s1, s2, s3;
        chunk_dot6<XT>(L0, qb.x, qb.y, xf, xo.x, xo.y, s0, s1);
        chunk_dot6<XT>(L1, qc.z, qc.w, xf + 4, xo.z, xo.w, s2, s3);
        // e_j = d16 sc_j: a 11-bit by 8-bit product, exact in fp32
        acc[r] = __builtin_fmaf(d * (float)(int8_t)(sc & 0xffu), s0, acc[r]);
        acc[r] = __builtin_fmaf(d * (float)(int8_t)((sc >> 8) & 0xffu), s1, acc[r]);
        acc[r] = __builtin_fmaf(d * (float)(int8_t)((sc >> 16) & 0xffu), s2, acc[r]);
        acc[r] = __builtin_fmaf(d * (float)(int8_t)(sc >> 24), s3, acc[r]);
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
    if constexpr (PRE) {
      // put_y's arithmetic: the fp32 sum, then the fp32 store
      if (writer && row < n) store_y(y, row, tot + res_cur, EB_F32);
      res_cur = res_load(gnext);
    } else if constexpr (R >= 2) {
      if (f.epi == EB_EPI_GLU) {
        // the up row (odd) of a pair is held R/2 ... lanes away, see reduce_rows
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

// One matrix per launch: one workgroup per CU (x is staged, and normalised,
// once per CU) of 16 waves, or 8 where a wave's weights and x parts would not
// fit the registers of four waves per SIMD without spilling (measured: up to
// 3 slots, 4 slot-rows).
__host__ __device__ constexpr int q6_m1_waves(int ns, int r) { return ns <= 3 && ns * r <= 4 ? 16 : 8; }

template <int XT, int NS, int R, int WG, bool PRE>
__global__ void __launch_bounds__(64 * WG) __attribute__((amdgpu_waves_per_eu(WG / 4)))
    gemv_q6_m1_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t sc_off,
                      int64_t d_off, int64_t ds, const void *__restrict__ x, void *__restrict__ y,
                      int yt, Fuse f) {
  extern __shared__ uint4 smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // group numbering as in gemv_m1_kernel
  q6_rows<XT, NS, R, kQ6Ring, PRE>(wdata, n, k, sc_off, d_off, ds, x, y, yt, f, 0,
                              (int64_t)blockIdx.x * WG + wave, (int64_t)wave * gridDim.x + blockIdx.x,
                              (n + R - 1) / R, (int64_t)gridDim.x * WG, smem);
}

// Several independent matrices (m == 1, same activation type, same slot count
// NS) in one persistent launch: the launch's units (rows weighted by their
// length) are cut into gridDim.x equal shares, each converted to whole R-row
// groups of the matrices it covers (neighbours round a shared boundary the
// same way, so every row is computed once).
constexpr int kQ6MultiWaves = 4;

template <int XT, int NS>
__global__ void __launch_bounds__(64 * kQ6MultiWaves) __attribute__((amdgpu_waves_per_eu(NS <= 1 ? 4 : 3)))
    gemv_q6_m1_multi_kernel(const M1Op *__restrict__ ops, int nops, int64_t units) {
  constexpr int R = q6_multi_rows(NS);
  extern __shared__ uint4 smem[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t G = gridDim.x;
  const int64_t u0 = units * (int64_t)blockIdx.x / G, u1 = units * ((int64_t)blockIdx.x + 1) / G;
  int lo = 0, hi = nops - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (ops[mid].unit_begin <= u0) lo = mid; else hi = mid - 1;
  }
  for (int op = lo; op < nops && ops[op].unit_begin < u1; ++op) {
    const M1Op o = ops[op];
    auto row_at = [&](int64_t u) {
      int64_t r = (u - o.unit_begin) / o.ku;
      r = r < 0 ? 0 : (r > o.n ? o.n : r);
      return r == o.n ? r : r / R * R;
    };
    const int64_t r0 = row_at(u0), r1 = row_at(u1);
    if (r0 >= r1) continue;  // uniform across the workgroup
    q6_rows<XT, NS, R, NS * R>(o.w, o.n, o.k, o.sc_off, o.d_off, o.ds, o.x, o.y, o.yt, o.f, r0 / R, wave, wave,
                          (r1 + R - 1) / R, kQ6MultiWaves, smem);
    __syncthreads();  // the next matrix restages LDS
  }
}

template <int XT, int NS>
hipError_t launch_m1_ns(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                        const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(EB_Q6_S, n, k);
  const int r = f.epi == EB_EPI_GLU ? 2 : 1;  // the gate/up product needs both rows in one wave
  const int wg = r == 2 ? q6_m1_waves(NS, 2) : q6_m1_waves(NS, 1);
  const int64_t groups = (n + r - 1) / r;
  int64_t grid = (groups + wg - 1) / wg;
  const int64_t cap = (int64_t)device_cu_count();
  if (grid > cap) grid = cap;
  const size_t lds = q6_m1_lds(NS, wg);
  // residual-adding ops with fp32 output preload their residuals
  const bool pre = f.epi == EB_EPI_ADD && yt == EB_F32;
  auto kern = r == 2 ? gemv_q6_m1_kernel<XT, NS, 2, q6_m1_waves(NS, 2), false>
                     : (pre ? gemv_q6_m1_kernel<XT, NS, 1, q6_m1_waves(NS, 1), true>
                            : gemv_q6_m1_kernel<XT, NS, 1, q6_m1_waves(NS, 1), false>);
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<(unsigned)grid, 64 * wg, lds, s>>>((const uint8_t *)wdata, n, k, L.sc_off, L.d_off, L.ds, x,
                                           y, yt, f);
  return hipGetLastError();
}

template <int XT>
hipError_t launch_m1(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                     const Fuse &f, hipStream_t s) {
  switch (q6_m1_slots(k)) {
    case 1: return launch_m1_ns<XT, 1>(wdata, n, k, x, y, yt, f, s);
    case 2: return launch_m1_ns<XT, 2>(wdata, n, k, x, y, yt, f, s);
    case 3: return launch_m1_ns<XT, 3>(wdata, n, k, x, y, yt, f, s);
    default: return launch_m1_ns<XT, 4>(wdata, n, k, x, y, yt, f, s);
  }
}

template <int XT, int NS>
hipError_t launch_multi_t(const M1Op *ops, int nops, int64_t units, int64_t rows, hipStream_t s) {
  int64_t grid = (int64_t)device_cu_count() * 4;
  const int64_t groups = rows / (kQ6MultiWaves * q6_multi_rows(NS));  // keep every wave busy
  if (grid > groups) grid = groups > 0 ? groups : 1;
  gemv_q6_m1_multi_kernel<XT, NS><<<(unsigned)grid, 64 * kQ6MultiWaves, q6_m1_lds(NS, kQ6MultiWaves), s>>>(
      ops, nops, units);
  return hipGetLastError();
}

template <int XT>
hipError_t launch_multi(const M1Op *ops, int nops, int64_t units, int64_t rows, int ns, hipStream_t s) {
  switch (ns) {
    case 1: return launch_multi_t<XT, 1>(ops, nops, units, rows, s);
    case 2: return launch_multi_t<XT, 2>(ops, nops, units, rows, s);
    case 3: return launch_multi_t<XT, 3>(ops, nops, units, rows, s);
    case 4: return launch_multi_t<XT, 4>(ops, nops, units, rows, s);
    default: return hipErrorInvalidValue;
  }
}

template <int MT>
hipError_t launch_mt(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt, int64_t m,
                     void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  const Layout L = layout_of(EB_Q6_S, n, k);
  const int64_t pairs = (n + 1) / 2;
  const unsigned grid = (unsigned)((pairs + kWaves - 1) / kWaves);
  const size_t lds = (size_t)MT * k * 2;
  auto kern = gemv_q6_kernel<MT>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
  }
  kern<<<grid, kThreads, lds, s>>>(static_cast<const uint8_t *>(wdata), n, k, L.sc_off,
                                                 L.d_off, L.ds, x, m, xt, y, yt, f);
  return hipGetLastError();
}

}  // namespace

int q6_m1_slots(int64_t k) { return (int)((k / kU6 + 63) / 64); }

bool q6_m1_fits(int64_t k) { return k > 0 && k % kQK6 == 0 && q6_m1_slots(k) <= kQ6M1MaxSlots; }

bool q6_m1_fusable(int64_t k, int32_t epi) {
  return q6_m1_fits(k) && (epi != EB_EPI_GLU || q6_multi_rows(q6_m1_slots(k)) >= 2);
}

int64_t q6_m1_fill(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                   const Fuse &f, int64_t unit_begin, M1Op *o) {
  const Layout L = layout_of(EB_Q6_S, n, k);
  o->w = (const uint8_t *)wdata;
  o->x = x;
  o->y = y;
  o->f = f;
  o->n = n;
  o->d_off = L.d_off;
  o->ds = L.ds;
  o->sc_off = L.sc_off;
  o->unit_begin = unit_begin;
  o->k = (int32_t)k;
  o->ku = (int32_t)(k / kU6);
  o->yt = yt;
  return n * (k / kU6);
}

hipError_t launch_gemv_q6_multi(int32_t xt, int ns, const M1Op *dev_ops, int nops, int64_t units,
                                int64_t rows, hipStream_t s) {
  if (xt == EB_F16) return launch_multi<EB_F16>(dev_ops, nops, units, rows, ns, s);
  return launch_multi<EB_BF16>(dev_ops, nops, units, rows, ns, s);
}

bool gemv_q6_fits(int64_t m, int64_t n, int64_t k) {
  const int64_t mt = m <= 1 ? 1 : (m <= 2 ? 2 : (m <= 4 ? 4 : 8));
  return m >= 1 && m <= kGemvMaxM && mt * k <= kGemvMaxMK && k % kQK6 == 0 &&
         (n + 1) / 2 <= (int64_t)0x7fffffff * kWaves;
}

hipError_t launch_gemv_q6(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt,
                          int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s) {
  if (!gemv_q6_fits(m, n, k)) return hipErrorInvalidValue;
  if (m == 1 && q6_m1_fits(k)) {
    if (xt == EB_F16) return launch_m1<EB_F16>(wdata, n, k, x, y, yt, f, s);
    return launch_m1<EB_BF16>(wdata, n, k, x, y, yt, f, s);
  }
  if (m <= 1) return launch_mt<1>(wdata, n, k, x, xt, m, y, yt, f, s);
  if (m <= 2) return launch_mt<2>(wdata, n, k, x, xt, m, y, yt, f, s);
  if (m <= 4) return launch_mt<4>(wdata, n, k, x, xt, m, y, yt, f, s);
  return launch_mt<8>(wdata, n, k, x, xt, m, y, yt, f, s);
}

}  // namespace eb
