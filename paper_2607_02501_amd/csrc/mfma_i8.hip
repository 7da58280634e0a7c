// mfma_i8.hip -- the low-precision prefill variant (paper section 3.2,
// backend-specific dispatch) on the integer matrix cores: activations
// quantized per 32-element block along k to int8 with a binary32 scale,
// Q8_0 / Q4_0 weight codes fed to v_mfma_i32_32x32x32_i8 as they are, one
// MFMA k-step per block, and each block's exact int32 tile scaled by
// s_ib * d_nb into fp32 accumulators.
//
// Activation step (one thread per row and block):
//   s = fl32(max |x| / 127) (0 for an all-zero block),
//   xq = clamp(round_half_away(x / s), -127, 127), the quotient in binary64
// (x has at most 11 significant bits and s 24: binary64 decides every
// rounding as the exact quotient would).  Codes go to xq[m][k] (int8, row
// major), scales to xs[k/32][ms] (block major, ms = m rounded up to 4), both
// in the caller's workspace.
//
// Product kernel: a workgroup of 4 waves owns a 128 (rows of x) x 128
// (weight rows) output tile; wave (wm, wn) owns 64 x 64 of it as 2 x 2
// MFMA tiles of 32 x 32.  Per block b a lane holds, for each of its x
// sub-tiles, the 16 codes k = 32 b + 16 (lane / 32) .. + 15 of row lane % 32
// (A operand), and for each weight sub-tile the same 16 weight codes of row
// lane % 32 (B operand; Q4_0 nibbles are unpacked to int8 c - 8 in
// registers).  The int32 result (lane: weight row lane % 32, x rows
// 8 (e / 4) + 4 (lane / 32) + e % 4) is converted to fp32 and added with
// weight s_ib d_nb: fma(float(P), s_ib d_nb, acc) -- three vector ALU
// operations per output element and block, which bound this kernel (the
// matrix cores take a quarter of that time).
#include <hip/hip_runtime.h>

#include "eb_internal.h"
#include "epilogue.h"
#include "mfma_common.h"

namespace eb {
namespace {

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v16i_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// ---- activation quantization ----

template <int XT>
__global__ void __launch_bounds__(256)
    quantize_x8_kernel(const uint16_t *__restrict__ x, int64_t m, int64_t k, int64_t ms,
                       int8_t *__restrict__ xq, float *__restrict__ xs) {
  const int64_t nb = k / kQK;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < ms * nb;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t % ms, b = t / ms;  // consecutive threads: consecutive rows of one block
    if (i >= m) {
      xs[b * ms + i] = 0.f;
      continue;
    }
    const uint16_t *src = x + i * k + b * kQK;
    float v[kQK];
    float a = 0.f;
#pragma unroll
    for (int j = 0; j < kQK; j += 8) {
      const uint4 w = *reinterpret_cast<const uint4 *>(src + j);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint16_t lo = (uint16_t)(ws[e] & 0xffffu), hi = (uint16_t)(ws[e] >> 16);
        v[j + 2 * e] = XT == EB_F16 ? (float)__builtin_bit_cast(_Float16, lo) : __uint_as_float((uint32_t)lo << 16);
        v[j + 2 * e + 1] = XT == EB_F16 ? (float)__builtin_bit_cast(_Float16, hi) : __uint_as_float((uint32_t)hi << 16);
      }
    }
#pragma unroll
    for (int j = 0; j < kQK; ++j) a = fmaxf(a, fabsf(v[j]));
    const float s = a / 127.0f;
    xs[b * ms + i] = s;
    uint32_t words[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      uint32_t word = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        int q = 0;
        if (s != 0.f) q = (int)fmin(fmax(round((double)v[4 * w + e] / (double)s), -127.0), 127.0);
        word |= (uint32_t)(uint8_t)(int8_t)q << (8 * e);
      }
      words[w] = word;
    }
    uint4 *dst = reinterpret_cast<uint4 *>(xq + i * k + b * kQK);
    dst[0] = make_uint4(words[0], words[1], words[2], words[3]);
    dst[1] = make_uint4(words[4], words[5], words[6], words[7]);
  }
}

// ---- product ----

constexpr int kBMi = 128, kBNi = 128;

// 16 Q4_0 nibbles (half h of a block's 16 bytes) -> int8 codes c - 8
__device__ inline v4i_t q4_codes(const uint4 raw, int h) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  v4i_t o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t v = (w[e] >> (4 * h)) & 0x0f0f0f0fu;
    // per byte (v | 0x80) - 8 stays in 120..135 (no borrow across bytes), and
    // the xor maps it to v - 8 modulo 256
    o[e] = (int)(((v | 0x80808080u) - 0x08080808u) ^ 0x80808080u);
  }
  return o;
}

template <int QT, int YT>
__global__ void __launch_bounds__(256)
    mm_i8_kernel(const uint8_t *__restrict__ wdata, int64_t n, int64_t k, int64_t d_off, int64_t ds,
                 const int8_t *__restrict__ xq, const float *__restrict__ xs, int64_t ms, int64_t m,
                 void *__restrict__ y, int yt, Fuse f) {
  constexpr int QSB = (QT == EB_Q8_0) ? 32 : 16;  // code bytes per block
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int r = lane & 31, h = lane >> 5;
  const int64_t n0 = (int64_t)blockIdx.x * kBNi, m0 = (int64_t)blockIdx.y * kBMi;
  const int rows_n = (int)min((int64_t)kBNi, n - n0), rows_m = (int)min((int64_t)kBMi, m - m0);
  const int nb = (int)(k / kQK);

  // descriptors over the tile's rows (rows past the end read zeros)
  const uint32_t qrow = (uint32_t)nb * QSB, drow = (uint32_t)ds * 2;
  const auto qr = rsrc(wdata + n0 * qrow, (uint32_t)rows_n * qrow);
  const auto dr = rsrc(wdata + d_off + n0 * drow, (uint32_t)rows_n * drow);
  const auto xr = rsrc(xq + m0 * k, (uint32_t)rows_m * (uint32_t)k);
  const auto sr = rsrc(xs, (uint32_t)(nb * ms * 4));
  uint32_t aoff[2], boff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    aoff[i] = (uint32_t)(64 * wm + 32 * i + r) * (uint32_t)k + 16u * h;
    boff[i] = (uint32_t)(64 * wn + 32 * i + r) * qrow + (QT == EB_Q8_0 ? 16u * h : 0u);
  }

  // Block scales of kGB blocks at a time, staged in LDS (two buffers): the
  // activation scales of the tile's 128 x rows and the weight scales of its
  // 128 weight rows, as fp32, block-major; a lane then reads its 16 x-row
  // scales per x sub-tile as four 16-byte LDS reads (lanes of a half-wave
  // read the same addresses) and one weight scale per weight sub-tile.
  constexpr int kGB = 8;
  __shared__ __align__(16) float s_lds[2][kGB][kBMi];
  __shared__ __align__(16) float d_lds[2][kGB][kBNi];
  const int t = threadIdx.x;
  auto stage = [&](int buf, int b0) __attribute__((always_inline)) {
    // activation scales: 8 blocks x 128 rows, 4 per thread, rows contiguous
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = t + 256 * q, bb = e / kBMi, row = e % kBMi;
      const uint32_t off = (uint32_t)((int64_t)(b0 + bb) * ms + m0 + row) * 4u;
      s_lds[buf][bb][row] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(sr, (int)(b0 + bb < nb ? off : 0x80000000u), 0, 0));
    }
    // weight scales: row t (t < 128) holds 8 consecutive binary16 scales
    if (t < kBNi) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(dr, (int)((uint32_t)t * drow + 2u * b0), 0, 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t w2 = v[q];
        d_lds[buf][2 * q][t] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w2 & 0xffffu));
        d_lds[buf][2 * q + 1][t] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w2 >> 16));
      }
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // operands of block b (zeros past the last block)
  struct Ops {
    v4i_t a[2], b[2];
  };
  auto load_ops = [&](Ops &o, int b) __attribute__((always_inline)) {
    const bool ok = b < nb;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const auto va = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)(ok ? aoff[i] + 32u * b : 0x80000000u), 0, 0);
      o.a[i] = __builtin_bit_cast(v4i_t, va);
      const auto vb = __builtin_amdgcn_raw_buffer_load_b128(qr, (int)(ok ? boff[i] + (uint32_t)QSB * b : 0x80000000u), 0, 0);
      if constexpr (QT == EB_Q8_0)
        o.b[i] = __builtin_bit_cast(v4i_t, vb);
      else
        o.b[i] = q4_codes(__builtin_bit_cast(uint4, vb), h);
    }
  };

  Ops cur, nxt;
  load_ops(cur, 0);
  stage(0, 0);
  __syncthreads();
  const int ngroups = (nb + kGB - 1) / kGB;
  for (int gi = 0; gi < ngroups; ++gi) {
    const int buf = gi & 1, b0 = gi * kGB;
    if (gi + 1 < ngroups) stage(buf ^ 1, b0 + kGB);  // next group's scales, read after the barrier
    const int nbg = min(kGB, nb - b0);
    // block scales of this lane, read from LDS one block ahead of their use
    f32x4_t sv[2][4], svn[2][4];
    float dv[2], dvn[2];
    auto read_scales = [&](f32x4_t (&S)[2][4], float (&D)[2], int bb) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
          S[i][g] = *reinterpret_cast<const f32x4_t *>(&s_lds[buf][bb][64 * wm + 32 * i + 8 * g + 4 * h]);
        D[i] = d_lds[buf][bb][64 * wn + 32 * i + r];
      }
    };
    read_scales(sv, dv, 0);
    for (int bb = 0; bb < nbg; ++bb) {
      load_ops(nxt, b0 + bb + 1);
      read_scales(svn, dvn, bb + 1 < kGB ? bb + 1 : bb);
      v16i_t p[2][2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const v16i_t zero = {};
          p[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(cur.a[i], cur.b[j], zero, 0, 0, 0);
        }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            acc[i][j][e] = __builtin_fmaf((float)p[i][j][e], sv[i][e >> 2][e & 3] * dv[j], acc[i][j][e]);
      cur = nxt;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int g = 0; g < 4; ++g) sv[i][g] = svn[i][g];
        dv[i] = dvn[i];
      }
    }
    __syncthreads();  // the next group's scales are in; this group's buffer is free
  }

  // epilogue: lane holds weight row (column of y) 64 wn + 32 j + r and x rows
  // 64 wm + 32 i + 8 (e / 4) + 4 h + e % 4
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int cl = 64 * wn + 32 * j + r;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rl = 64 * wm + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
        float v = acc[i][j][e];
        if (f.epi == EB_EPI_GLU) {  // rows 2c, 2c + 1 of the weights sit in lanes r, r ^ 1
          const float up = __shfl_xor(v, 1);
          if ((r & 1) == 0 && rl < rows_m && cl < rows_n)
            store_y(y, (m0 + rl) * (n / 2) + (n0 + cl) / 2, silu_mul(v, up), yt);
          continue;
        }
        if (rl < rows_m && cl < rows_n) put_y(y, (m0 + rl) * n + n0 + cl, v, yt, f);
      }
  }
}

inline unsigned grid1(int64_t threads) {
  int64_t g = (threads + 255) / 256;
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(g, 65536));
}

}  // namespace

size_t i8_workspace_bytes(int64_t m, int64_t k) {
  const int64_t ms = (m + 3) / 4 * 4;
  return (size_t)round_up(m * k, 256) + (size_t)round_up(k / kQK * ms * 4, 256);
}

bool i8_fits(int64_t m, int64_t n, int64_t k) {
  const int64_t ms = (m + 3) / 4 * 4;
  return m >= 1 && (int64_t)kBMi * k < 0x7fff0000LL && (int64_t)kBNi * (k / kQK) * 32 < 0x7fff0000LL &&
         (k / kQK) * ms * 4 < 0x7fff0000LL && (n + kBNi - 1) / kBNi <= 0x7fffffffLL &&
         (m + kBMi - 1) / kBMi <= 65535;
}

hipError_t launch_mfma_i8(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                          int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f, void *ws,
                          hipStream_t s) {
  if (!i8_fits(m, n, k)) return hipErrorInvalidValue;
  const int64_t ms = (m + 3) / 4 * 4, nb = k / kQK;
  int8_t *xq = static_cast<int8_t *>(ws);
  float *xsc = reinterpret_cast<float *>(static_cast<uint8_t *>(ws) + round_up(m * k, 256));
  const auto *xp = static_cast<const uint16_t *>(x);
  if (xt == EB_F16)
    quantize_x8_kernel<EB_F16><<<grid1(ms * nb), 256, 0, s>>>(xp, m, k, ms, xq, xsc);
  else
    quantize_x8_kernel<EB_BF16><<<grid1(ms * nb), 256, 0, s>>>(xp, m, k, ms, xq, xsc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const Layout L = layout_of(type, n, k);
  const dim3 grid((unsigned)((n + kBNi - 1) / kBNi), (unsigned)((m + kBMi - 1) / kBMi));
  const auto *wp = static_cast<const uint8_t *>(wdata);
  if (type == EB_Q8_0) {
    if (yt == EB_F32)
      mm_i8_kernel<EB_Q8_0, EB_F32><<<grid, 256, 0, s>>>(wp, n, k, L.d_off, L.ds, xq, xsc, ms, m, y, yt, f);
    else
      mm_i8_kernel<EB_Q8_0, EB_BF16><<<grid, 256, 0, s>>>(wp, n, k, L.d_off, L.ds, xq, xsc, ms, m, y, yt, f);
  } else {
    if (yt == EB_F32)
      mm_i8_kernel<EB_Q4_0, EB_F32><<<grid, 256, 0, s>>>(wp, n, k, L.d_off, L.ds, xq, xsc, ms, m, y, yt, f);
    else
      mm_i8_kernel<EB_Q4_0, EB_BF16><<<grid, 256, 0, s>>>(wp, n, k, L.d_off, L.ds, xq, xsc, ms, m, y, yt, f);
  }
  return hipGetLastError();
}

}  // namespace eb
