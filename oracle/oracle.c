/*
 * oracle.c -- plain, slow, obviously-correct CPU reference for block-quantized
 * linear layers.  TEST INFRASTRUCTURE ONLY: nothing in the product library may
 * link, load or call this file.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark use it.  It shares no code, header, table
 * or helper with the HIP implementation.
 *
 * What it computes (paper section 4, Table 3: the runtime is evaluated with
 * 8-bit and 4-bit quantized C++ configurations; section 3.2, "latency-first
 * fused execution", puts those quantized linear layers on the batch-1 path):
 *
 *   y[m][n] = sum_k x[m][k] * w_hat[n][k],   w_hat = dequant(quant(W))
 *
 * with the weights stored in the ggml-style Q8_0 / Q4_0 block formats:
 * blocks of 32 consecutive weights along k (the input-feature axis of W[n][k]),
 * each block carrying one IEEE binary16 scale.
 *
 *   Q8_0 block (34 bytes): d16 (little-endian binary16), then 32 int8 codes.
 *     amax = max_j |x_j|;  d32 = fl32(amax / 127);  d16 = binary16_RNE(d32)
 *     q_j  = clamp(round_half_away_from_zero(x_j / d16), -127, 127)
 *            (0 for every j when d16 == 0)
 *   Q4_0 block (18 bytes): d16, then 16 bytes of packed 4-bit codes.
 *     m = the signed element of largest magnitude (first index on ties,
 *         starting from +0.0);  d32 = fl32(m / -8);  d16 = binary16_RNE(d32)
 *     c_j = clamp(floor(x_j / d16 + 1/2), -8, 7)   (0 when d16 == 0)
 *     nibble_j = c_j + 8;  byte i (0..15) = nibble_i | nibble_{i+16} << 4
 *   Dequant: w_hat = q * d16 (Q8_0) or (nibble - 8) * d16 (Q4_0), exact in
 *   binary64.
 *
 *   Q6_S super-block (210 bytes, 256 weights = 16 sub-blocks of 16): the
 *   6-bit configuration of the same evaluation; the paper names no format, so
 *   this one is defined here (a two-level "super-block" scale):
 *     m_j = the signed element of largest magnitude of sub-block j (first
 *           index on ties, starting from +0.0);  s_j = fl32(m_j / -32)
 *     amax = max_j |s_j|;  d32 = fl32(amax / 127);  d16 = binary16_RNE(d32)
 *     sc_j = clamp(round_half_away_from_zero(s_j / d16), -127, 127)
 *            (0 for every j when d16 == 0)
 *     e_j  = d16 * sc_j   (exact: at most 11 + 7 significant bits)
 *     q_i  = clamp(floor(x_i / e_j + 1/2), -32, 31)   (0 when e_j == 0)
 *     u_i  = q_i + 32 in 0..63
 *   Bytes: d16, then sc_0..sc_15 as int8, then 8 chunks of 24 bytes, chunk c
 *   holding elements 32c .. 32c + 31 (local index i): byte i (0..15) =
 *   (u_i & 15) | (u_{i+16} & 15) << 4, byte 16 + t (t = 0..7) =
 *   (u_t >> 4) | (u_{t+8} >> 4) << 2 | (u_{t+16} >> 4) << 4 | (u_{t+24} >> 4) << 6.
 *   Dequant: w_hat_i = (u_i - 32) * d16 * sc_{i/16}, exact in binary64.
 *
 * Readings taken where the format description is silent (each is listed with
 * its reason in the design notes of the repository):
 *   - codes are rounded against the *stored* binary16 scale d16, so that every
 *     element satisfies |x - w_hat| <= |d16|/2 (saturated Q4_0 codes and
 *     underflowed scales excepted);
 *   - ties: Q8_0 rounds half away from zero, Q4_0 rounds half up;
 *   - x / d16 is evaluated in binary64: x has 24 significant bits and d16 at
 *     most 11, so the binary64 quotient can neither create nor destroy a tie
 *     and every rounding decision equals the one on the exact quotient; the
 *     same holds for s_j / d16 and x_i / e_j of Q6_S (e_j: at most 18 bits).
 *
 * Matmul: every product and sum in binary64, in plain k order, one output at
 * a time.  Alongside y it returns bound[m][n] = sum_k |x[m][k]| * |w_hat[n][k]|,
 * the scale against which an fp32-accumulating implementation's error is
 * normalised.  Threads (pthreads) only split the set of outputs; each output
 * is still one sequential binary64 loop.
 *
 * Low-precision prefill variant (section 3.2, backend-specific dispatch):
 * the activations quantized per 32-element block to int8 with a binary32
 * scale (s = fl32(max|x| / 127), codes rounded half away from zero against
 * s), each block's product an exact integer sum of code products scaled by
 * s * d16, and the bound of the activation-quantization error.
 *
 * Layer steps on either side of the product (section 3.2, operator fusion),
 * each in binary64: rounding to binary16 / bfloat16 (nearest, ties to even),
 * RMS normalisation h * gamma / sqrt(eps + mean h^2) and the SiLU-gated
 * product silu(g) * u, silu(t) = t / (1 + exp(-t)).
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -shared -fPIC -pthread
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)

#define ORACLE_Q8_0 1
#define ORACLE_Q4_0 2
#define ORACLE_Q6_S 3

#define ORACLE_X_F16 1
#define ORACLE_X_BF16 2

#define QK 32
#define QK6 256 /* weights per Q6_S super-block */
#define QS6 16  /* weights per Q6_S sub-block */

/* ---------------------------------------------------------------------- */
/* binary16 / bfloat16 encode and decode, written from the IEEE 754 formats */
/* ---------------------------------------------------------------------- */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
double oracle_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int f = h & 0x3ff;
  double v;
  if (e == 0x1f) {
    v = f ? NAN : INFINITY;
  } else if (e == 0) {
    v = ldexp((double)f, -24); /* subnormal: f * 2^-24 */
  } else {
    v = ldexp((double)(1024 + f), e - 25); /* (1 + f/1024) * 2^(e-15) */
  }
  return sign ? -v : v;
}

/* bfloat16: the upper 16 bits of an IEEE binary32. */
double oracle_bf16_to_double(uint16_t b) {
  int sign = (b >> 15) & 1;
  int e = (b >> 7) & 0xff;
  int f = b & 0x7f;
  double v;
  if (e == 0xff) {
    v = f ? NAN : INFINITY;
  } else if (e == 0) {
    v = ldexp((double)f, -133); /* subnormal: f * 2^-126 * 2^-7 */
  } else {
    v = ldexp((double)(128 + f), e - 134); /* (1 + f/128) * 2^(e-127) */
  }
  return sign ? -v : v;
}

/* Round a binary32 value to the nearest binary16, ties to even (the IEEE 754
 * default rounding), with gradual underflow and overflow to infinity. */
uint16_t oracle_float_to_half_rne(float f) {
  double a = fabs((double)f);
  uint16_t sign = signbit(f) ? 0x8000u : 0u;
  if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
  if (isinf(f)) return (uint16_t)(sign | 0x7c00u);
  if (a == 0.0) return sign;
  /* a lies in [2^E, 2^(E+1)); the binary16 spacing there is 2^(E-10), and
   * below the normal range (E < -14) it stays 2^-24. */
  int e2;
  (void)frexp(a, &e2);
  int E = e2 - 1;
  if (E < -14) E = -14;
  double spacing = ldexp(1.0, E - 10);
  double r = rint(a / spacing); /* a/spacing is exact; rint = ties-to-even */
  double v = r * spacing;       /* exact */
  if (v > 65504.0) return (uint16_t)(sign | 0x7c00u);
  uint16_t bits;
  if (v < ldexp(1.0, -14)) {
    bits = (uint16_t)(v * ldexp(1.0, 24)); /* subnormal fraction */
  } else {
    int ev;
    double m = frexp(v, &ev); /* v = m * 2^ev, m in [0.5, 1) */
    int biased = ev - 1 + 15;
    int frac = (int)((2.0 * m - 1.0) * 1024.0);
    bits = (uint16_t)((biased << 10) | frac);
  }
  return (uint16_t)(sign | bits);
}

/* ---------------------------------------------------------------------- */
/* Quantization to the canonical (array-of-blocks) byte layout             */
/* ---------------------------------------------------------------------- */

static void put_d16(uint8_t *dst, uint16_t d16) {
  dst[0] = (uint8_t)(d16 & 0xff);
  dst[1] = (uint8_t)(d16 >> 8);
}

static uint16_t get_d16(const uint8_t *src) {
  return (uint16_t)(src[0] | (src[1] << 8));
}

static void quantize_block_q8_0(const float *x, uint8_t *blk) {
  float amax = 0.0f;
  for (int j = 0; j < QK; ++j) {
    float a = fabsf(x[j]);
    if (a > amax) amax = a;
  }
  float d32 = amax / 127.0f;
  uint16_t d16 = oracle_float_to_half_rne(d32);
  double d = oracle_half_to_double(d16);
  put_d16(blk, d16);
  for (int j = 0; j < QK; ++j) {
    int q = 0;
    if (d != 0.0) {
      double t = round((double)x[j] / d); /* round() = half away from zero */
      if (t > 127.0) t = 127.0;
      if (t < -127.0) t = -127.0;
      q = (int)t;
    }
    blk[2 + j] = (uint8_t)(int8_t)q;
  }
}

static void quantize_block_q4_0(const float *x, uint8_t *blk) {
  float amax = 0.0f, m = 0.0f;
  for (int j = 0; j < QK; ++j) {
    float a = fabsf(x[j]);
    if (a > amax) {
      amax = a;
      m = x[j];
    }
  }
  float d32 = m / -8.0f;
  uint16_t d16 = oracle_float_to_half_rne(d32);
  double d = oracle_half_to_double(d16);
  put_d16(blk, d16);
  int nib[QK];
  for (int j = 0; j < QK; ++j) {
    int c = 0;
    if (d != 0.0) {
      double t = floor((double)x[j] / d + 0.5); /* round half up */
      if (t > 7.0) t = 7.0;
      if (t < -8.0) t = -8.0;
      c = (int)t;
    }
    nib[j] = c + 8;
  }
  for (int i = 0; i < QK / 2; ++i) blk[2 + i] = (uint8_t)(nib[i] | (nib[i + QK / 2] << 4));
}

static void quantize_block_q6_s(const float *x, uint8_t *blk) {
  float s[QK6 / QS6];
  float amax = 0.0f;
  for (int j = 0; j < QK6 / QS6; ++j) {
    float mag = 0.0f, m = 0.0f;
    for (int i = 0; i < QS6; ++i) {
      float a = fabsf(x[j * QS6 + i]);
      if (a > mag) {
        mag = a;
        m = x[j * QS6 + i];
      }
    }
    s[j] = m / -32.0f;
    if (fabsf(s[j]) > amax) amax = fabsf(s[j]);
  }
  float d32 = amax / 127.0f;
  uint16_t d16 = oracle_float_to_half_rne(d32);
  double d = oracle_half_to_double(d16);
  put_d16(blk, d16);
  int sc[QK6 / QS6];
  for (int j = 0; j < QK6 / QS6; ++j) {
    sc[j] = 0;
    if (d != 0.0) {
      double t = round((double)s[j] / d); /* half away from zero */
      if (t > 127.0) t = 127.0;
      if (t < -127.0) t = -127.0;
      sc[j] = (int)t;
    }
    blk[2 + j] = (uint8_t)(int8_t)sc[j];
  }
  int u[QK6];
  for (int i = 0; i < QK6; ++i) {
    double e = d * (double)sc[i / QS6]; /* exact */
    int q = 0;
    if (e != 0.0) {
      double t = floor((double)x[i] / e + 0.5); /* round half up */
      if (t > 31.0) t = 31.0;
      if (t < -32.0) t = -32.0;
      q = (int)t;
    }
    u[i] = q + 32;
  }
  for (int c = 0; c < QK6 / 32; ++c) {
    uint8_t *ch = blk + 2 + QK6 / QS6 + 24 * c;
    const int *uc = u + 32 * c;
    for (int i = 0; i < 16; ++i) ch[i] = (uint8_t)((uc[i] & 15) | (uc[i + 16] & 15) << 4);
    for (int t = 0; t < 8; ++t)
      ch[16 + t] = (uint8_t)((uc[t] >> 4) | (uc[t + 8] >> 4) << 2 | (uc[t + 16] >> 4) << 4 |
                             (uc[t + 24] >> 4) << 6);
  }
}

int64_t oracle_block_bytes(int qtype) {
  if (qtype == ORACLE_Q8_0) return 2 + QK;
  if (qtype == ORACLE_Q4_0) return 2 + QK / 2;
  if (qtype == ORACLE_Q6_S) return 2 + QK6 / QS6 + QK6 * 6 / 8;
  return -1;
}

/* Weights per block: 32, or 256 for the Q6_S super-block. */
int64_t oracle_block_elems(int qtype) {
  if (qtype == ORACLE_Q8_0 || qtype == ORACLE_Q4_0) return QK;
  if (qtype == ORACLE_Q6_S) return QK6;
  return -1;
}

typedef struct {
  int qtype;
  const float *w;
  int64_t k;
  uint8_t *out;
  int64_t begin, end; /* rows for this worker */
} qjob_t;

static void *run_qjob(void *arg) {
  qjob_t *J = (qjob_t *)arg;
  int64_t bb = oracle_block_bytes(J->qtype), be = oracle_block_elems(J->qtype);
  int64_t nb = J->k / be;
  for (int64_t r = J->begin; r < J->end; ++r)
    for (int64_t b = 0; b < nb; ++b) {
      const float *src = J->w + r * J->k + b * be;
      uint8_t *dst = J->out + (r * nb + b) * bb;
      if (J->qtype == ORACLE_Q8_0)
        quantize_block_q8_0(src, dst);
      else if (J->qtype == ORACLE_Q4_0)
        quantize_block_q4_0(src, dst);
      else
        quantize_block_q6_s(src, dst);
    }
  return NULL;
}

/* w: fp32 [n][k] row-major; out: n * (k/E) canonical blocks (E weights per
 * block), row by row.  Threads (nthreads <= 1: the calling thread) only split
 * the rows. */
int oracle_quantize(int qtype, const float *w, int64_t n, int64_t k, uint8_t *out, int nthreads) {
  int64_t bb = oracle_block_bytes(qtype), be = oracle_block_elems(qtype);
  if (bb < 0 || n < 0 || k < 0 || k % be != 0 || (!w && n * k) || (!out && n * k))
    return ORACLE_EINVAL;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > n) nthreads = n > 0 ? (int)n : 1;
  qjob_t jobs[256];
  pthread_t tids[256];
  if (nthreads > 256) nthreads = 256;
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].qtype = qtype;
    jobs[t].w = w;
    jobs[t].k = k;
    jobs[t].out = out;
    jobs[t].begin = n * t / nthreads;
    jobs[t].end = n * (t + 1) / nthreads;
  }
  if (nthreads == 1) {
    run_qjob(&jobs[0]);
    return ORACLE_OK;
  }
  int started = 0, rc = ORACLE_OK;
  for (int t = 0; t < nthreads; ++t) {
    if (pthread_create(&tids[t], NULL, run_qjob, &jobs[t]) != 0) {
      rc = ORACLE_EINVAL;
      break;
    }
    ++started;
  }
  for (int t = 0; t < started; ++t) pthread_join(tids[t], NULL);
  return rc;
}

/* ---------------------------------------------------------------------- */
/* Dequantization                                                          */
/* ---------------------------------------------------------------------- */

static double code_at(int qtype, const uint8_t *blk, int j) {
  if (qtype == ORACLE_Q8_0) return (double)(int8_t)blk[2 + j];
  int byte = blk[2 + (j % (QK / 2))];
  int nibble = (j < QK / 2) ? (byte & 0x0f) : (byte >> 4);
  return (double)(nibble - 8);
}

/* Code u_i (0..63) of element i of a Q6_S super-block. */
static int q6_code(const uint8_t *blk, int i) {
  const uint8_t *ch = blk + 2 + QK6 / QS6 + 24 * (i / 32);
  int l = i % 32;
  int lo = (l < 16) ? (ch[l] & 15) : (ch[l - 16] >> 4);
  int hi = (ch[16 + l % 8] >> (2 * (l / 8))) & 3;
  return lo | hi << 4;
}

/* One row of w_hat (k values) from the row's k/E blocks. */
static void dequant_row(int qtype, const uint8_t *row_blocks, int64_t k, double *dst) {
  int64_t bb = oracle_block_bytes(qtype);
  if (qtype == ORACLE_Q6_S) {
    for (int64_t b = 0; b < k / QK6; ++b) {
      const uint8_t *blk = row_blocks + b * bb;
      double d = oracle_half_to_double(get_d16(blk));
      for (int i = 0; i < QK6; ++i)
        dst[b * QK6 + i] = (double)(q6_code(blk, i) - 32) * (d * (double)(int8_t)blk[2 + i / QS6]);
    }
    return;
  }
  for (int64_t b = 0; b < k / QK; ++b) {
    const uint8_t *blk = row_blocks + b * bb;
    double d = oracle_half_to_double(get_d16(blk));
    for (int j = 0; j < QK; ++j) dst[b * QK + j] = code_at(qtype, blk, j) * d;
  }
}

int oracle_dequant(int qtype, const uint8_t *blocks, int64_t n, int64_t k, double *w_hat) {
  int64_t bb = oracle_block_bytes(qtype), be = oracle_block_elems(qtype);
  if (bb < 0 || n < 0 || k < 0 || k % be != 0) return ORACLE_EINVAL;
  for (int64_t r = 0; r < n; ++r) dequant_row(qtype, blocks + r * (k / be) * bb, k, w_hat + r * k);
  return ORACLE_OK;
}

/* ---------------------------------------------------------------------- */
/* Linear layer in binary64                                                */
/* ---------------------------------------------------------------------- */

typedef struct {
  int qtype;
  const uint8_t *blocks;
  int64_t k;
  const double *xd; /* [m][k] decoded activations */
  int64_t m;
  const int64_t *cols; /* output columns (rows of W) to compute */
  int64_t ncols;
  double *y, *bound; /* [m][ncols] */
  int64_t begin, end; /* slice of cols for this worker */
} job_t;

static void *run_job(void *arg) {
  job_t *J = (job_t *)arg;
  int64_t bb = oracle_block_bytes(J->qtype), be = oracle_block_elems(J->qtype);
  double *wrow = (double *)malloc(sizeof(double) * (size_t)(J->k ? J->k : 1));
  if (!wrow) return (void *)1;
  for (int64_t c = J->begin; c < J->end; ++c) {
    int64_t n = J->cols[c];
    dequant_row(J->qtype, J->blocks + n * (J->k / be) * bb, J->k, wrow);
    for (int64_t i = 0; i < J->m; ++i) {
      const double *xr = J->xd + i * J->k;
      double s = 0.0, b = 0.0;
      for (int64_t kk = 0; kk < J->k; ++kk) {
        double p = xr[kk] * wrow[kk];
        s += p;
        b += fabs(p);
      }
      J->y[i * J->ncols + c] = s;
      J->bound[i * J->ncols + c] = b;
    }
  }
  free(wrow);
  return NULL;
}

/*
 * y[i][c], bound[i][c] for i < m and c < ncols, output column cols[c] (a row
 * index of W in [0, n)).  x holds raw binary16 or bfloat16 words [m][k].
 * nthreads <= 1 runs on the calling thread.
 */
int oracle_qlinear(int qtype, const uint8_t *blocks, int64_t n, int64_t k, const uint16_t *x,
                   int xdtype, int64_t m, const int64_t *cols, int64_t ncols, double *y,
                   double *bound, int nthreads) {
  if (oracle_block_bytes(qtype) < 0 || k <= 0 || k % oracle_block_elems(qtype) != 0 || n <= 0 ||
      m < 0 || ncols < 0)
    return ORACLE_EINVAL;
  if (xdtype != ORACLE_X_F16 && xdtype != ORACLE_X_BF16) return ORACLE_EINVAL;
  for (int64_t c = 0; c < ncols; ++c)
    if (cols[c] < 0 || cols[c] >= n) return ORACLE_EINVAL;
  if (m == 0 || ncols == 0) return ORACLE_OK;
  double *xd = (double *)malloc(sizeof(double) * (size_t)(m * k));
  if (!xd) return ORACLE_EINVAL;
  for (int64_t i = 0; i < m * k; ++i)
    xd[i] = (xdtype == ORACLE_X_F16) ? oracle_half_to_double(x[i]) : oracle_bf16_to_double(x[i]);

  if (nthreads < 1) nthreads = 1;
  if (nthreads > ncols) nthreads = (int)ncols;
  job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
  pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
  int rc = ORACLE_OK;
  if (!jobs || !tids) {
    rc = ORACLE_EINVAL;
    goto done;
  }
  for (int t = 0; t < nthreads; ++t) {
    job_t *J = &jobs[t];
    J->qtype = qtype;
    J->blocks = blocks;
    J->k = k;
    J->xd = xd;
    J->m = m;
    J->cols = cols;
    J->ncols = ncols;
    J->y = y;
    J->bound = bound;
    J->begin = ncols * t / nthreads;
    J->end = ncols * (t + 1) / nthreads;
  }
  if (nthreads == 1) {
    if (run_job(&jobs[0])) rc = ORACLE_EINVAL;
  } else {
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
      if (pthread_create(&tids[t], NULL, run_job, &jobs[t]) != 0) {
        rc = ORACLE_EINVAL;
        break;
      }
      ++started;
    }
    for (int t = 0; t < started; ++t) {
      void *ret = NULL;
      pthread_join(tids[t], &ret);
      if (ret) rc = ORACLE_EINVAL;
    }
  }
done:
  free(jobs);
  free(tids);
  free(xd);
  return rc;
}

/* ---------------------------------------------------------------------- */
/* The steps on either side of the linear layer in a decoder layer (paper  */
/* section 3.2: operator fusion on the batch-1 path; the backbones of      */
/* section 2.1 / Table 1 are decoder stacks): RMS normalisation of the     */
/* residual stream before a projection, the SiLU-gated product of a        */
/* gate/up projection pair, and (in the Python layer) the residual         */
/* addition after a projection.                                            */
/* ---------------------------------------------------------------------- */

/* Nearest value of a binary floating-point format with p significant bits
 * (p - 1 stored fraction bits), exponent bias `bias` and normal exponents
 * 1 - bias .. bias, to v, ties to the even significand, with gradual
 * underflow and overflow to infinity; returns the 16-bit encoding. */
static uint16_t round_to_format16(double v, int p, int bias) {
  const int fb = p - 1;
  const int emin = 1 - bias, emax = bias;
  const uint16_t sign = signbit(v) ? 0x8000u : 0u;
  const uint16_t inf = (uint16_t)((2 * bias + 1) << fb);
  if (isnan(v)) return (uint16_t)(sign | inf | (1u << (fb - 1)));
  if (isinf(v)) return (uint16_t)(sign | inf);
  double a = fabs(v);
  if (a == 0.0) return sign;
  /* a lies in [2^E, 2^(E+1)); the format's spacing there is 2^(E - fb), and
   * below the normal range it stays 2^(emin - fb). */
  int e2;
  (void)frexp(a, &e2);
  int E = e2 - 1;
  if (E < emin) E = emin;
  double spacing = ldexp(1.0, E - fb);
  double r = rint(a / spacing); /* a / spacing is exact; rint rounds ties to even */
  double q = r * spacing;       /* exact */
  if (q >= ldexp(1.0, emax + 1)) return (uint16_t)(sign | inf);
  if (q < ldexp(1.0, emin)) return (uint16_t)(sign | (uint16_t)(q / ldexp(1.0, emin - fb)));
  int ev;
  double m = frexp(q, &ev); /* q = m * 2^ev, m in [0.5, 1) */
  int biased = ev - 1 + bias;
  int frac = (int)((2.0 * m - 1.0) * (double)(1 << fb));
  return (uint16_t)(sign | (biased << fb) | frac);
}

/* out[i] = the binary16 (xtype F16: 11 significant bits, bias 15) or
 * bfloat16 (BF16: 8 significant bits, bias 127) encoding nearest to v[i]. */
int oracle_round_x16(const double *v, int64_t count, int xtype, uint16_t *out) {
  if (count < 0 || (xtype != ORACLE_X_F16 && xtype != ORACLE_X_BF16)) return ORACLE_EINVAL;
  for (int64_t i = 0; i < count; ++i)
    out[i] = xtype == ORACLE_X_F16 ? round_to_format16(v[i], 11, 15) : round_to_format16(v[i], 8, 127);
  return ORACLE_OK;
}

/* RMS normalisation of every row of h[m][k] (binary32) with per-feature
 * weights gamma[k]: r_i = 1 / sqrt(eps + (1/k) sum_j h[i][j]^2) and
 * out[i][j] = h[i][j] * gamma[j] * r_i, all in binary64.  eps >= 0; a row of
 * zeros needs eps > 0. */
int oracle_rmsnorm(const float *h, const float *gamma, double eps, int64_t m, int64_t k,
                   double *out) {
  if (m < 0 || k <= 0 || !(eps >= 0.0)) return ORACLE_EINVAL;
  for (int64_t i = 0; i < m; ++i) {
    const float *row = h + i * k;
    double ss = 0.0;
    for (int64_t j = 0; j < k; ++j) ss += (double)row[j] * (double)row[j];
    double ms = ss / (double)k + eps;
    if (!(ms > 0.0)) return ORACLE_EINVAL;
    double r = 1.0 / sqrt(ms);
    for (int64_t j = 0; j < k; ++j) out[i * k + j] = (double)row[j] * (double)gamma[j] * r;
  }
  return ORACLE_OK;
}

/* out[i] = silu(g[i]) * u[i], silu(t) = t / (1 + exp(-t)) (the sigmoid-
 * weighted linear unit), in binary64. */
int oracle_silu_mul(const double *g, const double *u, int64_t count, double *out) {
  if (count < 0) return ORACLE_EINVAL;
  for (int64_t i = 0; i < count; ++i) out[i] = g[i] / (1.0 + exp(-g[i])) * u[i];
  return ORACLE_OK;
}

/* ---------------------------------------------------------------------- */
/* Low-precision prefill variant (section 3.2, backend-specific dispatch:  */
/* the large-m projections on the integer matrix cores).  The activations  */
/* are quantized per 32-element block along k to int8 with a binary32      */
/* scale; each block's product is a sum of integer code products, scaled  */
/* by the activation block scale and the weight block scale.               */
/* ---------------------------------------------------------------------- */

/* Per row i and block b of x[m][k] (binary16 or bfloat16 words):
 *   a = max_j |x_ij|,  s_ib = fl32(a / 127)  (0 when a == 0),
 *   xq_ij = clamp(round_half_away_from_zero(x_ij / s_ib), -127, 127)
 *           (0 when s_ib == 0),
 * the quotient in binary64 (x has at most 11 significant bits and s 24, so
 * it decides every rounding as the exact quotient would).  xq: int8 [m][k];
 * s: binary32 [m][k/32]. */
int oracle_quantize_x8(const uint16_t *x, int xdtype, int64_t m, int64_t k, int8_t *xq, float *s) {
  if (m < 0 || k <= 0 || k % QK != 0) return ORACLE_EINVAL;
  if (xdtype != ORACLE_X_F16 && xdtype != ORACLE_X_BF16) return ORACLE_EINVAL;
  for (int64_t i = 0; i < m; ++i)
    for (int64_t b = 0; b < k / QK; ++b) {
      double v[QK];
      float a = 0.0f;
      for (int j = 0; j < QK; ++j) {
        uint16_t w = x[i * k + b * QK + j];
        v[j] = xdtype == ORACLE_X_F16 ? oracle_half_to_double(w) : oracle_bf16_to_double(w);
        float av = (float)fabs(v[j]); /* exact: a 16-bit value fits binary32 */
        if (av > a) a = av;
      }
      float sc = a / 127.0f;
      s[i * (k / QK) + b] = sc;
      for (int j = 0; j < QK; ++j) {
        int q = 0;
        if (sc != 0.0f) {
          double t = round(v[j] / (double)sc); /* half away from zero */
          if (t > 127.0) t = 127.0;
          if (t < -127.0) t = -127.0;
          q = (int)t;
        }
        xq[i * k + b * QK + j] = (int8_t)q;
      }
    }
  return ORACLE_OK;
}

/* Integer code of weight j of a Q8_0 / Q4_0 block. */
static int int_code(int qtype, const uint8_t *blk, int j) {
  if (qtype == ORACLE_Q8_0) return (int8_t)blk[2 + j];
  int byte = blk[2 + (j % (QK / 2))];
  return ((j < QK / 2) ? (byte & 0x0f) : (byte >> 4)) - 8;
}

/* y[i][c] = sum_b s_ib * d_nb * P_inb, P_inb = sum_{j in block b} xq_ij * q_nj
 * (an exact integer), n = cols[c], the outer sum in binary64 in block order;
 * bound[i][c] = sum_j |s_ib xq_ij| |w_hat_nj| (the scale of an fp32
 * implementation's rounding error); qerr[i][c] = sum_b (s_ib / 2) sum_{j in b}
 * |w_hat_nj|, which bounds |y - x . w_hat| for the 16-bit x the codes came
 * from (every |x_ij - s_ib xq_ij| <= s_ib / 2).  Q8_0 and Q4_0 weights. */
int oracle_qlinear_x8(int qtype, const uint8_t *blocks, int64_t n, int64_t k, const int8_t *xq,
                      const float *s, int64_t m, const int64_t *cols, int64_t ncols, double *y,
                      double *bound, double *qerr) {
  if ((qtype != ORACLE_Q8_0 && qtype != ORACLE_Q4_0) || k <= 0 || k % QK != 0 || n <= 0 || m < 0 ||
      ncols < 0)
    return ORACLE_EINVAL;
  for (int64_t c = 0; c < ncols; ++c)
    if (cols[c] < 0 || cols[c] >= n) return ORACLE_EINVAL;
  const int64_t nb = k / QK, bb = oracle_block_bytes(qtype);
  for (int64_t c = 0; c < ncols; ++c) {
    const uint8_t *row = blocks + cols[c] * nb * bb;
    for (int64_t i = 0; i < m; ++i) {
      double acc = 0.0, bd = 0.0, qe = 0.0;
      for (int64_t b = 0; b < nb; ++b) {
        const uint8_t *blk = row + b * bb;
        const double d = oracle_half_to_double(get_d16(blk));
        const double sb = (double)s[i * nb + b];
        long long p = 0;
        double wsum = 0.0, xw = 0.0;
        for (int j = 0; j < QK; ++j) {
          const int q = int_code(qtype, blk, j);
          const int xv = xq[i * k + b * QK + j];
          p += (long long)xv * q;
          wsum += fabs((double)q * d);
          xw += fabs((double)xv) * fabs((double)q * d);
        }
        acc += sb * d * (double)p;
        bd += sb * xw;
        qe += sb / 2.0 * wsum;
      }
      y[i * ncols + c] = acc;
      bound[i * ncols + c] = bd;
      qerr[i * ncols + c] = qe;
    }
  }
  return ORACLE_OK;
}
