/*
 * eb.h -- C ABI of libeb: linear layers on block-quantized weights for
 * batch-1 embodied-model inference on AMD Instinct MI355X (gfx950).
 *
 * The operation is the quantized linear layer that the paper's runtime runs
 * in its backbone and head plugins (paper section 3.2, "latency-first fused
 * execution": operator fusion, backend-specific dispatch, buffer reuse and
 * graph replay for batch-1 inference) at the 8-bit and 4-bit C++
 * configurations it evaluates (section 4, Table 3):
 *
 *     y[m][n] = sum_k x[m][k] * w_hat[n][k],   w_hat = dequant(quant(W))
 *
 * Weight formats (ggml-style blocks of 32 consecutive weights along k, each
 * with one IEEE binary16 scale d16):
 *   EB_Q8_0: amax = max|w_j|, d16 = binary16_RNE(fl32(amax / 127)),
 *            q_j = clamp(round_half_away(w_j / d16), -127, 127); w_hat = q * d16.
 *   EB_Q4_0: m = signed element of largest |w_j| (first index wins),
 *            d16 = binary16_RNE(fl32(m / -8)),
 *            c_j = clamp(floor(w_j / d16 + 1/2), -8, 7); w_hat = c * d16.
 *   When d16 == 0 every code is 0.  Codes are rounded against the stored
 *   binary16 scale, exactly (the rounding decision equals the one on the exact
 *   quotient).
 *   EB_Q6_S (the 6-bit configuration; the paper names no format, this one is
 *            defined here): super-blocks of 256 weights in 16 sub-blocks of 16.
 *            m_j = signed element of largest |w| of sub-block j (first index
 *            wins), s_j = fl32(m_j / -32); d16 = binary16_RNE(fl32(max_j |s_j|
 *            / 127)); sc_j = clamp(round_half_away(s_j / d16), -127, 127)
 *            (0 when d16 == 0); e_j = d16 * sc_j;
 *            q_i = clamp(floor(w_i / e_j + 1/2), -32, 31) (0 when e_j == 0),
 *            stored as u_i = q_i + 32; w_hat = q * e_j.  k % 256 == 0.
 *
 * Canonical byte layout (array of blocks, row by row, k/32 blocks per row):
 *   Q8_0 block, 34 bytes: d16 little-endian, then q_0..q_31 as int8.
 *   Q4_0 block, 18 bytes: d16, then 16 bytes, byte i = (c_i + 8) | (c_{i+16} + 8) << 4.
 *   Q6_S super-block, 210 bytes (k/256 per row): d16, sc_0..sc_15 (int8),
 *     then 8 chunks of 24 bytes, chunk c holding weights 32c .. 32c + 31
 *     (local index i): byte i (0..15) = (u_i & 15) | (u_{i+16} & 15) << 4,
 *     byte 16 + t (t = 0..7) = (u_t >> 4) | (u_{t+8} >> 4) << 2 |
 *     (u_{t+16} >> 4) << 4 | (u_{t+24} >> 4) << 6.
 *
 * Device layout ("planar", what eb_quantize_* write and eb_qlinear reads),
 * inside one buffer of eb_qweights_bytes(type, n, k) bytes:
 *   qs plane at offset 0: row r, block b at byte (r * (k/32) + b) * QB, where
 *     QB = 32 (Q8_0, the 32 int8 codes) or 16 (Q4_0, the 16 packed bytes in
 *     the canonical order);
 *   d plane at byte offset d_off = round_up(n * (k/32) * QB, 256): row r, block
 *     b at binary16 index r * DS + b, DS = round_up(k/32, 8); entries b >= k/32
 *     are zero.
 *   Q6_S: qs plane of 24-byte chunks (QB = 24 per 32 weights, the chunk bytes
 *     above); int8 sub-scale plane at sc_off = round_up(n * (k/32) * 24, 256),
 *     row r at byte r * (k/16); d plane at round_up(sc_off + n * (k/16), 256),
 *     row stride DS = round_up(k/256, 8) binary16 entries.
 *   It holds the canonical bytes, rearranged; eb_qweights_to_canonical /
 *   eb_qweights_from_canonical convert in either direction.
 *
 * Conventions for every entry point:
 *   - All pointers are DEVICE pointers unless stated otherwise; the caller owns
 *     every buffer (weights, activations, outputs, and the workspaces that hold
 *     split-K partial sums, normalised activations and stack-plan tables:
 *     eb_qlinear_workspace_bytes, eb_qlinear_stack_workspace_bytes).  The
 *     library allocates no device memory and never synchronises the stream.
 *     Its cached state is the stack-plan cache of eb_qlinear_stack (host
 *     plans, their HIP graphs, one capture stream and one side stream per
 *     device, two events per plan that forks a side launch) and the compute
 *     unit count per device.
 *   - Work is enqueued on `stream` (0 = the null stream); EB_OK means the work
 *     was enqueued, not that it finished.
 *   - Arguments are validated on the host before anything is launched; on any
 *     error nothing is launched and the output buffers are untouched.
 *   - Inputs must be finite.  Quantization requires max|w| / 127 <= 65504 per
 *     block (the binary16 scale must not overflow).
 *   - Outputs must not overlap inputs (one exception: the residual of a
 *     residual-adding epilogue may be the output itself, see below).
 *   - Sizes: 1 <= n <= 2^31 - 1, 32 <= k <= 2^24 with k % 32 == 0 (k % 256
 *     == 0 for Q6_S),
 *     0 <= m <= 2^24 (m == 0 is a no-op).
 *   - Thread-compatible: concurrent calls must use different output buffers.
 */
#ifndef EB_H
#define EB_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t eb_status;
#define EB_OK 0
#define EB_ERR_INVALID (-1)     /* bad size, null pointer, bad enum value */
#define EB_ERR_ALIGN (-2)       /* pointer not aligned as required */
#define EB_ERR_UNSUPPORTED (-3) /* valid but unsupported combination (dtype pair, path) */
#define EB_ERR_HIP (-4)         /* the HIP runtime reported an error (no device, launch failure) */

/* quantization formats */
#define EB_Q8_0 1
#define EB_Q4_0 2
#define EB_Q6_S 3

/* element types */
#define EB_F32 0
#define EB_F16 1
#define EB_BF16 2

/* kernel paths for eb_qlinear_ex */
#define EB_PATH_AUTO 0 /* pick by m, qtype and shape (measured crossover) */
#define EB_PATH_GEMV 1 /* bandwidth-bound GEMV, requires m <= 8 and m' * k <= 65536, m' = m rounded up to 1, 2, 4 or 8 */
#define EB_PATH_MFMA 2 /* LDS-tiled dequantize-to-16-bit + MFMA, any m */
/* Low-precision prefill variant (section 3.2, backend-specific dispatch), Q8_0 /
 * Q4_0, opt-in only (EB_PATH_AUTO never takes it): x is quantized per
 * 32-element block along k to int8 (s = fl32(max|x| / 127), codes rounded half
 * away from zero against s, into the workspace: eb_qlinear_workspace_bytes),
 * the weight codes go to the int8 matrix cores as they are and each block's
 * exact integer product is scaled by s * d16 in fp32.  Accuracy: within 2e-3
 * of that method's exact value, normalised by sum |s xq||w_hat|; it differs
 * from the 16-bit product by at most sum_b (s_b / 2) sum_{k in b} |w_hat|.
 * No normalisation prologue (EB_ERR_UNSUPPORTED); epilogues as usual. */
#define EB_PATH_MFMA_I8 3

/* A quantized weight matrix W[n][k] in the planar device layout above.
 * `data` is a device pointer, 256-byte aligned, eb_qweights_bytes(type, n, k)
 * bytes; it is owned by the caller. */
typedef struct {
  int32_t type; /* EB_Q8_0 or EB_Q4_0 */
  int32_t reserved; /* must be 0 */
  int64_t n;    /* output features (rows of W) */
  int64_t k;    /* input features (columns of W), multiple of 32 */
  void *data;
} eb_qweights;

/* Byte offsets of the planar layout (all values in bytes except d_stride). */
typedef struct {
  int64_t qs_offset;     /* always 0 */
  int64_t qs_row_bytes;  /* (k/32) * QB */
  int64_t d_offset;      /* start of the binary16 scale plane */
  int64_t d_stride;      /* scale-plane row stride in binary16 elements (DS) */
  int64_t total_bytes;   /* == eb_qweights_bytes */
  int64_t canonical_bytes; /* size of the canonical form: n * (k/32) * (2 + QB), Q6_S n * (k/256) * 210 */
  int64_t sc_offset;     /* Q6_S: start of the int8 sub-scale plane (0 otherwise) */
  int64_t sc_stride;     /* Q6_S: its row stride in bytes, k/16 (0 otherwise) */
} eb_layout;

/* Steps of a decoder layer fused around one projection (paper section 3.2,
 * operator fusion on the batch-1 path; the backbones of section 2.1 are
 * decoder stacks whose projections sit between an RMS normalisation and a
 * residual addition, with a SiLU-gated feed-forward).
 *
 * Prologue EB_PRO_RMSNORM: x is the fp32 residual stream h[m][k]; the product
 *   takes x_hat[i][j] = round(h[i][j] * g[j] * r_i), r_i = 1 / sqrt(eps +
 *   (1/k) sum_j h[i][j]^2), rounded to nearest even in x_type, g = norm_weight.
 *   On the GEMV path every workgroup normalises while it stages x (no extra
 *   launch); on the MFMA path a row kernel writes x_hat first (one more launch)
 *   into the caller's workspace (m * k * 2 bytes, rounded up to 256, at its
 *   start); without a workspace that large such a call returns
 *   EB_ERR_UNSUPPORTED.
 * Epilogue EB_EPI_ADD: y = x_hat . w_hat^T + r, r = residual[m][n] of y_type;
 *   residual may be y itself (in-place update of the residual stream) but
 *   must not otherwise overlap y.
 * Epilogue EB_EPI_GLU: rows 2j and 2j + 1 of W are the gate and up rows of
 *   feature j (n even); y is [m][n/2] with y[i][j] = silu(gate) * up,
 *   silu(t) = t / (1 + exp(-t)) evaluated in fp32.
 * Accuracy: with e_g, e_u the accuracy bar of the two products (2e-3 of their
 *   sums of |x_hat||w_hat|, B_g and B_u), a GLU output is within
 *   2e-3 * (1.1 B_g |u| + |silu(g)| B_u + 0.0022 B_g B_u) (|silu'| < 1.1);
 *   an ADD output within the product's bar plus one fp32 rounding. */
#define EB_PRO_NONE 0
#define EB_PRO_RMSNORM 1
#define EB_EPI_NONE 0
#define EB_EPI_ADD 1
#define EB_EPI_GLU 2

/* One linear layer of a stack: y[m][n] = x[m][k] . w_hat^T, with optional
 * fused steps.  Fields after y_type may be left zero (no fused step). */
typedef struct {
  eb_qweights w;
  const void *x; /* device, row-major, 16-byte aligned: [m][k] of x_type, or fp32 [m][k]
                    with EB_PRO_RMSNORM */
  void *y;       /* device, [m][n] (EB_EPI_GLU: [m][n/2]) of y_type, row-major, 16-byte aligned */
  int64_t m;
  int32_t x_type; /* EB_F16 or EB_BF16: the activations the product consumes */
  int32_t y_type; /* EB_F32, EB_BF16 or EB_F16 */
  int32_t prologue;        /* EB_PRO_NONE or EB_PRO_RMSNORM */
  int32_t epilogue;        /* EB_EPI_NONE, EB_EPI_ADD or EB_EPI_GLU */
  const float *norm_weight; /* EB_PRO_RMSNORM: g[k], fp32, device, 16-byte aligned */
  const void *residual;    /* EB_EPI_ADD: [m][n] of y_type, device, 16-byte aligned */
  float norm_eps;          /* EB_PRO_RMSNORM: finite, >= 0 (a zero row needs eps > 0) */
  int32_t reserved;        /* must be 0 */
} eb_qlinear_op;

/* Library version string (static storage). */
const char *eb_version(void);

/* Human-readable name of a status code (static storage; never NULL). */
const char *eb_status_str(eb_status s);

/* Size in bytes of the planar device buffer for W[n][k] of format `type`
 * (a multiple of 256), or 0 if the arguments are invalid. Host-only. */
size_t eb_qweights_bytes(int32_t type, int64_t n, int64_t k);

/* Fills *out with the planar layout of W[n][k]. Host-only.
 * EB_ERR_INVALID on bad type/sizes or out == NULL. */
eb_status eb_qweights_layout(int32_t type, int64_t n, int64_t k, eb_layout *out);

/* Quantize fp32 W[n][k] (device, row-major, 16-byte aligned) into the planar
 * Q8_0 layout at `out` (device, 256-byte aligned, eb_qweights_bytes bytes).
 * Bit-exact with the definition above.  n == 0 is a no-op.
 * EB_ERR_INVALID: null pointer with n > 0, n < 0, k % 32 != 0 or out-of-range size.
 * EB_ERR_ALIGN: w not 16-byte aligned or out not 256-byte aligned. */
eb_status eb_quantize_q8_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream);

/* Same as eb_quantize_q8_0 for the Q4_0 format. */
eb_status eb_quantize_q4_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream);

/* Same as eb_quantize_q8_0 for the Q6_S format (k % 256 == 0, else
 * EB_ERR_INVALID).  Q6_S ops have GEMVs of their own (m <= 8; EB_PATH_AUTO
 * takes them up to m = 4; independent m == 1 ops share fused stack launches),
 * a matrix-core kernel of their own up to m = 128 (16 weight rows and up to 64
 * rows of x per workgroup, the whole of k; bfloat16 activations take w_hat as
 * hi/lo pairs, binary16 ones round it once), and the tile kernel of the other
 * formats beyond (k may be split); the accuracy of each path is as stated for
 * eb_qlinear.  They never join fused or grouped matrix-core stack launches. */
eb_status eb_quantize_q6_s(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream);

/* Write the canonical array-of-blocks bytes of *w into `dst` (device,
 * eb_layout.canonical_bytes bytes, no alignment requirement). */
eb_status eb_qweights_to_canonical(const eb_qweights *w, void *dst, hipStream_t stream);

/* Build the planar layout at `out` (device, 256-byte aligned,
 * eb_qweights_bytes bytes) from canonical blocks at `src` (device). */
eb_status eb_qweights_from_canonical(int32_t type, const void *src, int64_t n, int64_t k,
                                     void *out, hipStream_t stream);

/* eb_qlinear_fused_ws for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the scratch of the MFMA path -- the normalised activations of
 * a prologue, then the fp32 partial sums of a split of k -- lives in a
 * static device array of 32 MiB that the library holds on every GPU it runs
 * on until the process ends (its address is resolved on the first call on
 * each device).  No allocating routine is called.  The normalised
 * activations must fit the array (m * k * 2 bytes, rounded up to 256;
 * otherwise EB_ERR_UNSUPPORTED and nothing is launched); a split of k is
 * taken only when its partial sums fit the rest.  Nothing in the array needs
 * to start at zero (every element read is written earlier in the same call).
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, other threads, a graph replayed while another
 * call runs) race on it and give undefined results; calls on one stream are
 * ordered and safe.  Errors as eb_qlinear_fused, plus EB_ERR_HIP if the
 * array's device address cannot be resolved. */
eb_status eb_qlinear_fused_static(const eb_qlinear_op *op, int32_t path, hipStream_t stream);

/* y[m][n] = x[m][k] . w_hat[n][k]^T with fp32 accumulation, on the path chosen
 * automatically, with no workspace: the MFMA path then runs unsplit (see
 * eb_qlinear_fused_ws for the split of k a workspace allows).
 * x: device [m][k] of x_type (EB_F16 or EB_BF16); y: device [m][n] of y_type
 * (EB_F32, EB_BF16 or EB_F16, 16-bit outputs rounded to nearest even).
 * No bias.  Accuracy, with B = sum_k |x||w_hat| per output (plus the output
 * rounding when y_type is 16-bit):
 *   - GEMV path (m <= 8), any x_type: |y - y_exact| <= 2e-3 B;
 *   - MFMA path, EB_BF16 x, m <= 128: w_hat enters the matrix cores as a pair
 *     of bfloat16 values (hi + lo, within 2^-16 of w_hat): <= 2e-3 B;
 *   - MFMA path, EB_BF16 x, m > 128 (matrix-core bound): w_hat is rounded once
 *     to bfloat16 (8 significant bits): <= (2e-3 + 2^-8) B;
 *   - MFMA path, EB_F16 x: w_hat is rounded once to binary16 (11 significant
 *     bits, subnormal below 2^-14): <= 2e-3 B + 2^-25 sum_k |x|; requires
 *     |w_hat| <= 65504, i.e. max |w| <= 65504 in every block.
 *   (paper section 4, Table 3: the 8-/4-bit configurations are judged by the
 *   outputs they give; these bounds are this library's contract for them.)
 * EB_ERR_INVALID: w or its data NULL, bad type/sizes, an unknown x_type or
 * y_type, x/y NULL with m > 0, y overlapping x or the weights.
 * EB_ERR_ALIGN: x or y not 16-byte aligned, w->data not 256-byte aligned.
 * EB_ERR_UNSUPPORTED: x_type EB_F32. EB_ERR_HIP: launch failure. */
eb_status eb_qlinear(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                     int32_t y_type, hipStream_t stream);

/* One projection with its fused steps (eb_qlinear_op: prologue, epilogue),
 * on `path` (EB_PATH_*; AUTO picks as eb_qlinear does for the op's m, n, k),
 * with no workspace (as eb_qlinear_fused_ws with a null workspace).
 * Errors as eb_qlinear, and EB_ERR_INVALID for an unknown prologue or
 * epilogue, a missing norm_weight or residual, a negative or non-finite eps,
 * an odd n with EB_EPI_GLU, reserved != 0, or a residual overlapping y
 * without being y; EB_ERR_ALIGN for norm_weight or residual not 16-byte
 * aligned; EB_ERR_UNSUPPORTED as described for the prologue above. */
eb_status eb_qlinear_fused(const eb_qlinear_op *op, int32_t path, hipStream_t stream);

/* Bytes of workspace with which eb_qlinear_fused_ws runs *op on `path` as
 * planned (normalised activations of a prologue on the MFMA path, then the
 * fp32 partial sums of a split of k; at most m * k * 2 + 64 MiB).  0 when the
 * op needs none (GEMV path, m == 0) or is invalid.  Host-only. */
size_t eb_qlinear_workspace_bytes(const eb_qlinear_op *op, int32_t path);

/* eb_qlinear_fused with a caller workspace (paper section 3.2, buffer reuse:
 * the scratch of a projection is the caller's memory, reused across calls).
 * `workspace`: device, 256-byte aligned, `workspace_bytes` bytes, or NULL
 * with 0 bytes; it must not overlap the op's buffers.  A problem with too few
 * output tiles to fill the GPU (few rows and columns, long k) is split along
 * k when its partial sums fit the workspace after the normalised activations:
 * each split writes fp32 partials and a second kernel adds them in a fixed
 * order, so results are deterministic for a given workspace size (they can
 * differ with the size, by the order of summation).  The workspace is used
 * in stream order: calls that share one must be on one stream (or ordered).
 * Errors as eb_qlinear_fused, plus EB_ERR_INVALID for a non-null workspace
 * overlapping an operand or a null one with workspace_bytes > 0, and
 * EB_ERR_ALIGN for a workspace not 256-byte aligned. */
eb_status eb_qlinear_fused_ws(const eb_qlinear_op *op, int32_t path, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* eb_qlinear with an explicit kernel path (EB_PATH_*), for crossover
 * measurement and tests.  EB_ERR_UNSUPPORTED if the forced path cannot run
 * this shape (EB_PATH_GEMV with m > 8 or m' * k > 65536). */
eb_status eb_qlinear_ex(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                        int32_t y_type, int32_t path, hipStream_t stream);

/* Which path EB_PATH_AUTO takes for this problem (host-only, no launch). */
int32_t eb_qlinear_auto_path(int32_t type, int32_t x_type, int64_t m, int64_t n, int64_t k);

/* Bytes of workspace eb_qlinear_stack needs for this op list (the tables of
 * its fused and grouped launches, split-K partial sums and normalised
 * activations), 0 when it needs none or an op is invalid.  Host-only. */
size_t eb_qlinear_stack_workspace_bytes(const eb_qlinear_op *ops, int32_t n_ops);

/* Run ops[0..n_ops) on `stream` with the results of running them in order,
 * each as eb_qlinear_fused_ws would (paper section 3.2: graph replay,
 * operator fusion, buffer reuse).  `ops` is a HOST array.  All ops are
 * validated before anything is enqueued; n_ops == 0 is a no-op.
 *   Workspace: device, 256-byte aligned, at least
 *   eb_qlinear_stack_workspace_bytes(ops, n_ops) bytes (else EB_ERR_INVALID;
 *   NULL with 0 bytes when that is 0), overlapping no op's buffers.  A plan is
 *   cached per (op list, workspace pointer and size) and keeps its launch
 *   tables in the workspace: while the plan is cached (until
 *   eb_stack_cache_clear, or until a plan for another op list is built on an
 *   overlapping workspace, which drops it), the caller must not write to,
 *   free or reuse that workspace for anything else.
 *   Each op may carry fused steps (prologue, epilogue) as eb_qlinear_fused.
 *   Fusion: a run of consecutive ops in which no op reads or writes memory
 *   that an earlier op of the run writes (decided by address ranges of x, y,
 *   the weights, norm_weight and residual) is executed by fewer launches: m == 1
 *   ops with the same formats by one persistent GEMV launch per K size class,
 *   small-m MFMA ops (m <= 128) by one persistent launch, larger-m MFMA ops
 *   with the same formats by one grouped launch over all their output tiles
 *   (whose mostly-padded last row tiles may go to a small-m launch).  Results
 *   are those of running the ops in order; the m == 1 fusion is bitwise
 *   identical to single calls.  The small-m launch of split-off rows runs
 *   beside its grouped launch on a second, library-owned stream (default
 *   priority), forked from and joined back into `stream` inside the recorded
 *   graph.  EB_STACK_FUSE=0 disables fusion, EB_STACK_GROUP=0 the grouped
 *   launch, EB_STACK_SPLIT_TAIL=0 its tail split, EB_STACK_OVERLAP_TAIL=0 the
 *   second stream (the tail launch then follows the grouped one).
 *   Dependent chains: when an op on the MFMA path is split along k, writes
 *   fp32 output without the gated product, and the next op normalises that
 *   output (EB_PRO_RMSNORM with x == this y, same m, k == this n), the
 *   split's reduction also writes the next op's normalised activations, with
 *   the same bits as its own row kernel; EB_STACK_FUSE_NORM=0 keeps the row
 *   kernel.
 *   Graph replay: the first call with a given op list (same pointers, sizes,
 *   types) builds a plan, records it into a HIP graph on a library-owned
 *   stream and caches both; later calls replay the graph with one launch.
 *   EB_STACK_GRAPH=0 launches the plan directly instead; EB_STACK_DEBUG=1
 *   prints each plan's steps to stderr when it is built.  Called while
 *   `stream` itself is being captured, the ops are launched plainly into it.
 * Memory: the workspace holds the plan's device tables (about 100 bytes per
 * fused op, written once when the plan is built), a split-K area when one of
 * its ops is split, and, for EB_PRO_RMSNORM ops on the MFMA path, the
 * normalised activations (the largest total m * k * 2 bytes of one launch
 * step).  At most 64 plans are cached; beyond that the cache is cleared. */
eb_status eb_qlinear_stack(const eb_qlinear_op *ops, int32_t n_ops, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* Number of kernel launches eb_qlinear_stack makes for this op list (host
 * only; nothing is allocated or launched), or a negative eb_status if an op is
 * invalid. */
int32_t eb_qlinear_stack_launches(const eb_qlinear_op *ops, int32_t n_ops);

/* Drop every cached stack plan and graph (after the device has finished its
 * work); their workspaces are then the caller's again. */
eb_status eb_stack_cache_clear(void);

#ifdef __cplusplus
}
#endif

#endif /* EB_H */
