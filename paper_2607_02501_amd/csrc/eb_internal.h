// eb_internal.h -- declarations shared by the library's translation units.
// Host-side launchers live next to their kernels; eb_api.cpp validates
// arguments and dispatches to them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/eb.h"
#include "../../include/eb_tuning.h"

namespace eb {

constexpr int kQK = 32;    // weights per block (Q6_S: per 24-byte code chunk)
constexpr int kQK6 = 256;  // weights per Q6_S super-block

__host__ __device__ inline int64_t qs_bytes_per_block(int32_t type) {
  return type == EB_Q8_0 ? 32 : (type == EB_Q4_0 ? 16 : 24);
}
__host__ __device__ inline int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

struct Layout {
  int64_t nb;          // blocks (Q6_S: 32-weight code chunks) per row
  int64_t qs_row;      // bytes per qs row
  int64_t d_off;       // byte offset of the binary16 scale plane
  int64_t ds;          // scale-plane row stride (elements)
  int64_t total;       // total bytes
  int64_t sc_off = 0;  // Q6_S: byte offset of the int8 sub-block scale plane
  int64_t ss = 0;      // Q6_S: its row stride (bytes, k / 16)
};

inline Layout layout_of(int32_t type, int64_t n, int64_t k) {
  Layout L;
  L.nb = k / kQK;
  L.qs_row = L.nb * qs_bytes_per_block(type);
  if (type == EB_Q6_S) {
    L.sc_off = round_up(n * L.qs_row, 256);
    L.ss = k / 16;
    L.d_off = round_up(L.sc_off + n * L.ss, 256);
    L.ds = round_up(k / kQK6, 8);
  } else {
    L.d_off = round_up(n * L.qs_row, 256);
    L.ds = round_up(L.nb, 8);
  }
  L.total = round_up(L.d_off + n * L.ds * 2, 256);
  return L;
}

// weights per canonical block and bytes per canonical block
inline int64_t block_elems(int32_t type) { return type == EB_Q6_S ? kQK6 : kQK; }
inline int64_t canonical_block_bytes(int32_t type) {
  return type == EB_Q6_S ? 2 + 16 + 192 : 2 + qs_bytes_per_block(type);
}

// Fused steps of one op (EB_PRO_*, EB_EPI_*) as the kernels take them.  The
// GEMV kernels apply the RMS-normalisation prologue themselves while staging
// x (x is then the fp32 residual stream, `gamma` its weights); the MFMA
// kernels read activations normalised beforehand by launch_rmsnorm and only
// apply the epilogue.  `r` is the residual of EB_EPI_ADD ([m][n] of the
// output type, possibly the output itself).
// pro and epi are whole dwords: kernels that read an op's Fuse from a
// table in device memory then get them by scalar loads, whereas a 16-bit
// field takes a vector load, whose wait also waits for every vector load
// issued before it (the next tile's prefetch in the persistent kernels; no
// measurable change on the action-expert and VLM passes, which run few tiles
// per workgroup).
struct Fuse {
  const float *gamma;
  const void *r;
  float eps;
  int32_t pro, epi;
};

// ---- launchers (each returns hipSuccess or the launch error) ----
hipError_t launch_quantize(int32_t type, const float *w, int64_t n, int64_t k, void *out,
                           hipStream_t s);
hipError_t launch_to_canonical(int32_t type, const void *planar, int64_t n, int64_t k, void *dst,
                               hipStream_t s);
hipError_t launch_from_canonical(int32_t type, const void *src, int64_t n, int64_t k, void *out,
                                 hipStream_t s);

// GEMV path: m <= 8, (m rounded up to 1, 2, 4 or 8) * k <= kGemvMaxMK
constexpr int64_t kGemvMaxM = 8;
constexpr int64_t kGemvMaxMK = 65536;
hipError_t launch_gemv(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                       int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s);

// x_hat[i][j] = round_xt(h[i][j] * gamma[j] / sqrt(eps + mean_j h[i][j]^2)),
// h fp32 [m][k], x_hat [m][k] of xt (EB_F16 / EB_BF16); one workgroup per row.
hipError_t launch_rmsnorm(const float *h, const float *gamma, float eps, int64_t m, int64_t k,
                          int32_t xt, void *out, hipStream_t s);

// The normalisation prologue of the next projection, fused into the split-K
// reduction of a projection whose fp32 output h is that projection's input:
// the reduction writes h (+ the residual) as the plain reduction does, then
// x_hat = round_xt(h * gamma * r_i) into xout, with the same bits as
// launch_rmsnorm on that h.  One workgroup per row; n % 4 == 0.
struct NormOut {
  const float *gamma;
  float eps;
  int32_t xt;
  void *xout;
};
hipError_t launch_splitk_reduce_rmsnorm(const float *ws, int splits, int64_t ws_stride, int64_t m,
                                        int64_t n, float *y, const float *residual,
                                        const NormOut &no, hipStream_t s);

// Fused m == 1 GEMV over several independent matrices (one launch).  The
// table lives in device memory; unit_begin (prefix sum of n * ku) ascends.
struct M1Op {
  const uint8_t *w;   // planar weights
  const void *x;      // activations [k] (16-bit; fp32 h with the normalisation prologue)
  void *y;            // outputs [n] (gate/up epilogue: [n / 2])
  int64_t n;
  int64_t d_off;      // scale-plane offset
  int64_t ds;         // scale-plane row stride (elements)
  int64_t sc_off;     // Q6_S: sub-scale plane offset (unused otherwise)
  int64_t unit_begin; // work units before this matrix
  int32_t k;
  int32_t ku;         // work units per row: 16-byte code units (Q6_S: 64-weight units)
  int32_t yt;
  int32_t pad;
  Fuse f;
};
// An m == 1 op the fused GEMV launch takes (k within its slot range; the
// gate/up epilogue needs at least two rows per wave).
bool m1_fusable(int32_t type, int64_t m, int64_t k, int32_t epi);
int m1_slots(int32_t type, int64_t k);
// Fills *o for one matrix; returns its number of work units (n * ku).
int64_t m1_fill(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x, void *y,
                int32_t yt, const Fuse &f, int64_t unit_begin, M1Op *o);
// All matrices of one launch have the same slot count ns (m1_slots); units
// and rows are the totals over the table.
hipError_t launch_gemv_m1_multi(int32_t type, int32_t xt, int ns, const M1Op *dev_ops, int nops,
                                int64_t units, int64_t rows, hipStream_t s);

// MFMA path: any m.  A plan fixes the tile configuration and the split of K
// over workgroups; with splits > 1 the launch needs ws_bytes of fp32 workspace
// (partial sums, summed in order by a second kernel).
struct MfmaPlan {
  int cfg = 0;
  bool q6 = false;        // Q6_S weights: the Q6_S kernel (any m, no split)
  bool hl = false;        // bfloat16 activations at m <= 128: hi/lo weight tiles
  bool narrow = false;    // m <= kNarrowMaxM: the narrow kernel (splits > 1: plus the reduction)
  int splits = 1;
  int kts = 0;            // K-tiles of 64 per split
  int64_t ws_stride = 0;  // floats between the partial outputs of two splits
  size_t ws_bytes = 0;
};
// max_ws: bytes of partial-sum workspace the call may use (0: no split);
// force_cfg >= 0 / force_splits > 0 fix the tile configuration / split count
// (tuning and tests; a forced choice that does not fit is not taken).
MfmaPlan plan_mfma(int32_t type, int32_t xt, int64_t m, int64_t n, int64_t k, size_t max_ws,
                   int force_cfg = -1, int force_splits = 0);
constexpr size_t kMaxSplitWorkspace = size_t(64) << 20;  // partial sums a plan may ask for
// ws == nullptr runs the plan's configuration unsplit.  norm_next (split runs
// with an fp32 output and no gated product only) fuses the next projection's
// normalisation into the reduction.
hipError_t launch_mfma(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                       int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f,
                       const MfmaPlan &plan, float *ws, hipStream_t s,
                       const NormOut *norm_next = nullptr);
// One launch of the tile kernel for tile configuration `cfg` (hi/lo weight
// tiles when hl) over `sp` splits of k of kts K-tiles each (the reduction of
// the splits is not part of it).  Defined in mfma_tile.h and instantiated for
// each weight format and activation type in its own translation unit.
template <int QT, int XT>
hipError_t mfma_tile_launch(int cfg, bool hl, const void *wdata, int64_t n, int64_t k, const void *x,
                            int64_t m, void *y, int32_t yt, const Fuse &f, int sp, int kts,
                            float *ws, int64_t st, hipStream_t s);
// Lone small-m projections (m <= kNarrowMaxM) in one launch: 16 weight rows
// and the whole of k per workgroup, k split over its waves and the partial
// tiles added through LDS (mfma_narrow.hip).  hl: bfloat16 hi/lo pairs.
// When the 16-row workgroups do not fill the GPU, k is split (narrow_splits)
// and each split writes fp32 partial sums for the ordered reduction.
constexpr int64_t kNarrowMaxM = 64;
constexpr int64_t kNarrowMaxK = 2048;  // k per split
constexpr int kNarrowMaxSplits = 8;
bool narrow_fits(int64_t m, int64_t n, int64_t k, int splits);
int narrow_splits(int64_t n, int64_t k, int cus);
hipError_t launch_mfma_narrow(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                              int32_t xt, bool hl, int64_t m, void *y, int32_t yt, const Fuse &f,
                              int splits, float *ws, int64_t ws_stride, hipStream_t s);
// Q6_S weights, m <= 8 (gemv_q6.hip): a wave per pair of weight rows, lanes
// over 32-weight chunks, fp32 products of the 6-bit codes and x staged in LDS.
bool gemv_q6_fits(int64_t m, int64_t n, int64_t k);
// m == 1 Q6_S kernel (k up to 16384) and its fused multi-matrix launch, the
// counterparts of m1_slots / m1_fusable / m1_fill / launch_gemv_m1_multi
int q6_m1_slots(int64_t k);
bool q6_m1_fits(int64_t k);
bool q6_m1_fusable(int64_t k, int32_t epi);
int64_t q6_m1_fill(const void *wdata, int64_t n, int64_t k, const void *x, void *y, int32_t yt,
                   const Fuse &f, int64_t unit_begin, M1Op *o);
hipError_t launch_gemv_q6_multi(int32_t xt, int ns, const M1Op *dev_ops, int nops, int64_t units,
                                int64_t rows, hipStream_t s);
hipError_t launch_gemv_q6(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt,
                          int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s);
// Q6_S weights on the matrix cores, any m, one launch (mfma_q6.hip): 16
// weight rows and up to 64 rows of x per workgroup, k split over its waves.
// bfloat16 activations take w_hat as hi/lo pairs at every m.
bool q6_fits(int64_t m, int64_t n, int64_t k);
hipError_t launch_mfma_q6(const void *wdata, int64_t n, int64_t k, const void *x, int32_t xt,
                          int64_t m, void *y, int32_t yt, const Fuse &f, hipStream_t s);
// Low-precision prefill variant (mfma_i8.hip, Q8_0 / Q4_0): x quantized per
// 32-element block to int8 into the workspace (i8_workspace_bytes: the codes,
// then the block scales), then the int8 matrix-core product with per-block
// scaling.
size_t i8_workspace_bytes(int64_t m, int64_t k);
bool i8_fits(int64_t m, int64_t n, int64_t k);
hipError_t launch_mfma_i8(int32_t type, const void *wdata, int64_t n, int64_t k, const void *x,
                          int32_t xt, int64_t m, void *y, int32_t yt, const Fuse &f, void *ws,
                          hipStream_t s);
// Whether a workgroup's byte spans of a bm x bn tile fit 32-bit buffer offsets.
bool mfma_fits_offsets(int32_t type, int64_t n, int64_t k, int bm, int bn);
int mfma_tile_count();
int mfma_cfg_bm(int cfg);        // rows of a tile configuration
double mfma_cfg_rate(int cfg);   // its measured full-chip rate, TFLOP/s

// Grouped MFMA launch over independent ops with more rows than a fused
// small-m launch takes: one workgroup per output tile of any op, in a table
// ordered longest tiles first (section 3.2: fewer, fuller launches).
struct GOp {
  const uint8_t *w;   // quantized weights (planar layout)
  const uint16_t *x;  // activations [m][k]
  void *y;            // outputs [m][n]
  int64_t n, k, d_off, ds, m;
  int64_t sc_off;     // Q6_S sub-scale plane (not grouped; 0 otherwise)
  int32_t yt, pad;
  Fuse f;
};
// Chooses the tile configuration for the group and fills the workgroup table
// (op, tile); returns the configuration, or -1 when none fits every op.
int plan_grouped(int32_t type, const std::vector<GOp> &ops, std::vector<int2> &order);
hipError_t launch_mfma_grouped(int32_t type, int32_t xt, int cfg, const GOp *ops, const int2 *order,
                                int64_t entries, hipStream_t s);
template <int QT, int XT>
hipError_t mfma_tile_launch_grouped(int cfg, const GOp *ops, const int2 *order, int64_t entries,
                                    hipStream_t s);

// Fused MFMA launch over several independent ops of a stack: one persistent
// launch whose workgroups each run a contiguous range of output tiles
// (units), balanced by K-tile steps, as one continuous load/compute pipeline.
// The table and the per-workgroup unit ranges live in device memory.
struct MMOp {
  const uint8_t *w;    // planar weights
  const uint16_t *x;   // activations [m][k]
  void *y;             // outputs [m][n]
  int64_t d_off;       // scale-plane offset
  int64_t unit_end;    // tiles of this op and all ops before it
  int32_t ds, m, n, k; // ds: scale-plane row stride (elements)
  int32_t tiles_n, nk, yt, pad;
  Fuse f;
};
constexpr int64_t kMMaxK = int64_t(1) << 22;  // k < this keeps per-tile byte spans in 31 bits
int mm_cfg(int64_t max_m);                // tile configuration for a run
int64_t mm_tiles(int cfg, int64_t m, int64_t n);
int mm_bk(int cfg);                       // k covered by one step of the configuration
// The 128-wide-step fused kernel (configuration 0), in its own source file.
hipError_t launch_lds2(int32_t type, int32_t xt, bool hl, int32_t yt, const MMOp *ops, int nops,
                       const int64_t *wg, int groups, hipStream_t s);
// Fills the unit ranges wg[0..groups] (balanced by steps) for a table whose
// unit_end / nk are set; returns the number of workgroups to launch.
// Workgroup unit ranges of a fused small-m launch; max_groups > 0 caps the
// workgroup count (rounded to a multiple of 8).
int mm_partition(const std::vector<MMOp> &ops, int cfg, std::vector<int64_t> &wg,
                 int max_groups = 0);
// All ops of one launch share the weight format, x type and y type.
// groups must be a positive multiple of 8 (mm_partition's result).
// hl: bfloat16 activations with w_hat as hi/lo pairs (ignored for binary16);
// a launch of only the split-off rows of large-m ops runs without (the ops'
// bound is the large-m one, w_hat rounded once).
hipError_t launch_mfma_multi(int32_t type, int32_t xt, bool hl, int32_t yt, int cfg, const MMOp *dev_ops,
                             int nops, const int64_t *dev_wg, int groups, hipStream_t s);

// number of compute units of the current device (cached per device)
int device_cu_count();

}  // namespace eb
