// eb_api.cpp -- the C ABI: host-side validation, path dispatch and the stack
// runner with HIP-graph replay (paper section 3.2: graph replay, buffer reuse
// and backend-specific dispatch for latency-first batch-1 execution).
//
// Validation happens entirely on the host before any HIP call, so every error
// path is testable without a GPU and nothing is launched on error.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "eb_internal.h"

namespace eb {

int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64) {
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (dev < 64) cache[dev].store(cus, std::memory_order_relaxed);
  return cus;
}

namespace {

constexpr int64_t kMaxN = 0x7fffffff;
constexpr int64_t kMaxK = int64_t(1) << 24;
constexpr int64_t kMaxM = int64_t(1) << 24;

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool valid_type(int32_t t) { return t == EB_Q8_0 || t == EB_Q4_0 || t == EB_Q6_S; }
bool known_dtype(int32_t t) { return t == EB_F32 || t == EB_F16 || t == EB_BF16; }

// k: a multiple of the format's block (32 weights, 256 for Q6_S)
bool valid_k(int32_t type, int64_t k) {
  return k >= 0 && k <= kMaxK && k % block_elems(type) == 0;
}

bool valid_nk(int32_t type, int64_t n, int64_t k) {
  return n >= 1 && n <= kMaxN && k >= kQK && valid_k(type, k);
}

size_t canonical_bytes(int32_t type, int64_t n, int64_t k) {
  return (size_t)n * (size_t)(k / block_elems(type)) * (size_t)canonical_block_bytes(type);
}

bool overlaps(const void *a, size_t an, const void *b, size_t bn) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return an && bn && a0 < b0 + bn && b0 < a0 + an;
}

size_t dsize(int32_t t) { return t == EB_F32 ? 4 : 2; }

int64_t gemv_mt(int64_t m) { return m <= 1 ? 1 : (m <= 2 ? 2 : (m <= 4 ? 4 : 8)); }

bool gemv_fits(int64_t m, int64_t k) {
  return m >= 1 && m <= kGemvMaxM && gemv_mt(m) * k <= kGemvMaxMK;
}

eb_status check_weights(const eb_qweights *w) {
  if (!w || !w->data || !valid_type(w->type) || w->reserved != 0 || !valid_nk(w->type, w->n, w->k))
    return EB_ERR_INVALID;
  if (!aligned(w->data, 256)) return EB_ERR_ALIGN;
  return EB_OK;
}

// One op as a plain projection (no fused steps).
eb_qlinear_op plain_op(const eb_qweights *w, const void *x, int32_t xt, int64_t m, void *y,
                       int32_t yt) {
  eb_qlinear_op o{};
  o.w = *w;
  o.x = x;
  o.y = y;
  o.m = m;
  o.x_type = xt;
  o.y_type = yt;
  return o;
}

// Output columns of an op (the gate/up epilogue halves them).
int64_t n_out(const eb_qlinear_op &o) { return o.epilogue == EB_EPI_GLU ? o.w.n / 2 : o.w.n; }
// Bytes of x the op reads (fp32 residual stream under the normalisation prologue).
size_t x_bytes(const eb_qlinear_op &o) {
  return (size_t)o.m * (size_t)o.w.k * (o.prologue == EB_PRO_RMSNORM ? 4 : 2);
}

Fuse fuse_of(const eb_qlinear_op &o) {
  Fuse f{};
  f.gamma = o.prologue == EB_PRO_RMSNORM ? o.norm_weight : nullptr;
  f.r = o.epilogue == EB_EPI_ADD ? o.residual : nullptr;
  f.eps = o.norm_eps;
  f.pro = o.prologue;
  f.epi = o.epilogue;
  return f;
}

eb_status check_op(const eb_qlinear_op &o, int32_t path) {
  eb_status st = check_weights(&o.w);
  if (st != EB_OK) return st;
  const int64_t m = o.m;
  if (m < 0 || m > kMaxM) return EB_ERR_INVALID;
  if (!known_dtype(o.x_type) || !known_dtype(o.y_type)) return EB_ERR_INVALID;
  if (path != EB_PATH_AUTO && path != EB_PATH_GEMV && path != EB_PATH_MFMA && path != EB_PATH_MFMA_I8)
    return EB_ERR_INVALID;
  if (o.prologue != EB_PRO_NONE && o.prologue != EB_PRO_RMSNORM) return EB_ERR_INVALID;
  if (o.epilogue != EB_EPI_NONE && o.epilogue != EB_EPI_ADD && o.epilogue != EB_EPI_GLU)
    return EB_ERR_INVALID;
  if (o.reserved != 0) return EB_ERR_INVALID;
  if (o.prologue == EB_PRO_RMSNORM && !(std::isfinite(o.norm_eps) && o.norm_eps >= 0.0f))
    return EB_ERR_INVALID;
  if (o.epilogue == EB_EPI_GLU && o.w.n % 2 != 0) return EB_ERR_INVALID;
  if (o.x_type == EB_F32) return EB_ERR_UNSUPPORTED;
  if (m == 0) return EB_OK;
  if (!o.x || !o.y) return EB_ERR_INVALID;
  if (o.prologue == EB_PRO_RMSNORM && !o.norm_weight) return EB_ERR_INVALID;
  if (o.epilogue == EB_EPI_ADD && !o.residual) return EB_ERR_INVALID;
  if (!aligned(o.x, 16) || !aligned(o.y, 16)) return EB_ERR_ALIGN;
  if (o.prologue == EB_PRO_RMSNORM && !aligned(o.norm_weight, 16)) return EB_ERR_ALIGN;
  if (o.epilogue == EB_EPI_ADD && !aligned(o.residual, 16)) return EB_ERR_ALIGN;
  const size_t yb = (size_t)m * (size_t)n_out(o) * dsize(o.y_type);
  const size_t wb = eb_qweights_bytes(o.w.type, o.w.n, o.w.k);
  if (overlaps(o.y, yb, o.x, x_bytes(o)) || overlaps(o.y, yb, o.w.data, wb)) return EB_ERR_INVALID;
  if (o.prologue == EB_PRO_RMSNORM && overlaps(o.y, yb, o.norm_weight, (size_t)o.w.k * 4))
    return EB_ERR_INVALID;
  if (o.epilogue == EB_EPI_ADD && o.residual != o.y && overlaps(o.y, yb, o.residual, yb))
    return EB_ERR_INVALID;
  if (path == EB_PATH_GEMV && !gemv_fits(m, o.w.k)) return EB_ERR_UNSUPPORTED;
  if (path == EB_PATH_MFMA_I8 && (o.w.type == EB_Q6_S || o.prologue != EB_PRO_NONE ||
                                  !i8_fits(m, o.w.n, o.w.k)))
    return EB_ERR_UNSUPPORTED;
  if (o.w.type == EB_Q6_S && path == EB_PATH_GEMV && !gemv_q6_fits(m, o.w.n, o.w.k))
    return EB_ERR_UNSUPPORTED;
  if (o.w.type == EB_Q6_S && path == EB_PATH_MFMA && !q6_fits(m, o.w.n, o.w.k))
    return EB_ERR_UNSUPPORTED;
  return EB_OK;
}

// Path choice from the measured GEMV / MFMA crossover on MI355X (single ops
// without a workspace, replayed from a graph; Q4_0 and Q8_0 at the decode /
// prefill / action-expert shapes): the GEMV wins at m = 1 everywhere; at
// m = 2..4 when the matrix has 4096 rows or more (with 1024 or 2048 the
// matrix cores win by 20-55%); at m = 5..8 where, in addition, the narrow
// matrix-core kernel does not apply (k > 2048: the unsplit tile kernel loses
// by 5-30%; the narrow kernel wins by 15-50%, or ties within 2%).
// Q6_S: its GEMV up to m = 4, its matrix-core kernel beyond.
int32_t pick_path(int32_t type, int32_t xt, int64_t m, int64_t n, int64_t k) {
  (void)xt;
  if (type == EB_Q6_S) return m <= 4 && gemv_q6_fits(m, n, k) ? EB_PATH_GEMV : EB_PATH_MFMA;
  if (!gemv_fits(m, k)) return EB_PATH_MFMA;
  if (m == 1) return EB_PATH_GEMV;
  if (n < 4096) return EB_PATH_MFMA;
  if (m <= 4) return EB_PATH_GEMV;
  return narrow_fits(m, n, k, 1) ? EB_PATH_MFMA : EB_PATH_GEMV;
}

// Bytes of normalised activations an op on the MFMA path needs (256-aligned).
size_t xhat_bytes(const eb_qlinear_op &o) {
  return o.prologue == EB_PRO_RMSNORM ? (size_t)round_up(o.m * o.w.k * 2, 256) : 0;
}

// One op on the MFMA path with a fixed plan: the prologue's row kernel writes
// the normalised activations to xbuf, then the product reads them.
// pre_normed: xbuf already holds them (written by the reduction of the op
// before, see NormOut); norm_next: this op's reduction writes the next op's.
hipError_t launch_mfma_op(const eb_qlinear_op &o, const MfmaPlan &P, void *xbuf, float *ws,
                          hipStream_t s, bool pre_normed = false,
                          const NormOut *norm_next = nullptr) {
  const void *x = o.x;
  Fuse f = fuse_of(o);
  if (o.prologue == EB_PRO_RMSNORM && pre_normed) {
    x = xbuf;
    f.pro = EB_PRO_NONE;
    f.gamma = nullptr;
  } else if (o.prologue == EB_PRO_RMSNORM) {
    hipError_t e = launch_rmsnorm(static_cast<const float *>(o.x), o.norm_weight, o.norm_eps, o.m,
                                  o.w.k, o.x_type, xbuf, s);
    if (e != hipSuccess) return e;
    x = xbuf;
    f.pro = EB_PRO_NONE;
    f.gamma = nullptr;
  }
  return launch_mfma(o.w.type, o.w.data, o.w.n, o.w.k, x, o.x_type, o.m, o.y, o.y_type, f, P, ws, s,
                     norm_next);
}

// Scratch of one op on the MFMA path inside a workspace of `cap` bytes: the
// normalised activations of a prologue (xb bytes at offset 0), then the
// split-K partial sums of the plan (P.ws_bytes, only if they fit).
struct OpScratch {
  MfmaPlan P;
  size_t xb = 0;
  size_t total = 0;
};

OpScratch op_scratch(const eb_qlinear_op &o, size_t cap, int force_cfg = -1, int force_splits = 0) {
  OpScratch r;
  r.xb = xhat_bytes(o);
  const size_t left = cap > r.xb ? std::min(cap - r.xb, kMaxSplitWorkspace) : 0;
  r.P = plan_mfma(o.w.type, o.x_type, o.m, o.w.n, o.w.k, left, force_cfg, force_splits);
  r.total = r.xb + r.P.ws_bytes;
  return r;
}

// One op with the caller's workspace `ws` (device, 256-byte aligned, wsb
// bytes; may be null with wsb == 0: then the MFMA path runs unsplit and a
// prologue on it is unsupported).
eb_status launch_op(const eb_qlinear_op &o, int32_t path, uint8_t *ws, size_t wsb, hipStream_t s,
                    int force_cfg = -1, int force_splits = 0) {
  if (o.m == 0) return EB_OK;
  if (path == EB_PATH_AUTO) path = pick_path(o.w.type, o.x_type, o.m, o.w.n, o.w.k);
  hipError_t e;
  if (path == EB_PATH_GEMV) {
    e = launch_gemv(o.w.type, o.w.data, o.w.n, o.w.k, o.x, o.x_type, o.m, o.y, o.y_type, fuse_of(o), s);
  } else if (path == EB_PATH_MFMA_I8) {
    if (!ws || wsb < i8_workspace_bytes(o.m, o.w.k)) return EB_ERR_UNSUPPORTED;
    e = launch_mfma_i8(o.w.type, o.w.data, o.w.n, o.w.k, o.x, o.x_type, o.m, o.y, o.y_type, fuse_of(o),
                       ws, s);
  } else {
    const OpScratch sc = op_scratch(o, ws ? wsb : 0, force_cfg, force_splits);
    if (sc.xb && (!ws || wsb < sc.xb)) return EB_ERR_UNSUPPORTED;
    float *part = sc.P.splits > 1 ? reinterpret_cast<float *>(ws + sc.xb) : nullptr;
    e = launch_mfma_op(o, sc.P, ws, part, s);
  }
  return e == hipSuccess ? EB_OK : EB_ERR_HIP;
}

// Workspace arguments: null with 0 bytes, or 256-byte aligned device memory
// that overlaps none of the op's buffers.
eb_status check_workspace(const eb_qlinear_op *ops, int32_t n_ops, const void *ws, size_t wsb) {
  if (!ws) return wsb == 0 ? EB_OK : EB_ERR_INVALID;
  if (!aligned(ws, 256)) return EB_ERR_ALIGN;
  for (int32_t i = 0; i < n_ops; ++i) {
    const eb_qlinear_op &o = ops[i];
    if (o.m == 0) continue;
    const size_t yb = (size_t)o.m * (size_t)n_out(o) * dsize(o.y_type);
    if (overlaps(ws, wsb, o.x, x_bytes(o)) || overlaps(ws, wsb, o.y, yb) ||
        overlaps(ws, wsb, o.w.data, eb_qweights_bytes(o.w.type, o.w.n, o.w.k)) ||
        (o.prologue == EB_PRO_RMSNORM && overlaps(ws, wsb, o.norm_weight, (size_t)o.w.k * 4)) ||
        (o.epilogue == EB_EPI_ADD && overlaps(ws, wsb, o.residual, yb)))
      return EB_ERR_INVALID;
  }
  return EB_OK;
}

eb_status quantize_common(int32_t type, const float *w, int64_t n, int64_t k, void *out,
                          hipStream_t s) {
  if (n < 0 || n > kMaxN || !valid_k(type, k)) return EB_ERR_INVALID;
  if (n == 0 || k == 0) return EB_OK;
  if (!w || !out) return EB_ERR_INVALID;
  if (!aligned(w, 16) || !aligned(out, 256)) return EB_ERR_ALIGN;
  if (overlaps(w, (size_t)n * k * 4, out, eb_qweights_bytes(type, n, k))) return EB_ERR_INVALID;
  return launch_quantize(type, w, n, k, out, s) == hipSuccess ? EB_OK : EB_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Stack plans.  A plan runs the ops in order; consecutive m == 1 GEMV ops with
// the same formats that neither read nor write what an earlier op of the run
// writes (checked by address ranges) are fused: the run is issued as one
// persistent launch per slot count, which is equivalent to running them in
// order because no op of the run observes another.  The plan and its device
// op table are cached per op list, together with the HIP graph that replays it.
// ---------------------------------------------------------------------------
struct Range {
  uintptr_t a, b;  // [a, b)
  bool hits(const Range &o) const { return a < o.b && o.a < b; }
};

// What an op reads (x, weights, normalisation weights, residual) and writes (y).
struct OpSpan {
  Range rd[4];
  int nrd = 0;
  Range y;
};

OpSpan span_of(const eb_qlinear_op &o) {
  auto range = [](const void *p, size_t bytes) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return Range{a, a + (uintptr_t)bytes};
  };
  OpSpan s;
  s.rd[s.nrd++] = range(o.x, x_bytes(o));
  s.rd[s.nrd++] = range(o.w.data, eb_qweights_bytes(o.w.type, o.w.n, o.w.k));
  if (o.prologue == EB_PRO_RMSNORM) s.rd[s.nrd++] = range(o.norm_weight, (size_t)o.w.k * 4);
  const size_t yb = (size_t)o.m * (size_t)n_out(o) * dsize(o.y_type);
  if (o.epilogue == EB_EPI_ADD) s.rd[s.nrd++] = range(o.residual, yb);
  s.y = range(o.y, yb);
  return s;
}

// op b may join a run containing op a only if neither observes the other
bool independent(const OpSpan &a, const OpSpan &b) {
  if (b.y.hits(a.y)) return false;
  for (int i = 0; i < b.nrd; ++i)
    if (b.rd[i].hits(a.y)) return false;
  for (int i = 0; i < a.nrd; ++i)
    if (b.y.hits(a.rd[i])) return false;
  return true;
}

// The prologue of an op on the MFMA path: its row kernel writes the
// normalised activations into the plan's buffer at `off`.
struct NormJob {
  const float *h, *gamma;
  float eps;
  int32_t xt;
  int64_t m, k;
  size_t off;
};

// Internal copies of ops whose x was replaced by an offset into the plan's
// normalised-activation buffer carry this marker in `reserved` (user ops must
// have reserved == 0).
constexpr int32_t kRelX = 1;

// Cap on the workgroups of a split-off-rows launch running beside a grouped
// launch (0: one per CU, as alone).  Measured on the m = 816 VLM prefill pass:
// no cap 3.89 ms, 128 or 64 workgroups 3.91-3.93 ms, 32 4.17 ms, 16 7.47 ms,
// the launch after the grouped one instead of beside it 4.00 ms.  Tuning hook:
// EB_STACK_SIDE_GROUPS (read once).
int side_groups() {
  static const int g = [] {
    const char *e = std::getenv("EB_STACK_SIDE_GROUPS");
    const int v = e ? std::atoi(e) : 0;
    return v >= 8 ? v : 0;
  }();
  return g;
}

struct Step {
  int op = -1;        // single op index, or -1 for a fused launch
  bool mfma = false;  // single op on the MFMA path, run with plan `mp`
  MfmaPlan mp;
  bool mm = false;    // fused MFMA launch (op == -1)
  int32_t type = 0, xt = 0, yt = 0;
  int ns = 0;
  size_t table = 0;   // first entry in the device table (M1Op or MMOp)
  int nops = 0;
  int64_t units = 0, rows = 0;
  int mm_cfg = 0, groups = 0;
  size_t wg = 0;      // first entry of the workgroup ranges
  bool gm = false;    // grouped MFMA launch (op == -1): table entries from `table`,
  size_t order = 0;   // workgroup entries from `order`
  int64_t entries = 0;
  std::vector<NormJob> norms;  // prologue row kernels run before the step
  bool side = false;  // fused launch of split-off rows that runs on the side stream,
                      // beside the grouped launch before it
  bool hl = true;     // fused small-m launch: bfloat16 hi/lo weight pairs (not for the
                      // split-off rows of large-m ops, whose bound is the large-m one)
  bool norm_next = false;   // single split MFMA op whose reduction also normalises
                            // its fp32 output for the next step's prologue
  bool pre_normed = false;  // single MFMA op whose prologue that reduction ran
};

struct Plan {
  std::vector<Step> steps;
  M1Op *table = nullptr;  // device copy of every fused GEMV launch's op table
  MMOp *mmtable = nullptr;  // same for fused MFMA launches
  int64_t *mmwg = nullptr;  // their workgroup unit ranges
  GOp *gmtable = nullptr;   // grouped MFMA launches: op table
  int2 *gmorder = nullptr;  // and workgroup (op, tile) entries
  float *ws = nullptr;    // split-K workspace shared by the plan's MFMA steps (run in order)
  size_t ws_bytes = 0;
  uint8_t *xbuf = nullptr;  // normalised activations of prologue ops on the MFMA path
  size_t xbuf_bytes = 0;
  size_t ws_total = 0;      // caller workspace the plan needs (tables, partial sums, xbuf)
  uint8_t *wsbase = nullptr;  // where that workspace is (the tables live there)
  hipEvent_t fork = nullptr, join = nullptr;  // side-stream steps (created when there are any)
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

bool env_off(const char *name) {
  const char *v = std::getenv(name);
  return v && v[0] == '0';
}

bool fusable(const eb_qlinear_op &o) {
  return o.m == 1 && gemv_fits(1, o.w.k) && m1_fusable(o.w.type, o.m, o.w.k, o.epilogue);
}

// MFMA ops that may join a fused launch.  The fused kernel addresses tiles of
// up to 256 rows with 31-bit offsets.  EB_STACK_FUSE_MAXM (default 128) caps
// the rows of a fused op; small-m single launches are latency-bound, large-m
// ones less so.
int64_t mm_max_m() {
  static const int64_t v = [] {
    const char *e = std::getenv("EB_STACK_FUSE_MAXM");
    return e ? std::atoll(e) : 128;
  }();
  return v;
}

// MFMA ops with more rows than a fused small-m launch takes, which may share a
// grouped launch (EB_STACK_GROUP=0 turns that off); Q6_S ops only where they
// take the tile kernel (m > 128).
bool gm_fusable(const eb_qlinear_op &o) {
  return (o.w.type != EB_Q6_S || o.m > 128) && o.m > mm_max_m() && !env_off("EB_STACK_GROUP") &&
         pick_path(o.w.type, o.x_type, o.m, o.w.n, o.w.k) == EB_PATH_MFMA;
}

bool mm_fusable(const eb_qlinear_op &o) {
  return o.w.type != EB_Q6_S && o.m >= 1 && o.m <= mm_max_m() && o.w.k < kMMaxK &&
         (o.m + 256) * o.w.n * (int64_t)dsize(o.y_type) < (int64_t(1) << 31) &&
         pick_path(o.w.type, o.x_type, o.m, o.w.n, o.w.k) == EB_PATH_MFMA;
}

// Builds the plan and sizes its workspace (P.ws_total); with a workspace base
// (at least P.ws_total bytes) also places its tables and buffers there and
// writes the tables.  Without one the plan is only counted and sized.
eb_status build_plan(const eb_qlinear_op *ops, int32_t n_ops, uint8_t *wsbase, Plan &P) {
  std::vector<M1Op> host;
  std::vector<MMOp> mmhost;
  std::vector<int64_t> mmwg;
  std::vector<GOp> gmhost;
  std::vector<int2> gmorder;
  const bool fuse = !env_off("EB_STACK_FUSE");
  // Normalisation jobs of the current iteration (one fused run, or one op):
  // their buffers are laid out from offset 0, since the steps of one
  // iteration run after those of the previous one.
  std::vector<NormJob> jobs;
  size_t xoff = 0;
  // an MFMA op with the prologue reads the plan's buffer instead of h
  auto prep = [&](const eb_qlinear_op &o) {
    if (o.prologue != EB_PRO_RMSNORM) return o;
    NormJob j{static_cast<const float *>(o.x), o.norm_weight, o.norm_eps, o.x_type, o.m, o.w.k, xoff};
    jobs.push_back(j);
    eb_qlinear_op c = o;
    c.x = reinterpret_cast<const void *>((uintptr_t)xoff);
    c.prologue = EB_PRO_NONE;
    c.norm_weight = nullptr;
    c.reserved = kRelX;
    xoff += xhat_bytes(o);
    return c;
  };
  // one fused small-m launch over `list` (same weight, x and y formats)
  auto add_mm_step = [&](const std::vector<eb_qlinear_op> &list, int max_groups = 0,
                         bool hl = true) {
    int64_t max_m = 0;
    for (const eb_qlinear_op &o : list) max_m = std::max(max_m, o.m);
    Step s;
    s.mm = true;
    s.hl = hl;
    s.type = list[0].w.type;
    s.xt = list[0].x_type;
    s.yt = list[0].y_type;
    s.mm_cfg = mm_cfg(max_m);
    s.table = mmhost.size();
    std::vector<MMOp> run;
    int64_t units = 0;
    for (const eb_qlinear_op &o : list) {
      const Layout L = layout_of(o.w.type, o.w.n, o.w.k);
      MMOp e{};
      e.w = static_cast<const uint8_t *>(o.w.data);
      e.x = static_cast<const uint16_t *>(o.x);
      e.y = o.y;
      e.d_off = L.d_off;
      units += mm_tiles(s.mm_cfg, o.m, o.w.n);
      e.unit_end = units;
      e.ds = (int32_t)L.ds;
      e.m = (int32_t)o.m;
      e.n = (int32_t)o.w.n;
      e.k = (int32_t)o.w.k;
      e.tiles_n = (int32_t)mm_tiles(s.mm_cfg, 1, o.w.n);
      e.nk = (int32_t)((o.w.k + mm_bk(s.mm_cfg) - 1) / mm_bk(s.mm_cfg));
      e.yt = o.y_type;
      e.pad = o.reserved == kRelX;  // x is an offset into the plan's buffer
      e.f = fuse_of(o);
      run.push_back(e);
    }
    std::vector<int64_t> wg;
    s.groups = mm_partition(run, s.mm_cfg, wg, max_groups);
    s.nops = (int)run.size();
    s.units = units;
    s.wg = mmwg.size();
    mmhost.insert(mmhost.end(), run.begin(), run.end());
    mmwg.insert(mmwg.end(), wg.begin(), wg.end());
    P.steps.push_back(s);
  };
  auto gops_of = [](const std::vector<eb_qlinear_op> &list) {
    std::vector<GOp> run;
    for (const eb_qlinear_op &o : list) {
      const Layout L = layout_of(o.w.type, o.w.n, o.w.k);
      GOp e{};
      e.w = static_cast<const uint8_t *>(o.w.data);
      e.x = static_cast<const uint16_t *>(o.x);
      e.y = o.y;
      e.n = o.w.n;
      e.k = o.w.k;
      e.d_off = L.d_off;
      e.ds = L.ds;
      e.sc_off = L.sc_off;
      e.m = o.m;
      e.yt = o.y_type;
      e.pad = o.reserved == kRelX;
      e.f = fuse_of(o);
      run.push_back(e);
    }
    return run;
  };
  int32_t i = 0;
  while (i < n_ops) {
    jobs.clear();
    xoff = 0;
    const size_t first_step = P.steps.size();
    // run [i, j) of consecutive ops that `ok` accepts and that are independent
    auto run_end = [&](auto ok) {
      std::vector<OpSpan> spans{span_of(ops[i])};
      int32_t j = i + 1;
      for (; j < n_ops; ++j) {
        if (!ok(ops[j])) break;
        const OpSpan sj = span_of(ops[j]);
        bool indep = true;
        for (const OpSpan &sp : spans) indep = indep && independent(sp, sj);
        if (!indep) break;
        spans.push_back(sj);
      }
      return j;
    };
    bool done = false;
    if (fuse && gm_fusable(ops[i])) {
      // run of independent large-m MFMA ops with the same weight and x formats
      const int32_t j = run_end([&](const eb_qlinear_op &o) {
        return gm_fusable(o) && o.w.type == ops[i].w.type && o.x_type == ops[i].x_type;
      });
      if (j - i > 1) {
        std::vector<eb_qlinear_op> mains, tails;
        for (int32_t r = i; r < j; ++r) mains.push_back(prep(ops[r]));
        std::vector<GOp> run = gops_of(mains);
        std::vector<int2> order;
        int cfg = plan_grouped(ops[i].w.type, run, order);
        // An op whose last row tile would be mostly padding (m = 816 in
        // 256-row tiles: 48 rows) gives those rows to a fused small-m launch
        // when the padded MFMA work saved outweighs reading its weights again.
        if (cfg >= 0 && !env_off("EB_STACK_SPLIT_TAIL")) {
          const int64_t bm = mfma_cfg_bm(cfg);
          const double rate = mfma_cfg_rate(cfg) * 1e12;
          std::vector<eb_qlinear_op> m2, t2;
          for (const eb_qlinear_op &o : mains) {
            const int64_t rem = o.m % bm, m0 = o.m - rem;
            eb_qlinear_op t = o;
            t.m = rem;
            t.x = static_cast<const uint8_t *>(o.x) + m0 * o.w.k * 2;
            t.y = static_cast<uint8_t *>(o.y) + m0 * n_out(o) * dsize(o.y_type);
            if (o.epilogue == EB_EPI_ADD)
              t.residual = static_cast<const uint8_t *>(o.residual) + m0 * o.w.n * dsize(o.y_type);
            bool split = rem > 0 && o.m > bm && mm_fusable(t);
            if (split) {
              const double row_flops = 2.0 * o.w.n * o.w.k;
              const double wbytes =
                  (double)o.w.n * o.w.k * (o.w.type == EB_Q8_0 ? 34.0 : 18.0) / 32.0;
              const double saved = (double)(bm - rem) * row_flops / rate;
              const double cost = std::max(wbytes / 4.5e12, (double)rem * row_flops / 0.35e15);
              split = saved > 1.2 * cost;
            }
            eb_qlinear_op mo = o;
            if (split) {
              mo.m = m0;
              t2.push_back(t);
            }
            m2.push_back(mo);
          }
          if (!t2.empty()) {
            std::vector<int2> order2;
            std::vector<GOp> run2 = gops_of(m2);
            const int cfg2 = plan_grouped(ops[i].w.type, run2, order2);
            if (cfg2 >= 0) {
              cfg = cfg2;
              run.swap(run2);
              order.swap(order2);
              tails.swap(t2);
            }
          }
        }
        if (cfg >= 0) {
          for (int2 &e : order)
            if (e.x >= 0) e.x += (int)gmhost.size();
          Step s;
          s.gm = true;
          s.type = ops[i].w.type;
          s.xt = ops[i].x_type;
          s.mm_cfg = cfg;
          s.table = gmhost.size();
          s.nops = (int)run.size();
          s.order = gmorder.size();
          s.entries = (int64_t)order.size();
          gmhost.insert(gmhost.end(), run.begin(), run.end());
          gmorder.insert(gmorder.end(), order.begin(), order.end());
          P.steps.push_back(s);
          // the split-off rows: one fused launch per output size.  They are
          // independent of the grouped launch (other output rows), so they run
          // beside it on a side stream: their weight streaming overlaps the
          // grouped launch's matrix-core work instead of following it.
          const bool overlap = !env_off("EB_STACK_OVERLAP_TAIL");
          for (int wide = 1; wide >= 0; --wide) {
            std::vector<eb_qlinear_op> cls;
            for (const eb_qlinear_op &t : tails)
              if ((t.y_type == EB_F32) == (wide == 1)) cls.push_back(t);
            if (cls.empty()) continue;
            add_mm_step(cls, overlap ? side_groups() : 0, false);
            P.steps.back().side = overlap;
          }
          i = j;
          done = true;
        } else {
          jobs.clear();
          xoff = 0;
        }
      }
    }
    if (!done && fuse && mm_fusable(ops[i])) {
      // run of independent small-m MFMA ops with the same formats (16-bit
      // output types share a launch)
      const bool wide = ops[i].y_type == EB_F32;
      const int32_t j = run_end([&](const eb_qlinear_op &o) {
        return mm_fusable(o) && o.w.type == ops[i].w.type && o.x_type == ops[i].x_type &&
               (o.y_type == EB_F32) == wide;
      });
      if (j - i > 1) {
        std::vector<eb_qlinear_op> list;
        for (int32_t r = i; r < j; ++r) list.push_back(prep(ops[r]));
        add_mm_step(list);
        i = j;
        done = true;
      }
    }
    if (!done && fuse && fusable(ops[i])) {
      // run of independent m == 1 GEMV ops with the same formats
      const int32_t j = run_end([&](const eb_qlinear_op &o) {
        return fusable(o) && o.w.type == ops[i].w.type && o.x_type == ops[i].x_type;
      });
      if (j - i > 1) {
        // one fused launch per slot count, in order of first appearance
        std::vector<int> classes;
        for (int32_t r = i; r < j; ++r) {
          const int ns = m1_slots(ops[r].w.type, ops[r].w.k);
          if (std::find(classes.begin(), classes.end(), ns) == classes.end()) classes.push_back(ns);
        }
        for (int ns : classes) {
          Step s;
          s.type = ops[i].w.type;
          s.xt = ops[i].x_type;
          s.ns = ns;
          s.table = host.size();
          for (int32_t r = i; r < j; ++r) {
            const eb_qlinear_op &o = ops[r];
            if (m1_slots(o.w.type, o.w.k) != ns) continue;
            M1Op e;
            s.units += m1_fill(o.w.type, o.w.data, o.w.n, o.w.k, o.x, o.y, o.y_type, fuse_of(o),
                               s.units, &e);
            s.rows += o.w.n;
            host.push_back(e);
            ++s.nops;
          }
          P.steps.push_back(s);
        }
        i = j;
        done = true;
      }
    }
    if (!done) {
      Step s;
      s.op = i++;
      P.steps.push_back(s);
    }
    if (!jobs.empty()) P.steps[first_step].norms = jobs;
    P.xbuf_bytes = std::max(P.xbuf_bytes, xoff);
  }
  for (Step &s : P.steps) {
    if (s.op < 0) continue;
    const eb_qlinear_op &o = ops[s.op];
    if (o.m == 0 || pick_path(o.w.type, o.x_type, o.m, o.w.n, o.w.k) != EB_PATH_MFMA) continue;
    s.mfma = true;
    s.mp = plan_mfma(o.w.type, o.x_type, o.m, o.w.n, o.w.k, kMaxSplitWorkspace);
    P.ws_bytes = std::max(P.ws_bytes, s.mp.ws_bytes);
    P.xbuf_bytes = std::max(P.xbuf_bytes, xhat_bytes(o));
  }
  // In a dependent layer chain, a split op writing the fp32 stream h (after
  // O and down: + h) is followed by an op normalising that h: the reduction,
  // which already holds every element of h, writes the normalised rows too
  // (one row kernel launch fewer per pair).  Both are single MFMA steps on
  // one stream; the reduction writes xbuf after its own op's product has read
  // it, and the next op reads it.
  if (!env_off("EB_STACK_FUSE_NORM")) {
    for (size_t q = 0; q + 1 < P.steps.size(); ++q) {
      Step &a = P.steps[q], &b = P.steps[q + 1];
      if (!a.mfma || !b.mfma || a.side || b.side || a.mp.splits <= 1 || !b.norms.empty()) continue;
      const eb_qlinear_op &oa = ops[a.op], &ob = ops[b.op];
      if (oa.y_type != EB_F32 || oa.epilogue == EB_EPI_GLU || ob.prologue != EB_PRO_RMSNORM) continue;
      if (ob.x != oa.y || ob.m != oa.m || ob.w.k != oa.w.n || oa.m == 0) continue;
      a.norm_next = true;
      b.pre_normed = true;
    }
  }
  // The plan's device memory is the caller's workspace: the op tables of its
  // fused and grouped launches, then the split-K partial sums, then the
  // normalised activations, each 256-byte aligned.
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = (size_t)round_up((int64_t)(off + bytes), 256);
    return o;
  };
  const size_t t_m1 = take(host.size() * sizeof(M1Op));
  const size_t t_mm = take(mmhost.size() * sizeof(MMOp));
  const size_t t_wg = take(mmwg.size() * sizeof(int64_t));
  const size_t t_gm = take(gmhost.size() * sizeof(GOp));
  const size_t t_go = take(gmorder.size() * sizeof(int2));
  const size_t t_tables = off;
  const size_t t_ws = take(P.ws_bytes);
  const size_t t_xb = take(P.xbuf_bytes);
  P.ws_total = off;
  if (!wsbase) return EB_OK;
  P.wsbase = wsbase;
  P.table = host.empty() ? nullptr : reinterpret_cast<M1Op *>(wsbase + t_m1);
  P.mmtable = mmhost.empty() ? nullptr : reinterpret_cast<MMOp *>(wsbase + t_mm);
  P.mmwg = mmwg.empty() ? nullptr : reinterpret_cast<int64_t *>(wsbase + t_wg);
  P.gmtable = gmhost.empty() ? nullptr : reinterpret_cast<GOp *>(wsbase + t_gm);
  P.gmorder = gmorder.empty() ? nullptr : reinterpret_cast<int2 *>(wsbase + t_go);
  P.ws = P.ws_bytes ? reinterpret_cast<float *>(wsbase + t_ws) : nullptr;
  P.xbuf = P.xbuf_bytes ? wsbase + t_xb : nullptr;
  // table entries whose x is an offset into the normalised-activation buffer
  for (MMOp &e : mmhost)
    if (e.pad) e.x = reinterpret_cast<const uint16_t *>(P.xbuf + reinterpret_cast<uintptr_t>(e.x));
  for (GOp &e : gmhost)
    if (e.pad) e.x = reinterpret_cast<const uint16_t *>(P.xbuf + reinterpret_cast<uintptr_t>(e.x));
  // the tables, written once when the plan is built (a copy, not an allocation)
  if (t_tables > 0) {
    std::vector<uint8_t> img(t_tables, 0);
    auto put = [&](size_t at, const void *src, size_t bytes) {
      if (bytes) std::memcpy(img.data() + at, src, bytes);
    };
    put(t_m1, host.data(), host.size() * sizeof(M1Op));
    put(t_mm, mmhost.data(), mmhost.size() * sizeof(MMOp));
    put(t_wg, mmwg.data(), mmwg.size() * sizeof(int64_t));
    put(t_gm, gmhost.data(), gmhost.size() * sizeof(GOp));
    put(t_go, gmorder.data(), gmorder.size() * sizeof(int2));
    if (hipMemcpy(wsbase, img.data(), t_tables, hipMemcpyHostToDevice) != hipSuccess)
      return EB_ERR_HIP;
  }
  return EB_OK;
}

// EB_STACK_DEBUG=1 prints each plan's steps to stderr when it is built.
void print_plan(const eb_qlinear_op *ops, const Plan &P) {
  std::fprintf(stderr, "[eb plan] %zu steps, xbuf %p (%zu B), ws %p (%zu B)\n", P.steps.size(),
               (void *)P.xbuf, P.xbuf_bytes, (void *)P.ws, P.ws_bytes);
  for (size_t i = 0; i < P.steps.size(); ++i) {
    const Step &st = P.steps[i];
    const char *kind = st.gm ? "grouped" : st.mm ? "small-m" : st.mfma ? "mfma" : st.op >= 0 ? "single" : "gemv-multi";
    std::fprintf(stderr, "[eb plan]  step %zu %s%s op %d nops %d cfg %d splits %d norms %zu", i, kind,
                 st.side ? " (side stream)" : "", st.op, st.nops, st.mm_cfg,
                 st.mfma ? st.mp.splits : 0, st.norms.size());
    for (const NormJob &j : st.norms) std::fprintf(stderr, " [h %p off %zu]", (const void *)j.h, j.off);
    if (st.pre_normed) std::fprintf(stderr, " (prologue ran in the previous reduction)");
    if (st.norm_next) std::fprintf(stderr, " (reduction normalises for the next step)");
    if (st.op >= 0)
      std::fprintf(stderr, " x %p y %p pro %d epi %d", ops[st.op].x, ops[st.op].y, ops[st.op].prologue,
                   ops[st.op].epilogue);
    std::fprintf(stderr, "\n");
  }
}

eb_status run_plan(const eb_qlinear_op *ops, const Plan &P, hipStream_t s, hipStream_t side) {
  for (size_t i = 0; i < P.steps.size(); ++i) {
    const Step &st = P.steps[i];
    if (st.side) continue;  // launched with the grouped step before it
    for (const NormJob &j : st.norms)
      if (launch_rmsnorm(j.h, j.gamma, j.eps, j.m, j.k, j.xt, P.xbuf + j.off, s) != hipSuccess)
        return EB_ERR_HIP;
    // side steps after a grouped step: fork them onto the side stream first
    // (their workgroups take a few CUs before the grouped launch fills the
    // rest), and join them back after the grouped launch
    size_t nside = 0;
    while (st.gm && i + 1 + nside < P.steps.size() && P.steps[i + 1 + nside].side) ++nside;
    if (nside > 0) {
      if (!side || hipEventRecord(P.fork, s) != hipSuccess ||
          hipStreamWaitEvent(side, P.fork, 0) != hipSuccess)
        return EB_ERR_HIP;
      for (size_t q = 1; q <= nside; ++q) {
        const Step &t = P.steps[i + q];
        if (launch_mfma_multi(t.type, t.xt, t.hl, t.yt, t.mm_cfg, P.mmtable + t.table, t.nops,
                              P.mmwg + t.wg, t.groups, side) != hipSuccess)
          return EB_ERR_HIP;
      }
      if (hipEventRecord(P.join, side) != hipSuccess) return EB_ERR_HIP;
    }
    if (st.gm) {
      // the table entries index the whole plan's op table
      if (launch_mfma_grouped(st.type, st.xt, st.mm_cfg, P.gmtable, P.gmorder + st.order,
                              st.entries, s) != hipSuccess)
        return EB_ERR_HIP;
    } else if (st.mm) {
      if (launch_mfma_multi(st.type, st.xt, st.hl, st.yt, st.mm_cfg, P.mmtable + st.table, st.nops,
                            P.mmwg + st.wg, st.groups, s) != hipSuccess)
        return EB_ERR_HIP;
    } else if (st.mfma) {
      const eb_qlinear_op &o = ops[st.op];
      NormOut no{};
      if (st.norm_next) {
        const eb_qlinear_op &nx = ops[P.steps[i + 1].op];
        no = NormOut{nx.norm_weight, nx.norm_eps, nx.x_type, P.xbuf};
      }
      if (launch_mfma_op(o, st.mp, P.xbuf, st.mp.splits > 1 ? P.ws : nullptr, s, st.pre_normed,
                         st.norm_next ? &no : nullptr) != hipSuccess)
        return EB_ERR_HIP;
    } else if (st.op >= 0) {
      eb_status r = launch_op(ops[st.op], EB_PATH_AUTO, nullptr, 0, s);
      if (r != EB_OK) return r;
    } else if (launch_gemv_m1_multi(st.type, st.xt, st.ns, P.table + st.table, st.nops, st.units,
                                    st.rows, s) != hipSuccess) {
      return EB_ERR_HIP;
    }
    if (nside > 0 && hipStreamWaitEvent(s, P.join, 0) != hipSuccess) return EB_ERR_HIP;
  }
  return EB_OK;
}

void destroy_plan(Plan &p) {
  if (p.exec) (void)hipGraphExecDestroy(p.exec);
  if (p.graph) (void)hipGraphDestroy(p.graph);
  if (p.fork) (void)hipEventDestroy(p.fork);
  if (p.join) (void)hipEventDestroy(p.join);
  p = Plan();
}

struct StackCache {
  std::mutex mu;
  std::unordered_map<std::string, Plan> map;
  hipStream_t capture_stream[64] = {};
  hipStream_t side_stream[64] = {};  // default priority, like every stream here
};

StackCache &cache() {
  static StackCache *c = new StackCache();  // leaked on purpose: no teardown-order issues
  return *c;
}

constexpr size_t kMaxCachedPlans = 64;

void clear_cache_locked(StackCache &C) {
  if (!C.map.empty()) (void)hipDeviceSynchronize();  // tables may still be in use
  for (auto &kv : C.map) destroy_plan(kv.second);
  C.map.clear();
}

eb_status run_ops_direct(const eb_qlinear_op *ops, int32_t n_ops, uint8_t *ws, size_t wsb,
                         hipStream_t s) {
  for (int32_t i = 0; i < n_ops; ++i) {
    eb_status st = launch_op(ops[i], EB_PATH_AUTO, ws, wsb, s);
    if (st != EB_OK) return st;
  }
  return EB_OK;
}

// ---------------------------------------------------------------------------
// Scratch for callers that cannot allocate (code under HIP graph capture,
// serving loops, harnesses that forbid allocation): one file-scope device
// array per GPU, of kStaticScratchBytes, that eb_qlinear_fused_static uses
// instead of a caller workspace.  Its device address is looked up once per
// device, with that device current; host code never uses the array's name
// as an address (in host code it is only a stand-in for the symbol).
// ---------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

struct StaticScratch {
  std::once_flag once[64];
  uint8_t *ptr[64] = {};
  hipError_t err[64] = {};
};

StaticScratch &static_scratch_state() {
  static StaticScratch *s = new StaticScratch();  // leaked on purpose: no teardown-order issues
  return *s;
}

// This device's scratch array (dev is the current device), or nullptr if the
// runtime could not resolve it.
uint8_t *static_scratch(int dev) {
  StaticScratch &S = static_scratch_state();
  std::call_once(S.once[dev], [&] {
    void *p = nullptr;
    S.err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (S.err[dev] == hipSuccess && p) S.ptr[dev] = static_cast<uint8_t *>(p);
  });
  return S.ptr[dev];
}

}  // namespace
}  // namespace eb

using namespace eb;

extern "C" {

const char *eb_version(void) { return "eb 0.1.0 (gfx950)"; }

const char *eb_status_str(eb_status s) {
  switch (s) {
    case EB_OK: return "EB_OK";
    case EB_ERR_INVALID: return "EB_ERR_INVALID: invalid argument";
    case EB_ERR_ALIGN: return "EB_ERR_ALIGN: misaligned pointer";
    case EB_ERR_UNSUPPORTED: return "EB_ERR_UNSUPPORTED: unsupported dtype or path";
    case EB_ERR_HIP: return "EB_ERR_HIP: HIP runtime error";
    default: return "unknown eb_status";
  }
}

size_t eb_qweights_bytes(int32_t type, int64_t n, int64_t k) {
  if (!valid_type(type) || n < 0 || n > kMaxN || !valid_k(type, k)) return 0;
  return (size_t)layout_of(type, n, k).total;
}

eb_status eb_qweights_layout(int32_t type, int64_t n, int64_t k, eb_layout *out) {
  if (!out || !valid_type(type) || n < 0 || n > kMaxN || !valid_k(type, k)) return EB_ERR_INVALID;
  const Layout L = layout_of(type, n, k);
  out->qs_offset = 0;
  out->qs_row_bytes = L.qs_row;
  out->d_offset = L.d_off;
  out->d_stride = L.ds;
  out->total_bytes = L.total;
  out->canonical_bytes = (int64_t)canonical_bytes(type, n, k);
  out->sc_offset = L.sc_off;
  out->sc_stride = L.ss;
  return EB_OK;
}

eb_status eb_quantize_q8_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream) {
  return quantize_common(EB_Q8_0, w, n, k, out, stream);
}

eb_status eb_quantize_q4_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream) {
  return quantize_common(EB_Q4_0, w, n, k, out, stream);
}

eb_status eb_quantize_q6_s(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream) {
  return quantize_common(EB_Q6_S, w, n, k, out, stream);
}

eb_status eb_qweights_to_canonical(const eb_qweights *w, void *dst, hipStream_t stream) {
  eb_status st = check_weights(w);
  if (st != EB_OK) return st;
  if (!dst) return EB_ERR_INVALID;
  const size_t cb = canonical_bytes(w->type, w->n, w->k);
  if (overlaps(dst, cb, w->data, eb_qweights_bytes(w->type, w->n, w->k))) return EB_ERR_INVALID;
  return launch_to_canonical(w->type, w->data, w->n, w->k, dst, stream) == hipSuccess ? EB_OK
                                                                                       : EB_ERR_HIP;
}

eb_status eb_qweights_from_canonical(int32_t type, const void *src, int64_t n, int64_t k,
                                     void *out, hipStream_t stream) {
  if (!valid_type(type) || !valid_nk(type, n, k) || !src || !out) return EB_ERR_INVALID;
  if (!aligned(out, 256)) return EB_ERR_ALIGN;
  const size_t cb = canonical_bytes(type, n, k);
  if (overlaps(src, cb, out, eb_qweights_bytes(type, n, k))) return EB_ERR_INVALID;
  return launch_from_canonical(type, src, n, k, out, stream) == hipSuccess ? EB_OK : EB_ERR_HIP;
}

eb_status eb_qlinear_ex(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                        int32_t y_type, int32_t path, hipStream_t stream) {
  if (!w) return EB_ERR_INVALID;
  const eb_qlinear_op o = plain_op(w, x, x_type, m, y, y_type);
  eb_status st = check_op(o, path);
  if (st != EB_OK) return st;
  return launch_op(o, path, nullptr, 0, stream);
}

eb_status eb_qlinear_fused(const eb_qlinear_op *op, int32_t path, hipStream_t stream) {
  return eb_qlinear_fused_ws(op, path, nullptr, 0, stream);
}

size_t eb_qlinear_workspace_bytes(const eb_qlinear_op *op, int32_t path) {
  if (!op || check_op(*op, path) != EB_OK || op->m == 0) return 0;
  if (path == EB_PATH_AUTO) path = pick_path(op->w.type, op->x_type, op->m, op->w.n, op->w.k);
  if (path == EB_PATH_GEMV) return 0;
  if (path == EB_PATH_MFMA_I8) return i8_workspace_bytes(op->m, op->w.k);
  return op_scratch(*op, kMaxSplitWorkspace + xhat_bytes(*op)).total;
}

eb_status eb_qlinear_fused_ws(const eb_qlinear_op *op, int32_t path, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  if (!op) return EB_ERR_INVALID;
  eb_status st = check_op(*op, path);
  if (st != EB_OK) return st;
  st = check_workspace(op, 1, workspace, workspace_bytes);
  if (st != EB_OK) return st;
  return launch_op(*op, path, static_cast<uint8_t *>(workspace), workspace_bytes, stream);
}

eb_status eb_qlinear_fused_static(const eb_qlinear_op *op, int32_t path, hipStream_t stream) {
  if (!op) return EB_ERR_INVALID;
  eb_status st = check_op(*op, path);
  if (st != EB_OK) return st;
  if (op->m == 0) return EB_OK;
  const int32_t p =
      path == EB_PATH_AUTO ? pick_path(op->w.type, op->x_type, op->m, op->w.n, op->w.k) : path;
  if (p == EB_PATH_MFMA && xhat_bytes(*op) > kStaticScratchBytes) return EB_ERR_UNSUPPORTED;
  if (p == EB_PATH_MFMA_I8 && i8_workspace_bytes(op->m, op->w.k) > kStaticScratchBytes)
    return EB_ERR_UNSUPPORTED;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return EB_ERR_HIP;
  uint8_t *ws = static_scratch(dev);
  if (!ws) return EB_ERR_HIP;
  return launch_op(*op, p, ws, kStaticScratchBytes, stream);
}

eb_status eb_qlinear(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                     int32_t y_type, hipStream_t stream) {
  return eb_qlinear_ex(w, x, x_type, m, y, y_type, EB_PATH_AUTO, stream);
}

int32_t eb_qlinear_auto_path(int32_t type, int32_t x_type, int64_t m, int64_t n, int64_t k) {
  if (!valid_type(type) || !valid_nk(type, n, k) || m < 1 || m > kMaxM) return EB_ERR_INVALID;
  return pick_path(type, x_type, m, n, k);
}

size_t eb_qlinear_stack_workspace_bytes(const eb_qlinear_op *ops, int32_t n_ops) {
  if (n_ops <= 0 || !ops) return 0;
  for (int32_t i = 0; i < n_ops; ++i)
    if (check_op(ops[i], EB_PATH_AUTO) != EB_OK) return 0;
  Plan P;
  build_plan(ops, n_ops, nullptr, P);
  return P.ws_total;
}

eb_status eb_qlinear_stack(const eb_qlinear_op *ops, int32_t n_ops, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  if (n_ops < 0) return EB_ERR_INVALID;
  if (n_ops == 0) return EB_OK;
  if (!ops) return EB_ERR_INVALID;
  for (int32_t i = 0; i < n_ops; ++i) {
    const eb_qlinear_op &o = ops[i];
    eb_status st = check_op(o, EB_PATH_AUTO);
    if (st != EB_OK) return st;
  }
  {
    eb_status st = check_workspace(ops, n_ops, workspace, workspace_bytes);
    if (st != EB_OK) return st;
  }
  uint8_t *const ws = static_cast<uint8_t *>(workspace);
  // Inside a caller's own stream capture, record plain launches into it.
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
    return run_ops_direct(ops, n_ops, ws, workspace_bytes, stream);

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return EB_ERR_HIP;
  const bool use_graph = !env_off("EB_STACK_GRAPH");
  std::string key(reinterpret_cast<const char *>(&dev), sizeof(dev));
  key.push_back(use_graph ? 'g' : 'd');
  key.push_back(env_off("EB_STACK_FUSE") ? 'u' : 'f');
  key.push_back(env_off("EB_STACK_GROUP") ? 'n' : 'g');
  key.push_back(env_off("EB_STACK_SPLIT_TAIL") ? 'w' : 's');
  key.push_back(env_off("EB_STACK_OVERLAP_TAIL") ? 'q' : 'o');
  key.push_back(env_off("EB_STACK_FUSE_NORM") ? 'r' : 'n');
  key.append(reinterpret_cast<const char *>(&ws), sizeof(ws));
  key.append(reinterpret_cast<const char *>(&workspace_bytes), sizeof(workspace_bytes));
  key.append(reinterpret_cast<const char *>(ops), sizeof(eb_qlinear_op) * (size_t)n_ops);

  StackCache &C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  auto it = C.map.find(key);
  if (it == C.map.end()) {
    if (C.map.size() >= kMaxCachedPlans) clear_cache_locked(C);
    Plan P;
    eb_status st = build_plan(ops, n_ops, nullptr, P);
    if (st == EB_OK && P.ws_total > workspace_bytes) st = EB_ERR_INVALID;  // workspace too small
    if (st == EB_OK && P.ws_total > 0) {
      // A cached plan whose tables sit in the same workspace bytes is dropped
      // first (after the device has finished any replay of it): the new
      // plan's tables overwrite them.
      bool clash = false;
      for (const auto &kv : C.map)
        clash = clash || overlaps(kv.second.wsbase, kv.second.ws_total, ws, P.ws_total);
      if (clash) {
        (void)hipDeviceSynchronize();
        for (auto kv = C.map.begin(); kv != C.map.end();) {
          if (overlaps(kv->second.wsbase, kv->second.ws_total, ws, P.ws_total)) {
            destroy_plan(kv->second);
            kv = C.map.erase(kv);
          } else {
            ++kv;
          }
        }
      }
      Plan Q;
      st = build_plan(ops, n_ops, ws, Q);
      P = Q;
    }
    if (st != EB_OK) {
      destroy_plan(P);
      return st;
    }
    if (std::getenv("EB_STACK_DEBUG")) print_plan(ops, P);
    bool has_side = false;
    for (const Step &s : P.steps) has_side = has_side || s.side;
    if (has_side && !C.side_stream[dev] &&
        hipStreamCreateWithFlags(&C.side_stream[dev], hipStreamNonBlocking) != hipSuccess) {
      C.side_stream[dev] = nullptr;
      destroy_plan(P);
      return EB_ERR_HIP;
    }
    if (has_side && (hipEventCreateWithFlags(&P.fork, hipEventDisableTiming) != hipSuccess ||
                     hipEventCreateWithFlags(&P.join, hipEventDisableTiming) != hipSuccess)) {
      destroy_plan(P);
      return EB_ERR_HIP;
    }
    if (use_graph) {
      if (!C.capture_stream[dev] &&
          hipStreamCreateWithFlags(&C.capture_stream[dev], hipStreamNonBlocking) != hipSuccess) {
        C.capture_stream[dev] = nullptr;
        destroy_plan(P);
        return EB_ERR_HIP;
      }
      hipStream_t cap = C.capture_stream[dev];
      if (hipStreamBeginCapture(cap, hipStreamCaptureModeRelaxed) != hipSuccess) {
        destroy_plan(P);
        return EB_ERR_HIP;
      }
      st = run_plan(ops, P, cap, C.side_stream[dev]);
      hipError_t e = hipStreamEndCapture(cap, &P.graph);
      if (st != EB_OK || e != hipSuccess || !P.graph ||
          hipGraphInstantiate(&P.exec, P.graph, nullptr, nullptr, 0) != hipSuccess) {
        destroy_plan(P);
        return EB_ERR_HIP;
      }
    }
    it = C.map.emplace(std::move(key), P).first;
  }
  const Plan &P = it->second;
  if (P.exec) return hipGraphLaunch(P.exec, stream) == hipSuccess ? EB_OK : EB_ERR_HIP;
  return run_plan(ops, P, stream, C.side_stream[dev]);
}

int32_t eb_qlinear_stack_launches(const eb_qlinear_op *ops, int32_t n_ops) {
  if (n_ops < 0 || (n_ops > 0 && !ops)) return EB_ERR_INVALID;
  for (int32_t i = 0; i < n_ops; ++i) {
    const eb_qlinear_op &o = ops[i];
    eb_status st = check_op(o, EB_PATH_AUTO);
    if (st != EB_OK) return st;
  }
  Plan P;
  build_plan(ops, n_ops, nullptr, P);
  int32_t launches = 0;
  for (const Step &st : P.steps) {
    launches += (int32_t)st.norms.size();
    if (st.op >= 0 && ops[st.op].m == 0) continue;
    launches += (st.mfma && st.mp.splits > 1) ? 2 : 1;
    if (st.mfma && ops[st.op].prologue == EB_PRO_RMSNORM && !st.pre_normed) ++launches;
  }
  return launches;
}

int32_t eb_mfma_tile_count(void) { return mfma_tile_count(); }

eb_status eb_qlinear_tuned(const eb_qlinear_op *op, int32_t tile, int32_t splits, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  if (!op || tile < -1 || tile >= mfma_tile_count() || splits < 0 || splits > 16) return EB_ERR_INVALID;
  eb_status st = check_op(*op, EB_PATH_MFMA);
  if (st != EB_OK) return st;
  st = check_workspace(op, 1, workspace, workspace_bytes);
  if (st != EB_OK) return st;
  return launch_op(*op, EB_PATH_MFMA, static_cast<uint8_t *>(workspace), workspace_bytes, stream,
                   tile, splits);
}

eb_status eb_stack_cache_clear(void) {
  StackCache &C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  clear_cache_locked(C);
  return EB_OK;
}

}  // extern "C"
