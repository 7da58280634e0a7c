// eb_api.cpp -- the C ABI: host-side validation, path dispatch and the stack
// runner with HIP-graph replay (paper section 3.2: graph replay, buffer reuse
// and backend-specific dispatch for latency-first batch-1 execution).
//
// Validation happens entirely on the host before any HIP call, so every error
// path is testable without a GPU and nothing is launched on error.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdlib>
#include <cstring>
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

bool valid_type(int32_t t) { return t == EB_Q8_0 || t == EB_Q4_0; }
bool known_dtype(int32_t t) { return t == EB_F32 || t == EB_F16 || t == EB_BF16; }

bool valid_nk(int64_t n, int64_t k) {
  return n >= 1 && n <= kMaxN && k >= kQK && k <= kMaxK && k % kQK == 0;
}

bool overlaps(const void *a, size_t an, const void *b, size_t bn) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return an && bn && a0 < b0 + bn && b0 < a0 + an;
}

size_t dsize(int32_t t) { return t == EB_F32 ? 4 : 2; }

int64_t gemv_mt(int64_t m) { return m <= 1 ? 1 : (m <= 2 ? 2 : 4); }

bool gemv_fits(int64_t m, int64_t k) {
  return m >= 1 && m <= kGemvMaxM && gemv_mt(m) * k <= kGemvMaxMK;
}

eb_status check_weights(const eb_qweights *w) {
  if (!w || !w->data || !valid_type(w->type) || w->reserved != 0 || !valid_nk(w->n, w->k))
    return EB_ERR_INVALID;
  if (!aligned(w->data, 256)) return EB_ERR_ALIGN;
  return EB_OK;
}

eb_status check_linear(const eb_qweights *w, const void *x, int32_t xt, int64_t m, const void *y,
                       int32_t yt, int32_t path) {
  eb_status st = check_weights(w);
  if (st != EB_OK) return st;
  if (m < 0 || m > kMaxM) return EB_ERR_INVALID;
  if (!known_dtype(xt) || !known_dtype(yt)) return EB_ERR_INVALID;
  if (path != EB_PATH_AUTO && path != EB_PATH_GEMV && path != EB_PATH_MFMA) return EB_ERR_INVALID;
  if (xt == EB_F32 || yt == EB_F16) return EB_ERR_UNSUPPORTED;
  if (m == 0) return EB_OK;
  if (!x || !y) return EB_ERR_INVALID;
  if (!aligned(x, 16) || !aligned(y, 16)) return EB_ERR_ALIGN;
  const size_t xb = (size_t)m * (size_t)w->k * 2, yb = (size_t)m * (size_t)w->n * dsize(yt);
  const size_t wb = eb_qweights_bytes(w->type, w->n, w->k);
  if (overlaps(y, yb, x, xb) || overlaps(y, yb, w->data, wb)) return EB_ERR_INVALID;
  if (path == EB_PATH_GEMV && !gemv_fits(m, w->k)) return EB_ERR_UNSUPPORTED;
  return EB_OK;
}

int32_t pick_path(int32_t type, int32_t xt, int64_t m, int64_t n, int64_t k) {
  (void)type;
  (void)xt;
  (void)n;
  return gemv_fits(m, k) ? EB_PATH_GEMV : EB_PATH_MFMA;
}

eb_status launch_linear(const eb_qweights *w, const void *x, int32_t xt, int64_t m, void *y,
                        int32_t yt, int32_t path, hipStream_t s) {
  if (m == 0) return EB_OK;
  if (path == EB_PATH_AUTO) path = pick_path(w->type, xt, m, w->n, w->k);
  hipError_t e = (path == EB_PATH_GEMV)
                     ? launch_gemv(w->type, w->data, w->n, w->k, x, xt, m, y, yt, s)
                     : launch_mfma(w->type, w->data, w->n, w->k, x, xt, m, y, yt, s);
  return e == hipSuccess ? EB_OK : EB_ERR_HIP;
}

eb_status quantize_common(int32_t type, const float *w, int64_t n, int64_t k, void *out,
                          hipStream_t s) {
  if (n < 0 || n > kMaxN || k < 0 || k > kMaxK || k % kQK != 0) return EB_ERR_INVALID;
  if (n == 0 || k == 0) return EB_OK;
  if (!w || !out) return EB_ERR_INVALID;
  if (!aligned(w, 16) || !aligned(out, 256)) return EB_ERR_ALIGN;
  if (overlaps(w, (size_t)n * k * 4, out, eb_qweights_bytes(type, n, k))) return EB_ERR_INVALID;
  return launch_quantize(type, w, n, k, out, s) == hipSuccess ? EB_OK : EB_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Stack graph cache: op list bytes + device -> instantiated graph.
// ---------------------------------------------------------------------------
struct GraphEntry {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

struct StackCache {
  std::mutex mu;
  std::unordered_map<std::string, GraphEntry> map;
  hipStream_t capture_stream[64] = {};
};

StackCache &cache() {
  static StackCache *c = new StackCache();  // leaked on purpose: no teardown-order issues
  return *c;
}

constexpr size_t kMaxCachedGraphs = 64;

void destroy_entry(GraphEntry &g) {
  if (g.exec) (void)hipGraphExecDestroy(g.exec);
  if (g.graph) (void)hipGraphDestroy(g.graph);
  g.exec = nullptr;
  g.graph = nullptr;
}

bool graphs_enabled() {
  const char *v = std::getenv("EB_STACK_GRAPH");
  return !(v && v[0] == '0');
}

eb_status run_ops_direct(const eb_qlinear_op *ops, int32_t n_ops, hipStream_t s) {
  for (int32_t i = 0; i < n_ops; ++i) {
    const eb_qlinear_op &o = ops[i];
    eb_status st = launch_linear(&o.w, o.x, o.x_type, o.m, o.y, o.y_type, EB_PATH_AUTO, s);
    if (st != EB_OK) return st;
  }
  return EB_OK;
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
  if (!valid_type(type) || n < 0 || n > kMaxN || k < 0 || k > kMaxK || k % kQK != 0) return 0;
  return (size_t)layout_of(type, n, k).total;
}

eb_status eb_qweights_layout(int32_t type, int64_t n, int64_t k, eb_layout *out) {
  if (!out || !valid_type(type) || n < 0 || n > kMaxN || k < 0 || k > kMaxK || k % kQK != 0)
    return EB_ERR_INVALID;
  const Layout L = layout_of(type, n, k);
  out->qs_offset = 0;
  out->qs_row_bytes = L.qs_row;
  out->d_offset = L.d_off;
  out->d_stride = L.ds;
  out->total_bytes = L.total;
  out->canonical_bytes = n * L.nb * (2 + qs_bytes_per_block(type));
  return EB_OK;
}

eb_status eb_quantize_q8_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream) {
  return quantize_common(EB_Q8_0, w, n, k, out, stream);
}

eb_status eb_quantize_q4_0(const float *w, int64_t n, int64_t k, void *out, hipStream_t stream) {
  return quantize_common(EB_Q4_0, w, n, k, out, stream);
}

eb_status eb_qweights_to_canonical(const eb_qweights *w, void *dst, hipStream_t stream) {
  eb_status st = check_weights(w);
  if (st != EB_OK) return st;
  if (!dst) return EB_ERR_INVALID;
  const size_t cb = (size_t)w->n * (w->k / kQK) * (2 + qs_bytes_per_block(w->type));
  if (overlaps(dst, cb, w->data, eb_qweights_bytes(w->type, w->n, w->k))) return EB_ERR_INVALID;
  return launch_to_canonical(w->type, w->data, w->n, w->k, dst, stream) == hipSuccess ? EB_OK
                                                                                       : EB_ERR_HIP;
}

eb_status eb_qweights_from_canonical(int32_t type, const void *src, int64_t n, int64_t k,
                                     void *out, hipStream_t stream) {
  if (!valid_type(type) || !valid_nk(n, k) || !src || !out) return EB_ERR_INVALID;
  if (!aligned(out, 256)) return EB_ERR_ALIGN;
  const size_t cb = (size_t)n * (k / kQK) * (2 + qs_bytes_per_block(type));
  if (overlaps(src, cb, out, eb_qweights_bytes(type, n, k))) return EB_ERR_INVALID;
  return launch_from_canonical(type, src, n, k, out, stream) == hipSuccess ? EB_OK : EB_ERR_HIP;
}

eb_status eb_qlinear_ex(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                        int32_t y_type, int32_t path, hipStream_t stream) {
  eb_status st = check_linear(w, x, x_type, m, y, y_type, path);
  if (st != EB_OK) return st;
  return launch_linear(w, x, x_type, m, y, y_type, path, stream);
}

eb_status eb_qlinear(const eb_qweights *w, const void *x, int32_t x_type, int64_t m, void *y,
                     int32_t y_type, hipStream_t stream) {
  return eb_qlinear_ex(w, x, x_type, m, y, y_type, EB_PATH_AUTO, stream);
}

int32_t eb_qlinear_auto_path(int32_t type, int32_t x_type, int64_t m, int64_t n, int64_t k) {
  if (!valid_type(type) || !valid_nk(n, k) || m < 1 || m > kMaxM) return EB_ERR_INVALID;
  return pick_path(type, x_type, m, n, k);
}

eb_status eb_qlinear_stack(const eb_qlinear_op *ops, int32_t n_ops, hipStream_t stream) {
  if (n_ops < 0) return EB_ERR_INVALID;
  if (n_ops == 0) return EB_OK;
  if (!ops) return EB_ERR_INVALID;
  for (int32_t i = 0; i < n_ops; ++i) {
    const eb_qlinear_op &o = ops[i];
    eb_status st = check_linear(&o.w, o.x, o.x_type, o.m, o.y, o.y_type, EB_PATH_AUTO);
    if (st != EB_OK) return st;
  }
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (!graphs_enabled() || hipStreamIsCapturing(stream, &cs) != hipSuccess ||
      cs != hipStreamCaptureStatusNone)
    return run_ops_direct(ops, n_ops, stream);

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return run_ops_direct(ops, n_ops, stream);
  std::string key(reinterpret_cast<const char *>(&dev), sizeof(dev));
  key.append(reinterpret_cast<const char *>(ops), sizeof(eb_qlinear_op) * (size_t)n_ops);

  StackCache &C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  auto it = C.map.find(key);
  if (it == C.map.end()) {
    if (!C.capture_stream[dev] &&
        hipStreamCreateWithFlags(&C.capture_stream[dev], hipStreamNonBlocking) != hipSuccess) {
      C.capture_stream[dev] = nullptr;
      return EB_ERR_HIP;
    }
    hipStream_t cap = C.capture_stream[dev];
    if (hipStreamBeginCapture(cap, hipStreamCaptureModeRelaxed) != hipSuccess) return EB_ERR_HIP;
    eb_status st = run_ops_direct(ops, n_ops, cap);
    GraphEntry g;
    hipError_t e = hipStreamEndCapture(cap, &g.graph);
    if (st != EB_OK || e != hipSuccess || !g.graph) {
      destroy_entry(g);
      return EB_ERR_HIP;
    }
    if (hipGraphInstantiate(&g.exec, g.graph, nullptr, nullptr, 0) != hipSuccess) {
      destroy_entry(g);
      return EB_ERR_HIP;
    }
    if (C.map.size() >= kMaxCachedGraphs) {
      for (auto &kv : C.map) destroy_entry(kv.second);
      C.map.clear();
    }
    it = C.map.emplace(std::move(key), g).first;
  }
  return hipGraphLaunch(it->second.exec, stream) == hipSuccess ? EB_OK : EB_ERR_HIP;
}

eb_status eb_stack_cache_clear(void) {
  StackCache &C = cache();
  std::lock_guard<std::mutex> lock(C.mu);
  for (auto &kv : C.map) destroy_entry(kv.second);
  C.map.clear();
  return EB_OK;
}

}  // extern "C"
