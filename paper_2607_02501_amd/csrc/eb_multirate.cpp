// eb_multirate.cpp -- control ticks over modules with refresh policies (paper
// section 3.2, modular multi-rate execution).  A tick runs every due module
// in order, each its `repeats` times, through eb_qlinear_stack on the
// module's own slice of the caller's workspace: every module keeps its cached
// plan (and graph) from tick to tick, and a module that is not due costs
// nothing -- its outputs from the last refresh stay in the caller's buffers
// for the modules that read them.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/eb_multirate.h"

namespace {

size_t up256(size_t v) { return (v + 255) / 256 * 256; }

bool valid_module(const eb_module &m) {
  return m.ops && m.n_ops >= 1 && m.period >= 1 && m.phase >= 0 && m.phase < m.period &&
         m.repeats >= 1;
}

bool due(const eb_module &m, int64_t tick) { return tick % m.period == m.phase; }

// Workspace slice sizes of the modules; false when a module or op is invalid.
bool slices(const eb_module *mods, int32_t n_mods, size_t *sizes) {
  for (int32_t i = 0; i < n_mods; ++i) {
    if (!valid_module(mods[i])) return false;
    // an op list the stack rejects gives a negative launch count
    if (eb_qlinear_stack_launches(mods[i].ops, mods[i].n_ops) < 0) return false;
    sizes[i] = up256(eb_qlinear_stack_workspace_bytes(mods[i].ops, mods[i].n_ops));
  }
  return true;
}

constexpr int32_t kMaxModules = 64;

// Slice sizes of a module list, cached by the modules' contents (policy
// fields and every op), so that a tick costs no plan building on the host.
std::mutex g_mu;
std::unordered_map<std::string, std::vector<size_t>> g_sizes;

bool cached_slices(const eb_module *mods, int32_t n_mods, size_t *sizes) {
  std::string key;
  for (int32_t i = 0; i < n_mods; ++i) {
    const eb_module &m = mods[i];
    if (!valid_module(m)) return false;
    key.append(reinterpret_cast<const char *>(&m.n_ops), sizeof(m.n_ops));
    key.append(reinterpret_cast<const char *>(m.ops), sizeof(eb_qlinear_op) * (size_t)m.n_ops);
  }
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_sizes.find(key);
    if (it != g_sizes.end()) {
      for (int32_t i = 0; i < n_mods; ++i) sizes[i] = it->second[i];
      return true;
    }
  }
  if (!slices(mods, n_mods, sizes)) return false;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_sizes.size() > 256) g_sizes.clear();
  g_sizes[key] = std::vector<size_t>(sizes, sizes + n_mods);
  return true;
}

}  // namespace

extern "C" {

size_t eb_multirate_workspace_bytes(const eb_module *mods, int32_t n_mods) {
  if (!mods || n_mods < 1 || n_mods > kMaxModules) return 0;
  size_t sizes[kMaxModules];
  if (!slices(mods, n_mods, sizes)) return 0;
  size_t total = 0;
  for (int32_t i = 0; i < n_mods; ++i) total += sizes[i];
  return total;
}

eb_status eb_multirate_tick(const eb_module *mods, int32_t n_mods, int64_t tick, void *workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  if (!mods || n_mods < 1 || n_mods > kMaxModules || tick < 0) return EB_ERR_INVALID;
  size_t sizes[kMaxModules];
  if (!cached_slices(mods, n_mods, sizes)) return EB_ERR_INVALID;
  size_t total = 0;
  for (int32_t i = 0; i < n_mods; ++i) total += sizes[i];
  if (total > workspace_bytes || (total > 0 && !workspace)) return EB_ERR_INVALID;
  if (workspace && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return EB_ERR_ALIGN;
  uint8_t *base = static_cast<uint8_t *>(workspace);
  size_t off = 0;
  for (int32_t i = 0; i < n_mods; ++i) {
    const eb_module &m = mods[i];
    if (due(m, tick)) {
      for (int32_t r = 0; r < m.repeats; ++r) {
        const eb_status st = eb_qlinear_stack(m.ops, m.n_ops, sizes[i] ? base + off : nullptr,
                                              sizes[i], stream);
        if (st != EB_OK) return st;
      }
    }
    off += sizes[i];
  }
  return EB_OK;
}

int32_t eb_multirate_launches(const eb_module *mods, int32_t n_mods, int64_t tick) {
  if (!mods || n_mods < 1 || n_mods > kMaxModules || tick < 0) return EB_ERR_INVALID;
  int32_t total = 0;
  for (int32_t i = 0; i < n_mods; ++i) {
    const eb_module &m = mods[i];
    if (!valid_module(m)) return EB_ERR_INVALID;
    const int32_t l = eb_qlinear_stack_launches(m.ops, m.n_ops);
    if (l < 0) return l;
    if (due(m, tick)) total += l * m.repeats;
  }
  return total;
}

}  // extern "C"
