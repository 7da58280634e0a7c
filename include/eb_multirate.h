/*
 * eb_multirate.h -- modular multi-rate execution of projection stacks (paper
 * section 3.1, first challenge, and section 3.2, first principle: components
 * of an embodied model run at different rates inside one control loop, as
 * explicit execution units with shared state and configurable refresh
 * policies).
 *
 * A module is one execution unit: a stack of projections (eb_qlinear_stack)
 * with a refresh policy.  A control tick runs, in module order, every module
 * that is due on that tick, each `repeats` times in a row.  For a
 * VLM-backboned policy with a flow-matching action expert: the backbone
 * module (the prefill of the observation, period R: refreshed every R ticks)
 * writes its outputs -- the residual stream and the projections that feed the
 * expert's attention -- into buffers that persist between ticks (the shared
 * state), and the expert module (period 1, repeats = the denoising steps)
 * reads them on every tick; between refreshes the backbone's state is reused,
 * not recomputed.
 *
 * Ownership and state: the caller owns the op arrays, every buffer they
 * name and the workspace; the library keeps only the stack-plan cache of
 * eb_qlinear_stack.  Each module gets its own 256-byte aligned slice of the
 * workspace (in module order, each as large as eb_qlinear_stack_workspace_bytes
 * of the module's ops), so the plans of all modules stay cached side by side.
 * The modules of a tick run in order on `stream`; EB_OK means enqueued.
 */
#ifndef EB_MULTIRATE_H
#define EB_MULTIRATE_H

#include "eb.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  const eb_qlinear_op *ops; /* host array of n_ops ops (as for eb_qlinear_stack) */
  int32_t n_ops;            /* >= 1 */
  int32_t period;           /* refresh policy: due on ticks t with t % period == phase; >= 1 */
  int32_t phase;            /* 0 <= phase < period */
  int32_t repeats;          /* runs per due tick, one after another; >= 1 */
} eb_module;

/* Workspace bytes for eb_multirate_tick over these modules (the sum of the
 * modules' stack workspaces, each rounded up to 256); 0 for invalid modules. */
size_t eb_multirate_workspace_bytes(const eb_module *mods, int32_t n_mods);

/* Run control tick `tick` (>= 0): every due module, in order, `repeats`
 * times.  workspace: device memory, 256-byte aligned, at least
 * eb_multirate_workspace_bytes bytes (may be null when that is 0), the same
 * pointer on every tick so that cached plans are reused.
 * EB_ERR_INVALID: null or empty module list, a bad policy field, tick < 0, a
 * workspace too small, or any op that eb_qlinear_stack rejects (nothing is
 * launched then). */
eb_status eb_multirate_tick(const eb_module *mods, int32_t n_mods, int64_t tick, void *workspace,
                            size_t workspace_bytes, hipStream_t stream);

/* Kernel launches control tick `tick` makes (host only), or a negative
 * eb_status for invalid arguments. */
int32_t eb_multirate_launches(const eb_module *mods, int32_t n_mods, int64_t tick);

#ifdef __cplusplus
}
#endif

#endif /* EB_MULTIRATE_H */
