/*
 * eb_tuning.h -- tuning and test entry points of libeb, beside the ABI in
 * eb.h: measuring the MFMA path's tile configurations and splits of k one by
 * one (paper section 3.2, backend-specific dispatch: the automatic choice of
 * eb_qlinear is a cost model over these configurations, checked against such
 * measurements).  No process-wide state: the choice is an argument per call.
 */
#ifndef EB_TUNING_H
#define EB_TUNING_H

#include "eb.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Number of tile configurations of the MFMA path (host-only). */
int32_t eb_mfma_tile_count(void);

/* *op on the MFMA path with tile configuration `tile` (0 ..
 * eb_mfma_tile_count() - 1, or -1 for the automatic choice) and `splits`
 * splits of k (1 .. 16, or 0 for the automatic choice), with the caller's
 * workspace as in eb_qlinear_fused_ws.  A forced choice the problem cannot
 * take is replaced by the automatic one: a split with fewer than 4 K-tiles of
 * 64 per split or whose partial sums do not fit the workspace, a tile without
 * the hi/lo weight tiles that bfloat16 activations at m <= 128 use.
 * Errors as eb_qlinear_fused_ws, and EB_ERR_INVALID for tile or splits out of
 * range. */
eb_status eb_qlinear_tuned(const eb_qlinear_op *op, int32_t tile, int32_t splits, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* EB_TUNING_H */
