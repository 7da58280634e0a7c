"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import torch

from oracle import oracle as O

QT = {"q8_0": O.Q8_0, "q4_0": O.Q4_0, "q6_s": O.Q6_S}
XT = {torch.float16: O.X_F16, torch.bfloat16: O.X_BF16}

# Error bound of the method: fp32 accumulation of 16-bit inputs, normalised by
# sum_k |x||w_hat| per output.  A bfloat16 output adds one round-to-nearest of
# |y| <= bound: bfloat16 keeps 8 significant bits, so up to 2^-8 relative.
TOL_F32 = 2e-3
TOL_BF16 = 2e-3 + 2.0 ** -8 * (1 + 2e-3)
# The large-m tile kernel with bfloat16 activations (m > 128, matrix-core
# bound) multiplies w_hat rounded once to bfloat16 (8 significant bits: up to
# 2^-8 relative per weight, which a one-hot x exposes whole); its bound is the
# method's 2e-3 plus that rounding.  Every other path meets 2e-3.
TOL_TILE_BF16 = 2e-3 + 2.0 ** -8

# Worst normalised error seen per check label (the text before the first
# space), printed at the end of the session by conftest.py.
WORST = {}


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def oracle_reference(orc, qtype, w_rows_f32: np.ndarray, x: torch.Tensor):
    """Oracle y and bound for all rows of x against the given fp32 weight rows."""
    blocks = orc.quantize(QT[qtype], w_rows_f32, nthreads=O.available_cores())
    n, k = w_rows_f32.shape
    y, bound = orc.qlinear(QT[qtype], blocks, n, k, bits16(x), XT[x.dtype],
                           nthreads=O.available_cores())
    return blocks, y, bound


DTYPE_TAG = {torch.float32: "f32", torch.bfloat16: "bf16", torch.float16: "f16"}


def assert_parity(y_gpu, y_ref, bound, tol, what="", slack=None):
    """Every output within tol * bound of the oracle (exactly equal where the
    bound is 0).  slack: an optional absolute allowance per output, added to
    the error budget before normalising (a path's documented absolute term)."""
    tag = DTYPE_TAG.get(y_gpu.dtype, "?") if isinstance(y_gpu, torch.Tensor) else "np"
    y = y_gpu.detach().double().cpu().numpy() if isinstance(y_gpu, torch.Tensor) else y_gpu
    assert y.shape == y_ref.shape, (y.shape, y_ref.shape)
    assert np.all(np.isfinite(y)), what
    zero = bound == 0
    assert np.all(y[zero] == 0), f"{what}: nonzero output where the bound is 0"
    if (~zero).any():
        err = np.abs(y[~zero] - y_ref[~zero])
        if slack is not None:
            err = np.maximum(err - np.broadcast_to(slack, y.shape)[~zero], 0.0)
        rel = err / bound[~zero]
        worst = float(rel.max())
        label = (what.split(" ")[0] if what else "unlabelled") + "/" + tag
        WORST[label] = max(WORST.get(label, 0.0), worst)
        assert worst <= tol, f"{what}: max normalised error {worst:.3e} > {tol:.3e}"
        return worst
    return 0.0
