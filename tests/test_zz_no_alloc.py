"""The no-allocation entry point (eb_qlinear_fused_static) against the entry
point it varies (eb_qlinear_fused_ws), through the C ABI: two calls in a row
on one device, the second with a smaller input, each with a normalisation
prologue on the MFMA path (its scratch holds the normalised activations), the
first also with a split of k (its scratch then holds the partial sums too)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import TOL_F32

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _case(eb, seed, m, n, k, qtype, epi):
    w = W.normal((n, k), seed, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), qtype)
    h = (W.normal((m, k), seed + 1, "cpu") * 2.0).to(DEV)
    g = (1.0 + 0.1 * W.normal((k,), seed + 2, "cpu")).to(DEV)
    n_out = n // 2 if epi == "glu" else n
    r = W.normal((m, n_out), seed + 3, "cpu").to(DEV) if epi == "add" else None
    return qw, h, g, r, n_out


def _op(eb, qw, h, g, r, y, epi):
    return eb.make_op(qw, h, y, x_dtype=torch.bfloat16, prologue="rmsnorm", norm_weight=g,
                      eps=1e-5, epilogue=epi, residual=r)


@pytest.mark.parametrize("qtype,epi", [("q8_0", "add"), ("q4_0", "glu")])
def test_static_scratch_matches_workspace_entry(eb, qtype, epi):
    stream = torch.cuda.current_stream().cuda_stream
    # m = 100, k = 4096 -> n = 1024: split along k on the MFMA path (partial
    # sums after the normalised activations); then m = 20, k = 1024 -> n =
    # 4096 (one narrow launch whose workgroups fill the GPU: normalised
    # activations only)
    for i, (m, n, k) in enumerate(((100, 1024, 4096), (20, 4096, 1024))):
        print(f"[no-alloc] {qtype} {epi} call {i}: m={m} n={n} k={k}", flush=True)
        qw, h, g, r, n_out = _case(eb, 7000 + 10 * i, m, n, k, qtype, epi)
        y_ws = torch.full((m, n_out), float("nan"), device=DEV)
        y_st = torch.full((m, n_out), float("nan"), device=DEV)
        op_ws = _op(eb, qw, h, g, r, y_ws, epi)
        op_st = _op(eb, qw, h, g, r, y_st, epi)
        nbytes = int(eb.lib.eb_qlinear_workspace_bytes(ctypes.byref(op_ws), eb.EB_PATH_MFMA))
        assert nbytes > m * k * 2 if i == 0 else nbytes == m * k * 2
        ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
        assert eb.lib.eb_qlinear_fused_ws(ctypes.byref(op_ws), eb.EB_PATH_MFMA, ws.data_ptr(),
                                          nbytes, stream) == eb.EB_OK
        assert eb.lib.eb_qlinear_fused_static(ctypes.byref(op_st), eb.EB_PATH_MFMA,
                                              stream) == eb.EB_OK
        torch.cuda.synchronize()
        assert torch.isfinite(y_st).all()
        # the same plan (tiles, split) on the same inputs: the same bits
        assert torch.equal(y_st, y_ws), (m, n, k)
        scale = (y_ws.abs() + 1e-30)
        assert float(((y_st - y_ws).abs() / scale).max()) <= TOL_F32


def test_static_scratch_rejects_oversized_prologue(eb):
    """Normalised activations larger than the 32 MiB array are refused before
    anything is launched."""
    qw = eb.empty_qweights("q8_0", 256, 16384, DEV)
    m, k = 1100, 16384  # 1100 * 16384 * 2 bytes > 32 MiB
    h = torch.zeros((m, k), device=DEV)
    g = torch.ones((k,), device=DEV)
    y = torch.empty((m, 256), device=DEV)
    op = eb.make_op(qw, h, y, x_dtype=torch.bfloat16, prologue="rmsnorm", norm_weight=g, eps=1e-5)
    st = eb.lib.eb_qlinear_fused_static(ctypes.byref(op), eb.EB_PATH_MFMA,
                                        torch.cuda.current_stream().cuda_stream)
    assert st == eb.EB_ERR_UNSUPPORTED
