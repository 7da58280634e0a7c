"""GPU parity of the low-precision prefill variant (EB_PATH_MFMA_I8) through
the C ABI, against the oracle's int8-activation method.

Bars: the int8 activation codes and block scales are bit-exact with the
oracle's; every output is within 2e-3 of the method's exact value normalised
by sum |s xq||w_hat| (plus one rounding for a 16-bit output); and the
difference from the 16-bit product stays within the method's stated
activation-quantization bound (the oracle's qerr) plus that tolerance.
"""
import ctypes

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import QT, TOL_BF16, TOL_F32, XT, assert_parity, bits16, oracle_reference

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _run_i8(eb, qw, x, out_dtype=torch.float32, epilogue=None, residual=None):
    """One call on the int8 path with a workspace of exactly the reported size;
    returns (y, workspace)."""
    m = x.shape[0]
    n_out = qw.n // 2 if epilogue == "glu" else qw.n
    y = torch.empty((m, n_out), dtype=out_dtype, device=DEV)
    op = eb.make_op(qw, x, y, epilogue=epilogue, residual=residual)
    nbytes = int(eb.lib.eb_qlinear_workspace_bytes(ctypes.byref(op), eb.EB_PATH_MFMA_I8))
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    st = eb.lib.eb_qlinear_fused_ws(ctypes.byref(op), eb.EB_PATH_MFMA_I8, ws.data_ptr(), nbytes,
                                    torch.cuda.current_stream().cuda_stream)
    assert st == eb.EB_OK, st
    torch.cuda.synchronize()
    return y, ws


def _x8_reference(oracle, qtype, w_rows, x, rows=None):
    blocks = oracle.quantize(QT[qtype], w_rows, nthreads=O.available_cores())
    xb = bits16(x if rows is None else x[rows])
    xq, s = oracle.quantize_x8(xb, XT[x.dtype])
    n, k = w_rows.shape
    y8, b8, qerr = oracle.qlinear_x8(QT[qtype], blocks, n, k, xq, s)
    y16, b16 = oracle.qlinear(QT[qtype], blocks, n, k, xb, XT[x.dtype], nthreads=O.available_cores())
    return y8, b8, qerr, y16, b16, xq, s


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_i8_codes_bit_exact_and_parity(eb, oracle, qtype, xdtype):
    """Ragged m and n around the 128 x 128 tiles, 65 blocks of k."""
    n, k = 300, 2080
    w = W.normal((n, k), 1500, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), qtype)
    for m in (1, 37, 128, 129, 300):
        x = W.normal((m, k), 1501 + m, "cpu").to(xdtype)
        y, ws = _run_i8(eb, qw, x.to(DEV))
        y8, b8, qerr, y16, b16, xq, s = _x8_reference(oracle, qtype, w.numpy(), x)
        # the activation step: codes [m][k] at offset 0, block scales [k/32][ms] after
        ms = (m + 3) // 4 * 4
        raw = ws.cpu().numpy()
        got_q = raw[:m * k].view(np.int8).reshape(m, k)
        off = (m * k + 255) // 256 * 256
        got_s = raw[off:off + 4 * (k // 32) * ms].view(np.float32).reshape(k // 32, ms)[:, :m].T
        assert np.array_equal(got_q, xq), m
        assert np.array_equal(got_s, s), m
        assert_parity(y, y8, b8, TOL_F32, f"i8 m={m}")
        # against the 16-bit product: within the stated activation-rounding bound
        err = np.abs(y.double().cpu().numpy() - y16)
        assert np.all(err <= qerr + TOL_F32 * b8 + 1e-30), m
    y, _ = _run_i8(eb, qw, x.to(DEV), out_dtype=torch.bfloat16)
    assert_parity(y, y8, b8, TOL_BF16, "i8 bf16 out")


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_i8_epilogues(eb, oracle, qtype):
    n, k, m = 258, 1024, 150
    w = W.normal((n, k), 1600, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), qtype)
    x = W.normal((m, k), 1601, "cpu").to(torch.bfloat16)
    y8, b8, _, _, _, _, _ = _x8_reference(oracle, qtype, w.numpy(), x)
    r = W.normal((m, n), 1602, "cpu")
    y, _ = _run_i8(eb, qw, x.to(DEV), epilogue="add", residual=r.to(DEV))
    assert_parity(y, y8 + r.double().numpy(), b8, TOL_F32, "i8_add")
    y, _ = _run_i8(eb, qw, x.to(DEV), epilogue="glu")
    g, u = y8[:, 0::2], y8[:, 1::2]
    ref = oracle.silu_mul(g, u)
    silu = oracle.silu_mul(g, np.ones_like(g))
    scale = 1.1 * b8[:, 0::2] * np.abs(u) + np.abs(silu) * b8[:, 1::2] + 0.0022 * b8[:, 0::2] * b8[:, 1::2]
    assert_parity(y, ref, scale, TOL_F32, "i8_glu")


@pytest.mark.parametrize("kind", ["onehot", "outlier", "sparse"])
def test_i8_structured_activations(eb, oracle, kind):
    n, k, m = 256, 1536, 130
    w = W.normal((n, k), 1700, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), "q8_0")
    gen = {"onehot": W.onehot_rows, "sparse": W.sparse_rows, "outlier": W.outlier_rows}[kind]
    x = gen(m, k, 1701).to(torch.bfloat16)
    y, _ = _run_i8(eb, qw, x.to(DEV))
    y8, b8, qerr, y16, _, _, _ = _x8_reference(oracle, "q8_0", w.numpy(), x)
    assert_parity(y, y8, b8, TOL_F32, f"i8_{kind}")
    assert np.all(np.abs(y.double().cpu().numpy() - y16) <= qerr + TOL_F32 * b8 + 1e-30)


def test_i8_refusals(eb):
    qw = eb.quantize(W.normal((64, 512), 1800, DEV, W.WEIGHT_STD), "q6_s")
    x = W.normal((64, 512), 1801, DEV).to(torch.bfloat16)
    y = torch.empty((64, 64), device=DEV)
    op = eb.make_op(qw, x, y)
    assert eb.lib.eb_qlinear_fused_ws(ctypes.byref(op), eb.EB_PATH_MFMA_I8, None, 0, None) == \
        eb.EB_ERR_UNSUPPORTED
    qw = eb.quantize(W.normal((64, 512), 1802, DEV, W.WEIGHT_STD), "q8_0")
    h = W.normal((64, 512), 1803, DEV)
    op = eb.make_op(qw, h, y, x_dtype=torch.bfloat16, prologue="rmsnorm",
                    norm_weight=torch.ones(512, device=DEV), eps=1e-5)
    assert eb.lib.eb_qlinear_fused_ws(ctypes.byref(op), eb.EB_PATH_MFMA_I8, None, 0, None) == \
        eb.EB_ERR_UNSUPPORTED
    op = eb.make_op(qw, x, y)   # no workspace
    assert eb.lib.eb_qlinear_fused_ws(ctypes.byref(op), eb.EB_PATH_MFMA_I8, None, 0, None) == \
        eb.EB_ERR_UNSUPPORTED


@pytest.mark.parametrize("name", ["q8_0_vlm_prefill_816", "q4_0_video_wam_4096"])
def test_i8_workload_sampled(eb, oracle, name):
    """The prefill workloads' widest projection at full size, sampled outputs."""
    wl = W.WORKLOADS[name]
    rng = np.random.default_rng(79)
    p = max(range(len(wl.projections)), key=lambda i: wl.projections[i][2] * wl.projections[i][1])
    pname, k, n = wl.projections[p]
    print(f"[parity] i8 {name} {pname} m={wl.m} n={n} k={k}", flush=True)
    w = W.weights(wl, 0, p, DEV)
    x = W.activations(wl, 0, p, DEV)
    qw = eb.quantize(w, wl.qtype)
    y, _ = _run_i8(eb, qw, x)
    cols = np.array(sorted({0, n - 1, 127, 128} | set(rng.choice(n, 40, replace=False).tolist())))
    rows = np.array(sorted({0, wl.m - 1, 127, 128} | set(rng.choice(wl.m, 20, replace=False).tolist())))
    wrows = w[torch.from_numpy(cols).to(DEV)].cpu().numpy()
    xr = x[torch.from_numpy(rows).to(DEV)].cpu()
    y8, b8, qerr, y16, _, _, _ = _x8_reference(oracle, wl.qtype, wrows, xr)
    got = y[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)]
    assert_parity(got, y8, b8, TOL_F32, f"i8_{name}")
    assert np.all(np.abs(got.double().cpu().numpy() - y16) <= qerr + TOL_F32 * b8 + 1e-30)
    del w, qw, y
    torch.cuda.empty_cache()
