"""GPU parity on structured activations: one-hot, sparse and outlier-channel
rows, and weights whose block scales span the binary16 range.

Dense N(0, 1) rows let rounding errors of different terms cancel; these
inputs do not.  A one-hot row makes one product the whole output, so any
rounding of w_hat shows at full size; sparse rows keep a few terms; outlier
channels (a few feature columns a thousand times larger than the rest, as
backbone activations have) stress any decode whose fp32 error grows with
sum |x| rather than with sum |x||w_hat|.  Every kernel path is compared with
the binary64 oracle element by element at the method's bar (2e-3 of
sum_k |x||w_hat|), except the bfloat16 large-m tile kernel, whose documented
bar adds the one bfloat16 rounding of w_hat (2^-8).
"""
import numpy as np
import pytest
import torch

from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import TOL_F32, TOL_TILE_BF16, assert_parity, oracle_reference

pytestmark = pytest.mark.gpu

DEV = "cuda"
N, K = 264, 1056           # ragged n, 33 blocks (odd block count, K tail)
N2, K2 = 136, 2080         # second op of the stacked cases
M_MAX = 300


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _x(kind, m, k, seed, xdtype):
    if kind == "onehot":
        x = W.onehot_rows(m, k, seed)
    elif kind == "sparse":
        x = W.sparse_rows(m, k, seed)
    elif kind == "outlier":
        x = W.outlier_rows(m, k, seed)
    else:
        raise ValueError(kind)
    return x.to(xdtype)


def _tol(xdtype, path, m):
    return TOL_TILE_BF16 if (xdtype == torch.bfloat16 and path in ("tile", "grouped") and m > 128) else TOL_F32


@pytest.mark.parametrize("kind", ["onehot", "sparse", "outlier"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_structured_activations_every_path(eb, oracle, qtype, xdtype, kind, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    monkeypatch.delenv("EB_STACK_GROUP", raising=False)
    seed = 4000 + 7 * (qtype == "q4_0") + 3 * (xdtype == torch.bfloat16)
    w = W.normal((N, K), seed, "cpu", W.WEIGHT_STD)
    w2 = W.normal((N2, K2), seed + 1, "cpu", W.WEIGHT_STD)
    x = _x(kind, M_MAX, K, seed + 2, xdtype)
    x2 = _x(kind, M_MAX, K2, seed + 3, xdtype)
    qw, qw2 = eb.quantize(w.to(DEV), qtype), eb.quantize(w2.to(DEV), qtype)
    _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
    _, y_ref2, bound2 = oracle_reference(oracle, qtype, w2.numpy(), x2)
    xd, xd2 = x.to(DEV), x2.to(DEV)
    tag = f"{qtype} {xdtype} {kind}"
    print(f"[adversarial] {tag}", flush=True)
    # GEMV path
    for m in (1, 4):
        y = eb.qlinear(qw, xd[:m], path="gemv")
        assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"adv_gemv m={m} {tag}")
    # single-op MFMA path: small m (HBM-bound tiles) and large m
    for m in (50, 128, 300):
        y = eb.qlinear(qw, xd[:m], path="mfma")
        assert_parity(y, y_ref[:m], bound[:m], _tol(xdtype, "tile", m), f"adv_tile m={m} {tag}")
    # fused small-m launches (m <= 64 and 64 < m <= 128) and the grouped
    # large-m launch: two independent ops per stack
    for m, path in ((50, "fused"), (100, "fused"), (300, "grouped")):
        ya = torch.full((m, N), float("nan"), device=DEV)
        yb = torch.full((m, N2), float("nan"), device=DEV)
        ops = eb.make_ops([(qw, xd[:m], ya), (qw2, xd2[:m], yb)])
        assert eb.stack_launches(ops) <= 3
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        tol = _tol(xdtype, path, m)
        assert_parity(ya, y_ref[:m], bound[:m], tol, f"adv_{path} m={m} {tag}")
        assert_parity(yb, y_ref2[:m], bound2[:m], tol, f"adv_{path} m={m} {tag} (op 2)")
    eb.stack_cache_clear()


def _extreme_scale_weights(n, k, seed):
    """N(0, 0.02) rows whose blocks are rescaled: every third block to
    max |w| = 60000 (binary16 range of w_hat kept), every fifth to about 1e-6
    (binary16-subnormal scales)."""
    w = W.normal((n, k), seed, "cpu", W.WEIGHT_STD).view(n, k // 32, 32)
    amax = w.abs().amax(dim=2, keepdim=True).clamp_min(1e-30)
    nb = k // 32
    big = torch.zeros(nb, dtype=torch.bool)
    big[0::3] = True
    tiny = torch.zeros(nb, dtype=torch.bool)
    tiny[1::5] = True
    w = torch.where(big.view(1, nb, 1), w / amax * 60000.0, w)
    w = torch.where(tiny.view(1, nb, 1), w / amax * 1e-6, w)
    return w.reshape(n, k).contiguous()


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_extreme_block_scales_every_path(eb, oracle, qtype, xdtype, monkeypatch):
    """Blocks with max |w| up to 60000 and down to 1e-6 in one row.  On the
    MFMA path with binary16 activations w_hat is rounded to binary16, whose
    subnormal spacing is 2^-24: the documented bound there adds 2^-25 sum_k |x|
    per output.  bfloat16 keeps the binary32 exponent range, so no term is
    added on the bfloat16 paths."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    seed = 4100 + 7 * (qtype == "q4_0") + 3 * (xdtype == torch.bfloat16)
    w = _extreme_scale_weights(N, K, seed)
    x = W.normal((M_MAX, K), seed + 1, "cpu").to(xdtype)
    qw = eb.quantize(w.to(DEV), qtype)
    _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
    xd = x.to(DEV)
    sum_abs_x = x.double().abs().sum(dim=1, keepdim=True).numpy()
    slack = 2.0 ** -25 * sum_abs_x if xdtype == torch.float16 else None
    tag = f"{qtype} {xdtype}"
    for m in (1, 4):
        y = eb.qlinear(qw, xd[:m], path="gemv")
        assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"adv_scale_gemv m={m} {tag}")
    for m in (50, 300):
        y = eb.qlinear(qw, xd[:m], path="mfma")
        assert_parity(y, y_ref[:m], bound[:m], _tol(xdtype, "tile", m), f"adv_scale_tile m={m} {tag}",
                      slack=None if slack is None else slack[:m])
    ya = torch.full((50, N), float("nan"), device=DEV)
    yb = torch.full((50, N), float("nan"), device=DEV)
    ops = eb.make_ops([(qw, xd[:50], ya), (qw, xd[50:100], yb)])
    eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    assert_parity(ya, y_ref[:50], bound[:50], TOL_F32, f"adv_scale_fused m=50 {tag}",
                  slack=None if slack is None else slack[:50])
    assert_parity(yb, y_ref[50:100], bound[50:100], TOL_F32, f"adv_scale_fused m=50 {tag} (op 2)",
                  slack=None if slack is None else slack[50:100])
    eb.stack_cache_clear()


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_constant_blocks_closed_form(eb, qtype, xdtype):
    """A row whose every block holds one value c (sign alternating by block):
    Q8_0 codes are all 127 sign(c) and Q4_0 codes all -8 (the extreme element
    maps to -8), so y = 127 sign(c) d16 sum_j x_j (Q8_0) or -8 d16 sum_j x_j
    (Q4_0) per block, with d16 the binary16 rounding of |c| / 127 or c / -8."""
    n, k = 40, 512
    nb = k // 32
    mags = torch.linspace(0.01, 0.05, n).view(n, 1, 1)
    sgn = torch.tensor([1.0 if b % 2 == 0 else -1.0 for b in range(nb)]).view(1, nb, 1)
    w = (mags * sgn).expand(n, nb, 32).reshape(n, k).contiguous().float()
    x = W.normal((64, k), 4200, "cpu").to(xdtype)
    qw = eb.quantize(w.to(DEV), qtype)
    # closed form in binary64 from binary16 scales computed by torch's own conversion
    c = (mags * sgn).view(n, nb).double()
    if qtype == "q8_0":
        d16 = (c.abs().float() / 127.0).half().double()
        coef = 127.0 * torch.sign(c) * d16            # w_hat of every element of block b
    else:
        d16 = (c.float() / -8.0).half().double()
        coef = -8.0 * d16
    xs = x.double().view(64, nb, 32).sum(dim=2)       # sum of x over each block
    y_cf = (xs @ coef.t()).numpy()                     # [m, n]
    bound = (x.double().abs().view(64, nb, 32).sum(dim=2) @ coef.abs().t()).numpy()
    for m, path in ((1, "gemv"), (4, "gemv"), (64, "mfma")):
        y = eb.qlinear(qw, x[:m].to(DEV), path=path)
        assert_parity(y, y_cf[:m], bound[:m], TOL_F32, f"closed_form_const m={m} {qtype} {xdtype}")
