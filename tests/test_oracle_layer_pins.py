"""Pins of the oracle's decoder-layer steps around the linear layer (no GPU).

The fused prologue and epilogues of a projection (paper section 3.2: operator
fusion on the batch-1 path) are RMS normalisation of the residual stream, the
SiLU-gated product of a gate/up projection pair and the residual addition.
Each oracle function is fixed here by a route independent of oracle.c:
  * rounding to binary16   -> numpy's float64 -> float16 conversion (library routine)
  * rounding to bfloat16   -> brute force over every finite bfloat16 value decoded by
                              torch, with the ties-to-even rule; torch's own
                              float32 -> bfloat16 conversion for float32 inputs
  * RMS normalisation      -> closed forms (constant rows, one-hot rows, a 3-4-5 case),
                              exact power-of-two scale invariance, unit mean square
  * SiLU-gated product     -> closed forms (silu(0) = 0, silu(t) - silu(-t) = t,
                              silu(ln 3) = (3/4) ln 3, saturation) and linearity in u
  * composition            -> the interleaved gate/up convention and the residual
                              addition against plain oracle products of single rows
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O

# ---------------------------------------------------------------------------
# rounding float64 -> binary16 / bfloat16
# ---------------------------------------------------------------------------


def _f16_specials():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    fin = h[np.isfinite(h)].astype(np.float64)
    fin = np.unique(fin)
    mids = (fin[:-1] + fin[1:]) / 2  # exact: neighbours differ by one spacing
    return np.concatenate([fin, mids, np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)])


def test_round_f16_matches_numpy(oracle):
    rng = np.random.default_rng(3)
    v = np.concatenate([
        _f16_specials(),
        rng.standard_normal(20000) * np.exp2(rng.integers(-30, 18, 20000)),
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 70000.0, -65520.0, 2.0 ** -25,
                  2.0 ** -26, 3 * 2.0 ** -26, np.inf, -np.inf]),
    ])
    got = oracle.round_x16(v, O.X_F16)
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def _bf16_grid():
    w = torch.arange(1 << 16, dtype=torch.int32).to(torch.int16)
    vals = w.view(torch.bfloat16).double().numpy()
    bits = w.numpy().view(np.uint16)
    ok = np.isfinite(vals) & (vals >= 0) & ~((vals == 0) & (bits != 0))  # +0 and positives
    order = np.argsort(vals[ok])
    return vals[ok][order], bits[ok][order]


def _bf16_brute(v, grid, gbits):
    """Nearest finite bfloat16 (ties to the even encoding), overflow to infinity."""
    out = np.empty(v.shape, np.uint16)
    top = grid[-1]
    half_ulp_top = (2.0 ** 128 - top) / 2  # the spacing above the largest finite value
    for i, x in enumerate(v):
        s = 0x8000 if math.copysign(1.0, x) < 0 else 0
        a = abs(x)
        if a >= top + half_ulp_top:
            out[i] = s | 0x7F80
            continue
        j = np.searchsorted(grid, a)  # grid[j-1] < a <= grid[j]
        if j < len(grid) and grid[j] == a:
            out[i] = s | gbits[j]
            continue
        if j == len(grid):  # above the largest finite value but below the rounding boundary
            out[i] = s | gbits[-1]
            continue
        lo, hi = grid[j - 1], grid[j]
        dl, dh = a - lo, hi - a  # exact (Sterbenz)
        if dl < dh or (dl == dh and gbits[j - 1] % 2 == 0):
            out[i] = s | gbits[j - 1]
        else:
            out[i] = s | gbits[j]
    return out


def test_round_bf16_brute_force(oracle):
    grid, gbits = _bf16_grid()
    rng = np.random.default_rng(4)
    mids = (grid[:-1] + grid[1:]) / 2
    pick = rng.choice(len(mids), 3000, replace=False)
    v = np.concatenate([
        mids[pick], -mids[pick], np.nextafter(mids[pick], 0), np.nextafter(mids[pick], np.inf),
        rng.standard_normal(3000) * np.exp2(rng.integers(-140, 120, 3000)),
        grid[rng.choice(len(grid), 500)],
        np.array([0.0, -0.0, 3.0e38, 3.39e38, 3.3961e38, 3.4e38, 2.0 ** -134, 3 * 2.0 ** -135]),
    ])
    assert np.array_equal(oracle.round_x16(v, O.X_BF16), _bf16_brute(v, grid, gbits))


def test_round_bf16_matches_torch_for_float32_inputs(oracle):
    rng = np.random.default_rng(5)
    f = (rng.standard_normal(50000) * np.exp2(rng.integers(-120, 120, 50000))).astype(np.float32)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.round_x16(f.astype(np.float64), O.X_BF16), ref)


# ---------------------------------------------------------------------------
# RMS normalisation
# ---------------------------------------------------------------------------


def test_rmsnorm_constant_rows_give_signed_gamma(oracle):
    rng = np.random.default_rng(6)
    k = 64  # powers of two keep every step exact: k c^2, its mean, the root, 1/|c|
    gamma = rng.standard_normal(k).astype(np.float32)
    c = np.array([4.0, -0.25, 2.0 ** -70, -(2.0 ** 60)], np.float32)
    h = np.repeat(c[:, None], k, axis=1)
    out = oracle.rmsnorm(h, gamma, 0.0)
    assert np.array_equal(out, np.sign(c)[:, None] * gamma.astype(np.float64)[None, :])


def test_rmsnorm_one_hot_row(oracle):
    k = 256  # sqrt(k) = 16 exactly
    gamma = np.linspace(0.5, 1.5, k).astype(np.float32)
    h = np.zeros((2, k), np.float32)
    h[0, 17] = 5.5
    h[1, 200] = -0.75
    out = oracle.rmsnorm(h, gamma, 0.0)
    ref = np.zeros((2, k))
    ref[0, 17] = 16.0 * float(gamma[17])
    ref[1, 200] = -16.0 * float(gamma[200])
    assert np.array_equal(out, ref)


def test_rmsnorm_eps_inside_the_root(oracle):
    """h = 3 everywhere, eps = 16: 3 / sqrt(9 + 16) = 0.6."""
    k = 8
    gamma = np.full(k, 2.0, np.float32)
    out = oracle.rmsnorm(np.full((1, k), 3.0, np.float32), gamma, 16.0)
    assert np.allclose(out, 1.2, rtol=1e-15, atol=0)
    # a zero row with eps > 0 normalises to zeros
    assert np.array_equal(oracle.rmsnorm(np.zeros((1, k), np.float32), gamma, 1e-6), np.zeros((1, k)))


def test_rmsnorm_scale_invariance_and_unit_mean_square(oracle):
    rng = np.random.default_rng(7)
    m, k = 5, 1000
    h = rng.standard_normal((m, k)).astype(np.float32)
    gamma = (rng.random(k) + 0.5).astype(np.float32)
    a = oracle.rmsnorm(h, gamma, 0.0)
    b = oracle.rmsnorm(h * np.float32(2.0 ** 37), gamma, 0.0)
    assert np.array_equal(a, b)
    ms = np.mean((a / gamma.astype(np.float64)) ** 2, axis=1)
    assert np.allclose(ms, 1.0, rtol=1e-12, atol=0)


def test_rmsnorm_rejects_zero_row_without_eps(oracle):
    with pytest.raises(ValueError):
        oracle.rmsnorm(np.zeros((1, 32), np.float32), np.ones(32, np.float32), 0.0)


# ---------------------------------------------------------------------------
# SiLU-gated product
# ---------------------------------------------------------------------------


def test_silu_closed_forms(oracle):
    t = np.array([0.0, math.log(3.0), 40.0, -40.0, 800.0, -800.0])
    s = oracle.silu_mul(t, np.ones_like(t))
    assert s[0] == 0.0
    assert math.isclose(s[1], 0.75 * math.log(3.0), rel_tol=1e-15)
    assert s[2] == 40.0  # 40 / (1 + e^-40) rounds to 40
    assert -1e-15 < s[3] < 0.0
    assert s[4] == 800.0 and s[5] == -0.0
    rng = np.random.default_rng(8)
    g = rng.standard_normal(1000) * 4
    odd = oracle.silu_mul(g, np.ones_like(g)) - oracle.silu_mul(-g, np.ones_like(g))
    assert np.allclose(odd, g, rtol=1e-14, atol=1e-15)
    u = rng.standard_normal(1000)
    assert np.allclose(oracle.silu_mul(g, u), oracle.silu_mul(g, np.ones_like(g)) * u,
                       rtol=1e-15, atol=0)


# ---------------------------------------------------------------------------
# composition around the linear layer
# ---------------------------------------------------------------------------


def _setup(rng, qtype, n, k, m):
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    blocks = O.get().quantize(qtype, w)
    x = rng.standard_normal((m, k)).astype(np.float32)
    return blocks, x


def test_fused_glu_pairs_interleaved_rows(oracle):
    rng = np.random.default_rng(9)
    n, k, m = 12, 64, 3
    blocks, x = _setup(rng, O.Q8_0, n, k, m)
    xw = torch.from_numpy(x).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    y, scale, _ = oracle.fused_qlinear(O.Q8_0, blocks, n, k, xw, O.X_F16, epilogue="glu")
    assert y.shape == (m, n // 2)
    bb = oracle.block_bytes(O.Q8_0)
    for j in range(n // 2):
        g, bg = oracle.qlinear(O.Q8_0, blocks[2 * j:2 * j + 1], 1, k, xw, O.X_F16)
        u, bu = oracle.qlinear(O.Q8_0, blocks[2 * j + 1:2 * j + 2], 1, k, xw, O.X_F16)
        g, u, bg, bu = g[:, 0], u[:, 0], bg[:, 0], bu[:, 0]
        assert np.array_equal(y[:, j], g / (1 + np.exp(-g)) * u)
        assert np.all(scale[:, j] >= 1.1 * bg * np.abs(u))
    assert bb == 34


def test_fused_add_and_rmsnorm_prologue(oracle):
    rng = np.random.default_rng(10)
    n, k, m = 8, 128, 4
    blocks, h = _setup(rng, O.Q4_0, n, k, m)
    gamma = (rng.random(k) + 0.5).astype(np.float32)
    r = rng.standard_normal((m, n))
    y, scale, xw = oracle.fused_qlinear(O.Q4_0, blocks, n, k, h, O.X_BF16, prologue="rmsnorm",
                                        gamma=gamma, eps=1e-5, epilogue="add", residual=r)
    # the product takes the normalised activations rounded to bfloat16
    xref = oracle.round_x16(oracle.rmsnorm(h, gamma, 1e-5), O.X_BF16)
    assert np.array_equal(xw, xref)
    y0, b0 = oracle.qlinear(O.Q4_0, blocks, n, k, xref, O.X_BF16)
    assert np.array_equal(y, y0 + r) and np.array_equal(scale, b0)
    # a subset of rows computes the same rows
    ys, _, _ = oracle.fused_qlinear(O.Q4_0, blocks, n, k, h, O.X_BF16, prologue="rmsnorm",
                                    gamma=gamma, eps=1e-5, epilogue="add", residual=r, rows=[3, 1])
    assert np.array_equal(ys, y[[3, 1]])
