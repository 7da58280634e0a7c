"""Pins of the oracle's int8-activation prefill variant (runs without a GPU).

The variant (section 3.2, backend-specific dispatch) quantizes the
activations per 32-element block along k to int8 against a binary32 scale
s = fl32(max|x| / 127), codes rounded half away from zero; a block's product
is an exact integer sum of code products, scaled by s * d16.  Fixed here by
routes independent of oracle.c:
  * scales            -> numpy float32 arithmetic
  * codes             -> brute-force argmin over every code, exact rationals,
                         with the tie rule; hand-worked ties and saturation
  * product           -> exact rational sums (fractions.Fraction)
  * error bound       -> |y8 - x . w_hat| <= sum_b (s/2) sum |w_hat| against
                         the (separately pinned) binary64 16-bit-x product
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O


def _f16(vals):
    return np.asarray(vals, np.float16).reshape(1, -1).view(np.uint16)


def test_x8_golden_ties_and_saturation(oracle):
    # a = 127 -> s = fl32(127 / 127) = 1: x / s is x itself.  2.5 -> 3 and
    # -2.5 -> -3 (half away from zero), 0.5 -> 1, -0.5 -> -1, 126.5 -> 127,
    # 1.25 -> 1; the second block is all zeros: s = 0, codes 0.
    blk = [127.0, 2.5, -2.5, 0.5, -0.5, 126.5, 1.25] + [0.0] * 25
    xq, s = oracle.quantize_x8(_f16(blk + [0.0] * 32), O.X_F16)
    assert s.tolist() == [[1.0, 0.0]]
    assert xq[0, :7].tolist() == [127, 3, -3, 1, -1, 127, 1]
    assert not xq[0, 7:].any()
    # bfloat16 words: -3 is the largest magnitude -> s = fl32(3 / 127) =
    # 0.023622047 (just below 3/127), so 1.5 / s = 63.50000024 -> 64, not a
    # tie; -3 / s = -127.0000005 -> -127 (clamped)
    x = np.zeros(32, np.float32)
    x[0], x[1] = -3.0, 1.5
    bits = (x.view(np.uint32) >> 16).astype(np.uint16).reshape(1, -1)
    xq, s = oracle.quantize_x8(bits, O.X_BF16)
    s32 = np.float32(3.0) / np.float32(127.0)
    assert s[0, 0] == s32
    assert xq[0, 0] == -127
    assert Fraction(float(s32)) < Fraction(3, 127)
    assert xq[0, 1] == 64


def _brute(xv, s):
    if s == 0:
        return 0
    xf, sf = Fraction(float(xv)), Fraction(float(s))
    best, bc = None, None
    for c in range(-127, 128):
        dist = abs(xf - c * sf)
        if best is None or dist < best or (dist == best and abs(c) > abs(bc)):
            best, bc = dist, c
    return bc


@pytest.mark.parametrize("xdt", [O.X_F16, O.X_BF16])
def test_x8_scales_and_codes_brute_force(oracle, xdt):
    rng = np.random.default_rng(81 + xdt)
    x = rng.standard_normal((6, 128)).astype(np.float32)
    x[1, :32] = 0.0
    x[2, 40] = 1000.0                      # outlier channel
    x[3] *= 1e-4
    x[4, 64:96] = np.float32(0.75)         # constant block
    if xdt == O.X_F16:
        bits = x.astype(np.float16).view(np.uint16)
        xv = bits.view(np.float16).astype(np.float64)
    else:
        u = x.view(np.uint32).astype(np.uint64)
        bits = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        xv = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    xq, s = oracle.quantize_x8(bits, xdt)
    for i in range(6):
        for b in range(4):
            blk = xv[i, 32 * b:32 * b + 32]
            s_ref = np.float32(np.abs(blk).max()) / np.float32(127.0)
            assert s[i, b] == s_ref, (i, b)
            for j in range(32):
                assert xq[i, 32 * b + j] == _brute(blk[j], s_ref), (i, b, j)


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
def test_x8_product_exact_rational(oracle, qtype):
    rng = np.random.default_rng(90 + qtype)
    n, k, m = 3, 96, 2
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    bits = rng.standard_normal((m, k)).astype(np.float16).view(np.uint16)
    blocks = oracle.quantize(qtype, w)
    xq, s = oracle.quantize_x8(bits, O.X_F16)
    y, bound, qerr = oracle.qlinear_x8(qtype, blocks, n, k, xq, s)
    what = oracle.dequant(qtype, blocks, n, k)
    for i in range(m):
        for c in range(n):
            exact = Fraction(0)
            bexact = Fraction(0)
            for b in range(k // 32):
                sb = Fraction(float(s[i, b]))
                for j in range(32 * b, 32 * b + 32):
                    t = sb * int(xq[i, j]) * Fraction(float(what[c, j]))
                    exact += t
                    bexact += abs(t)
            tol = Fraction(k * 2.0 ** -52) * bexact
            assert abs(Fraction(y[i, c]) - exact) <= tol
            assert abs(Fraction(bound[i, c]) - bexact) <= tol


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
@pytest.mark.parametrize("xdt", [O.X_F16, O.X_BF16])
def test_x8_error_bound_against_16bit_product(oracle, qtype, xdt):
    """|y8 - x . w_hat| <= qerr: the activation rounding, |x - s xq| <= s / 2,
    is the only difference from the 16-bit-x product (pinned elsewhere)."""
    rng = np.random.default_rng(95)
    n, k, m = 48, 512, 9
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    x = rng.standard_normal((m, k)).astype(np.float32)
    x[:, 7] *= 300.0
    if xdt == O.X_F16:
        bits = x.astype(np.float16).view(np.uint16)
    else:
        u = x.view(np.uint32).astype(np.uint64)
        bits = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    blocks = oracle.quantize(qtype, w)
    y16, b16 = oracle.qlinear(qtype, blocks, n, k, bits, xdt)
    xq, s = oracle.quantize_x8(bits, xdt)
    y8, b8, qerr = oracle.qlinear_x8(qtype, blocks, n, k, xq, s)
    assert np.all(np.abs(y8 - y16) <= qerr * (1 + 1e-9) + 1e-12 * b16)
    # every code within range and every block's largest element at +-127
    assert np.abs(xq.astype(np.int64)).max() <= 127
    nz = s > 0
    mx = np.abs(xq.astype(np.int64)).reshape(m, k // 32, 32).max(axis=2)
    assert np.all(mx[nz] == 127)
