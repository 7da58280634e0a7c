"""Pins of the CPU oracle against things other than itself (runs without a GPU).

Each test fixes part of the oracle by a route independent of oracle.c:
  * binary16 / bfloat16 conversion  -> numpy's own IEEE conversions (library routine)
  * packed bytes of special blocks   -> values worked out by hand from the block
                                        format definition (closed form)
  * scales                           -> recomputed with numpy float32 / float16 arithmetic
  * codes                            -> brute-force argmin over every code, in exact
                                        rational arithmetic, with the tie rule
  * round trip                       -> |x - w_hat| <= |d16|/2 invariant
  * matmul                           -> exact rational sums (fractions.Fraction) and
                                        numpy float64 BLAS
The block formats are the Q8_0 / Q4_0 layouts (32 weights per block along k,
one binary16 scale) behind the paper's 8-bit and 4-bit configurations
(section 4, Table 3).
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O

# ---------------------------------------------------------------------------
# binary16 / bfloat16 conversions
# ---------------------------------------------------------------------------


def test_half_decode_every_code(oracle):
    codes = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = codes.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(c)) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_bf16_decode_every_code(oracle):
    codes = np.arange(1 << 16, dtype=np.uint32)
    ref = (codes << 16).astype(np.uint32).view(np.float32).astype(np.float64)
    got = np.array([oracle.bf16_to_double(int(c)) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def _float_cases(rng):
    # random binary32 bit patterns over the whole range, plus the places where
    # binary16 rounding is delicate: exact ties, the subnormal range, the
    # normal/subnormal border and the overflow threshold.
    cases = [rng.integers(0, 1 << 32, 20000, dtype=np.uint64).astype(np.uint32).view(np.float32)]
    h = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float32)
    cases.append(h)                                           # every finite binary16 value
    mid = ((h[:-1].astype(np.float64) + h[1:].astype(np.float64)) / 2).astype(np.float32)
    cases.append(mid)                                         # exact midpoints (ties)
    cases.append(np.nextafter(mid, np.float32(0)))
    cases.append(np.nextafter(mid, np.float32(np.inf)))
    cases.append(np.array([65504.0, 65519.0, 65519.996, 65520.0, 65536.0, 1e30, 2.0 ** -24,
                           2.0 ** -25, np.nextafter(np.float32(2.0 ** -25), np.float32(1)),
                           2.0 ** -26, 2.0 ** -14, 1.0 / 127.0, 0.0, -0.0, np.inf, -np.inf],
                          dtype=np.float32))
    out = np.concatenate(cases)
    out = out[~np.isnan(out)]
    return np.concatenate([out, -out])


def test_float_to_half_matches_numpy(oracle):
    rng = np.random.default_rng(1234)
    xs = _float_cases(rng)
    with np.errstate(over="ignore"):
        ref = xs.astype(np.float16).view(np.uint16)
    got = np.array([oracle.float_to_half(float(x)) for x in xs], dtype=np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(float(xs[i]), hex(got[i]), hex(ref[i])) for i in bad[:10]]


# ---------------------------------------------------------------------------
# Packed bytes of special blocks, worked out by hand from the definition
# ---------------------------------------------------------------------------


def _q(oracle, qtype, block):
    return oracle.quantize(qtype, np.asarray(block, np.float32).reshape(1, 32)).tobytes()


def _hex(s):
    return bytes.fromhex(s.replace(" ", ""))


def test_golden_all_zero(oracle):
    z = np.zeros(32, np.float32)
    # Q8_0: amax = 0 -> d32 = +0 -> d16 = 0x0000; every code 0.
    assert _q(oracle, O.Q8_0, z) == _hex("0000" + "00" * 32)
    # Q4_0: signed max starts at +0.0 -> d32 = +0/-8 = -0.0 -> d16 = 0x8000 (stored 00 80);
    # d16 == 0 so every code is 0 -> nibble 8 -> bytes 0x88.
    assert _q(oracle, O.Q4_0, z) == _hex("0080" + "88" * 16)
    # negative zeros do not change the scan (|-0| > 0 is false)
    assert _q(oracle, O.Q4_0, -z) == _hex("0080" + "88" * 16)


def test_golden_spikes(oracle):
    e0 = np.zeros(32, np.float32)
    e0[0] = 1.0
    # Q8_0: d32 = fl32(1/127) = 0.0078740157..; binary16 spacing in [2^-7, 2^-6) is 2^-17,
    # (d32 - 2^-7) / 2^-17 = 8.06 -> fraction 8 -> d16 = 0x2008 = 0.00787353515625;
    # q0 = round(1 / 0.00787353515625) = round(127.0078) = 127 = 0x7F.
    assert _q(oracle, O.Q8_0, e0) == _hex("0820" + "7f" + "00" * 31)
    # Q4_0: m = +1 -> d = -0.125 = 0xB000; c0 = floor(-8 + 0.5) = -8 -> nibble 0;
    # zeros -> c = 0 -> nibble 8.  byte0 = nib0 | nib16 << 4 = 0x80, the rest 0x88.
    assert _q(oracle, O.Q4_0, e0) == _hex("00b0" + "80" + "88" * 15)

    e17 = np.zeros(32, np.float32)
    e17[17] = 1.0
    assert _q(oracle, O.Q8_0, e17) == _hex("0820" + "00" * 17 + "7f" + "00" * 14)
    # element 17 is the high nibble of byte 1: byte1 = nib1 | nib17 << 4 = 0x08
    assert _q(oracle, O.Q4_0, e17) == _hex("00b0" + "88" + "08" + "88" * 14)

    # Q8_0: -1 -> same scale, q = -127 = 0x81.  Q4_0: m = -1 -> d = +0.125 = 0x3000,
    # c = floor(-1/0.125 + 0.5) = -8 -> nibble 0 again.
    assert _q(oracle, O.Q8_0, -e0) == _hex("0820" + "81" + "00" * 31)
    assert _q(oracle, O.Q4_0, -e0) == _hex("0030" + "80" + "88" * 15)


def test_golden_ties_and_saturation(oracle):
    # Q8_0 with amax = 127 * 2^-7 gives d32 = 2^-7 exactly, d16 = 0x2000.
    b = np.zeros(32, np.float32)
    b[0] = 127 * 2.0 ** -7
    b[1] = 2.5 * 2.0 ** -7       # exact tie 2.5 -> 3 (half away from zero)
    b[2] = -2.5 * 2.0 ** -7      # -2.5 -> -3
    b[3] = 0.5 * 2.0 ** -7       # 0.5 -> 1
    b[4] = -0.5 * 2.0 ** -7      # -0.5 -> -1
    got = _q(oracle, O.Q8_0, b)
    assert got[:2] == _hex("0020")
    assert list(np.frombuffer(got[2:7], np.int8)) == [127, 3, -3, 1, -1]

    # Q4_0 with m = -1 -> d = 0.125 (0x3000).  x/d: 2.5 -> floor(3.0) = 3,
    # -2.5 -> floor(-2.0) = -2 (half up), 0.99/0.125 = 7.92 -> 8 -> saturates to 7.
    c = np.zeros(32, np.float32)
    c[0] = -1.0
    c[1] = 0.3125
    c[2] = -0.3125
    c[3] = np.float32(0.99)
    c[4] = 0.0625                 # 0.5 -> floor(1.0) = 1
    c[5] = -0.0625                # -0.5 -> floor(0.0) = 0
    got = _q(oracle, O.Q4_0, c)
    assert got[:2] == _hex("0030")
    nib = [(got[2 + (j % 16)] >> (4 * (j // 16))) & 0xF for j in range(32)]
    assert [n - 8 for n in nib[:6]] == [-8, 3, -2, 7, 1, 0]


def test_golden_q4_max_magnitude_tie_first_index_wins(oracle):
    b = np.zeros(32, np.float32)
    b[0], b[5] = 1.0, -1.0
    got = _q(oracle, O.Q4_0, b)
    assert got[:2] == _hex("00b0")   # m = +1 (first) -> d = -0.125
    b[0], b[5] = -1.0, 1.0
    got = _q(oracle, O.Q4_0, b)
    assert got[:2] == _hex("0030")   # m = -1 (first) -> d = +0.125
    # the +1 then sits at x/d = 8 -> floor(8.5) = 8 -> saturates to code 7 (nibble 15)
    assert (got[2 + 5] & 0xF) == 15


# ---------------------------------------------------------------------------
# Scales, codes and round trip against independent recomputation
# ---------------------------------------------------------------------------


def _adversarial_blocks(rng):
    blocks = []
    blocks.append(rng.standard_normal(32).astype(np.float32) * np.float32(0.02))
    blocks.append(rng.standard_normal(32).astype(np.float32))
    blocks.append(rng.standard_normal(32).astype(np.float32) * np.float32(1e-6))   # tiny -> d16 underflow
    blocks.append(rng.standard_normal(32).astype(np.float32) * np.float32(2e-5))   # subnormal d16
    blocks.append(rng.standard_normal(32).astype(np.float32) * np.float32(1000.0))
    x = np.zeros(32, np.float32)
    x[7] = -3.0
    blocks.append(x)
    x = np.full(32, 0.25, np.float32)
    blocks.append(x)
    x = np.full(32, -0.25, np.float32)
    blocks.append(x)
    # ties against a power-of-two scale
    x = (np.arange(32, dtype=np.float32) - 16) * np.float32(0.5) * np.float32(2.0 ** -7)
    x[0] = 127 * 2.0 ** -7
    blocks.append(x.astype(np.float32))
    x = (np.arange(32, dtype=np.float32) - 16) * np.float32(0.0625)
    x[31] = -1.0
    blocks.append(x.astype(np.float32))
    # max-magnitude tie in both signs
    x = rng.standard_normal(32).astype(np.float32) * np.float32(0.1)
    x[3], x[20] = 0.5, -0.5
    blocks.append(x)
    return np.stack(blocks)


def _expected_scale(qtype, blk):
    a = np.abs(blk.astype(np.float32))
    if qtype == O.Q8_0:
        d32 = np.float32(a.max()) / np.float32(127.0)
    else:
        m = np.float32(0.0) if a.max() == 0 else blk[int(np.argmax(a))]  # argmax = first index
        d32 = np.float32(m) / np.float32(-8.0)
    return np.array([d32], np.float32).astype(np.float16).view(np.uint16)[0]


def _brute_force_code(qtype, x, d16bits):
    d = Fraction(float(np.uint16(d16bits).view(np.float16)))
    if d == 0:
        return 0
    lo, hi = (-127, 127) if qtype == O.Q8_0 else (-8, 7)
    xf = Fraction(float(x))
    best, best_c = None, None
    for c in range(lo, hi + 1):
        dist = abs(xf - c * d)
        if best is None or dist < best:
            best, best_c = dist, c
        elif dist == best:
            # tie: Q8_0 takes the code farther from zero, Q4_0 the larger code
            if qtype == O.Q8_0:
                if abs(c) > abs(best_c):
                    best_c = c
            else:
                best_c = max(best_c, c)
    return best_c


def _decode_codes(qtype, blocks_bytes):
    nb = blocks_bytes.shape[0]
    if qtype == O.Q8_0:
        return blocks_bytes[:, 2:].view(np.int8).astype(np.int64)
    qs = blocks_bytes[:, 2:].astype(np.int64)
    codes = np.empty((nb, 32), np.int64)
    codes[:, :16] = (qs & 0xF) - 8
    codes[:, 16:] = (qs >> 4) - 8
    return codes


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
def test_codes_brute_force(oracle, qtype):
    rng = np.random.default_rng(7)
    blocks = np.concatenate([_adversarial_blocks(rng),
                             rng.standard_normal((16, 32)).astype(np.float32) * np.float32(0.02)])
    q = oracle.quantize(qtype, blocks)  # one row per block (k = 32)
    q = q.reshape(blocks.shape[0], -1)
    codes = _decode_codes(qtype, q)
    for i, blk in enumerate(blocks):
        d16 = int(q[i, 0]) | (int(q[i, 1]) << 8)
        assert d16 == int(_expected_scale(qtype, blk)), (i, hex(d16))
        for j in range(32):
            assert codes[i, j] == _brute_force_code(qtype, blk[j], d16), (i, j, blk[j])


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
def test_round_trip_bound(oracle, qtype):
    rng = np.random.default_rng(11)
    w = (rng.standard_normal((256, 4096)) * 0.02).astype(np.float32)
    q = oracle.quantize(qtype, w)
    what = oracle.dequant(qtype, q, 256, 4096)
    d = q[:, :, :2].copy().view(np.uint16)[..., 0].view(np.float16).astype(np.float64)
    dd = np.repeat(np.abs(d), 32, axis=1)
    err = np.abs(w.astype(np.float64) - what)
    codes = _decode_codes(qtype, q.reshape(-1, q.shape[-1])).reshape(256, 4096)
    if qtype == O.Q8_0:
        assert np.all(err <= dd / 2)
    else:
        sat = (codes == 7) & (w.astype(np.float64) / np.where(dd > 0, np.repeat(d, 32, axis=1), 1) >= 7.5)
        assert np.all(err[~sat] <= dd[~sat] / 2)
        assert np.all(err[sat] <= dd[sat] * (1 + 2.0 ** -7))
        assert sat.mean() < 0.02
    # dequantized values are code * d16 exactly
    assert np.array_equal(what, codes * np.repeat(d, 32, axis=1))


# ---------------------------------------------------------------------------
# The binary64 linear layer
# ---------------------------------------------------------------------------


def _xbits(rng, m, k, dtype):
    x = rng.standard_normal((m, k)).astype(np.float32)
    if dtype == O.X_F16:
        return x.astype(np.float16).view(np.uint16)
    # bfloat16, ties-to-even, written as integer arithmetic on the binary32 bits
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _decode_x(bits, dtype):
    if dtype == O.X_F16:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
@pytest.mark.parametrize("xdt", [O.X_F16, O.X_BF16])
def test_qlinear_exact_rational_k32(oracle, qtype, xdt):
    """4 x 32 x 4 cases: binary64 sums against exact rational sums."""
    rng = np.random.default_rng(3 + qtype * 10 + xdt)
    for trial in range(6):
        w = (rng.standard_normal((4, 32)) * 0.02).astype(np.float32)
        xb = _xbits(rng, 4, 32, xdt)
        q = oracle.quantize(qtype, w)
        y, bound = oracle.qlinear(qtype, q, 4, 32, xb, xdt)
        what = oracle.dequant(qtype, q, 4, 32)
        xv = _decode_x(xb, xdt)
        for i in range(4):
            for n in range(4):
                exact = sum(Fraction(float(xv[i, k])) * Fraction(float(what[n, k])) for k in range(32))
                bexact = sum(abs(Fraction(float(xv[i, k])) * Fraction(float(what[n, k]))) for k in range(32))
                tol = 32 * 2.0 ** -53 * float(bexact)
                assert abs(Fraction(y[i, n]) - exact) <= Fraction(tol)
                assert abs(Fraction(bound[i, n]) - bexact) <= Fraction(tol)


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
def test_qlinear_vs_numpy_blas(oracle, qtype):
    rng = np.random.default_rng(5)
    n, k, m = 96, 352, 7  # 11 blocks per row
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    xb = _xbits(rng, m, k, O.X_F16)
    q = oracle.quantize(qtype, w)
    y, bound = oracle.qlinear(qtype, q, n, k, xb, O.X_F16)
    what = oracle.dequant(qtype, q, n, k)
    xv = _decode_x(xb, O.X_F16)
    ref = xv @ what.T
    assert np.all(np.abs(y - ref) <= 1e-12 * bound + 1e-300)
    assert np.allclose(bound, np.abs(xv) @ np.abs(what).T, rtol=1e-12, atol=0)


def test_qlinear_column_subset_and_threads_agree(oracle):
    rng = np.random.default_rng(9)
    n, k, m = 64, 256, 3
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    xb = _xbits(rng, m, k, O.X_BF16)
    q = oracle.quantize(O.Q4_0, w)
    y1, b1 = oracle.qlinear(O.Q4_0, q, n, k, xb, O.X_BF16, nthreads=1)
    y4, b4 = oracle.qlinear(O.Q4_0, q, n, k, xb, O.X_BF16, nthreads=4)
    cols = np.array([63, 0, 17, 17])
    ys, bs = oracle.qlinear(O.Q4_0, q, n, k, xb, O.X_BF16, cols=cols, nthreads=2)
    assert np.array_equal(y1, y4) and np.array_equal(b1, b4)
    assert np.array_equal(ys, y1[:, cols]) and np.array_equal(bs, b1[:, cols])


def test_qlinear_onehot_reads_out_weights(oracle):
    """x = e_k gives y[:, n] = w_hat[n, k] exactly (closed form)."""
    rng = np.random.default_rng(13)
    n, k = 8, 64
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    for qtype in (O.Q8_0, O.Q4_0):
        q = oracle.quantize(qtype, w)
        what = oracle.dequant(qtype, q, n, k)
        xb = np.zeros((k, k), np.uint16)
        xb[np.arange(k), np.arange(k)] = 0x3C00  # binary16 1.0
        y, _ = oracle.qlinear(qtype, q, n, k, xb, O.X_F16)
        assert np.array_equal(y, what.T)


@pytest.mark.parametrize("qtype", [O.Q8_0, O.Q4_0])
def test_qlinear_constant_blocks_closed_form(oracle, qtype):
    """Blocks holding one value c each: every Q8_0 code is 127 sign(c) with
    d16 = binary16(|c| / 127), every Q4_0 code -8 with d16 = binary16(c / -8)
    (the extreme element maps to -8), so y = sum_b coef_b * sum_{j in b} x_j
    with coef_b = 127 sign(c) d16 or -8 d16 (closed form; the binary16
    roundings come from numpy)."""
    rng = np.random.default_rng(29)
    n, k = 6, 256
    nb = k // 32
    c = (rng.uniform(0.005, 0.08, (n, nb)) * rng.choice([-1.0, 1.0], (n, nb))).astype(np.float32)
    w = np.repeat(c, 32, axis=1)
    q = oracle.quantize(qtype, w)
    if qtype == O.Q8_0:
        d16 = (np.abs(c) / np.float32(127)).astype(np.float16).astype(np.float64)
        coef = 127.0 * np.sign(c) * d16
    else:
        d16 = (c / np.float32(-8)).astype(np.float16).astype(np.float64)
        coef = -8.0 * d16
    x = rng.standard_normal((5, k)).astype(np.float16)
    xs = x.astype(np.float64).reshape(5, nb, 32).sum(axis=2)
    y, bound = oracle.qlinear(qtype, q, n, k, x.view(np.uint16), O.X_F16)
    ref = xs @ coef.T
    assert np.allclose(y, ref, rtol=0, atol=1e-12 * np.abs(bound).max())
    assert np.allclose(bound, np.abs(x.astype(np.float64)).reshape(5, nb, 32).sum(axis=2) @ np.abs(coef).T,
                       rtol=1e-13, atol=0)


def test_oracle_rejects_bad_arguments(oracle):
    with pytest.raises(ValueError):
        oracle.quantize(O.Q8_0, np.zeros((2, 33), np.float32))
    with pytest.raises(ValueError):
        oracle.quantize(3, np.zeros((2, 32), np.float32))
