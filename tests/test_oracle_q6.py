"""Pins of the oracle's Q6_S super-block format (runs without a GPU).

The paper evaluates a 6-bit configuration beside the 8- and 4-bit ones
(section 4, Table 3) but names no format; Q6_S is defined in oracle.c's
header: 256 weights in 16 sub-blocks of 16, a sub-block scale s_j = m_j / -32
from the sub-block's signed largest element, the 16 scales coded as int8
against one binary16 super-scale d16, and 6-bit codes against e_j = d16 * sc_j.

Each part is fixed by a route independent of oracle.c:
  * packed bytes of hand-built super-blocks -> worked out by hand from the
    definition (the derivation is in each test)
  * d16                                    -> numpy float32 / float16 arithmetic
  * sub-scales and codes                   -> brute-force argmin over every value,
    in exact rational arithmetic, with the tie rules
  * round trip                             -> |x - w_hat| <= |e_j| / 2 off the clamp
  * unpacking                              -> bit arithmetic written here
  * matmul                                 -> numpy float64 BLAS
"""
from fractions import Fraction

import numpy as np

from oracle import oracle as O


def _q6(oracle, x):
    x = np.asarray(x, np.float32).reshape(1, -1)
    return oracle.quantize(O.Q6_S, x).reshape(-1, 210)


def _hex(s):
    return bytes.fromhex(s.replace(" ", ""))


def _unpack(blocks):
    """(nb, 210) canonical super-blocks -> d16 bits (nb,), sc (nb, 16), u (nb, 256)."""
    blocks = np.asarray(blocks, np.uint8).reshape(-1, 210)
    d16 = blocks[:, 0].astype(np.uint16) | (blocks[:, 1].astype(np.uint16) << 8)
    sc = blocks[:, 2:18].view(np.int8).astype(np.int64)
    ch = blocks[:, 18:].reshape(-1, 8, 24).astype(np.int64)
    lo = np.concatenate([ch[:, :, :16] & 15, ch[:, :, :16] >> 4], axis=2)       # (nb, 8, 32)
    hb = ch[:, :, 16:]                                                            # (nb, 8, 8)
    hi = np.concatenate([(hb >> (2 * s)) & 3 for s in range(4)], axis=2)          # index 8 s + t
    u = (lo | (hi << 4)).reshape(-1, 256)
    return d16, sc, u


def test_q6_block_size(oracle):
    assert oracle.block_bytes(O.Q6_S) == 210        # 2 + 16 + 256 * 6 / 8
    assert O.BLOCK_ELEMS[O.Q6_S] == 256


def test_q6_golden_all_zero(oracle):
    # every m_j = +0 -> s_j = -0, amax = 0 -> d16 = 0x0000 -> sc_j = 0, e_j = 0,
    # codes 0 -> u = 32 (low nibble 0, high bits 2): low bytes 0x00, high bytes
    # 2 | 2 << 2 | 2 << 4 | 2 << 6 = 0xAA.
    expect = "0000" + "00" * 16 + ("00" * 16 + "aa" * 8) * 8
    assert _q6(oracle, np.zeros(256)).tobytes() == _hex(expect)


def test_q6_golden_one_hot(oracle):
    # x_0 = 1: m_0 = 1 -> s_0 = -1/32; amax = 2^-5 -> d32 = fl32(2^-5 / 127) =
    # 2.4606299e-4 in [2^-12, 2^-11), binary16 spacing 2^-22: 1032.06 spacings
    # -> d16 = 1032 * 2^-22 (exponent -12 -> biased 3, fraction 8) = 0x0C08.
    # sc_0 = round(-2^-5 / (1032 * 2^-22)) = round(-127.008) = -127 (0x81);
    # e_0 = -127 * 1032 * 2^-22; q_0 = floor(1 / e_0 + 1/2) = floor(-31.502) =
    # -32 -> u_0 = 0.  Every other code is 0 (u = 32).
    # chunk 0: low bytes all 0; high byte 0 = hi(u_0) | hi(u_8) << 2 | hi(u_16) << 4
    # | hi(u_24) << 6 = 0 | 8 | 32 | 128 = 0xA8, the rest 0xAA.
    x = np.zeros(256)
    x[0] = 1.0
    expect = "080c" + "81" + "00" * 15 + "00" * 16 + "a8" + "aa" * 7 + ("00" * 16 + "aa" * 8) * 7
    assert _q6(oracle, x).tobytes() == _hex(expect)


def test_q6_golden_ramp_subnormal_scale(oracle):
    # x_i = ((i mod 16) - 8) * 2^-6: every sub-block's largest is -8 * 2^-6
    # (index 0, first) -> s_j = 2^-8 for all j; d32 = fl32(2^-8 / 127) =
    # 3.0757874e-5, below 2^-14: binary16 subnormal spacing 2^-24 -> 516.03
    # -> d16 = 516 * 2^-24 (0x0204); sc_j = round(2^-8 / (516 * 2^-24)) =
    # round(127.008) = 127 (0x7F); e = 127 * 516 * 2^-24 = 65532 * 2^-24;
    # x_i / e = (i - 8) * 2^18 / 65532 = 4.000244 (i - 8) -> q = 4 (i - 8) for
    # every i (the excess is below 1/2), u = 4 (i mod 16).
    # chunk low byte i = lo(4 i) | lo(4 i) << 4 -> 00 44 88 cc repeated;
    # high byte t: hi(4 t) = t >> 2, hi(4 (t + 8)) = (t + 8) >> 2 ->
    # t < 4: 0 | 2 << 2 | 0 << 4 | 2 << 6 = 0x88; t >= 4: 1 | 3 << 2 | 1 << 4 | 3 << 6 = 0xDD.
    x = np.array([((i % 16) - 8) * 2.0 ** -6 for i in range(256)])
    chunk = "004488cc" * 4 + "88" * 4 + "dd" * 4
    assert _q6(oracle, x).tobytes() == _hex("0402" + "7f" * 16 + chunk * 8)


def test_q6_golden_ties_and_saturation(oracle):
    # d16 = 2^-10 (0x1400) from amax = 127 * 2^-10, i.e. m_0 = -127 * 2^-5.
    # sub-block 0: sc_0 = 127, e_0 = 127 * 2^-10; x_1 = 2.5 e_0 -> floor(3.0) = 3
    #   (u 35); x_2 = -2.5 e_0 -> floor(-2.0) = -2 (u 30); x_3 = 31.5 e_0 ->
    #   floor(32) = 32 -> clamped to 31 (u 63); x_0 -> -32 (u 0).
    # sub-block 1: m_1 = -2.5 * 2^-5 -> s_1 = 2.5 * 2^-10 -> sc_1 = round(2.5) = 3
    #   (half away from zero); e_1 = 3 * 2^-10; x_16 / e_1 = -26.67 -> -27 (u 5).
    # sub-block 2: m_2 = +2.5 * 2^-5 -> s_2 = -2.5 * 2^-10 -> sc_2 = -3 (0xFD);
    #   x_32 / e_2 = -26.67 -> -27 (u 5).
    # chunk 0 low bytes: lo(u_0) | lo(u_16) << 4 = 0 | 5 << 4 = 0x50; lo(35) = 3;
    #   lo(30) = 14; lo(63) = 15; high bytes: t=0: 0 | 2<<2 | hi(5)=0 | 2<<6 = 0x88;
    #   t=1: hi(35)=2 -> 0xAA; t=2: hi(30)=1 -> 0xA9; t=3: hi(63)=3 -> 0xAB; 0xAA.
    # chunk 1: low byte 0 = lo(5) = 0x05; high byte 0 = hi(5) = 0 -> 0xA8.
    x = np.zeros(256)
    e0 = 127 * 2.0 ** -10
    x[0] = -127 * 2.0 ** -5
    x[1], x[2], x[3] = 2.5 * e0, -2.5 * e0, 31.5 * e0
    x[16] = -2.5 * 2.0 ** -5
    x[32] = 2.5 * 2.0 ** -5
    chunk0 = "50030e0f" + "00" * 12 + "88aaa9ab" + "aa" * 4
    chunk1 = "05" + "00" * 15 + "a8" + "aa" * 7
    rest = ("00" * 16 + "aa" * 8) * 6
    expect = "0014" + "7f03fd" + "00" * 13 + chunk0 + chunk1 + rest
    assert _q6(oracle, x).tobytes() == _hex(expect)


# ---------------------------------------------------------------------------
# scales and codes against exact rational brute force
# ---------------------------------------------------------------------------


def _super_blocks(rng):
    out = [rng.standard_normal(256) * 0.02,
           rng.standard_normal(256),
           rng.standard_normal(256) * 1e-6,          # d16 subnormal
           rng.standard_normal(256) * 1e-9,          # d16 underflows to 0
           rng.standard_normal(256) * 300.0]
    x = rng.standard_normal(256) * 0.02
    x[16:32] = 0.0                                   # an all-zero sub-block
    x[40], x[45] = 0.3, -0.3                         # max-magnitude tie within a sub-block
    x[70] = 5.0                                      # one sub-block far larger than the rest
    out.append(x)
    x = rng.standard_normal(256) * 0.02
    x[::16] *= 40.0                                  # outliers at each sub-block's start
    out.append(x)
    x = np.repeat(rng.standard_normal(16), 16) * 0.05  # constant sub-blocks
    out.append(x)
    return np.stack(out).astype(np.float32)


def _expected_d16(blk):
    s = []
    for j in range(16):
        sub = blk[16 * j:16 * j + 16]
        a = np.abs(sub)
        m = np.float32(0.0) if a.max() == 0 else sub[int(np.argmax(a))]  # first index
        s.append(np.float32(m) / np.float32(-32.0))
    s = np.array(s, np.float32)
    amax = np.float32(np.abs(s).max())
    d32 = amax / np.float32(127.0)
    return s, int(np.array([d32], np.float32).astype(np.float16).view(np.uint16)[0])


def _argmin(target, step, lo, hi, tie_away_from_zero):
    if step == 0:
        return 0
    best, best_c = None, None
    for c in range(lo, hi + 1):
        dist = abs(target - c * step)
        if best is None or dist < best:
            best, best_c = dist, c
        elif dist == best:
            if tie_away_from_zero:
                if abs(c) > abs(best_c):
                    best_c = c
            else:
                best_c = max(best_c, c)   # half up
    return best_c


def test_q6_scales_and_codes_brute_force(oracle):
    rng = np.random.default_rng(61)
    blocks = _super_blocks(rng)
    q = oracle.quantize(O.Q6_S, blocks)          # one row per super-block (k = 256)
    d16, sc, u = _unpack(q)
    for b, blk in enumerate(blocks):
        s, d_expect = _expected_d16(blk)
        assert int(d16[b]) == d_expect, (b, hex(int(d16[b])), hex(d_expect))
        d = Fraction(float(np.uint16(d_expect).view(np.float16)))
        for j in range(16):
            sc_expect = _argmin(Fraction(float(s[j])), d, -127, 127, True)
            assert sc[b, j] == sc_expect, (b, j)
            e = d * sc_expect
            for i in range(16 * j, 16 * j + 16):
                q_expect = _argmin(Fraction(float(blk[i])), e, -32, 31, False)
                assert u[b, i] - 32 == q_expect, (b, i, float(blk[i]))


def test_q6_round_trip_and_dequant(oracle):
    rng = np.random.default_rng(62)
    n, k = 64, 2048
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    q = oracle.quantize(O.Q6_S, w)
    assert q.shape == (n, k // 256, 210)
    what = oracle.dequant(O.Q6_S, q, n, k)
    d16, sc, u = _unpack(q)
    d = d16.view(np.float16).astype(np.float64)                    # (n * k/256,)
    e = (d[:, None] * sc).reshape(n, k // 16)                      # per sub-block
    ee = np.repeat(e, 16, axis=1)
    codes = (u - 32).reshape(n, k)
    # dequantized values are code * d16 * sc exactly
    assert np.array_equal(what, codes * ee)
    err = np.abs(w.astype(np.float64) - what)
    clamped = (codes == -32) | (codes == 31)
    assert np.all(err[~clamped] <= np.abs(ee[~clamped]) / 2)
    # at the ends of the code range: |e_j - s_j| <= d16 / 2 (sc_j is the
    # nearest integer to s_j / d16), so the sub-block's largest element, at
    # -32 s_j, is off by at most 32 d16 / 2 beyond its own rounding; an element
    # of the other sign close to it in magnitude saturates at +31 (the code
    # range is asymmetric, as in Q4_0), off by at most |e_j| + 16 d16
    dd = np.repeat(d, 256).reshape(n, k)
    assert np.all(err[clamped] <= np.abs(ee[clamped]) + 16 * dd[clamped])
    sat = clamped & (err > np.abs(ee) / 2)
    assert sat.mean() < 0.005
    # 6.5625 bits per weight
    assert q.nbytes * 8 / (n * k) == 6.5625


def test_q6_qlinear_vs_numpy_blas(oracle):
    rng = np.random.default_rng(63)
    n, k, m = 40, 768, 5
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    x = rng.standard_normal((m, k)).astype(np.float32).astype(np.float16)
    q = oracle.quantize(O.Q6_S, w)
    y, bound = oracle.qlinear(O.Q6_S, q, n, k, x.view(np.uint16), O.X_F16)
    d16, sc, u = _unpack(q)
    d = d16.view(np.float16).astype(np.float64)
    what = ((u - 32) * np.repeat(d[:, None] * sc, 16, axis=1)).reshape(n, k)
    xv = x.astype(np.float64)
    assert np.all(np.abs(y - xv @ what.T) <= 1e-12 * bound + 1e-300)
    assert np.allclose(bound, np.abs(xv) @ np.abs(what).T, rtol=1e-12, atol=0)
