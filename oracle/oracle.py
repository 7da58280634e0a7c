"""ctypes binding of the CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY.  The product library never imports this module;
only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` do.  It shares no code with the HIP path: it builds and loads its
own shared object from ``oracle.c`` with gcc.

Every function follows the definition in the header of ``oracle.c``: the
Q8_0 / Q4_0 block formats (32 weights per block along k, one binary16 scale)
and the Q6_S super-block format (256 weights, 16 int8 sub-block scales under
one binary16 scale, 6-bit codes) that realise the paper's 8-, 4- and 6-bit
configurations (section 4, Table 3),
and the binary64 linear layer y = x . w_hat^T, plus the decoder-layer steps
fused around it (section 3.2, operator fusion): RMS normalisation before a
projection, the SiLU-gated product of a gate/up pair and the residual addition
after one (``fused_qlinear``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

Q8_0 = 1
Q4_0 = 2
Q6_S = 3
X_F16 = 1
X_BF16 = 2
QK = 32
BLOCK_ELEMS = {Q8_0: 32, Q4_0: 32, Q6_S: 256}

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-std=c99", "-D_GNU_SOURCE",
           "-shared", "-fPIC", "-pthread"]


def build(force: bool = False, out: str | None = None, extra: list[str] | None = None) -> str:
    """Compile oracle.c with gcc (IEEE arithmetic: no fast-math, no FMA contraction)."""
    out = out or _LIB
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", *_CFLAGS, *(extra or []), _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


class Oracle:
    def __init__(self, path: str | None = None):
        self.lib = ctypes.CDLL(path or build())
        L = self.lib
        L.oracle_half_to_double.restype = ctypes.c_double
        L.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_double.restype = ctypes.c_double
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_float_to_half_rne.restype = ctypes.c_uint16
        L.oracle_float_to_half_rne.argtypes = [ctypes.c_float]
        L.oracle_block_bytes.restype = ctypes.c_int64
        L.oracle_block_bytes.argtypes = [ctypes.c_int]
        L.oracle_block_elems.restype = ctypes.c_int64
        L.oracle_block_elems.argtypes = [ctypes.c_int]
        L.oracle_quantize.restype = ctypes.c_int
        L.oracle_quantize.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_int]
        L.oracle_dequant.restype = ctypes.c_int
        L.oracle_dequant.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_int64, ctypes.c_void_p]
        L.oracle_qlinear.restype = ctypes.c_int
        L.oracle_qlinear.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                     ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        L.oracle_round_x16.restype = ctypes.c_int
        L.oracle_round_x16.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_void_p]
        L.oracle_rmsnorm.restype = ctypes.c_int
        L.oracle_rmsnorm.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double,
                                     ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        L.oracle_quantize_x8.restype = ctypes.c_int
        L.oracle_quantize_x8.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        L.oracle_qlinear_x8.restype = ctypes.c_int
        L.oracle_qlinear_x8.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.oracle_silu_mul.restype = ctypes.c_int
        L.oracle_silu_mul.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_void_p]

    # -- scalar format helpers ------------------------------------------------
    def half_to_double(self, h: int) -> float:
        return self.lib.oracle_half_to_double(int(h) & 0xFFFF)

    def bf16_to_double(self, b: int) -> float:
        return self.lib.oracle_bf16_to_double(int(b) & 0xFFFF)

    def float_to_half(self, f: float) -> int:
        return int(self.lib.oracle_float_to_half_rne(float(np.float32(f))))

    def block_bytes(self, qtype: int) -> int:
        return int(self.lib.oracle_block_bytes(qtype))

    # -- quantize / dequantize -----------------------------------------------
    def quantize(self, qtype: int, w: np.ndarray, nthreads: int = 1) -> np.ndarray:
        """fp32 W[n, k] -> canonical blocks, uint8 [n, k/E, block_bytes], E =
        BLOCK_ELEMS[qtype] weights per block."""
        w = np.ascontiguousarray(w, dtype=np.float32)
        n, k = w.shape
        bb = self.block_bytes(qtype)
        out = np.zeros((n, k // BLOCK_ELEMS[qtype], bb), dtype=np.uint8)
        rc = self.lib.oracle_quantize(qtype, w.ctypes.data, n, k, out.ctypes.data, int(nthreads))
        if rc != 0:
            raise ValueError("oracle_quantize rejected the arguments")
        return out

    def dequant(self, qtype: int, blocks: np.ndarray, n: int, k: int) -> np.ndarray:
        blocks = np.ascontiguousarray(blocks, dtype=np.uint8)
        assert blocks.size == n * (k // BLOCK_ELEMS[qtype]) * self.block_bytes(qtype)
        out = np.empty((n, k), dtype=np.float64)
        rc = self.lib.oracle_dequant(qtype, blocks.ctypes.data, n, k, out.ctypes.data)
        if rc != 0:
            raise ValueError("oracle_dequant rejected the arguments")
        return out

    def qlinear(self, qtype: int, blocks: np.ndarray, n: int, k: int, x_bits: np.ndarray,
                xdtype: int, cols=None, nthreads: int = 1):
        """x_bits: uint16 [m, k] raw binary16/bfloat16 words.

        Returns (y, bound), float64 [m, len(cols)] (all n columns when cols is None).
        """
        blocks = np.ascontiguousarray(blocks, dtype=np.uint8)
        assert blocks.size == n * (k // BLOCK_ELEMS[qtype]) * self.block_bytes(qtype)
        x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
        if x_bits.ndim == 1:
            x_bits = x_bits.reshape(1, -1)
        m = x_bits.shape[0]
        assert x_bits.shape[1] == k
        cols = np.arange(n, dtype=np.int64) if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
        y = np.zeros((m, cols.size), dtype=np.float64)
        bound = np.zeros((m, cols.size), dtype=np.float64)
        rc = self.lib.oracle_qlinear(qtype, blocks.ctypes.data, n, k, x_bits.ctypes.data, xdtype,
                                     m, cols.ctypes.data, cols.size, y.ctypes.data,
                                     bound.ctypes.data, int(nthreads))
        if rc != 0:
            raise ValueError("oracle_qlinear rejected the arguments")
        return y, bound


    # -- low-precision prefill variant: int8 activation blocks --------------
    def quantize_x8(self, x_bits: np.ndarray, xdtype: int):
        """uint16 [m, k] activation words -> (int8 codes [m, k], binary32 scales [m, k/32])."""
        x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
        if x_bits.ndim == 1:
            x_bits = x_bits.reshape(1, -1)
        m, k = x_bits.shape
        xq = np.zeros((m, k), dtype=np.int8)
        s = np.zeros((m, k // QK), dtype=np.float32)
        if self.lib.oracle_quantize_x8(x_bits.ctypes.data, xdtype, m, k, xq.ctypes.data,
                                       s.ctypes.data) != 0:
            raise ValueError("oracle_quantize_x8 rejected the arguments")
        return xq, s

    def qlinear_x8(self, qtype: int, blocks: np.ndarray, n: int, k: int, xq: np.ndarray,
                   s: np.ndarray, cols=None):
        """The int8-activation product.  Returns (y, bound, qerr), float64
        [m, len(cols)]: y = sum_b s d (integer block dot), bound = sum |x~||w_hat|
        with x~ = s xq, qerr = the activation-quantization error bound."""
        blocks = np.ascontiguousarray(blocks, dtype=np.uint8)
        assert blocks.size == n * (k // QK) * self.block_bytes(qtype)
        xq = np.ascontiguousarray(xq, dtype=np.int8)
        s = np.ascontiguousarray(s, dtype=np.float32)
        m = xq.shape[0]
        assert xq.shape == (m, k) and s.shape == (m, k // QK)
        cols = np.arange(n, dtype=np.int64) if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
        y = np.zeros((m, cols.size)); bound = np.zeros((m, cols.size)); qerr = np.zeros((m, cols.size))
        if self.lib.oracle_qlinear_x8(qtype, blocks.ctypes.data, n, k, xq.ctypes.data, s.ctypes.data,
                                      m, cols.ctypes.data, cols.size, y.ctypes.data,
                                      bound.ctypes.data, qerr.ctypes.data) != 0:
            raise ValueError("oracle_qlinear_x8 rejected the arguments")
        return y, bound, qerr

    # -- the steps around the linear layer in a decoder layer ---------------
    def round_x16(self, v: np.ndarray, xdtype: int) -> np.ndarray:
        """Nearest binary16 (X_F16) or bfloat16 (X_BF16) words to float64 values, ties to even."""
        v = np.ascontiguousarray(v, dtype=np.float64)
        out = np.empty(v.shape, dtype=np.uint16)
        if self.lib.oracle_round_x16(v.ctypes.data, v.size, xdtype, out.ctypes.data) != 0:
            raise ValueError("oracle_round_x16 rejected the arguments")
        return out

    def rmsnorm(self, h: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
        """float64 h[i][j] * gamma[j] / sqrt(eps + mean_j h[i][j]^2) for binary32 h [m, k]."""
        h = np.ascontiguousarray(h, dtype=np.float32)
        if h.ndim == 1:
            h = h.reshape(1, -1)
        gamma = np.ascontiguousarray(gamma, dtype=np.float32)
        m, k = h.shape
        assert gamma.shape == (k,)
        out = np.empty((m, k), dtype=np.float64)
        if self.lib.oracle_rmsnorm(h.ctypes.data, gamma.ctypes.data, float(eps), m, k,
                                   out.ctypes.data) != 0:
            raise ValueError("oracle_rmsnorm rejected the arguments")
        return out

    def silu_mul(self, g: np.ndarray, u: np.ndarray) -> np.ndarray:
        """float64 silu(g) * u, silu(t) = t / (1 + exp(-t))."""
        g = np.ascontiguousarray(g, dtype=np.float64)
        u = np.ascontiguousarray(u, dtype=np.float64)
        assert g.shape == u.shape
        out = np.empty(g.shape, dtype=np.float64)
        if self.lib.oracle_silu_mul(g.ctypes.data, u.ctypes.data, g.size, out.ctypes.data) != 0:
            raise ValueError("oracle_silu_mul rejected the arguments")
        return out

    def fused_qlinear(self, qtype: int, blocks: np.ndarray, n: int, k: int, x, xdtype: int,
                      prologue: str = "none", gamma=None, eps: float = 0.0,
                      epilogue: str = "none", residual=None, rows=None, nthreads: int = 1):
        """One projection of a decoder layer with its neighbouring steps.

        prologue "none": x is uint16 [m, k] raw activation words of xdtype.
        prologue "rmsnorm": x is binary32 h [m, k]; the product takes
            round_x16(rmsnorm(h, gamma, eps)), the normalised activations in
            the activation type the linear layer consumes.
        epilogue "none": y = x . w_hat^T; "add": y + residual (float64 [m, n]);
        "glu": rows 2j and 2j + 1 of W are the gate and up rows of feature j,
            y[:, j] = silu(gate) * up, shape [m, n / 2].
        rows: which rows of x (the others are not computed).

        Returns (y, scale, x_words): the error of an fp32-accumulating
        implementation is measured against scale (|x||w_hat| summed over k for
        "none" and "add"; for "glu", with Bg, Bu those sums of the gate and up
        outputs g, u: 1.1 Bg |u| + |silu(g)| Bu + 0.0022 Bg Bu, the first-order
        propagation of errors tau Bg, tau Bu through silu (|silu'| < 1.1) and
        the product, plus their product term for tau <= 2e-3).
        """
        if prologue == "rmsnorm":
            h = np.asarray(x, dtype=np.float32)
            h = h if rows is None else h[rows]
            xw = self.round_x16(self.rmsnorm(h, gamma, eps), xdtype)
        elif prologue == "none":
            xw = np.asarray(x, dtype=np.uint16)
            xw = xw if rows is None else xw[rows]
        else:
            raise ValueError(prologue)
        y, bound = self.qlinear(qtype, blocks, n, k, xw, xdtype, nthreads=nthreads)
        if epilogue == "none":
            return y, bound, xw
        if epilogue == "add":
            r = np.asarray(residual, dtype=np.float64)
            r = r if rows is None else r[rows]
            return y + r, bound, xw
        if epilogue == "glu":
            assert n % 2 == 0
            g, u = y[:, 0::2], y[:, 1::2]
            bg, bu = bound[:, 0::2], bound[:, 1::2]
            s = self.silu_mul(g, u)
            silu = self.silu_mul(g, np.ones_like(g))
            scale = 1.1 * bg * np.abs(u) + np.abs(silu) * bu + 0.0022 * bg * bu
            return s, scale, xw
        raise ValueError(epilogue)


_ORACLE = None


def get() -> Oracle:
    global _ORACLE
    if _ORACLE is None:
        _ORACLE = Oracle()
    return _ORACLE


def available_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1
