"""ctypes binding of the CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY.  The product library never imports this module;
only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` do.  It shares no code with the HIP path: it builds and loads its
own shared object from ``oracle.c`` with gcc.

Every function follows the definition in the header of ``oracle.c``: the
Q8_0 / Q4_0 block formats (32 weights per block along k, one binary16 scale)
that realise the paper's 8-bit and 4-bit configurations (section 4, Table 3),
and the binary64 linear layer y = x . w_hat^T.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

Q8_0 = 1
Q4_0 = 2
X_F16 = 1
X_BF16 = 2
QK = 32

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
        """fp32 W[n, k] -> canonical blocks, uint8 [n, k/32, block_bytes]."""
        w = np.ascontiguousarray(w, dtype=np.float32)
        n, k = w.shape
        bb = self.block_bytes(qtype)
        out = np.zeros((n, k // QK, bb), dtype=np.uint8)
        rc = self.lib.oracle_quantize(qtype, w.ctypes.data, n, k, out.ctypes.data, int(nthreads))
        if rc != 0:
            raise ValueError("oracle_quantize rejected the arguments")
        return out

    def dequant(self, qtype: int, blocks: np.ndarray, n: int, k: int) -> np.ndarray:
        blocks = np.ascontiguousarray(blocks, dtype=np.uint8)
        assert blocks.size == n * (k // QK) * self.block_bytes(qtype)
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
        assert blocks.size == n * (k // QK) * self.block_bytes(qtype)
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
