"""Hash of the sources a kernel family is built from (used to tell whether
recorded profiler counters still describe the current kernels)."""
import hashlib
import os

_CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
_COMMON = ("epilogue.h", "eb_internal.h", "eb_api.cpp")
_FILES = {
    # GEMV kernels (m <= 8)
    "gemv": ("gemv.hip", "gemv_common.h") + _COMMON,
    # tile kernel of the MFMA path (single ops, split-K, grouped launches)
    "mfma": ("mfma.hip", "mfma_tile.h", "mfma_narrow.hip", "mfma_q8_0_bf16.hip", "mfma_q8_0_f16.hip",
             "mfma_q4_0_bf16.hip", "mfma_q4_0_f16.hip", "mfma_q6_s_bf16.hip", "mfma_q6_s_f16.hip",
             "mfma_common.h", "norm.hip") + _COMMON,
    # fused small-m MFMA kernels (m <= 128)
    "mm": ("mfma_lds2.hip", "mfma_multi.hip", "mfma_common.h", "mm_common.h", "norm.hip") + _COMMON,
    # the Q6_S kernel (every m)
    "q6": ("mfma_q6.hip", "mfma_common.h", "norm.hip") + _COMMON,
    "gemv_q6": ("gemv_q6.hip", "gemv_common.h") + _COMMON,
    "i8": ("mfma_i8.hip", "mfma_common.h") + _COMMON,
}


def family(symbol: str) -> str:
    """Kernel family of a kernel symbol (as the profiler names it)."""
    if symbol.startswith("gemv_q6"):
        return "gemv_q6"
    if symbol.startswith("gemv"):
        return "gemv"
    if symbol.startswith("mm_i8") or symbol.startswith("quantize_x8"):
        return "i8"
    if symbol.startswith("mm_q6"):
        return "q6"
    if symbol.startswith("mm_narrow"):
        return "mfma"
    if symbol.startswith("mm_"):
        return "mm"
    return "mfma"


def kernel_sources_sha(fam: str) -> str:
    h = hashlib.sha256()
    for f in _FILES[fam]:
        with open(os.path.join(_CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]
