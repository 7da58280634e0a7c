"""Hash of the sources a kernel family is built from (used to tell whether
recorded profiler counters still describe the current kernels)."""
import hashlib
import os

_CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
_FILES = {
    "gemv": ("gemv.hip", "epilogue.h", "eb_internal.h", "eb_api.cpp"),
    "mfma": ("mfma.hip", "mfma_multi.hip", "mfma_lds2.hip", "mfma_common.h", "mm_common.h", "norm.hip",
             "epilogue.h",
             "eb_internal.h", "eb_api.cpp"),
}


def kernel_sources_sha(path: str) -> str:
    h = hashlib.sha256()
    for f in _FILES[path]:
        with open(os.path.join(_CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]
