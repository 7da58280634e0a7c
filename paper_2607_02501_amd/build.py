"""Build libeb.so (HIP kernels for gfx950 + the C ABI) in-tree with hipcc.

    python -m paper_2607_02501_amd.build      # or build() from Python

Every HIP source is compiled with packed-fp32 instructions disabled and with
IEEE-exact fp32 division / denormals; quantize.hip also without FMA
contraction, so that packing is bit-exact with the format definition.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libeb.so")

ARCH = "gfx950"
SOURCES = ["eb_api.cpp", "eb_multirate.cpp", "quantize.hip", "gemv.hip", "norm.hip", "mfma.hip", "mfma_q8_0_bf16.hip",
           "mfma_q8_0_f16.hip", "mfma_q4_0_bf16.hip", "mfma_q4_0_f16.hip", "mfma_q6_s_bf16.hip", "mfma_q6_s_f16.hip", "mfma_multi.hip",
           "mfma_lds2.hip", "mfma_narrow.hip", "mfma_q6.hip", "gemv_q6.hip", "mfma_i8.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
          "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas"]
PER_FILE = {"quantize.hip": ["-ffp-contract=off"],
            # keep MFMA accumulators in VGPRs in the fused persistent kernel
            "mfma_multi.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the HIP toolchain is required to build libeb.so")


def _compile(src: str, obj: str) -> None:
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = [hipcc(), *COMMON, *PER_FILE.get(os.path.basename(src), []), *lang, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link paper_2607_02501_amd/libeb.so."""
    with tempfile.TemporaryDirectory(prefix="eb_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", "8")))
        with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
            list(ex.map(lambda so: _compile(os.path.join(CSRC, so[0]), so[1]), zip(SOURCES, objs)))
        out = LIB + ".tmp%d" % os.getpid()
        cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        os.replace(out, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    try:
        build(verbose=True)
    except RuntimeError as e:
        print(e, file=sys.stderr)
        sys.exit(1)
    sys.exit(0)
