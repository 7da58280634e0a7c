"""Python binding of libeb (argument marshalling only).

Every computation runs in the HIP kernels of libeb.so; this module only
allocates outputs and workspaces with torch (the library allocates no device
memory), passes raw device pointers and the current HIP stream, and turns
status codes into exceptions.  It raises at import time if libeb.so has not
been built (there is no fallback path).

Names follow the C ABI in include/eb.h and include/eb_tuning.h.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeb.so")

EB_OK = 0
EB_ERR_INVALID = -1
EB_ERR_ALIGN = -2
EB_ERR_UNSUPPORTED = -3
EB_ERR_HIP = -4

EB_Q8_0 = 1
EB_Q4_0 = 2
EB_Q6_S = 3
EB_F32 = 0
EB_F16 = 1
EB_BF16 = 2
EB_PATH_AUTO = 0
EB_PATH_GEMV = 1
EB_PATH_MFMA = 2
EB_PATH_MFMA_I8 = 3
EB_PRO_NONE = 0
EB_PRO_RMSNORM = 1
EB_EPI_NONE = 0
EB_EPI_ADD = 1
EB_EPI_GLU = 2

QTYPES = {"q8_0": EB_Q8_0, "q4_0": EB_Q4_0, "q6_s": EB_Q6_S}
# weights and canonical bytes per block of each format
BLOCK_ELEMS = {"q8_0": 32, "q4_0": 32, "q6_s": 256}
BLOCK_BYTES = {"q8_0": 34, "q4_0": 18, "q6_s": 210}
DTYPES = {torch.float32: EB_F32, torch.float16: EB_F16, torch.bfloat16: EB_BF16}
PATHS = {"auto": EB_PATH_AUTO, "gemv": EB_PATH_GEMV, "mfma": EB_PATH_MFMA, "mfma_i8": EB_PATH_MFMA_I8}
PROLOGUES = {None: EB_PRO_NONE, "none": EB_PRO_NONE, "rmsnorm": EB_PRO_RMSNORM}
EPILOGUES = {None: EB_EPI_NONE, "none": EB_EPI_NONE, "add": EB_EPI_ADD, "glu": EB_EPI_GLU}


class eb_qweights(ctypes.Structure):
    _fields_ = [("type", ctypes.c_int32), ("reserved", ctypes.c_int32), ("n", ctypes.c_int64),
                ("k", ctypes.c_int64), ("data", ctypes.c_void_p)]


class eb_layout(ctypes.Structure):
    _fields_ = [("qs_offset", ctypes.c_int64), ("qs_row_bytes", ctypes.c_int64),
                ("d_offset", ctypes.c_int64), ("d_stride", ctypes.c_int64),
                ("total_bytes", ctypes.c_int64), ("canonical_bytes", ctypes.c_int64),
                ("sc_offset", ctypes.c_int64), ("sc_stride", ctypes.c_int64)]


class eb_qlinear_op(ctypes.Structure):
    _fields_ = [("w", eb_qweights), ("x", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("m", ctypes.c_int64), ("x_type", ctypes.c_int32), ("y_type", ctypes.c_int32),
                ("prologue", ctypes.c_int32), ("epilogue", ctypes.c_int32),
                ("norm_weight", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("norm_eps", ctypes.c_float), ("reserved", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"libeb.so not found at {LIB_PATH}: build it first "
                      "(python -m paper_2607_02501_amd.build); there is no fallback path")

lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
lib.eb_version.restype = ctypes.c_char_p
lib.eb_version.argtypes = []
lib.eb_status_str.restype = ctypes.c_char_p
lib.eb_status_str.argtypes = [_i32]
lib.eb_qweights_bytes.restype = ctypes.c_size_t
lib.eb_qweights_bytes.argtypes = [_i32, _i64, _i64]
lib.eb_qweights_layout.restype = _i32
lib.eb_qweights_layout.argtypes = [_i32, _i64, _i64, ctypes.POINTER(eb_layout)]
for _name in ("eb_quantize_q8_0", "eb_quantize_q4_0", "eb_quantize_q6_s"):
    getattr(lib, _name).restype = _i32
    getattr(lib, _name).argtypes = [_vp, _i64, _i64, _vp, _vp]
lib.eb_qweights_to_canonical.restype = _i32
lib.eb_qweights_to_canonical.argtypes = [ctypes.POINTER(eb_qweights), _vp, _vp]
lib.eb_qweights_from_canonical.restype = _i32
lib.eb_qweights_from_canonical.argtypes = [_i32, _vp, _i64, _i64, _vp, _vp]
lib.eb_qlinear.restype = _i32
lib.eb_qlinear.argtypes = [ctypes.POINTER(eb_qweights), _vp, _i32, _i64, _vp, _i32, _vp]
lib.eb_qlinear_ex.restype = _i32
lib.eb_qlinear_ex.argtypes = [ctypes.POINTER(eb_qweights), _vp, _i32, _i64, _vp, _i32, _i32, _vp]
lib.eb_qlinear_fused.restype = _i32
lib.eb_qlinear_fused.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32, _vp]
lib.eb_qlinear_auto_path.restype = _i32
lib.eb_qlinear_auto_path.argtypes = [_i32, _i32, _i64, _i64, _i64]
lib.eb_qlinear_stack.restype = _i32
lib.eb_qlinear_stack.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32, _vp, ctypes.c_size_t, _vp]
lib.eb_qlinear_stack_workspace_bytes.restype = ctypes.c_size_t
lib.eb_qlinear_stack_workspace_bytes.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32]
lib.eb_qlinear_workspace_bytes.restype = ctypes.c_size_t
lib.eb_qlinear_workspace_bytes.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32]
lib.eb_qlinear_fused_ws.restype = _i32
lib.eb_qlinear_fused_ws.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32, _vp, ctypes.c_size_t, _vp]
lib.eb_qlinear_fused_static.restype = _i32
lib.eb_qlinear_fused_static.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32, _vp]
lib.eb_qlinear_tuned.restype = _i32
lib.eb_qlinear_tuned.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32, _i32, _vp, ctypes.c_size_t, _vp]
lib.eb_qlinear_stack_launches.restype = _i32
lib.eb_qlinear_stack_launches.argtypes = [ctypes.POINTER(eb_qlinear_op), _i32]


class eb_module(ctypes.Structure):
    _fields_ = [("ops", ctypes.POINTER(eb_qlinear_op)), ("n_ops", _i32), ("period", _i32),
                ("phase", _i32), ("repeats", _i32)]


lib.eb_multirate_workspace_bytes.restype = ctypes.c_size_t
lib.eb_multirate_workspace_bytes.argtypes = [ctypes.POINTER(eb_module), _i32]
lib.eb_multirate_tick.restype = _i32
lib.eb_multirate_tick.argtypes = [ctypes.POINTER(eb_module), _i32, _i64, _vp, ctypes.c_size_t, _vp]
lib.eb_multirate_launches.restype = _i32
lib.eb_multirate_launches.argtypes = [ctypes.POINTER(eb_module), _i32, _i64]
lib.eb_stack_cache_clear.restype = _i32
lib.eb_stack_cache_clear.argtypes = []
lib.eb_mfma_tile_count.restype = _i32
lib.eb_mfma_tile_count.argtypes = []


class EBError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {lib.eb_status_str(status).decode()}")
        self.status = status


def _check(status: int, what: str) -> None:
    if status != EB_OK:
        raise EBError(status, what)


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def version() -> str:
    return lib.eb_version().decode()


def qweights_bytes(qtype: str, n: int, k: int) -> int:
    return int(lib.eb_qweights_bytes(QTYPES[qtype], n, k))


def layout(qtype: str, n: int, k: int) -> eb_layout:
    out = eb_layout()
    _check(lib.eb_qweights_layout(QTYPES[qtype], n, k, ctypes.byref(out)), "eb_qweights_layout")
    return out


class QWeights:
    """A quantized weight matrix W[n, k] held in a caller-owned device buffer."""

    def __init__(self, qtype: str, n: int, k: int, buf: torch.Tensor):
        assert buf.dtype == torch.uint8 and buf.is_cuda
        self.qtype, self.n, self.k, self.buf = qtype, n, k, buf

    @property
    def c(self) -> eb_qweights:
        return eb_qweights(QTYPES[self.qtype], 0, self.n, self.k, self.buf.data_ptr())

    @property
    def device(self):
        return self.buf.device

    def nbytes(self) -> int:
        return qweights_bytes(self.qtype, self.n, self.k)


def empty_qweights(qtype: str, n: int, k: int, device="cuda") -> QWeights:
    nbytes = qweights_bytes(qtype, n, k)
    if nbytes == 0:
        raise EBError(EB_ERR_INVALID, "eb_qweights_bytes")
    # torch's caching allocator returns 512-byte aligned blocks
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return QWeights(qtype, n, k, buf)


def quantize(w: torch.Tensor, qtype: str, out: QWeights | None = None) -> QWeights:
    """fp32 W[n, k] (device) -> QWeights in the planar layout."""
    assert w.dtype == torch.float32 and w.is_cuda and w.dim() == 2
    w = w.contiguous()
    n, k = w.shape
    out = out or empty_qweights(qtype, n, k, w.device)
    fn = {"q8_0": lib.eb_quantize_q8_0, "q4_0": lib.eb_quantize_q4_0,
          "q6_s": lib.eb_quantize_q6_s}[qtype]
    _check(fn(w.data_ptr(), n, k, out.buf.data_ptr(), _stream(w.device)), fn.__name__)
    return out


def to_canonical(qw: QWeights) -> torch.Tensor:
    """Canonical array-of-blocks bytes (device uint8 tensor [n, k/E, block_bytes],
    E = BLOCK_ELEMS[qtype])."""
    dst = torch.empty((qw.n, qw.k // BLOCK_ELEMS[qw.qtype], BLOCK_BYTES[qw.qtype]),
                      dtype=torch.uint8, device=qw.device)
    c = qw.c
    _check(lib.eb_qweights_to_canonical(ctypes.byref(c), dst.data_ptr(), _stream(qw.device)),
           "eb_qweights_to_canonical")
    return dst


def from_canonical(blocks: torch.Tensor, qtype: str, n: int, k: int) -> QWeights:
    assert blocks.dtype == torch.uint8 and blocks.is_cuda
    blocks = blocks.contiguous()
    out = empty_qweights(qtype, n, k, blocks.device)
    _check(lib.eb_qweights_from_canonical(QTYPES[qtype], blocks.data_ptr(), n, k,
                                          out.buf.data_ptr(), _stream(blocks.device)),
           "eb_qweights_from_canonical")
    return out


_SCRATCH = {}


def scratch(device, nbytes: int):
    """A caller-owned workspace of at least nbytes on `device` for direct calls
    on the current stream (one growing torch buffer per device and stream;
    calls on one stream run in order, so they may share it)."""
    if nbytes <= 0:
        return None
    device = torch.device(device)
    key = (device.index if device.index is not None else torch.cuda.current_device(),
           _stream(device))
    buf = _SCRATCH.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.empty(max(nbytes, 4 << 20), dtype=torch.uint8, device=device)
        _SCRATCH[key] = buf
    return buf


def _run_op(op: eb_qlinear_op, path: int, device, tile=None, splits=0) -> None:
    nbytes = int(lib.eb_qlinear_workspace_bytes(ctypes.byref(op), path if tile is None else EB_PATH_MFMA))
    if tile is not None:
        nbytes += 64 << 20  # room for any forced split (also where the automatic plan needs none)
    ws = scratch(device, nbytes)
    wp, wb = (ws.data_ptr(), ws.numel()) if ws is not None else (None, 0)
    if tile is None:
        _check(lib.eb_qlinear_fused_ws(ctypes.byref(op), path, wp, wb, _stream(device)),
               "eb_qlinear_fused_ws")
    else:
        _check(lib.eb_qlinear_tuned(ctypes.byref(op), tile, splits, wp, wb, _stream(device)),
               "eb_qlinear_tuned")


def qlinear(qw: QWeights, x: torch.Tensor, out_dtype=torch.float32, path: str = "auto",
            out: torch.Tensor | None = None) -> torch.Tensor:
    """y[m, n] = x[m, k] . w_hat^T on the GPU (fp32 accumulation), with a
    workspace from scratch() so that the MFMA path may split k."""
    assert x.is_cuda and x.dim() == 2 and x.shape[1] == qw.k
    x = x.contiguous()
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, qw.n), dtype=out_dtype, device=x.device)
    _run_op(make_op(qw, x, out), PATHS[path], x.device)
    return out


def qlinear_tuned(qw: QWeights, x: torch.Tensor, tile: int = -1, splits: int = 0,
                  out_dtype=torch.float32, out: torch.Tensor | None = None) -> torch.Tensor:
    """qlinear on the MFMA path with a forced tile configuration / split of k
    (-1 / 0: automatic), for tuning and tests (eb_qlinear_tuned)."""
    assert x.is_cuda and x.dim() == 2 and x.shape[1] == qw.k
    x = x.contiguous()
    if out is None:
        out = torch.empty((x.shape[0], qw.n), dtype=out_dtype, device=x.device)
    _run_op(make_op(qw, x, out), EB_PATH_MFMA, x.device, tile=tile, splits=splits)
    return out


def auto_path(qtype: str, x_dtype, m: int, n: int, k: int) -> str:
    p = lib.eb_qlinear_auto_path(QTYPES[qtype], DTYPES[x_dtype], m, n, k)
    return {EB_PATH_GEMV: "gemv", EB_PATH_MFMA: "mfma"}.get(p, "invalid")


def make_op(qw: QWeights, x: torch.Tensor, y: torch.Tensor, x_dtype=None, prologue=None,
            norm_weight: torch.Tensor | None = None, eps: float = 0.0, epilogue=None,
            residual: torch.Tensor | None = None) -> eb_qlinear_op:
    """One eb_qlinear_op.  With prologue="rmsnorm", x is the fp32 residual
    stream and x_dtype the 16-bit type the product consumes (default bf16)."""
    if x_dtype is None:
        x_dtype = torch.bfloat16 if x.dtype == torch.float32 else x.dtype
    return eb_qlinear_op(qw.c, x.data_ptr(), y.data_ptr(), x.shape[0], DTYPES[x_dtype],
                         DTYPES[y.dtype], PROLOGUES[prologue], EPILOGUES[epilogue],
                         norm_weight.data_ptr() if norm_weight is not None else None,
                         residual.data_ptr() if residual is not None else None, float(eps), 0)


def make_ops(entries) -> ctypes.Array:
    """entries: iterable of (QWeights, x, y) or (QWeights, x, y, {make_op keywords}).
    Returns a ctypes eb_qlinear_op array."""
    entries = list(entries)
    arr = (eb_qlinear_op * len(entries))()
    for i, e in enumerate(entries):
        arr[i] = make_op(*e[:3], **(e[3] if len(e) > 3 else {}))
    return arr


def qlinear_fused(qw: QWeights, x: torch.Tensor, out_dtype=torch.float32, x_dtype=None,
                  prologue=None, norm_weight=None, eps: float = 0.0, epilogue=None,
                  residual=None, path: str = "auto", out: torch.Tensor | None = None,
                  tile: int | None = None, splits: int = 0) -> torch.Tensor:
    """One projection with fused steps (eb_qlinear_fused): optional RMS
    normalisation of x before the product, residual addition ("add") or the
    SiLU-gated product of interleaved gate/up rows ("glu", output n / 2).
    tile / splits force the MFMA path's tile configuration / split of k
    (eb_qlinear_tuned; -1 / 0: automatic)."""
    assert x.is_cuda and x.dim() == 2 and x.shape[1] == qw.k
    x = x.contiguous()
    m = x.shape[0]
    if out is None:
        n_out = qw.n // 2 if epilogue == "glu" else qw.n
        out = torch.empty((m, n_out), dtype=out_dtype, device=x.device)
    op = make_op(qw, x, out, x_dtype, prologue, norm_weight, eps, epilogue, residual)
    if tile is None and not splits:
        _run_op(op, PATHS[path], x.device)
    else:
        _run_op(op, EB_PATH_MFMA, x.device, tile=-1 if tile is None else tile, splits=splits)
    return out


def stack_workspace_bytes(ops: ctypes.Array) -> int:
    return int(lib.eb_qlinear_stack_workspace_bytes(ops, len(ops)))


def qlinear_stack(ops: ctypes.Array, device=None) -> None:
    """eb_qlinear_stack with a workspace that belongs to this op array (kept
    on it: the cached plan keeps its tables there while it is cached)."""
    nbytes = stack_workspace_bytes(ops)
    ws = getattr(ops, "_eb_workspace", None)
    if nbytes and (ws is None or ws.numel() < nbytes):
        ws = torch.empty(nbytes, dtype=torch.uint8,
                         device=device if device is not None else torch.cuda.current_device())
        ops._eb_workspace = ws
    wp, wb = (ws.data_ptr(), ws.numel()) if (nbytes and ws is not None) else (None, 0)
    _check(lib.eb_qlinear_stack(ops, len(ops), wp, wb, _stream(device)), "eb_qlinear_stack")


def stack_launches(ops: ctypes.Array) -> int:
    """Kernel launches eb_qlinear_stack makes for this op list (host-only)."""
    n = lib.eb_qlinear_stack_launches(ops, len(ops))
    if n < 0:
        raise EBError(n, "eb_qlinear_stack_launches")
    return n


def stack_cache_clear() -> None:
    _check(lib.eb_stack_cache_clear(), "eb_stack_cache_clear")


def mfma_tile_count() -> int:
    return int(lib.eb_mfma_tile_count())


def make_modules(specs) -> ctypes.Array:
    """specs: iterable of (ops array from make_ops, period, phase, repeats).
    The op arrays are kept on the result (the modules point into them)."""
    specs = list(specs)
    arr = (eb_module * len(specs))()
    for i, (ops, period, phase, repeats) in enumerate(specs):
        arr[i] = eb_module(ctypes.cast(ops, ctypes.POINTER(eb_qlinear_op)), len(ops), period, phase,
                           repeats)
    arr._eb_ops = [s[0] for s in specs]
    return arr


def multirate_tick(mods: ctypes.Array, tick: int, device=None) -> None:
    """eb_multirate_tick with a workspace that belongs to this module array."""
    nbytes = int(lib.eb_multirate_workspace_bytes(mods, len(mods)))
    ws = getattr(mods, "_eb_workspace", None)
    if nbytes and (ws is None or ws.numel() < nbytes):
        ws = torch.empty(nbytes, dtype=torch.uint8,
                         device=device if device is not None else torch.device("cuda"))
        mods._eb_workspace = ws
    dev = ws.device if ws is not None else torch.device("cuda")
    _check(lib.eb_multirate_tick(mods, len(mods), tick, ws.data_ptr() if nbytes else None, nbytes,
                                 _stream(dev)), "eb_multirate_tick")


def multirate_launches(mods: ctypes.Array, tick: int) -> int:
    n = lib.eb_multirate_launches(mods, len(mods), tick)
    if n < 0:
        raise EBError(n, "eb_multirate_launches")
    return n
