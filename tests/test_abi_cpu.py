"""The C ABI without a GPU: libeb.so loads, exports every symbol include/eb.h
declares, its host-only layout functions are right, and argument validation
rejects bad calls before anything reaches the HIP runtime."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eb.h")


@pytest.fixture(scope="module")
def eb():
    lib = os.path.join(ROOT, "paper_2607_02501_amd", "libeb.so")
    if not os.path.exists(lib):
        from paper_2607_02501_amd import build

        build.build()
    from paper_2607_02501_amd import eb as _eb

    return _eb


def declared_functions():
    text = "".join(open(os.path.join(ROOT, "include", h)).read()
                   for h in sorted(os.listdir(os.path.join(ROOT, "include"))) if h.endswith(".h"))
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eb_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("eb_quantize_q8_0", "eb_quantize_q4_0", "eb_quantize_q6_s", "eb_qlinear",
                     "eb_qlinear_stack"):
        assert required in names


def test_library_resolves_every_symbol_at_load(eb):
    # RTLD_NOW binds every reference (kernel launch stubs included) at load time
    ctypes.CDLL(eb.LIB_PATH, mode=os.RTLD_NOW)


def test_every_declared_symbol_is_exported(eb):
    lib = ctypes.CDLL(eb.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(eb):
    for s in (0, -1, -2, -3, -4, 17):
        assert eb.lib.eb_status_str(s)
    assert eb.version().startswith("eb ")


@pytest.mark.parametrize("qtype,qb", [("q8_0", 32), ("q4_0", 16)])
@pytest.mark.parametrize("n,k", [(1, 32), (7, 96), (4096, 4096), (4096, 11008), (3, 288)])
def test_layout(eb, qtype, qb, n, k):
    L = eb.layout(qtype, n, k)
    nb = k // 32
    assert L.qs_offset == 0 and L.qs_row_bytes == nb * qb
    assert L.d_offset % 256 == 0 and L.d_offset >= n * nb * qb and L.d_offset - n * nb * qb < 256
    assert L.d_stride % 8 == 0 and nb <= L.d_stride < nb + 8
    assert L.total_bytes % 256 == 0 and L.total_bytes >= L.d_offset + 2 * n * L.d_stride
    assert L.canonical_bytes == n * nb * (2 + qb)
    assert eb.qweights_bytes(qtype, n, k) == L.total_bytes


@pytest.mark.parametrize("n,k", [(1, 256), (7, 768), (4096, 4096), (4096, 11008), (3, 2304)])
def test_layout_q6(eb, n, k):
    """Q6_S planar layout: 24-byte code chunks per 32 weights, the int8
    sub-scale plane (k/16 bytes per row), the binary16 scale plane
    (round_up(k/256, 8) entries per row), each 256-byte aligned."""
    if k % 256:
        assert eb.lib.eb_qweights_bytes(eb.EB_Q6_S, n, k) == 0
        return
    L = eb.layout("q6_s", n, k)
    nb = k // 32
    assert L.qs_offset == 0 and L.qs_row_bytes == nb * 24
    assert L.sc_offset % 256 == 0 and 0 <= L.sc_offset - n * nb * 24 < 256
    assert L.sc_stride == k // 16
    assert L.d_offset % 256 == 0 and 0 <= L.d_offset - (L.sc_offset + n * k // 16) < 256
    assert L.d_stride % 8 == 0 and k // 256 <= L.d_stride < k // 256 + 8
    assert L.total_bytes % 256 == 0 and 0 <= L.total_bytes - (L.d_offset + 2 * n * L.d_stride) < 256
    assert L.canonical_bytes == n * (k // 256) * 210
    assert eb.qweights_bytes("q6_s", n, k) == L.total_bytes
    # Q8_0 / Q4_0 layouts have no sub-scale plane
    assert eb.layout("q8_0", n, k).sc_offset == 0 and eb.layout("q4_0", n, k).sc_stride == 0


def test_q6_validation(eb):
    L = eb.lib
    assert L.eb_quantize_q6_s(0x200000, 4, 128, 0x100000, None) == -1   # k % 256
    assert L.eb_quantize_q6_s(0x200000, 4, 256, 0x100080, None) == -2   # out misaligned
    assert L.eb_quantize_q6_s(None, 0, 256, None, None) == 0            # empty: no-op
    assert L.eb_qweights_from_canonical(eb.EB_Q6_S, 0x200000, 4, 288, 0x100000, None) == -1
    w = _w(eb, eb.EB_Q6_S, n=64, k=512)
    # its GEMV up to m = 4, the matrix cores beyond; the GEMV takes m <= 8
    for m, path in ((1, eb.EB_PATH_GEMV), (4, eb.EB_PATH_GEMV), (5, eb.EB_PATH_MFMA),
                    (50, eb.EB_PATH_MFMA), (300, eb.EB_PATH_MFMA)):
        assert L.eb_qlinear_auto_path(eb.EB_Q6_S, eb.EB_BF16, m, 64, 512) == path, m
    assert L.eb_qlinear_ex(ctypes.byref(w), X, eb.EB_F16, 9, Y, eb.EB_F32, eb.EB_PATH_GEMV,
                           None) == eb.EB_ERR_UNSUPPORTED
    bad = _w(eb, eb.EB_Q6_S, n=64, k=288)
    assert L.eb_qlinear(ctypes.byref(bad), X, eb.EB_F16, 1, Y, eb.EB_F32, None) == -1
    # no split along k: no workspace, except for a prologue's normalised rows
    # on the matrix-core path (the GEMV normalises while it stages x)
    op = eb.eb_qlinear_op(_w(eb, eb.EB_Q6_S, n=1024, k=4096, data=1 * GB), 8 * GB, 9 * GB, 50,
                          eb.EB_BF16, eb.EB_F32)
    assert L.eb_qlinear_workspace_bytes(ctypes.byref(op), eb.EB_PATH_AUTO) == 0
    normed = eb.eb_qlinear_op(_w(eb, eb.EB_Q6_S, n=1024, k=4096, data=1 * GB), 8 * GB, 9 * GB, 50,
                              eb.EB_BF16, eb.EB_F32, eb.EB_PRO_RMSNORM, 0, G, None, 1e-5, 0)
    assert L.eb_qlinear_workspace_bytes(ctypes.byref(normed), eb.EB_PATH_AUTO) == 50 * 4096 * 2
    # in a stack independent m == 1 Q6_S ops share one fused GEMV launch (k up
    # to 16384); with more rows, or longer rows, every op is a launch of its own
    def q6ops(m, k):
        return [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (1 << 20), 9 * GB + i * (1 << 20),
                    k=k, n=2048, m=m, qtype=eb.EB_Q6_S, xt=eb.EB_F16) for i in range(4)]
    assert _launches(eb, q6ops(1, 1024)) == 1
    assert _launches(eb, q6ops(1, 16384)) == 1
    assert _launches(eb, q6ops(2, 1024)) == 4
    assert _launches(eb, q6ops(1, 16640)) == 4
    # one fused launch per slot count (64-weight units per lane: k = 4096 -> 1, 11008 -> 3)
    assert _launches(eb, q6ops(1, 4096)[:2] + q6ops(1, 11008)[2:]) == 2
    # beyond 128 rows the tile kernel of the other formats: a lone op may split
    # k (many tiles: unsplit), independent ops share one grouped launch
    op = eb.eb_qlinear_op(_w(eb, eb.EB_Q6_S, n=4096, k=4096, data=1 * GB), 8 * GB, 9 * GB, 4096,
                          eb.EB_BF16, eb.EB_F32)
    assert L.eb_qlinear_workspace_bytes(ctypes.byref(op), eb.EB_PATH_AUTO) == 0
    for m, n, k in ((129, 4096, 4096), (816, 2048, 2048), (4096, 4096, 4096)):
        ops = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (64 << 20), 12 * GB + i * (128 << 20),
                   k=k, n=n, m=m, qtype=eb.EB_Q6_S, xt=eb.EB_BF16) for i in range(3)]
        assert _launches(eb, ops) == 1, (m, n, k)
        assert _launches(eb, ops[:1]) in (1, 2), (m, n, k)   # the op alone, split or not
    # up to 128 rows its own kernel, one launch per op
    assert _launches(eb, [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (64 << 20),
                              12 * GB + i * (128 << 20), k=2048, n=2048, m=128, qtype=eb.EB_Q6_S,
                              xt=eb.EB_BF16) for i in range(3)]) == 3


def test_bytes_rejects_bad_sizes(eb):
    assert eb.lib.eb_qweights_bytes(eb.EB_Q8_0, 4, 33) == 0
    assert eb.lib.eb_qweights_bytes(4, 4, 32) == 0
    assert eb.lib.eb_qweights_bytes(eb.EB_Q6_S, 4, 32) == 0
    assert eb.lib.eb_qweights_bytes(eb.EB_Q4_0, -1, 32) == 0
    assert eb.lib.eb_qweights_layout(eb.EB_Q4_0, 4, 32, None) == eb.EB_ERR_INVALID


def _w(eb, qtype=None, n=64, k=64, data=0x100000, reserved=0):
    return eb.eb_qweights(qtype or eb.EB_Q8_0, reserved, n, k, data)


# Fake, never-dereferenced addresses: every call below must be rejected on the host.
X, Y = 0x200000, 0x400000


@pytest.mark.parametrize("case,expect", [
    ("null_w", -1), ("null_data", -1), ("bad_type", -1), ("reserved", -1), ("k33", -1),
    ("k0", -1), ("n0", -1), ("m_neg", -1), ("bad_xt", -1), ("bad_path", -1), ("x_null", -1),
    ("w_misaligned", -2), ("x_misaligned", -2), ("y_misaligned", -2), ("x_f32", -3),
    ("bad_yt", -1), ("gemv_m9", -3), ("gemv_big_k", -3), ("overlap", -1),
])
def test_qlinear_validation(eb, case, expect):
    w = _w(eb)
    x, y, m, xt, yt, path = X, Y, 4, eb.EB_F16, eb.EB_F32, eb.EB_PATH_AUTO
    wp = ctypes.byref(w)
    if case == "null_w":
        wp = None
    elif case == "null_data":
        w.data = None
    elif case == "bad_type":
        w.type = 7
    elif case == "reserved":
        w.reserved = 1
    elif case == "k33":
        w.k = 33
    elif case == "k0":
        w.k = 0
    elif case == "n0":
        w.n = 0
    elif case == "m_neg":
        m = -1
    elif case == "bad_xt":
        xt = 9
    elif case == "bad_path":
        path = 5
    elif case == "x_null":
        x = None
    elif case == "w_misaligned":
        w.data = 0x100010
    elif case == "x_misaligned":
        x = X + 8
    elif case == "y_misaligned":
        y = Y + 4
    elif case == "x_f32":
        xt = eb.EB_F32
    elif case == "bad_yt":
        yt = 7
    elif case == "gemv_m9":
        m, path = 9, eb.EB_PATH_GEMV
    elif case == "gemv_big_k":
        w.k, m, path = 65536, 2, eb.EB_PATH_GEMV
        y = 0x10000000  # clear of the (fake) 4.4 MB weight range
    elif case == "overlap":
        y = X + 64
    assert eb.lib.eb_qlinear_ex(wp, x, xt, m, y, yt, path, None) == expect


G, R = 0x600000, 0x800000  # fake norm-weight and residual addresses


@pytest.mark.parametrize("case,expect", [
    ("bad_prologue", -1), ("bad_epilogue", -1), ("reserved", -1), ("no_gamma", -1),
    ("neg_eps", -1), ("nan_eps", -1), ("inf_eps", -1), ("no_residual", -1), ("glu_odd_n", -1),
    ("gamma_misaligned", -2), ("residual_misaligned", -2), ("residual_overlaps_y", -1),
    ("y_overlaps_gamma", -1), ("y_overlaps_h", -1), ("x_f32", -3), ("gemv_m9", -3),
])
def test_fused_validation(eb, case, expect):
    """eb_qlinear_fused rejects bad fused-step fields on the host (nothing launches)."""
    w = _w(eb)
    op = eb.eb_qlinear_op(w, X, Y, 4, eb.EB_BF16, eb.EB_F32, eb.EB_PRO_RMSNORM, eb.EB_EPI_ADD,
                          G, R, 1e-5, 0)
    path = eb.EB_PATH_AUTO
    if case == "bad_prologue":
        op.prologue = 2
    elif case == "bad_epilogue":
        op.epilogue = 3
    elif case == "reserved":
        op.reserved = 1
    elif case == "no_gamma":
        op.norm_weight = None
    elif case == "neg_eps":
        op.norm_eps = -1e-6
    elif case == "nan_eps":
        op.norm_eps = float("nan")
    elif case == "inf_eps":
        op.norm_eps = float("inf")
    elif case == "no_residual":
        op.residual = None
    elif case == "glu_odd_n":
        op.w.n, op.epilogue = 63, eb.EB_EPI_GLU
    elif case == "gamma_misaligned":
        op.norm_weight = G + 4
    elif case == "residual_misaligned":
        op.residual = R + 8
    elif case == "residual_overlaps_y":
        op.residual = Y + 16  # not y itself, but inside y's 4 x 64 fp32 outputs
    elif case == "y_overlaps_gamma":
        op.norm_weight = Y + 32
    elif case == "y_overlaps_h":
        op.y = X + 4 * 64 * 3  # h is fp32 under the prologue: 4 rows x 64 x 4 bytes
    elif case == "x_f32":
        op.x_type = eb.EB_F32
    elif case == "gemv_m9":
        op.m, path = 9, eb.EB_PATH_GEMV
    assert eb.lib.eb_qlinear_fused(ctypes.byref(op), path, None) == expect
    assert eb.lib.eb_qlinear_fused(None, path, None) == eb.EB_ERR_INVALID


def test_fused_m0_is_noop_and_still_validated(eb):
    """m == 0 with fused steps launches nothing (null x, y, norm weight and
    residual are allowed), but enum and shape fields are still checked."""
    w = _w(eb)
    op = eb.eb_qlinear_op(w, None, None, 0, eb.EB_BF16, eb.EB_F32, eb.EB_PRO_RMSNORM,
                          eb.EB_EPI_ADD, None, None, 1e-5, 0)
    assert eb.lib.eb_qlinear_fused(ctypes.byref(op), eb.EB_PATH_AUTO, None) == eb.EB_OK
    arr = (eb.eb_qlinear_op * 2)(op, op)
    assert eb.lib.eb_qlinear_stack_launches(arr, 2) == 0
    op.epilogue = 7
    assert eb.lib.eb_qlinear_fused(ctypes.byref(op), eb.EB_PATH_AUTO, None) == eb.EB_ERR_INVALID
    op.epilogue, op.norm_eps = eb.EB_EPI_GLU, -1.0
    assert eb.lib.eb_qlinear_fused(ctypes.byref(op), eb.EB_PATH_AUTO, None) == eb.EB_ERR_INVALID
    op.norm_eps, op.w.n = 1e-5, 63  # odd n with the gate/up epilogue
    assert eb.lib.eb_qlinear_fused(ctypes.byref(op), eb.EB_PATH_AUTO, None) == eb.EB_ERR_INVALID


def test_fused_stack_counts_prologue_launches(eb):
    """A normalisation prologue costs a row-kernel launch on the MFMA path and
    nothing on the GEMV path; dependencies through the residual stream split runs."""
    k, n = 256, 512
    WB = eb.lib.eb_qweights_bytes(eb.EB_Q8_0, n, k)
    ws = [0x10000000 + i * ((WB + 4095) // 4096 * 4096) for i in range(4)]
    H, A, Q, GU, ACT = 0x20000000, 0x21000000, 0x22000000, 0x23000000, 0x24000000

    def op(i, x, y, m, pro=0, epi=0, res=None, nn=n, kk=k, yt=None):
        w = eb.eb_qweights(eb.EB_Q8_0, 0, nn, kk, ws[i])
        return eb.eb_qlinear_op(w, x, y, m, eb.EB_BF16, eb.EB_F32 if yt is None else yt, pro, epi,
                                G if pro else None, res, 1e-5, 0)

    def launches(lst):
        arr = (eb.eb_qlinear_op * len(lst))(*lst)
        return eb.lib.eb_qlinear_stack_launches(arr, len(lst))

    # one decoder layer at m = 1: normalised QKV, O adding into h, normalised
    # gate/up with the gated product, down adding into h
    for m, pro_cost in ((1, 0), (50, 1)):
        layer = [op(0, H, Q, m, pro=1),
                 op(1, A, H, m, epi=1, res=H),
                 op(2, H, GU, m, pro=1, epi=2, yt=eb.EB_BF16),
                 op(3, GU, H, m, epi=1, res=H, kk=n // 2)]
        # every op depends on the one before (h, then the gate/up output), so
        # nothing fuses: 4 launches plus the prologue row kernels
        assert launches(layer) == 4 + 2 * pro_cost, m
    # two independent normalised projections of one h fuse into one launch
    for m, expect in ((1, 1), (50, 3)):
        two = [op(0, H, Q, m, pro=1), op(2, H, GU, m, pro=1)]
        assert launches(two) == expect, m


def test_reduction_runs_next_prologue(eb, monkeypatch):
    """In a dependent layer chain the split-K reduction that writes the fp32
    stream h (O and down, + h) also normalises it for the next projection, so
    those prologues cost no row-kernel launch; EB_STACK_FUSE_NORM=0 keeps them.
    At m <= 64 the projections run on the narrow kernel; those whose 16-row
    workgroups would not fill the GPU (O and down: 1024 rows) split k and are
    reduced, and those reductions normalise for the next projection."""
    d, f = 1024, 4096   # the action-expert layer shape

    def chain(m, stream16=False):
        H, A, Q, GU = 0x20000000, 0x21000000, 0x22000000, 0x23000000
        ops, base = [], 0x10000000
        for _ in range(2):
            for n, k, x, y, pro, epi, res, yt in ((3 * d, d, H, Q, 1, 0, None, eb.EB_BF16),
                                                  (d, d, A, H, 0, 1, H, eb.EB_F32),
                                                  (2 * f, d, H, GU, 1, 2, None, eb.EB_BF16),
                                                  (d, f, GU, H, 0, 1, H, eb.EB_F32)):
                w = eb.eb_qweights(eb.EB_Q8_0, 0, n, k, base)
                base += (eb.lib.eb_qweights_bytes(eb.EB_Q8_0, n, k) + 4095) // 4096 * 4096
                if stream16 and epi == 1:
                    yt = eb.EB_BF16
                ops.append(eb.eb_qlinear_op(w, x, y, m, eb.EB_BF16, yt, pro, epi,
                                            G if pro else None, res, 1e-5, 0))
        return (eb.eb_qlinear_op * len(ops))(*ops)

    # m = 50: 8 narrow launches, 4 reductions (O and down split k: 64
    # workgroups of 16 rows would leave most CUs idle) and 4 prologue row
    # kernels; fused, every prologue after a split O or down runs in its
    # reduction, leaving the first layer's QKV prologue
    monkeypatch.setenv("EB_STACK_FUSE_NORM", "0")
    assert eb.lib.eb_qlinear_stack_launches(chain(50), 8) == 8 + 4 + 4
    monkeypatch.delenv("EB_STACK_FUSE_NORM")
    assert eb.lib.eb_qlinear_stack_launches(chain(50), 8) == 8 + 4 + 1
    # m = 100: split projections; every prologue after a split O or down costs nothing
    monkeypatch.setenv("EB_STACK_FUSE_NORM", "0")
    unfused = eb.lib.eb_qlinear_stack_launches(chain(100), 8)
    monkeypatch.delenv("EB_STACK_FUSE_NORM")
    fused = eb.lib.eb_qlinear_stack_launches(chain(100), 8)
    assert 8 + 4 < fused < unfused, (fused, unfused)
    # a 16-bit stream (no fp32 h to reduce into) keeps the row kernels
    assert eb.lib.eb_qlinear_stack_launches(chain(100, stream16=True), 8) == unfused


def test_qlinear_m0_is_noop(eb):
    w = _w(eb)
    assert eb.lib.eb_qlinear(ctypes.byref(w), None, eb.EB_F16, 0, None, eb.EB_F32, None) == 0


def test_quantize_validation(eb):
    L = eb.lib
    assert L.eb_quantize_q8_0(None, 0, 64, None, None) == 0          # empty: no-op
    assert L.eb_quantize_q8_0(None, 4, 64, 0x100000, None) == -1    # null w
    assert L.eb_quantize_q4_0(0x200000, 4, 48, 0x100000, None) == -1  # k % 32
    assert L.eb_quantize_q4_0(0x200004, 4, 64, 0x100000, None) == -2  # w misaligned
    assert L.eb_quantize_q4_0(0x200000, 4, 64, 0x100080, None) == -2  # out misaligned
    assert L.eb_quantize_q8_0(0x200000, -1, 64, 0x100000, None) == -1


def test_canonical_validation(eb):
    w = _w(eb)
    assert eb.lib.eb_qweights_to_canonical(ctypes.byref(w), None, None) == -1
    assert eb.lib.eb_qweights_from_canonical(eb.EB_Q4_0, 0x200000, 4, 40, 0x100000, None) == -1
    assert eb.lib.eb_qweights_from_canonical(eb.EB_Q4_0, 0x200000, 4, 64, 0x100040, None) == -2


def test_stack_validation(eb):
    ops = (eb.eb_qlinear_op * 2)()
    ops[0] = eb.eb_qlinear_op(_w(eb), X, Y, 1, eb.EB_F16, eb.EB_F32)
    ops[1] = eb.eb_qlinear_op(_w(eb, k=33), X, Y, 1, eb.EB_F16, eb.EB_F32)
    assert eb.lib.eb_qlinear_stack(ops, 2, None, 0, None) == -1   # second op invalid -> nothing launched
    assert eb.lib.eb_qlinear_stack(ops, 0, None, 0, None) == 0
    assert eb.lib.eb_qlinear_stack(ops, -1, None, 0, None) == -1
    assert eb.lib.eb_qlinear_stack(None, 3, None, 0, None) == -1


def test_auto_path(eb):
    f = eb.lib.eb_qlinear_auto_path
    assert f(eb.EB_Q4_0, eb.EB_F16, 1, 4096, 4096) == eb.EB_PATH_GEMV
    assert f(eb.EB_Q8_0, eb.EB_BF16, 816, 2560, 2048) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q8_0, eb.EB_BF16, 50, 2048, 1024) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q8_0, eb.EB_F16, 1, 4096, 1 << 20) == eb.EB_PATH_MFMA  # x too large for LDS
    # measured crossover: GEMV for m = 2..4 when n >= 4096, for m = 5..8 when
    # also k is past the narrow matrix-core kernel (k > 2048)
    assert f(eb.EB_Q4_0, eb.EB_F16, 4, 4096, 4096) == eb.EB_PATH_GEMV
    assert f(eb.EB_Q8_0, eb.EB_BF16, 4, 1024, 4096) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q8_0, eb.EB_BF16, 3, 2048, 2048) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q8_0, eb.EB_BF16, 2, 8192, 1024) == eb.EB_PATH_GEMV
    assert f(eb.EB_Q4_0, eb.EB_F16, 5, 4096, 4096) == eb.EB_PATH_GEMV
    assert f(eb.EB_Q4_0, eb.EB_F16, 8, 12288, 4096) == eb.EB_PATH_GEMV
    assert f(eb.EB_Q8_0, eb.EB_BF16, 6, 8192, 1024) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q8_0, eb.EB_BF16, 8, 32768, 2048) == eb.EB_PATH_MFMA
    assert f(eb.EB_Q4_0, eb.EB_F16, 5, 4096, 16384) == eb.EB_PATH_MFMA  # x too large for the GEMV
    assert f(eb.EB_Q8_0, eb.EB_F16, 0, 64, 64) == eb.EB_ERR_INVALID


# ---------------------------------------------------------------------------
# Stack plans: which runs of ops are fused (host-only; addresses are fake)
# ---------------------------------------------------------------------------

def _op(eb, data, x, y, k=4096, n=4096, m=1, qtype=None, xt=None, yt=None):
    return eb.eb_qlinear_op(eb.eb_qweights(qtype or eb.EB_Q4_0, 0, n, k, data), x, y, m,
                            xt or eb.EB_F16, yt or eb.EB_F32)


def _launches(eb, ops):
    arr = (eb.eb_qlinear_op * len(ops))(*ops)
    return eb.lib.eb_qlinear_stack_launches(arr, len(ops))


GB = 1 << 30


def test_stack_fuses_independent_decode_ops(eb, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    ops = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * 65536, 9 * GB + i * 65536) for i in range(12)]
    assert _launches(eb, ops) == 1
    # two K size classes (4096: 2 slots, 11008: 6 slots) -> one launch each
    ops += [_op(eb, 3 * GB + i * (64 << 20), 10 * GB + i * 65536, 11 * GB + i * 65536, k=11008)
            for i in range(4)]
    assert _launches(eb, ops) == 2
    monkeypatch.setenv("EB_STACK_FUSE", "0")
    assert _launches(eb, ops) == len(ops)


def test_stack_respects_dependencies(eb, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    W0, W1, W2 = 1 * GB, 2 * GB, 3 * GB
    X, Y0, Y1 = 8 * GB, 9 * GB, 10 * GB
    # read-after-write: op1 reads op0's output (bf16 y feeding the next x)
    raw = [_op(eb, W0, X, Y0, yt=eb.EB_BF16), _op(eb, W1, Y0, Y1, xt=eb.EB_BF16)]
    assert _launches(eb, raw) == 2
    # write-after-read: op1 overwrites op0's input
    war = [_op(eb, W0, X, Y0), _op(eb, W1, 20 * GB, X, xt=eb.EB_BF16, yt=eb.EB_BF16)]
    assert _launches(eb, war) == 2
    # write-after-write on the same output
    waw = [_op(eb, W0, X, Y0), _op(eb, W1, X + 65536, Y0)]
    assert _launches(eb, waw) == 2
    # independent again after the dependency: [a, b | c, d] -> 2 launches
    bf = eb.EB_BF16
    chain = [_op(eb, W0, X, Y0, xt=bf, yt=bf), _op(eb, W1, X + 65536, Y1, xt=bf),
             _op(eb, W2, Y0, 11 * GB, xt=bf), _op(eb, 4 * GB, X + 2 * 65536, 12 * GB, xt=bf)]
    assert _launches(eb, chain) == 2


def test_stack_breaks_runs_on_format_and_m(eb, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    a = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * 65536, 9 * GB + i * 65536) for i in range(3)]
    q8 = _op(eb, 5 * GB, 10 * GB, 11 * GB, qtype=eb.EB_Q8_0)
    b = [_op(eb, 6 * GB + i * (64 << 20), 12 * GB + i * 65536, 13 * GB + i * 65536) for i in range(3)]
    assert _launches(eb, a + [q8] + b) == 3
    m4 = _op(eb, 5 * GB, 10 * GB, 11 * GB, m=4)
    assert _launches(eb, a + [m4] + b) == 3
    m0 = _op(eb, 5 * GB, 10 * GB, 11 * GB, m=0)
    assert _launches(eb, a + [m0] + b) == 2  # an empty op launches nothing
    assert _launches(eb, [a[0]]) == 1
    bad = a + [_op(eb, 5 * GB, 10 * GB, 11 * GB, k=33)]
    assert _launches(eb, bad) == eb.EB_ERR_INVALID


def test_tuned_validation(eb):
    """eb_qlinear_tuned (include/eb_tuning.h) takes the tile and split per
    call and rejects values out of range on the host."""
    count = eb.lib.eb_mfma_tile_count()
    assert count >= 1
    op = eb.eb_qlinear_op(_w(eb), X, Y, 64, eb.EB_F16, eb.EB_F32)
    f = eb.lib.eb_qlinear_tuned
    for tile, splits in ((-2, 0), (count, 0), (0, 17), (0, -1)):
        assert f(ctypes.byref(op), tile, splits, None, 0, None) == eb.EB_ERR_INVALID
    assert f(None, -1, 0, None, 0, None) == eb.EB_ERR_INVALID


def test_no_process_wide_setters_in_the_abi():
    """The public header declares no setter of global state (the tile / split
    choice is a per-call argument of the tuning header)."""
    names = declared_functions()
    assert not [n for n in names if "force" in n or n.startswith("eb_set")], names
    # tuning entry points live in eb_tuning.h, not in the public eb.h
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    assert "eb_qlinear_tuned" not in text


def test_library_imports_no_allocator(eb):
    """libeb.so allocates no device or host memory through the HIP runtime:
    its dynamic symbol table references no HIP allocation or free routine
    (the caller passes every buffer and workspace)."""
    import subprocess

    out = subprocess.run(["nm", "-D", "--undefined-only", eb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    hip = sorted({line.split()[-1] for line in out.splitlines() if "hip" in line.lower()})
    assert hip, "expected HIP runtime imports"
    alloc = [n for n in hip if re.search(r"malloc|free|alloc", n, re.I)]
    assert not alloc, alloc


def test_stack_counts_split_k_reduction(eb):
    # a long-k op at m = 100 or 50 is split (product + ordered reduction);
    # at m = 50 the narrow kernel takes the whole of k in one launch when its
    # 16-row workgroups fill the GPU (n = 4096: 256 of them); a large prefill
    # op fills the GPU unsplit
    for m in (100, 50):
        split = [_op(eb, 1 * GB, 8 * GB, 9 * GB, k=4096, n=1024, m=m, qtype=eb.EB_Q8_0,
                     xt=eb.EB_BF16)]
        assert _launches(eb, split) == 2, m
    narrow = [_op(eb, 1 * GB, 8 * GB, 9 * GB, k=2048, n=4096, m=50, qtype=eb.EB_Q8_0,
                  xt=eb.EB_BF16)]
    assert _launches(eb, narrow) == 1
    whole = [_op(eb, 1 * GB, 8 * GB, 9 * GB, k=3072, n=9216, m=4096, qtype=eb.EB_Q4_0,
                 xt=eb.EB_BF16)]
    assert _launches(eb, whole) == 1


def test_workspace_sizes(eb):
    """Workspace queries: none for the GEMV path, normalised activations plus
    split-K partial sums on the MFMA path, tables and buffers for a stack."""
    q = eb.lib.eb_qlinear_workspace_bytes
    gemv = eb.eb_qlinear_op(_w(eb, k=4096, n=4096), 8 * GB, 9 * GB, 1, eb.EB_F16, eb.EB_F32)
    assert q(ctypes.byref(gemv), eb.EB_PATH_AUTO) == 0
    plain = eb.eb_qlinear_op(_w(eb, k=4096, n=1024, data=1 * GB), 8 * GB, 9 * GB, 100, eb.EB_BF16,
                             eb.EB_F32)
    partial = q(ctypes.byref(plain), eb.EB_PATH_AUTO)
    assert partial > 0 and partial % 256 == 0  # split along k: fp32 partials
    normed = eb.eb_qlinear_op(_w(eb, k=4096, n=1024, data=1 * GB), 8 * GB, 9 * GB, 100, eb.EB_BF16,
                              eb.EB_F32, eb.EB_PRO_RMSNORM, 0, G, None, 1e-5, 0)
    assert q(ctypes.byref(normed), eb.EB_PATH_AUTO) == partial + 100 * 4096 * 2
    # m <= 64, k <= 2048, n = 4096: the narrow kernel needs no partial sums
    small = eb.eb_qlinear_op(_w(eb, k=2048, n=4096, data=1 * GB), 8 * GB, 9 * GB, 50, eb.EB_BF16,
                             eb.EB_F32)
    assert q(ctypes.byref(small), eb.EB_PATH_AUTO) == 0
    bad = eb.eb_qlinear_op(_w(eb, k=33), X, Y, 4, eb.EB_F16, eb.EB_F32)
    assert q(ctypes.byref(bad), eb.EB_PATH_AUTO) == 0
    # a fused run of small-m ops needs its table (and nothing else)
    ops = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (1 << 20), 9 * GB + i * (1 << 20),
               k=1024, n=2048, m=50, qtype=eb.EB_Q8_0, xt=eb.EB_BF16) for i in range(8)]
    arr = (eb.eb_qlinear_op * len(ops))(*ops)
    sb = eb.lib.eb_qlinear_stack_workspace_bytes(arr, len(ops))
    assert 0 < sb < 8 * 1024 and sb % 256 == 0
    assert eb.lib.eb_qlinear_stack_workspace_bytes(arr, 0) == 0


def test_workspace_validation(eb):
    """A workspace must be 256-byte aligned, overlap no operand, and be given
    whenever its size is; a prologue on the MFMA path needs one."""
    f = eb.lib.eb_qlinear_fused_ws
    op = eb.eb_qlinear_op(_w(eb, k=4096, n=1024, data=1 * GB), 8 * GB, 9 * GB, 50, eb.EB_BF16,
                          eb.EB_F32)
    assert f(ctypes.byref(op), eb.EB_PATH_AUTO, 10 * GB + 64, 1 << 20, None) == eb.EB_ERR_ALIGN
    assert f(ctypes.byref(op), eb.EB_PATH_AUTO, None, 4096, None) == eb.EB_ERR_INVALID
    assert f(ctypes.byref(op), eb.EB_PATH_AUTO, 8 * GB, 1 << 20, None) == eb.EB_ERR_INVALID  # on x
    assert f(ctypes.byref(op), eb.EB_PATH_AUTO, 1 * GB, 1 << 20, None) == eb.EB_ERR_INVALID  # on w
    normed = eb.eb_qlinear_op(_w(eb, k=4096, n=1024, data=1 * GB), 8 * GB, 9 * GB, 50, eb.EB_BF16,
                              eb.EB_F32, eb.EB_PRO_RMSNORM, 0, G, None, 1e-5, 0)
    assert eb.lib.eb_qlinear_fused(ctypes.byref(normed), eb.EB_PATH_MFMA, None) == eb.EB_ERR_UNSUPPORTED
    assert f(ctypes.byref(normed), eb.EB_PATH_MFMA, 10 * GB, 4096, None) == eb.EB_ERR_UNSUPPORTED
    arr = (eb.eb_qlinear_op * 1)(op)
    assert eb.lib.eb_qlinear_stack(arr, 1, 10 * GB + 8, 4096, None) == eb.EB_ERR_ALIGN
    assert eb.lib.eb_qlinear_stack(arr, 1, None, 4096, None) == eb.EB_ERR_INVALID


def test_stack_fuses_independent_small_m_mfma_ops(eb, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    bf = eb.EB_BF16
    ops = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (1 << 20), 9 * GB + i * (1 << 20),
               k=1024, n=2048, m=50, qtype=eb.EB_Q8_0, xt=bf) for i in range(8)]
    assert _launches(eb, ops) == 1
    # a different output type starts a new run (the lone op may be split-K: 2 launches)
    odd = _op(eb, 5 * GB, 10 * GB, 11 * GB, k=1024, n=2048, m=50, qtype=eb.EB_Q8_0, xt=bf, yt=bf)
    assert _launches(eb, ops[:4] + [odd] + ops[4:]) == 2 + _launches(eb, [odd])
    # m above the fused limit runs alone
    big = _op(eb, 5 * GB, 10 * GB, 11 * GB, k=1024, n=2048, m=200, qtype=eb.EB_Q8_0, xt=bf)
    assert _launches(eb, ops[:4] + [big] + ops[4:]) == 2 + _launches(eb, [big])
    # read-after-write: the second op reads the first one's output
    W0, W1 = 1 * GB, 2 * GB
    raw = [_op(eb, W0, 8 * GB, 9 * GB, k=1024, n=1024, m=50, qtype=eb.EB_Q8_0, xt=bf, yt=bf),
           _op(eb, W1, 9 * GB, 10 * GB, k=1024, n=1024, m=50, qtype=eb.EB_Q8_0, xt=bf)]
    assert _launches(eb, raw) == _launches(eb, raw[:1]) + _launches(eb, raw[1:])
    monkeypatch.setenv("EB_STACK_FUSE", "0")
    assert _launches(eb, ops) == 8 * _launches(eb, ops[:1])


def test_stack_groups_independent_large_m_mfma_ops(eb, monkeypatch):
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    monkeypatch.delenv("EB_STACK_GROUP", raising=False)
    bf = eb.EB_BF16
    # four projections of one layer with large m: one grouped launch, output
    # types may differ within it
    shapes = [(2048, 2560), (2048, 2048), (2048, 32768), (16384, 2048)]
    ops = [_op(eb, (1 + 2 * i) * GB, 16 * GB + i * GB, 24 * GB + i * GB, k=k, n=n, m=816,
               qtype=eb.EB_Q8_0, xt=bf, yt=(bf if i == 1 else eb.EB_F32))
           for i, (k, n) in enumerate(shapes)]
    assert _launches(eb, ops) == 1
    # a different activation format starts a new group
    f16 = _op(eb, 12 * GB, 40 * GB, 41 * GB, k=2048, n=2048, m=816, qtype=eb.EB_Q8_0,
              xt=eb.EB_F16)
    assert _launches(eb, ops[:2] + [f16] + ops[2:]) == 2 + _launches(eb, [f16])
    # read-after-write: the second op reads the first one's output
    raw = [_op(eb, 1 * GB, 8 * GB, 9 * GB, k=1024, n=1024, m=512, qtype=eb.EB_Q4_0, xt=bf, yt=bf),
           _op(eb, 2 * GB, 9 * GB, 10 * GB, k=1024, n=1024, m=512, qtype=eb.EB_Q4_0, xt=bf)]
    assert _launches(eb, raw) == _launches(eb, raw[:1]) + _launches(eb, raw[1:])
    monkeypatch.setenv("EB_STACK_GROUP", "0")
    assert _launches(eb, ops) == sum(_launches(eb, [o]) for o in ops)
    monkeypatch.delenv("EB_STACK_GROUP")
    # a whole 18-layer pass picks 256-row tiles; m = 816 leaves 48 rows in the
    # last row tile, which go to fused small-m launches (one per output type)
    full = [_op(eb, (1 + 3 * i) * GB, (2 + 3 * i) * GB, (3 + 3 * i) * GB, k=k, n=n, m=816,
                qtype=eb.EB_Q8_0, xt=bf, yt=(bf if i % 4 == 1 else eb.EB_F32))
            for i, (k, n) in enumerate(shapes * 18)]
    assert _launches(eb, full) == 3
    monkeypatch.setenv("EB_STACK_SPLIT_TAIL", "0")
    assert _launches(eb, full) == 1


def test_multirate_policy_and_counts(eb):
    """Control ticks (include/eb_multirate.h): a module runs on ticks t with
    t % period == phase, `repeats` times; the tick's launches are the due
    modules' stack launches; each module gets its own workspace slice."""
    backbone = [_op(eb, 1 * GB + i * (64 << 20), 8 * GB + i * (1 << 20), 9 * GB + i * (1 << 20),
                    k=1024, n=2048, m=100, qtype=eb.EB_Q8_0, xt=eb.EB_BF16) for i in range(2)]
    expert = [_op(eb, 2 * GB + i * (64 << 20), 10 * GB + i * (1 << 20), 11 * GB + i * (1 << 20),
                  k=1024, n=1024, m=1, qtype=eb.EB_Q4_0) for i in range(3)]
    b_ops = (eb.eb_qlinear_op * 2)(*backbone)
    e_ops = (eb.eb_qlinear_op * 3)(*expert)
    lb, le = _launches(eb, backbone), _launches(eb, expert)
    mods = eb.make_modules([(b_ops, 4, 1, 1), (e_ops, 1, 0, 10)])
    for t in range(8):
        assert eb.multirate_launches(mods, t) == (lb if t % 4 == 1 else 0) + 10 * le, t
    ws = eb.lib.eb_multirate_workspace_bytes(mods, 2)
    sb = eb.lib.eb_qlinear_stack_workspace_bytes(b_ops, 2)
    se = eb.lib.eb_qlinear_stack_workspace_bytes(e_ops, 3)
    assert ws == (sb + 255) // 256 * 256 + (se + 255) // 256 * 256
    # bad policies, ticks and workspaces are refused before anything runs
    L = eb.lib
    for period, phase, repeats in ((0, 0, 1), (2, 2, 1), (2, -1, 1), (1, 0, 0)):
        bad = eb.make_modules([(e_ops, period, phase, repeats)])
        assert L.eb_multirate_launches(bad, 1, 0) == eb.EB_ERR_INVALID
        assert L.eb_multirate_workspace_bytes(bad, 1) == 0
        assert L.eb_multirate_tick(bad, 1, 0, None, 0, None) == eb.EB_ERR_INVALID
    assert L.eb_multirate_launches(mods, 2, -1) == eb.EB_ERR_INVALID
    assert L.eb_multirate_tick(None, 1, 0, None, 0, None) == eb.EB_ERR_INVALID
    assert L.eb_multirate_tick(mods, 0, 0, None, 0, None) == eb.EB_ERR_INVALID
    if ws:
        assert L.eb_multirate_tick(mods, 2, 0, None, 0, None) == eb.EB_ERR_INVALID
        assert L.eb_multirate_tick(mods, 2, 0, 12 * GB, ws - 1, None) == eb.EB_ERR_INVALID
        assert L.eb_multirate_tick(mods, 2, 0, 12 * GB + 16, ws, None) == eb.EB_ERR_ALIGN


def test_int8_path_validation(eb):
    """The int8-activation prefill path: Q8_0 / Q4_0 only, no prologue, a
    workspace for the codes (m * k bytes, 256-aligned) and block scales
    (k/32 * round_up(m, 4) floats); never chosen by the automatic path."""
    L = eb.lib
    q = L.eb_qlinear_workspace_bytes
    for m in (1, 37, 816):
        op = eb.eb_qlinear_op(_w(eb, eb.EB_Q8_0, n=2048, k=4096, data=1 * GB), 8 * GB, 9 * GB, m,
                              eb.EB_BF16, eb.EB_F32)
        expect = (m * 4096 + 255) // 256 * 256 + (128 * ((m + 3) // 4 * 4) * 4 + 255) // 256 * 256
        assert q(ctypes.byref(op), eb.EB_PATH_MFMA_I8) == expect, m
        assert L.eb_qlinear_auto_path(eb.EB_Q8_0, eb.EB_BF16, m, 2048, 4096) != eb.EB_PATH_MFMA_I8
        # no workspace: refused before anything runs
        assert L.eb_qlinear_fused_ws(ctypes.byref(op), eb.EB_PATH_MFMA_I8, None, 0, None) == \
            eb.EB_ERR_UNSUPPORTED
    q6 = eb.eb_qlinear_op(_w(eb, eb.EB_Q6_S, n=2048, k=4096, data=1 * GB), 8 * GB, 9 * GB, 100,
                          eb.EB_BF16, eb.EB_F32)
    assert L.eb_qlinear_fused_ws(ctypes.byref(q6), eb.EB_PATH_MFMA_I8, None, 0, None) == \
        eb.EB_ERR_UNSUPPORTED
    normed = eb.eb_qlinear_op(_w(eb, eb.EB_Q4_0, n=2048, k=4096, data=1 * GB), 8 * GB, 9 * GB, 100,
                              eb.EB_BF16, eb.EB_F32, eb.EB_PRO_RMSNORM, 0, G, None, 1e-5, 0)
    assert L.eb_qlinear_fused_ws(ctypes.byref(normed), eb.EB_PATH_MFMA_I8, None, 0, None) == \
        eb.EB_ERR_UNSUPPORTED
    assert L.eb_qlinear_ex(ctypes.byref(_w(eb)), X, eb.EB_F16, 4, Y, eb.EB_F32, 4, None) == \
        eb.EB_ERR_INVALID   # unknown path

