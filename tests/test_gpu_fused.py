"""GPU parity of the fused decoder-layer steps around a projection (through the C ABI).

The steps (paper section 3.2, operator fusion) are the RMS-normalisation
prologue, the residual-addition epilogue and the SiLU-gated product of
interleaved gate/up rows.  Every output is compared with the oracle's
``fused_qlinear`` (binary64, the normalised activations rounded to the
activation type as the product consumes them) against its error scale S:
|y - y_ref| <= 2e-3 S + u_out (|y_ref| + 2e-3 S), u_out the unit roundoff of
the output type (2^-24 fp32, 2^-11 fp16, 2^-8 bf16); where S is 0 the output
must equal the oracle's exactly.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import QT, WORST, XT, bits16

pytestmark = pytest.mark.gpu

DEV = "cuda"
TAU = 2e-3
U_OUT = {torch.float32: 2.0 ** -24, torch.float16: 2.0 ** -11, torch.bfloat16: 2.0 ** -8}


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def assert_fused(y_gpu, y_ref, scale, what):
    y = y_gpu.detach().double().cpu().numpy()
    assert y.shape == y_ref.shape, (what, y.shape, y_ref.shape)
    assert np.all(np.isfinite(y)), what
    u = U_OUT[y_gpu.dtype]
    err = np.abs(y - y_ref)
    zero = scale == 0
    # exactly representable references (a residual passed through) stay exact
    assert np.all(err[zero] <= u * np.abs(y_ref[zero])), f"{what}: inexact where the scale is 0"
    allowed = TAU * scale + u * (np.abs(y_ref) + TAU * scale)
    bad = err > allowed
    assert not bad.any(), f"{what}: {int(bad.sum())} outputs out of bounds, worst excess " \
                          f"{float((err - allowed)[bad].max()):.3e}"
    if (~zero).any():
        worst = float((err[~zero] / scale[~zero]).max())
        label = what.split(" ")[0]
        WORST[label] = max(WORST.get(label, 0.0), worst)


class Case:
    """One projection with its inputs on the host and the device."""

    def __init__(self, eb, seed, qtype, n, k, m, xdtype, pro, epi, ydtype):
        self.qtype, self.n, self.k, self.m = qtype, n, k, m
        self.xdtype, self.pro, self.epi, self.ydtype = xdtype, pro, epi, ydtype
        self.w = W.normal((n, k), seed, "cpu", W.WEIGHT_STD)
        self.qw = eb.quantize(self.w.to(DEV), qtype)
        if pro == "rmsnorm":
            self.x = W.normal((m, k), seed + 1, "cpu") * 3.0  # the residual stream, fp32
            self.gamma = 1.0 + 0.25 * W.normal((k,), seed + 2, "cpu")
        else:
            self.x = W.normal((m, k), seed + 1, "cpu").to(xdtype)
            self.gamma = None
        self.n_out = n // 2 if epi == "glu" else n
        self.r = W.normal((m, n), seed + 3, "cpu").to(ydtype) if epi == "add" else None
        self.xd = self.x.to(DEV)
        self.gd = self.gamma.to(DEV) if self.gamma is not None else None
        self.rd = self.r.to(DEV) if self.r is not None else None

    def run(self, eb, path="auto", out=None, residual=None, splits=0):
        return eb.qlinear_fused(self.qw, self.xd, out_dtype=self.ydtype, x_dtype=self.xdtype,
                                prologue=self.pro, norm_weight=self.gd, eps=1e-5,
                                epilogue=self.epi, residual=self.rd if residual is None else residual,
                                path=path, out=out, splits=splits)

    def reference(self, orc, rows=None):
        blocks = orc.quantize(QT[self.qtype], self.w.numpy(), nthreads=O.available_cores())
        x = self.x.numpy() if self.pro == "rmsnorm" else bits16(self.x)
        r = self.r.double().numpy() if self.r is not None else None
        y, scale, _ = orc.fused_qlinear(QT[self.qtype], blocks, self.n, self.k, x, XT[self.xdtype],
                                        prologue=self.pro or "none",
                                        gamma=self.gamma.numpy() if self.gamma is not None else None,
                                        eps=1e-5, epilogue=self.epi or "none", residual=r, rows=rows,
                                        nthreads=O.available_cores())
        return y, scale


# ---------------------------------------------------------------------------
# single calls on both paths
# ---------------------------------------------------------------------------

FUSIONS = [("rmsnorm", None), (None, "add"), (None, "glu"), ("rmsnorm", "glu"), ("rmsnorm", "add")]


@pytest.mark.parametrize("pro,epi", FUSIONS)
@pytest.mark.parametrize("qtype,xdtype,ydtype", [
    ("q4_0", torch.float16, torch.float32), ("q8_0", torch.bfloat16, torch.bfloat16),
    ("q4_0", torch.bfloat16, torch.float16)])
def test_fused_single_calls(eb, oracle, pro, epi, qtype, xdtype, ydtype):
    """m = 1 (one-row GEMV kernel), m = 3 (general GEMV kernel), m = 20 and
    m = 150 (tiled MFMA kernel, with its own epilogue and with a split of k
    forced, whose reduction applies the epilogue), on a ragged shape: n = 198
    (99 gate/up pairs), k = 1184 (37 blocks)."""
    n, k = 198, 1184
    for m, path, splits in ((1, "gemv", 0), (3, "gemv", 0), (20, "mfma", 0), (150, "mfma", 1),
                            (150, "mfma", 4)):
        c = Case(eb, 1000 + m, qtype, n, k, m, xdtype, pro, epi, ydtype)
        y = c.run(eb, path, splits=splits)
        torch.cuda.synchronize()
        y_ref, scale = c.reference(oracle)
        assert_fused(y, y_ref, scale, f"fused_{pro}_{epi} {qtype} m={m} {path} splits={splits}")


def test_glu_on_long_rows_uses_paired_rows(eb, oracle):
    """m = 1 with k = 9216 (Q4_0: 288 units, one row per wave in the one-row
    kernel): the gate/up product runs on the general GEMV kernel instead."""
    c = Case(eb, 1100, "q4_0", 64, 9216, 1, torch.float16, "rmsnorm", "glu", torch.float16)
    y = c.run(eb, "gemv")
    torch.cuda.synchronize()
    y_ref, scale = c.reference(oracle)
    assert_fused(y, y_ref, scale, "fused_glu_long m=1")


@pytest.mark.parametrize("qtype", ["q4_0", "q8_0", "q6_s"])
@pytest.mark.parametrize("pro,epi", [(None, None), ("rmsnorm", "glu"), (None, "add")])
def test_m1_lone_launch_partial_last_round(eb, oracle, qtype, pro, epi):
    """Lone m = 1 launches with more row groups than waves (one 16-wave
    workgroup per compute unit, 4096 waves on 256 CUs): 9426 rows are two
    whole rounds of one-row groups and a partial third, or one whole round of
    gate/up pairs and a partial second; the partial round's groups are
    numbered differently from the whole rounds'.  k = 256: one unit slot per
    lane."""
    n, k = 9426, 256
    c = Case(eb, 1300, qtype, n, k, 1, torch.float16, pro, epi, torch.float32)
    y = c.run(eb, "gemv")
    torch.cuda.synchronize()
    y_ref, scale = c.reference(oracle)
    assert_fused(y, y_ref, scale, f"m1_lone_rounds {qtype} {pro} {epi}")


@pytest.mark.parametrize("qtype,k,pro,epi", [
    ("q4_0", 4096, "rmsnorm", "glu"),   # 2 slots x 2 rows: 4 items in flight
    ("q4_0", 8192, None, None),         # 4 slots: 4 items
    ("q4_0", 8192, None, "add"),
    ("q4_0", 11008, None, "add"),       # 6 slots: 3 items
    ("q4_0", 16384, "rmsnorm", None),   # 8 slots: 4 items
    ("q8_0", 2048, "rmsnorm", "glu"),   # 2 slots x 2 rows
    ("q8_0", 4096, None, "add"),        # 4 slots
    ("q8_0", 8192, None, None),         # 8 slots
])
def test_m1_lone_launch_item_rings(eb, oracle, qtype, k, pro, epi):
    """Lone m = 1 launches whose waves keep 3 or 4 items (1 KiB each) in flight
    (part of the first group requested before x is staged, the rest after),
    with more row groups than waves (4096 on 256 CUs), so that waves run the
    group loop more than once; residual-adding ops with fp32 output read each
    row's residual ahead of its weights."""
    n = 9000 if epi == "glu" else 4200
    c = Case(eb, 1400 + k // 32, qtype, n, k, 1, torch.float16, pro, epi, torch.float32)
    y = c.run(eb, "gemv")
    torch.cuda.synchronize()
    y_ref, scale = c.reference(oracle)
    assert_fused(y, y_ref, scale, f"m1_rings {qtype} k={k} {pro} {epi}")


def test_residual_in_place(eb, oracle):
    """residual == y: the residual stream is updated in place, on both paths
    (m = 150: the tile kernel's own epilogue, and with a split of k its
    reduction's)."""
    for m, path, splits in ((1, "gemv", 0), (3, "gemv", 0), (40, "mfma", 0), (150, "mfma", 1),
                            (150, "mfma", 3)):
        c = Case(eb, 1200 + m + splits, "q8_0", 256, 512, m, torch.bfloat16, None, "add", torch.float32)
        h = c.rd.clone()
        eb.qlinear_fused(c.qw, c.xd, out_dtype=torch.float32, epilogue="add", residual=h, out=h,
                         path=path, splits=splits)
        torch.cuda.synchronize()
        y_ref, scale = c.reference(oracle)
        assert_fused(h, y_ref, scale, f"fused_inplace m={m} {path} splits={splits}")


def test_zero_stream_and_zero_weights(eb):
    """Closed forms: a zero residual stream normalises to zero activations
    (eps > 0), so the product is exactly 0 and an added residual passes through
    unchanged; zero weights make the gate/up product exactly 0."""
    n, k = 128, 256
    qw = eb.quantize(W.normal((n, k), 1300, DEV, W.WEIGHT_STD), "q4_0")
    gamma = torch.ones(k, device=DEV)
    for m, path in ((1, "gemv"), (2, "gemv"), (70, "mfma")):
        h = torch.zeros((m, k), device=DEV)
        r = W.normal((m, n), 1301, DEV).to(torch.bfloat16)
        y = eb.qlinear_fused(qw, h, out_dtype=torch.bfloat16, x_dtype=torch.bfloat16,
                             prologue="rmsnorm", norm_weight=gamma, eps=1e-6, epilogue="add",
                             residual=r, path=path)
        torch.cuda.synchronize()
        assert torch.equal(y, r), (m, path)
    qz = eb.quantize(torch.zeros((n, k), device=DEV), "q8_0")
    for m, path in ((1, "gemv"), (70, "mfma")):
        x = W.normal((m, k), 1302, DEV).to(torch.float16)
        y = eb.qlinear_fused(qz, x, epilogue="glu", path=path)
        torch.cuda.synchronize()
        assert y.shape == (m, n // 2) and torch.count_nonzero(y) == 0


# ---------------------------------------------------------------------------
# stacks: a dependent decoder-layer chain and fused runs of independent ops
# ---------------------------------------------------------------------------

def _layer_chain(eb, seed, qtype, xdtype, m, d, f):
    """One decoder layer: normalised QKV, O adding into h (attention itself is
    outside the path: its output is a seeded input), normalised gate/up with
    the gated product, down adding into h."""
    h = W.normal((m, d), seed, DEV) * 2.0
    attn = W.normal((m, d), seed + 1, DEV).to(xdtype)
    g1 = 1.0 + 0.2 * W.normal((d,), seed + 2, DEV)
    g2 = 1.0 + 0.2 * W.normal((d,), seed + 3, DEV)
    ws = [W.normal((n, k), seed + 10 + i, "cpu", W.WEIGHT_STD)
          for i, (n, k) in enumerate(((3 * d, d), (d, d), (2 * f, d), (d, f)))]
    qws = [eb.quantize(w.to(DEV), qtype) for w in ws]
    qkv = torch.empty((m, 3 * d), device=DEV, dtype=xdtype)
    act = torch.empty((m, f), device=DEV, dtype=xdtype)
    ops = eb.make_ops([
        (qws[0], h, qkv, dict(x_dtype=xdtype, prologue="rmsnorm", norm_weight=g1, eps=1e-5)),
        (qws[1], attn, h, dict(epilogue="add", residual=h)),
        (qws[2], h, act, dict(x_dtype=xdtype, prologue="rmsnorm", norm_weight=g2, eps=1e-5,
                               epilogue="glu")),
        (qws[3], act, h, dict(epilogue="add", residual=h)),
    ])
    # the op table holds raw pointers: keep every buffer it names alive
    return dict(h=h, attn=attn, g1=g1, g2=g2, ws=ws, qws=qws, qkv=qkv, act=act, ops=ops)


def _chain_reference(orc, L, qtype, xdtype, h0):
    """Step by step on the oracle, feeding each step the GPU's own intermediate
    (qkv, the activations) rounded as the GPU stored them."""
    q = QT[qtype]
    d = h0.shape[1]
    blocks = [orc.quantize(q, w.numpy(), nthreads=O.available_cores()) for w in L["ws"]]
    nth = O.available_cores()
    qkv_ref, s_qkv, _ = orc.fused_qlinear(q, blocks[0], 3 * d, d, h0, XT[xdtype], prologue="rmsnorm",
                                          gamma=L["g1"].cpu().numpy(), eps=1e-5, nthreads=nth)
    h1_ref, s_h1, _ = orc.fused_qlinear(q, blocks[1], d, d, bits16(L["attn"]), XT[xdtype],
                                        epilogue="add", residual=h0.astype(np.float64), nthreads=nth)
    return blocks, (qkv_ref, s_qkv), (h1_ref, s_h1)


@pytest.mark.parametrize("qtype,xdtype,m,d,f", [("q4_0", torch.float16, 1, 512, 704),
                                                ("q8_0", torch.bfloat16, 50, 512, 704),
                                                ("q4_0", torch.bfloat16, 100, 512, 704),
                                                ("q8_0", torch.bfloat16, 300, 512, 704),
                                                ("q8_0", torch.bfloat16, 50, 1024, 4096),
                                                ("q4_0", torch.float16, 50, 1024, 4096),
                                                ("q8_0", torch.bfloat16, 40, 2048, 1024),
                                                ("q8_0", torch.bfloat16, 100, 1024, 4096),
                                                ("q4_0", torch.bfloat16, 100, 3072, 1024),
                                                ("q8_0", torch.bfloat16, 72, 5120, 1024),
                                                ("q6_s", torch.float16, 1, 512, 768),
                                                ("q6_s", torch.bfloat16, 50, 512, 768),
                                                ("q6_s", torch.bfloat16, 300, 512, 768),
                                                ("q6_s", torch.float16, 200, 1024, 2048)])
def test_decoder_layer_chain(eb, oracle, qtype, xdtype, m, d, f, monkeypatch):
    """The four projections of a layer as one stack: results equal the ops run
    one by one through eb_qlinear_fused, bit for bit (with and without the
    gate/up normalisation fused into the split O projection's reduction, which
    the layers whose O projection is split get: rows of 1024, 3072 -- a
    partial last chunk of the register-held row -- and 5120 outputs, past the
    register form; at m <= 64 O is split when its 16-row workgroups would not
    fill the GPU), and each step is
    within the oracle bound given its (GPU) inputs."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    L = _layer_chain(eb, 1400 + m, qtype, xdtype, m, d, f)
    h0 = L["h"].clone()
    # reference run: the same ops one at a time
    ref_h = h0.clone()
    ref_qkv = torch.empty_like(L["qkv"])
    ref_act = torch.empty_like(L["act"])
    qws = L["qws"]
    eb.qlinear_fused(qws[0], ref_h, out_dtype=xdtype, x_dtype=xdtype, prologue="rmsnorm",
                     norm_weight=L["g1"], eps=1e-5, out=ref_qkv)
    eb.qlinear_fused(qws[1], L["attn"], epilogue="add", residual=ref_h, out=ref_h)
    h1_gpu = ref_h.clone()
    eb.qlinear_fused(qws[2], ref_h, out_dtype=xdtype, x_dtype=xdtype, prologue="rmsnorm",
                     norm_weight=L["g2"], eps=1e-5, epilogue="glu", out=ref_act)
    eb.qlinear_fused(qws[3], ref_act, epilogue="add", residual=ref_h, out=ref_h)
    # the stack, in every mode
    counts = {}
    for fuse_norm in ("1", "0"):
        monkeypatch.setenv("EB_STACK_FUSE_NORM", fuse_norm)
        eb.stack_cache_clear()
        counts[fuse_norm] = eb.stack_launches(L["ops"])
        for mode in ("1", "1", "0"):
            monkeypatch.setenv("EB_STACK_GRAPH", mode)
            L["h"].copy_(h0)
            eb.qlinear_stack(L["ops"])
            torch.cuda.synchronize()
            assert torch.equal(L["qkv"], ref_qkv), (fuse_norm, mode)
            assert torch.equal(L["act"], ref_act), (fuse_norm, mode)
            assert torch.equal(L["h"], ref_h), (fuse_norm, mode)
    eb.stack_cache_clear()
    # when O is split along k (a single O op takes two launches), its
    # reduction normalises for gate/up: one launch fewer
    o_split = eb.stack_launches(eb.make_ops([(L["qws"][1], L["attn"], L["h"],
                                              dict(epilogue="add", residual=L["h"]))])) == 2
    assert counts["1"] == counts["0"] - (1 if o_split else 0), (counts, o_split)
    # each step against the oracle
    hn = h0.cpu().numpy()
    blocks, (qkv_ref, s_qkv), (h1_ref, s_h1) = _chain_reference(oracle, L, qtype, xdtype, hn)
    assert_fused(ref_qkv, qkv_ref, s_qkv, f"chain_qkv m={m}")
    assert_fused(h1_gpu, h1_ref, s_h1, f"chain_o m={m}")
    h1 = h1_gpu.cpu().numpy()
    act_ref, s_act, _ = oracle.fused_qlinear(QT[qtype], blocks[2], 2 * f, d, h1, XT[xdtype],
                                             prologue="rmsnorm", gamma=L["g2"].cpu().numpy(),
                                             eps=1e-5, epilogue="glu", nthreads=O.available_cores())
    assert_fused(ref_act, act_ref, s_act, f"chain_glu m={m}")
    h2_ref, s_h2, _ = oracle.fused_qlinear(QT[qtype], blocks[3], d, f, bits16(ref_act), XT[xdtype],
                                           epilogue="add", residual=h1.astype(np.float64),
                                           nthreads=O.available_cores())
    assert_fused(ref_h, h2_ref, s_h2, f"chain_down m={m}")


@pytest.mark.parametrize("qtype,xdtype,m", [("q4_0", torch.float16, 1), ("q8_0", torch.bfloat16, 40),
                                            ("q4_0", torch.bfloat16, 96), ("q8_0", torch.bfloat16, 260)])
def test_fused_runs_with_steps(eb, oracle, qtype, xdtype, m, monkeypatch):
    """Independent ops with fused steps share one launch (GEMV at m = 1, the
    small-m MFMA kernels at m = 40 / 96, the grouped tile kernel at m = 260):
    two normalised projections of one stream (one with the gated product)
    and two residual additions into separate streams."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    monkeypatch.delenv("EB_STACK_GROUP", raising=False)
    d = 1024
    # ordered so that ops with fp32 and with 16-bit outputs form two runs
    cases = [Case(eb, 1500, qtype, 768, d, m, xdtype, "rmsnorm", None, torch.float32),
             Case(eb, 1520, qtype, 512, d, m, xdtype, None, "add", torch.float32),
             Case(eb, 1510, qtype, 1280, d, m, xdtype, "rmsnorm", "glu", torch.bfloat16),
             Case(eb, 1530, qtype, 384, d, m, xdtype, None, "add", torch.bfloat16)]
    cases[2].x, cases[2].xd = cases[0].x, cases[0].xd  # both normalise the same stream
    outs = [torch.full((m, c.n_out), float("nan"), device=DEV, dtype=c.ydtype) for c in cases]
    entries = []
    for c, y in zip(cases, outs):
        kw = dict(x_dtype=c.xdtype, prologue=c.pro, norm_weight=c.gd, eps=1e-5, epilogue=c.epi,
                  residual=c.rd)
        entries.append((c.qw, c.xd, y, kw))
    ops = eb.make_ops(entries)
    launches = eb.stack_launches(ops)
    # m = 1: one GEMV launch; m <= 128: a row kernel per prologue and one
    # launch per run; m = 260: the row kernels, one grouped launch and at most
    # one small-m launch per output size for split-off last rows
    assert launches == (1 if m == 1 else 4) if m <= 128 else launches <= 5, launches
    eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    for c, y in zip(cases, outs):
        y_ref, scale = c.reference(oracle)
        assert_fused(y, y_ref, scale, f"fused_run_{c.pro}_{c.epi} m={m}")
    eb.stack_cache_clear()
