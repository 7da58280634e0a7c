"""GPU parity of the Q6_S (6-bit super-block) path through the C ABI.

Q6_S realises the 6-bit configuration the paper evaluates beside 8- and
4-bit (section 4, Table 3).  Bars as for the other formats: packed bytes
bit-exact with the oracle; every output within 2e-3 of the binary64 oracle,
normalised by sum_k |x||w_hat| (plus one rounding for a 16-bit output;
(2e-3 + 2^-8) on the tile kernel with bfloat16 x, m > 128, where w_hat is
rounded once to bfloat16); outputs whose bound is 0 exactly 0; stacks
bitwise equal to single calls.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import TOL_BF16, TOL_F32, TOL_TILE_BF16, assert_parity, bits16, oracle_reference
from tests.test_gpu_fused import Case, assert_fused

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _special_super_blocks():
    rng = np.random.default_rng(71)
    rows = [np.zeros(256), np.eye(1, 256, 0)[0], -np.eye(1, 256, 200)[0],
            np.array([((i % 16) - 8) * 2.0 ** -6 for i in range(256)])]
    x = np.zeros(256)
    e0 = 127 * 2.0 ** -10
    x[0] = -127 * 2.0 ** -5
    x[1], x[2], x[3] = 2.5 * e0, -2.5 * e0, 31.5 * e0
    x[16], x[32] = -2.5 * 2.0 ** -5, 2.5 * 2.0 ** -5
    rows.append(x)
    for scale in (0.02, 1.0, 1e-6, 1e-9, 300.0):
        rows.append(rng.standard_normal(256) * scale)
    x = rng.standard_normal(256) * 0.02
    x[16:32] = 0.0
    x[40], x[45] = 0.3, -0.3
    x[70] = 5.0
    rows.append(x)
    x = rng.standard_normal(256) * 0.02
    x[::16] *= 40.0
    rows.append(x)
    rows.append(np.repeat(rng.standard_normal(16), 16) * 0.05)
    return np.stack(rows).astype(np.float32)


def test_q6_packing_special_blocks_bit_exact(eb, oracle):
    w = _special_super_blocks()
    qw = eb.quantize(torch.from_numpy(w).to(DEV), "q6_s")
    got = eb.to_canonical(qw).cpu().numpy()
    ref = oracle.quantize(O.Q6_S, w)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("n,k", [(1, 256), (37, 768), (300, 2304), (64, 11008)])
def test_q6_packing_random_bit_exact(eb, oracle, n, k):
    w = W.normal((n, k), 500 + n + k, "cpu", 0.02)
    qw = eb.quantize(w.to(DEV), "q6_s")
    got = eb.to_canonical(qw).cpu().numpy()
    ref = oracle.quantize(O.Q6_S, w.numpy(), nthreads=O.available_cores())
    assert np.array_equal(got, ref)
    # padding and gaps of the planar layout are zero
    L = eb.layout("q6_s", n, k)
    raw = qw.buf.cpu().numpy()
    d = raw[L.d_offset:L.d_offset + 2 * n * L.d_stride].view(np.uint16).reshape(n, L.d_stride)
    assert np.all(d[:, k // 256:] == 0)
    assert np.all(raw[n * L.qs_row_bytes:L.sc_offset] == 0)
    assert np.all(raw[L.sc_offset + n * L.sc_stride:L.d_offset] == 0)


def test_q6_canonical_round_trip(eb, oracle):
    n, k = 129, 1280
    w = W.normal((n, k), 77, "cpu", 0.02).numpy()
    ref = oracle.quantize(O.Q6_S, w)
    qw = eb.from_canonical(torch.from_numpy(ref).to(DEV), "q6_s", n, k)
    assert np.array_equal(eb.to_canonical(qw).cpu().numpy(), ref)
    qw2 = eb.quantize(torch.from_numpy(w).to(DEV), "q6_s")
    assert torch.equal(qw.buf, qw2.buf)


MS = [1, 3, 8, 16, 17, 33, 64, 65, 130]


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("n,k", [(37, 768), (515, 2304), (130, 256)])
def test_q6_qlinear_parity(eb, oracle, xdtype, n, k):
    """Every m-block count (1, 2, 4 rows of 16 and several 64-row tiles; 130
    rows take the tile kernel), ragged n, k of 1, 3 and 9 super-blocks
    (uneven shares of k over the eight waves), fp32 and bfloat16 outputs."""
    w = W.normal((n, k), 600 + n, "cpu", W.WEIGHT_STD)
    x = W.normal((max(MS), k), 601 + n, "cpu").to(xdtype)
    qw = eb.quantize(w.to(DEV), "q6_s")
    _, y_ref, bound = oracle_reference(oracle, "q6_s", w.numpy(), x)
    tile = TOL_TILE_BF16 if xdtype == torch.bfloat16 else TOL_F32
    for m in MS:
        y = eb.qlinear(qw, x[:m].to(DEV))
        assert_parity(y, y_ref[:m], bound[:m], tile if m > 128 else TOL_F32, f"q6 m={m} n={n} k={k}")
    y = eb.qlinear(qw, x.to(DEV), out_dtype=torch.bfloat16)
    assert_parity(y, y_ref, bound, tile + TOL_BF16 - TOL_F32, "q6 bf16 out")


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_q6_every_tile_and_split(eb, oracle, xdtype):
    """m > 128 runs on the tile kernel: every tile shape, unsplit and k split
    3 ways, on ragged m and n with 36 K-tiles (9 super-blocks); 70 rows keep
    the Q6_S kernel whatever tile is asked for."""
    m, n, k = 300, 520, 2304
    w = W.normal((n, k), 1900, "cpu", W.WEIGHT_STD)
    x = W.normal((m, k), 1901, "cpu").to(xdtype)
    qw = eb.quantize(w.to(DEV), "q6_s")
    _, y_ref, bound = oracle_reference(oracle, "q6_s", w.numpy(), x)
    xd = x.to(DEV)
    tol = TOL_TILE_BF16 if xdtype == torch.bfloat16 else TOL_F32
    for tile in range(eb.mfma_tile_count()):
        for splits in (1, 3):
            y = eb.qlinear_tuned(qw, xd, tile, splits)
            assert_parity(y, y_ref, bound, tol, f"q6 tile {tile} splits {splits}")
        y = eb.qlinear_tuned(qw, xd[:70], tile, 4, out_dtype=torch.bfloat16)
        assert_parity(y, y_ref[:70], bound[:70], TOL_BF16, f"q6 tile {tile} m=70 bf16 out")


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("kind", ["onehot", "sparse", "outlier"])
def test_q6_structured_activations(eb, oracle, xdtype, kind):
    """One-hot rows read single weights out (the rounding of w_hat to the
    activation type is the whole error), sparse rows and outlier channels
    (x 1000) at m = 1, m = 80 and m = 200 (the tile kernel: bfloat16 x then
    carries w_hat rounded once, the (2e-3 + 2^-8) bound)."""
    n, k = 256, 1536
    w = W.normal((n, k), 700, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), "q6_s")
    for m in (1, 80, 200):
        gen = {"onehot": W.onehot_rows, "sparse": W.sparse_rows, "outlier": W.outlier_rows}[kind]
        x = gen(m, k, 701 + m).to(xdtype)
        _, y_ref, bound = oracle_reference(oracle, "q6_s", w.numpy(), x)
        y = eb.qlinear(qw, x.to(DEV))
        tol = TOL_TILE_BF16 if (m > 128 and xdtype == torch.bfloat16) else TOL_F32
        assert_parity(y, y_ref, bound, tol, f"q6_{kind} m={m}")


FUSIONS = [("rmsnorm", None), (None, "add"), (None, "glu"), ("rmsnorm", "glu"), ("rmsnorm", "add")]


@pytest.mark.parametrize("pro,epi", FUSIONS)
@pytest.mark.parametrize("xdtype,ydtype", [(torch.float16, torch.float32),
                                           (torch.bfloat16, torch.bfloat16)])
def test_q6_fused_steps(eb, oracle, pro, epi, xdtype, ydtype):
    n, k = 198, 1280
    for m, splits in ((1, 0), (20, 0), (150, 0), (150, 3)):
        c = Case(eb, 1200 + m, "q6_s", n, k, m, xdtype, pro, epi, ydtype)
        y = c.run(eb, splits=splits)   # 150 rows: the tile kernel, k split 3 ways in the second run
        torch.cuda.synchronize()
        y_ref, scale = c.reference(oracle)
        assert_fused(y, y_ref, scale, f"q6_fused_{pro}_{epi} m={m} splits={splits}")


def test_q6_zero_weights_and_determinism(eb):
    qw = eb.quantize(torch.zeros((64, 512), device=DEV), "q6_s")
    x = W.normal((40, 512), 800, DEV).to(torch.bfloat16)
    assert torch.count_nonzero(eb.qlinear(qw, x)) == 0
    w = W.normal((300, 2048), 801, DEV, W.WEIGHT_STD)
    qw = eb.quantize(w, "q6_s")
    for m in (1, 50, 200):
        x = W.normal((m, 2048), 802 + m, DEV).to(torch.bfloat16)
        a, b = eb.qlinear(qw, x), eb.qlinear(qw, x)
        assert torch.equal(a, b), m


def test_q6_stack_matches_single_calls(eb, monkeypatch):
    """A layer of Q6_S projections with the fused steps as one stack, in
    capture, replay and direct modes: bitwise equal to the ops run one by one."""
    d, f, m = 512, 1536, 24
    ws = [W.normal(s, 900 + i, DEV, W.WEIGHT_STD) for i, s in
          enumerate(((3 * d, d), (d, d), (2 * f, d), (d, f)))]
    qws = [eb.quantize(w, "q6_s") for w in ws]
    h0 = W.normal((m, d), 905, DEV) * 2.0
    g1 = (1.0 + 0.1 * W.normal((d,), 906, DEV))
    g2 = (1.0 + 0.1 * W.normal((d,), 907, DEV))
    attn = W.normal((m, d), 908, DEV).to(torch.bfloat16)

    def run(h, qkv, act, stack):
        specs = [(qws[0], h, qkv, dict(x_dtype=torch.bfloat16, prologue="rmsnorm", norm_weight=g1, eps=1e-5)),
                 (qws[1], attn, h, dict(epilogue="add", residual=h)),
                 (qws[2], h, act, dict(x_dtype=torch.bfloat16, prologue="rmsnorm", norm_weight=g2,
                                       eps=1e-5, epilogue="glu")),
                 (qws[3], act, h, dict(epilogue="add", residual=h))]
        if stack:
            eb.qlinear_stack(eb.make_ops(specs))
        else:
            for qw, x, y, kw in specs:
                eb.qlinear_fused(qw, x, out=y, out_dtype=y.dtype, **kw)
        torch.cuda.synchronize()

    ref_h, ref_qkv = h0.clone(), torch.empty((m, 3 * d), dtype=torch.bfloat16, device=DEV)
    ref_act = torch.empty((m, f), dtype=torch.bfloat16, device=DEV)
    run(ref_h, ref_qkv, ref_act, False)
    for mode in ("1", "1", "0"):
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        h, qkv, act = h0.clone(), torch.empty_like(ref_qkv), torch.empty_like(ref_act)
        run(h, qkv, act, True)
        assert torch.equal(qkv, ref_qkv) and torch.equal(act, ref_act) and torch.equal(h, ref_h), mode
    eb.stack_cache_clear()


# m == 1: units of 64 weights, one per lane per slot; k from one slot to four,
# each with a ragged last slot (units past the row's end meet zero x) and full
M1_KS = [256, 4096, 4352, 8192, 11008, 12544, 16384]


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("k", M1_KS)
def test_q6_m1_every_slot_count(eb, oracle, xdtype, k):
    n = 77
    w = W.normal((n, k), 1300 + k, "cpu", W.WEIGHT_STD)
    qw = eb.quantize(w.to(DEV), "q6_s")
    for kind, x in (("normal", W.normal((1, k), 1301 + k, "cpu")),
                    ("outlier", W.outlier_rows(1, k, 1302 + k)),
                    ("onehot", W.onehot_rows(1, k, 1303 + k))):
        x = x.to(xdtype)
        _, y_ref, bound = oracle_reference(oracle, "q6_s", w.numpy(), x)
        y = eb.qlinear(qw, x.to(DEV))
        assert_parity(y, y_ref, bound, TOL_F32, f"q6 m=1 k={k} {kind}")


@pytest.mark.parametrize("pro,epi", FUSIONS)
@pytest.mark.parametrize("k", [4352, 11008])
def test_q6_m1_fused_steps_long_rows(eb, oracle, pro, epi, k):
    """The fused steps at two and three slots per lane (the gate/up product
    takes two rows per wave, which at three slots runs 8-wave workgroups)."""
    for xdtype, ydtype in ((torch.float16, torch.float32), (torch.bfloat16, torch.bfloat16)):
        c = Case(eb, 1400 + k, "q6_s", 130, k, 1, xdtype, pro, epi, ydtype)
        y = c.run(eb)
        torch.cuda.synchronize()
        y_ref, scale = c.reference(oracle)
        assert_fused(y, y_ref, scale, f"q6_m1_{pro}_{epi} k={k} {xdtype}")


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_q6_m1_fused_launch_matches_single_calls(eb, oracle, xdtype, monkeypatch):
    """Independent m == 1 projections of several slot counts (k = 1024, 4096,
    4352, 11008) with every fused step share fused launches in a stack:
    bitwise equal to single calls, and each within the oracle's bar."""
    shapes = [(3 * 512, 4096, "rmsnorm", None), (4096, 4096, None, "add"), (2 * 600, 4352, "rmsnorm", "glu"),
              (4096, 11008, None, "add"), (1030, 1024, None, None), (96, 11008, "rmsnorm", None)]
    cases = [Case(eb, 1500 + i, "q6_s", n, k, 1, xdtype, pro, epi, torch.float32)
             for i, (n, k, pro, epi) in enumerate(shapes)]
    singles = [c.run(eb) for c in cases]
    torch.cuda.synchronize()
    for c, y in zip(cases, singles):
        y_ref, scale = c.reference(oracle)
        assert_fused(y, y_ref, scale, f"q6_m1 fused {c.n}x{c.k} {c.pro} {c.epi}")
    outs = [torch.empty_like(y) for y in singles]
    specs = []
    for c, o in zip(cases, outs):
        kw = dict(x_dtype=c.xdtype, epilogue=c.epi)
        if c.pro:
            kw.update(prologue="rmsnorm", norm_weight=c.gd, eps=1e-5)
        if c.epi == "add":
            kw.update(residual=c.rd)
        specs.append((c.qw, c.xd, o, kw))
    ops = eb.make_ops(specs)
    assert eb.stack_launches(ops) == 3   # slot counts 1, 2 and 3
    for mode in ("1", "1", "0"):
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        for o in outs:
            o.fill_(float("nan"))
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        for y, o in zip(singles, outs):
            assert torch.equal(y, o), mode
    eb.stack_cache_clear()


def _extreme_q6_weights(n, k, seed):
    """N(0, 0.02) rows whose super-blocks are rescaled: every third to
    max |w| = 60000, every fifth to about 1e-6 (a binary16-subnormal or zero
    super-scale), and inside every other super-block one sub-block 100x
    smaller than the rest (sub-scales far below the super-scale)."""
    w = W.normal((n, k), seed, "cpu", W.WEIGHT_STD).view(n, k // 256, 256)
    amax = w.abs().amax(dim=2, keepdim=True).clamp_min(1e-30)
    ns = k // 256
    big = torch.zeros(ns, dtype=torch.bool)
    big[0::3] = True
    tiny = torch.zeros(ns, dtype=torch.bool)
    tiny[1::5] = True
    w = torch.where(big.view(1, ns, 1), w / amax * 60000.0, w)
    w = torch.where(tiny.view(1, ns, 1), w / amax * 1e-6, w)
    w[:, 0::2, 32:48] *= 0.01
    return w.reshape(n, k).contiguous()


@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_q6_extreme_scales_every_path(eb, oracle, xdtype, monkeypatch):
    """Super-blocks with max |w| from 1e-6 to 60000 in one row and sub-blocks
    far below their super-scale, on every Q6_S path: the m = 1 GEMV (lone and
    in a fused launch), the m <= 8 GEMV, the Q6_S matrix-core kernel and the
    tile kernel (binary16 x: w_hat rounded to binary16 adds 2^-25 sum_k |x|;
    bfloat16 x: the tile bound)."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    n, k = 200, 2560
    w = _extreme_q6_weights(n, k, 2000 + (xdtype == torch.bfloat16))
    x = W.normal((300, k), 2010, "cpu").to(xdtype)
    qw = eb.quantize(w.to(DEV), "q6_s")
    _, y_ref, bound = oracle_reference(oracle, "q6_s", w.numpy(), x)
    xd = x.to(DEV)
    sum_abs_x = x.double().abs().sum(dim=1, keepdim=True).numpy()
    f16 = xdtype == torch.float16
    for m in (1, 4):
        y = eb.qlinear(qw, xd[:m], path="gemv")
        assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"q6_scale_gemv m={m}")
    for m in (50, 300):
        y = eb.qlinear(qw, xd[:m], path="mfma")
        tol = TOL_TILE_BF16 if (m > 128 and not f16) else TOL_F32
        assert_parity(y, y_ref[:m], bound[:m], tol, f"q6_scale_mfma m={m}",
                      slack=2.0 ** -25 * sum_abs_x[:m] if f16 else None)
    # two independent m = 1 ops in one fused launch
    ya = torch.full((1, n), float("nan"), device=DEV)
    yb = torch.full((1, n), float("nan"), device=DEV)
    ops = eb.make_ops([(qw, xd[:1], ya), (qw, xd[1:2], yb)])
    assert eb.stack_launches(ops) == 1
    eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    assert_parity(ya, y_ref[:1], bound[:1], TOL_F32, "q6_scale_fused m=1")
    assert_parity(yb, y_ref[1:2], bound[1:2], TOL_F32, "q6_scale_fused m=1 (op 2)")
    eb.stack_cache_clear()
