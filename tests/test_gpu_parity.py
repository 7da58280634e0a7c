"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: packed weights bit-exact; every output within 2e-3 of the binary64
oracle, normalised by sum_k |x||w_hat| (plus one bf16 rounding for bf16
outputs); outputs whose bound is 0 are exactly 0.
"""
import os

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2607_02501_amd import workloads as W
from tests.gpu_helpers import TOL_BF16, TOL_F32, TOL_TILE_BF16, assert_parity, bits16, oracle_reference

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _case(seed, n, k, m, xdtype, wscale=W.WEIGHT_STD):
    w = W.normal((n, k), seed, "cpu", wscale)
    x = W.normal((m, k), seed + 1, "cpu").to(xdtype)
    return w, x


# ---------------------------------------------------------------------------
# Packing
# ---------------------------------------------------------------------------

def _special_blocks():
    rng = np.random.default_rng(21)
    rows = []
    z = np.zeros(32, np.float32)
    rows.append(z)
    e = z.copy(); e[0] = 1.0; rows.append(e)
    e = z.copy(); e[17] = 1.0; rows.append(e)
    rows.append(-rows[1])
    t = z.copy(); t[0] = 127 * 2.0 ** -7; t[1] = 2.5 * 2.0 ** -7; t[2] = -2.5 * 2.0 ** -7; rows.append(t)
    t = z.copy(); t[0] = -1.0; t[1] = 0.3125; t[2] = -0.3125; t[3] = 0.99; rows.append(t)
    t = z.copy(); t[0], t[5] = 1.0, -1.0; rows.append(t)
    rows.append(rng.standard_normal(32).astype(np.float32) * np.float32(1e-6))
    rows.append(rng.standard_normal(32).astype(np.float32) * np.float32(2e-5))
    rows.append(rng.standard_normal(32).astype(np.float32) * np.float32(1000))
    rows.append((np.arange(32, dtype=np.float32) - 16) * np.float32(0.0625))
    return np.stack(rows).reshape(-1, 32)


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_packing_special_blocks_bit_exact(eb, oracle, qtype):
    w = _special_blocks()
    qw = eb.quantize(torch.from_numpy(w).to(DEV), qtype)
    got = eb.to_canonical(qw).cpu().numpy()
    ref = oracle.quantize(O.Q8_0 if qtype == "q8_0" else O.Q4_0, w)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("n,k", [(1, 32), (37, 96), (300, 1056), (64, 11008)])
def test_packing_random_bit_exact(eb, oracle, qtype, n, k):
    w = W.normal((n, k), 100 + n + k, "cpu", 0.02)
    qw = eb.quantize(w.to(DEV), qtype)
    got = eb.to_canonical(qw).cpu().numpy()
    ref = oracle.quantize(O.Q8_0 if qtype == "q8_0" else O.Q4_0, w.numpy())
    assert np.array_equal(got, ref)
    # the planar scale-plane padding is zero
    L = eb.layout(qtype, n, k)
    raw = qw.buf.cpu().numpy()
    d = raw[L.d_offset:L.d_offset + 2 * n * L.d_stride].view(np.uint16).reshape(n, L.d_stride)
    assert np.all(d[:, k // 32:] == 0)


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_from_canonical_round_trip(eb, oracle, qtype):
    n, k = 129, 352
    w = W.normal((n, k), 5, "cpu", 0.02).numpy()
    ref = oracle.quantize(O.Q8_0 if qtype == "q8_0" else O.Q4_0, w)
    qw = eb.from_canonical(torch.from_numpy(ref).to(DEV), qtype, n, k)
    assert np.array_equal(eb.to_canonical(qw).cpu().numpy(), ref)
    qw2 = eb.quantize(torch.from_numpy(w).to(DEV), qtype)
    assert torch.equal(qw.buf, qw2.buf)


# ---------------------------------------------------------------------------
# qlinear on small ragged shapes, every path
# ---------------------------------------------------------------------------

SHAPES = [(37, 96), (515, 1056), (130, 2080)]
MS_GEMV = [1, 2, 3, 4, 5, 8]
MS_MFMA = [1, 5, 9, 50, 64, 65, 130]


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("n,k", SHAPES)
def test_qlinear_gemv_parity(eb, oracle, qtype, xdtype, n, k):
    w, x = _case(1000 + n, n, k, max(MS_GEMV), xdtype)
    qw = eb.quantize(w.to(DEV), qtype)
    _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
    for m in MS_GEMV:
        y = eb.qlinear(qw, x[:m].to(DEV), path="gemv")
        assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"gemv m={m}")
    y = eb.qlinear(qw, x[:1].to(DEV), out_dtype=torch.bfloat16, path="gemv")
    assert_parity(y, y_ref[:1], bound[:1], TOL_BF16, "gemv bf16 out")


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("n,k", SHAPES)
def test_qlinear_mfma_parity(eb, oracle, qtype, xdtype, n, k):
    w, x = _case(2000 + n, n, k, max(MS_MFMA), xdtype)
    qw = eb.quantize(w.to(DEV), qtype)
    _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
    for m in MS_MFMA:
        y = eb.qlinear(qw, x[:m].to(DEV), path="mfma")
        assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"mfma m={m}")
    y = eb.qlinear(qw, x.to(DEV), out_dtype=torch.bfloat16, path="mfma")
    assert_parity(y, y_ref, bound, TOL_BF16, "mfma bf16 out")


@pytest.mark.parametrize("qtype,xdtype", [("q8_0", torch.bfloat16), ("q4_0", torch.float16)])
def test_narrow_kernel_edges(eb, oracle, qtype, xdtype):
    """Lone small-m MFMA projections at the edges of the narrow kernel: every
    count of 16-row blocks of m (1, 2, 4) and the m just past each, a ragged
    last group of 16 weight rows, k at its limit (2048 = 64 blocks over 8
    waves) and one block past it (the tiled kernel with a split of k), and an
    uneven share of k between the waves (k = 11 blocks)."""
    n = 1000 + 3
    for k in (352, 2048, 2080):
        w, x = _case(3000 + k, n, k, 64, xdtype)
        qw = eb.quantize(w.to(DEV), qtype)
        _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
        for m in (1, 16, 17, 32, 33, 63, 64):
            y = eb.qlinear(qw, x[:m].to(DEV), path="mfma")
            assert_parity(y, y_ref[:m], bound[:m], TOL_F32, f"narrow m={m} k={k}")
        y = eb.qlinear(qw, x[:40].to(DEV), out_dtype=torch.bfloat16, path="mfma")
        assert_parity(y, y_ref[:40], bound[:40], TOL_BF16, f"narrow bf16 out k={k}")


@pytest.mark.parametrize("qtype,xdtype", [("q8_0", torch.bfloat16), ("q4_0", torch.float16),
                                          ("q4_0", torch.bfloat16)])
def test_every_mfma_tile_and_split(eb, oracle, qtype, xdtype):
    # ragged m and n for every tile shape, an odd block count (K tail), 33 K-tiles
    m, n, k = 300, 520, 2080
    w, x = _case(77, n, k, m, xdtype)
    qw = eb.quantize(w.to(DEV), qtype)
    _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
    xd = x.to(DEV)
    tol = TOL_TILE_BF16 if xdtype == torch.bfloat16 else TOL_F32
    for tile in range(eb.mfma_tile_count()):
        for splits in (1, 3):
            y = eb.qlinear_tuned(qw, xd, tile, splits)
            assert_parity(y, y_ref, bound, tol, f"tile {tile} splits {splits}")
        # m = 70: bfloat16 activations take the hi/lo tiles (the forced tile
        # applies where it has them)
        y = eb.qlinear_tuned(qw, xd[:70], tile, 4, out_dtype=torch.bfloat16)
        assert_parity(y, y_ref[:70], bound[:70], TOL_BF16, f"tile {tile} splits 4 bf16 out")


def test_split_k_deterministic_and_matches_unsplit(eb):
    n, k = 384, 8192
    w, x = _case(43, n, k, 96, torch.bfloat16)
    qw = eb.quantize(w.to(DEV), "q8_0")
    xd = x.to(DEV)
    whole = eb.qlinear_tuned(qw, xd, 1, 1)
    a = eb.qlinear_tuned(qw, xd, 1, 6)
    b = eb.qlinear_tuned(qw, xd, 1, 6)
    assert torch.equal(a, b)
    # same products, summed in another order: close, not necessarily equal
    scale = (x.float().abs() @ w.abs().t()).to(DEV)
    assert float(((a - whole).abs() / scale).max()) < 1e-4


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_qlinear_auto_matches_forced_path(eb, qtype):
    n, k = 300, 1024
    w, x = _case(7, n, k, 70, torch.bfloat16)
    qw = eb.quantize(w.to(DEV), qtype)
    xd = x.to(DEV)
    for m in (1, 4, 5, 70):
        want = eb.auto_path(qtype, torch.bfloat16, m, n, k)
        assert torch.equal(eb.qlinear(qw, xd[:m]), eb.qlinear(qw, xd[:m], path=want))


# ---------------------------------------------------------------------------
# Closed forms and invariants
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_onehot_reads_out_weights(eb, oracle, qtype, xdtype):
    n, k = 96, 128
    w = W.normal((n, k), 31, "cpu", 0.02)
    qw = eb.quantize(w.to(DEV), qtype)
    blocks = oracle.quantize(O.Q8_0 if qtype == "q8_0" else O.Q4_0, w.numpy())
    what = oracle.dequant(O.Q8_0 if qtype == "q8_0" else O.Q4_0, blocks, n, k)  # [n, k] float64
    eye = torch.eye(k, dtype=xdtype, device=DEV)
    # GEMV path: exact w_hat (code * d16 is exact in fp32)
    for j in range(0, k, 4):
        y = eb.qlinear(qw, eye[j:j + 4], path="gemv").double().cpu().numpy()
        assert np.array_equal(y, what[:, j:j + 4].T)
    # MFMA path (m = k = 128): each output is one product, so the bar applies
    # to w_hat itself -- binary16 holds it to 2^-11, bfloat16 hi/lo pairs to 2^-16
    y = eb.qlinear(qw, eye, path="mfma")
    assert_parity(y, what.T.copy(), np.abs(what.T), TOL_F32, f"onehot_mfma {qtype} {xdtype}")


def test_zero_weights_give_exact_zero(eb):
    n, k = 70, 256
    qw = eb.quantize(torch.zeros((n, k), device=DEV), "q4_0")
    x = torch.randn(9, k, device=DEV).to(torch.float16)
    for path, m in (("gemv", 3), ("mfma", 9)):
        y = eb.qlinear(qw, x[:m], path=path)
        assert torch.count_nonzero(y) == 0


@pytest.mark.parametrize("path,m", [("gemv", 1), ("gemv", 4), ("mfma", 50), ("mfma", 200)])
def test_deterministic(eb, path, m):
    n, k = 1000, 2048
    w, x = _case(41, n, k, m, torch.bfloat16)
    qw = eb.quantize(w.to(DEV), "q8_0")
    xd = x.to(DEV)
    a = eb.qlinear(qw, xd, path=path)
    b = eb.qlinear(qw, xd, path=path)
    assert torch.equal(a, b)


def test_minimum_and_empty_shapes(eb, oracle):
    w, x = _case(3, 1, 32, 4, torch.float16)
    for qtype in ("q8_0", "q4_0"):
        qw = eb.quantize(w.to(DEV), qtype)
        _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
        for path, m in (("gemv", 1), ("gemv", 4), ("mfma", 4)):
            assert_parity(eb.qlinear(qw, x[:m].to(DEV), path=path), y_ref[:m], bound[:m], TOL_F32)
        y = eb.qlinear(qw, x[:0].to(DEV))
        assert y.shape == (0, 1)


# ---------------------------------------------------------------------------
# Stack: graph replay and direct launches give the single-call results
# ---------------------------------------------------------------------------

def test_stack_matches_single_calls(eb, monkeypatch):
    shapes = [("q4_0", torch.float16, 1, 300, 512), ("q8_0", torch.bfloat16, 50, 200, 1024),
              ("q4_0", torch.bfloat16, 130, 260, 352), ("q8_0", torch.float16, 3, 96, 4096),
              ("q8_0", torch.bfloat16, 64, 256, 8192), ("q4_0", torch.bfloat16, 100, 192, 6144)]
    entries, refs = [], []
    for i, (qt, xdt, m, n, k) in enumerate(shapes):
        w, x = _case(500 + i, n, k, m, xdt)
        qw = eb.quantize(w.to(DEV), qt)
        xd = x.to(DEV)
        y = torch.full((m, n), float("nan"), device=DEV)
        entries.append((qw, xd, y))
        refs.append(eb.qlinear(qw, xd))
    ops = eb.make_ops(entries)
    for mode in ("1", "1", "0"):  # capture, replay, direct
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        for _, _, y in entries:
            y.fill_(float("nan"))
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        for (_, _, y), r in zip(entries, refs):
            assert torch.equal(y, r)
    eb.stack_cache_clear()


@pytest.mark.parametrize("qtype", ["q4_0", "q8_0"])
@pytest.mark.parametrize("xdtype", [torch.float16, torch.bfloat16])
def test_fused_decode_stack_matches_single_calls(eb, qtype, xdtype, monkeypatch):
    """Independent m == 1 ops of several K classes run as fused launches and
    give bitwise the same outputs as one call per op."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    shapes = [(512, 300), (4096, 1000), (1024, 64), (11008 if qtype == "q4_0" else 6144, 257),
              (4096, 4097), (32, 5), (2048, 2048), (1024, 640)]
    entries, refs = [], []
    for i, (k, n) in enumerate(shapes):
        w, x = _case(800 + i, n, k, 1, xdtype)
        qw = eb.quantize(w.to(DEV), qtype)
        xd = x.to(DEV)
        y = torch.full((1, n), float("nan"), device=DEV, dtype=torch.bfloat16 if i % 3 == 2 else torch.float32)
        entries.append((qw, xd, y))
        refs.append(eb.qlinear(qw, xd, out_dtype=y.dtype))
    ops = eb.make_ops(entries)
    assert eb.stack_launches(ops) < len(shapes)
    for mode in ("1", "1", "0"):
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        for _, _, y in entries:
            y.fill_(float("nan"))
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        for (_, _, y), r in zip(entries, refs):
            assert torch.equal(y, r)
    eb.stack_cache_clear()


@pytest.mark.parametrize("qtype,xdtype,ydtype,ms", [
    ("q8_0", torch.bfloat16, torch.float32, (50, 64, 20, 50)),
    ("q4_0", torch.float16, torch.bfloat16, (100, 128, 70, 5)),
    ("q4_0", torch.bfloat16, torch.float32, (33, 1, 64, 9)),
    ("q8_0", torch.float16, torch.bfloat16, (64, 7, 128, 65)),
])
def test_fused_mfma_stack(eb, oracle, qtype, xdtype, ydtype, ms, monkeypatch):
    """Independent small-m MFMA ops run as one persistent launch (weights
    dequantized into MFMA registers): every output within the oracle bound,
    the same bits on every run and in every stack mode, and the single-call
    results up to summation order."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    shapes = [(300, 1056), (128, 96), (1000, 2080), (130, 4096)]  # odd block counts, ragged n
    entries, cases = [], []
    for i, ((n, k), m) in enumerate(zip(shapes, ms)):
        w, x = _case(900 + i, n, k, m, xdtype)
        qw = eb.quantize(w.to(DEV), qtype)
        y = torch.full((m, n), float("nan"), device=DEV, dtype=ydtype)
        entries.append((qw, x.to(DEV), y))
        cases.append((w, x))
    ops = eb.make_ops(entries)
    if min(ms) > 4:
        assert eb.stack_launches(ops) == 1
    first = None
    for mode in ("1", "1", "0"):  # capture, replay, direct
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        for _, _, y in entries:
            y.fill_(float("nan"))
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        outs = [y.clone() for _, _, y in entries]
        if first is None:
            first = outs
        for a, b in zip(first, outs):
            assert torch.equal(a, b)
    tol = TOL_F32 if ydtype == torch.float32 else TOL_BF16
    for (w, x), (qw, xd, y) in zip(cases, entries):
        _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
        assert_parity(y, y_ref, bound, tol, f"fused m={x.shape[0]}")
        single = eb.qlinear(qw, xd, out_dtype=ydtype)
        scale = torch.from_numpy(bound).to(DEV).float().clamp_min(1e-30)
        assert float(((y.float() - single.float()).abs() / scale).max()) <= 2 * tol
    eb.stack_cache_clear()


@pytest.mark.parametrize("qtype,xdtype,ms", [
    ("q8_0", torch.bfloat16, (129, 300, 257, 520)),
    ("q4_0", torch.float16, (816, 130, 200, 384)),
])
def test_grouped_mfma_stack(eb, oracle, qtype, xdtype, ms, monkeypatch):
    """Independent large-m MFMA ops run as one grouped launch of the tile
    kernel: every output within the oracle bound, the same bits on every run
    and in every stack mode, and the unsplit single-call results up to the
    order of summation over k (the two may use tile shapes that walk k in
    different orders)."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    monkeypatch.delenv("EB_STACK_GROUP", raising=False)
    shapes = [(300, 1056), (128, 96), (1000, 2080), (130, 4096)]  # odd block counts, ragged n
    ydt = [torch.float32, torch.bfloat16, torch.float32, torch.bfloat16]
    entries, cases = [], []
    for i, ((n, k), m) in enumerate(zip(shapes, ms)):
        w, x = _case(950 + i, n, k, m, xdtype)
        qw = eb.quantize(w.to(DEV), qtype)
        y = torch.full((m, n), float("nan"), device=DEV, dtype=ydt[i])
        entries.append((qw, x.to(DEV), y))
        cases.append((w, x))
    ops = eb.make_ops(entries)
    # one grouped launch, plus a fused small-m launch per output type for rows
    # split off mostly-padded last row tiles
    assert 1 <= eb.stack_launches(ops) <= 3
    first = None
    # capture, replay, direct; then the split-off rows after the grouped launch
    # instead of beside it on the second stream, recorded and direct
    for mode, overlap in (("1", "1"), ("1", "1"), ("0", "1"), ("1", "0"), ("0", "0")):
        monkeypatch.setenv("EB_STACK_GRAPH", mode)
        monkeypatch.setenv("EB_STACK_OVERLAP_TAIL", overlap)
        for _, _, y in entries:
            y.fill_(float("nan"))
        eb.qlinear_stack(ops)
        torch.cuda.synchronize()
        outs = [y.clone() for _, _, y in entries]
        if first is None:
            first = outs
        for a, b in zip(first, outs):
            assert torch.equal(a, b), (mode, overlap)
    monkeypatch.delenv("EB_STACK_OVERLAP_TAIL", raising=False)
    for (w, x), (qw, xd, y) in zip(cases, entries):
        tol = TOL_F32 if y.dtype == torch.float32 else TOL_BF16
        if xdtype == torch.bfloat16:
            tol += TOL_TILE_BF16 - TOL_F32
        _, y_ref, bound = oracle_reference(oracle, qtype, w.numpy(), x)
        assert_parity(y, y_ref, bound, tol, f"grouped m={x.shape[0]}")
        single = eb.qlinear_tuned(qw, xd, -1, 1, out_dtype=y.dtype)
        scale = torch.from_numpy(bound).to(DEV).float().clamp_min(1e-30)
        assert float(((y.float() - single.float()).abs() / scale).max()) <= 2 * tol
    eb.stack_cache_clear()


def test_stack_dependent_chain(eb, oracle, monkeypatch):
    """op 1 reads op 0's bf16 output: the plan must not fuse them."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    k0, n0, n1 = 1024, 512, 384
    w0, x0 = _case(900, n0, k0, 1, torch.bfloat16)
    w1, _ = _case(901, n1, n0, 1, torch.bfloat16)
    q0, q1 = eb.quantize(w0.to(DEV), "q4_0"), eb.quantize(w1.to(DEV), "q4_0")
    xd = x0.to(DEV)
    y0 = torch.empty((1, n0), dtype=torch.bfloat16, device=DEV)
    y1 = torch.empty((1, n1), dtype=torch.float32, device=DEV)
    ops = eb.make_ops([(q0, xd, y0), (q1, y0, y1)])
    assert eb.stack_launches(ops) == 2
    eb.qlinear_stack(ops)
    torch.cuda.synchronize()
    ref0 = eb.qlinear(q0, xd, out_dtype=torch.bfloat16)
    assert torch.equal(y0, ref0)
    _, y_ref, bound = oracle_reference(oracle, "q4_0", w1.numpy(), ref0)
    assert_parity(y1, y_ref, bound, TOL_F32, "chained op")
    eb.stack_cache_clear()


# ---------------------------------------------------------------------------
# Full-size workloads (the shapes the benchmark times), sampled outputs
# ---------------------------------------------------------------------------

def _sample_idx(total, count, rng, extra=()):
    base = {0, total - 1, *[e for e in extra if 0 <= e < total]}
    pool = rng.choice(total, size=min(total, count), replace=False)
    return np.array(sorted(base | set(int(v) for v in pool)), dtype=np.int64)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_sampled_parity(eb, oracle, name):
    wl = W.WORKLOADS[name]
    rng = np.random.default_rng(77)
    for layer in sorted({0, wl.layers - 1}):
        for p, (pname, k, n) in enumerate(wl.projections):
            print(f"[parity] {name} layer={layer} proj={pname} m={wl.m} n={n} k={k}", flush=True)
            w = W.weights(wl, layer, p, DEV)
            x = W.activations(wl, layer, p, DEV)
            qw = eb.quantize(w, wl.qtype)
            y = eb.qlinear(qw, x)                        # auto path, as timed by the benchmark
            cols = _sample_idx(n, 48, rng, extra=(127, 128, 255, 256))
            rows = _sample_idx(wl.m, 24, rng, extra=(63, 64, 127, 128))
            wrows = w[torch.from_numpy(cols).to(DEV)].cpu().numpy()
            blocks, y_ref, bound = oracle_reference(oracle, wl.qtype, wrows, x[torch.from_numpy(rows).to(DEV)])
            # packing of the sampled rows is bit-exact
            canon = eb.to_canonical(qw)[torch.from_numpy(cols).to(DEV)].cpu().numpy()
            assert np.array_equal(canon, blocks), f"{name} {pname}: packed bytes differ"
            got = y[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)]
            assert_parity(got, y_ref, bound, TOL_F32, f"{name} layer {layer} {pname}")
            del w, qw, y
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_stack_sampled_parity(eb, oracle, name, monkeypatch):
    """A whole pass of the workload through eb_qlinear_stack, in the launch
    configuration the benchmark times (fused launches, graph replay), checked
    on sampled outputs of the first and last layer (and step) of every
    projection."""
    monkeypatch.delenv("EB_STACK_FUSE", raising=False)
    monkeypatch.delenv("EB_STACK_GRAPH", raising=False)
    wl = W.WORKLOADS[name]
    rng = np.random.default_rng(78)
    qws, entries, where = {}, [], {}
    for layer in range(wl.layers):
        for p, (_, k, n) in enumerate(wl.projections):
            qws[layer, p] = eb.quantize(W.weights(wl, layer, p, DEV), wl.qtype)
    for step in range(wl.steps):
        for layer in range(wl.layers):
            for p, (_, k, n) in enumerate(wl.projections):
                x = W.activations(wl, layer, p, DEV, step=step)
                y = torch.full((wl.m, n), float("nan"), device=DEV)
                where[step, layer, p] = len(entries)
                entries.append((qws[layer, p], x, y))
    ops = eb.make_ops(entries)
    print(f"[parity] {name}: {len(entries)} ops in {eb.stack_launches(ops)} launches", flush=True)
    eb.qlinear_stack(ops)
    eb.qlinear_stack(ops)  # second call replays the cached graph
    torch.cuda.synchronize()
    for step in sorted({0, wl.steps - 1}):
        for layer in sorted({0, wl.layers - 1}):
            for p, (pname, k, n) in enumerate(wl.projections):
                qw, x, y = entries[where[step, layer, p]]
                cols = _sample_idx(n, 24, rng, extra=(127, 128, 255, 256))
                # tile edges, including the rows a grouped launch hands to a
                # fused small-m launch (m = 816: rows 768..815)
                rows = _sample_idx(wl.m, 12, rng, extra=(49, 63, 64, 255, 256, 767, 768, 769))
                wrows = W.weights(wl, layer, p, DEV, rows=torch.from_numpy(cols).to(DEV)).cpu().numpy()
                _, y_ref, bound = oracle_reference(oracle, wl.qtype, wrows,
                                                   x[torch.from_numpy(rows).to(DEV)])
                got = y[torch.from_numpy(rows).to(DEV)][:, torch.from_numpy(cols).to(DEV)]
                assert_parity(got, y_ref, bound, TOL_F32, f"{name} step {step} layer {layer} {pname}")
    del entries, qws, ops
    eb.stack_cache_clear()
    torch.cuda.empty_cache()
