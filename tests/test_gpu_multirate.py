"""Multi-rate execution (paper section 3.2, modular multi-rate execution):
control ticks over a backbone module refreshed every R ticks and an action
expert module run every tick for several denoising steps, through the C ABI.

Bar: after every tick, every buffer equals the result of running the due
modules' stacks one by one in the same order (bit for bit), and a module that
is not due leaves its outputs -- the state the expert reads -- untouched.
"""
import ctypes

import pytest
import torch

from paper_2607_02501_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def eb():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02501_amd import eb as _eb

    return _eb


def _layer(eb, seed, qtype, m, d, f, h, attn, qkv, act, xdt):
    """Stack entries of one decoder layer on the fp32 stream h."""
    qws = [eb.quantize(W.normal((n, k), seed + i, DEV, W.WEIGHT_STD), qtype)
           for i, (n, k) in enumerate(((3 * d, d), (d, d), (2 * f, d), (d, f)))]
    g1 = 1.0 + 0.1 * W.normal((d,), seed + 10, DEV)
    g2 = 1.0 + 0.1 * W.normal((d,), seed + 11, DEV)
    return [(qws[0], h, qkv, dict(x_dtype=xdt, prologue="rmsnorm", norm_weight=g1, eps=1e-5)),
            (qws[1], attn, h, dict(epilogue="add", residual=h)),
            (qws[2], h, act, dict(x_dtype=xdt, prologue="rmsnorm", norm_weight=g2, eps=1e-5,
                                  epilogue="glu")),
            (qws[3], act, h, dict(epilogue="add", residual=h))]


@pytest.mark.parametrize("period,repeats", [(2, 3), (3, 1)])
def test_ticks_match_module_stacks(eb, period, repeats, monkeypatch):
    monkeypatch.delenv("EB_STACK_GRAPH", raising=False)
    m, d, f = 24, 256, 512
    bf = torch.bfloat16
    # backbone: two layers on its own stream hb, then a context projection
    # ctx = proj(hb) that the expert's attention stand-in reads (the shared state)
    hb = W.normal((m, d), 11, DEV)
    qkv_b = torch.empty((m, 3 * d), dtype=bf, device=DEV)
    act_b = torch.empty((m, f), dtype=bf, device=DEV)
    attn_b = W.normal((m, d), 12, DEV).to(bf)
    ctx = torch.zeros((m, d), dtype=bf, device=DEV)
    backbone = (_layer(eb, 100, "q8_0", m, d, f, hb, attn_b, qkv_b, act_b, bf)
                + _layer(eb, 200, "q8_0", m, d, f, hb, attn_b, qkv_b, act_b, bf))
    wctx = eb.quantize(W.normal((d, d), 300, DEV, W.WEIGHT_STD), "q6_s")
    backbone.append((wctx, hb, ctx, dict(x_dtype=bf, prologue="rmsnorm",
                                         norm_weight=torch.ones(d, device=DEV), eps=1e-5)))
    # expert: one layer on its stream he whose O projection reads ctx
    he = W.normal((m, d), 13, DEV)
    qkv_e = torch.empty((m, 3 * d), dtype=bf, device=DEV)
    act_e = torch.empty((m, f), dtype=bf, device=DEV)
    expert = _layer(eb, 400, "q4_0", m, d, f, he, ctx, qkv_e, act_e, bf)
    b_ops, e_ops = eb.make_ops(backbone), eb.make_ops(expert)
    mods = eb.make_modules([(b_ops, period, 0, 1), (e_ops, 1, 0, repeats)])

    bufs = [hb, qkv_b, act_b, ctx, he, qkv_e, act_e]
    init = [b.clone() for b in bufs]
    # reference: the due modules' stacks run directly, tick by tick
    ref = []
    for t in range(2 * period):
        if t % period == 0:
            eb.qlinear_stack(b_ops)
        for _ in range(repeats):
            eb.qlinear_stack(e_ops)
        torch.cuda.synchronize()
        ref.append([b.clone() for b in bufs])
    for b, v in zip(bufs, init):
        b.copy_(v)
    torch.cuda.synchronize()
    for t in range(2 * period):
        before_ctx = ctx.clone()
        expect = eb.multirate_launches(mods, t)
        assert expect == (eb.stack_launches(b_ops) if t % period == 0 else 0) + \
            repeats * eb.stack_launches(e_ops)
        eb.multirate_tick(mods, t)
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(bufs, ref[t])):
            assert torch.equal(got, want), (t, i)
        if t % period:
            assert torch.equal(ctx, before_ctx), t   # the backbone's state is reused
    eb.stack_cache_clear()
