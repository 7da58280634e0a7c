"""Seeded synthetic inputs and the workload shapes they come in.

This module holds no arithmetic of the method: it only names shapes and draws
random numbers.  Both the HIP path's tests/benchmark and the CPU oracle take
their inputs from here, so the two sides always see identical bytes.

The shapes stand in for the model families the paper evaluates (section 2.1,
Table 1 taxonomy; section 4, Tables 3-4): an autoregressive-token VLA decoding
one action token at a time, a VLM-backboned VLA prefilling image and text
tokens, its flow-matching action expert denoising an action chunk, and a
shared-backbone video world-action model.  The paper publishes no weights or
activations for them, so the distributions are synthetic: weights ~ N(0, 0.02)
in fp32, activations ~ N(0, 1) drawn in fp32 and rounded (ties-to-even) to the
activation dtype.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

Q8_0 = "q8_0"
Q4_0 = "q4_0"
Q6_S = "q6_s"


@dataclass(frozen=True)
class Workload:
    name: str
    qtype: str
    x_dtype: torch.dtype
    m: int
    layers: int
    steps: int
    # (name, k, n) per projection, in execution order within one layer
    projections: tuple = field(default_factory=tuple)
    wid: int = 0  # distinct id mixed into every seed

    def ops_per_pass(self) -> int:
        return self.layers * self.steps * len(self.projections)


WORKLOADS = {
    # one Q8_0 linear layer, batch-1 decode, 2048 -> 2048, fp16 activations
    # 128 distinct copies of the one 2048x2048 layer (the first has seed 0) run
    # back to back, so that a pass streams 570 MB rather than one 4.5 MB matrix
    # that the 256 MB last-level cache would hold
    "q8_0_m1_2048": Workload("q8_0_m1_2048", Q8_0, torch.float16, 1, 128, 1,
                             (("linear", 2048, 2048),), wid=0),
    # 7B-class decoder, batch-1 decode of one token through 32 layers, Q4_0
    "q4_0_decode_7b": Workload("q4_0_decode_7b", Q4_0, torch.float16, 1, 32, 1,
                               (("qkv", 4096, 12288), ("o", 4096, 4096),
                                ("gate_up", 4096, 22016), ("down", 11008, 4096)), wid=1),
    # the same decoder in the 6-bit format (Q6_S super-blocks)
    "q6_s_decode_7b": Workload("q6_s_decode_7b", Q6_S, torch.float16, 1, 32, 1,
                               (("qkv", 4096, 12288), ("o", 4096, 4096),
                                ("gate_up", 4096, 22016), ("down", 11008, 4096)), wid=5),
    # VLM backbone prefill: 3 camera views x 256 patch tokens + 48 text tokens
    "q8_0_vlm_prefill_816": Workload("q8_0_vlm_prefill_816", Q8_0, torch.bfloat16, 816, 18, 1,
                                     (("qkv", 2048, 2560), ("o", 2048, 2048),
                                      ("gate_up", 2048, 32768), ("down", 16384, 2048)), wid=2),
    # the same prefill in the 6-bit format
    "q6_s_vlm_prefill_816": Workload("q6_s_vlm_prefill_816", Q6_S, torch.bfloat16, 816, 18, 1,
                                     (("qkv", 2048, 2560), ("o", 2048, 2048),
                                      ("gate_up", 2048, 32768), ("down", 16384, 2048)), wid=6),
    # flow-matching action expert: 50 action tokens, 10 denoising steps, same weights each step
    "q8_0_action_expert_50x10": Workload("q8_0_action_expert_50x10", Q8_0, torch.bfloat16, 50, 18,
                                         10, (("qkv", 1024, 2048), ("o", 1024, 1024),
                                              ("gate_up", 1024, 8192), ("down", 4096, 1024)),
                                         wid=3),
    # DiT-style video world-action backbone: 16 frames x 256 latent tokens
    "q4_0_video_wam_4096": Workload("q4_0_video_wam_4096", Q4_0, torch.bfloat16, 4096, 28, 1,
                                    (("qkv", 3072, 9216), ("o", 3072, 3072),
                                     ("mlp_up", 3072, 12288), ("mlp_down", 12288, 3072)), wid=4),
}

WEIGHT_STD = 0.02


def seed_of(wid: int, layer: int, proj: int, kind: int, step: int = 0) -> int:
    """Deterministic seed; the single 2048x2048 layer's weights use seed 0."""
    return (((wid * 4096 + layer) * 16 + proj) * 4 + kind) * 64 + step


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def normal(shape, seed: int, device="cpu", std: float = 1.0) -> torch.Tensor:
    """fp32 N(0, std^2) samples from torch's generator on `device`."""
    t = torch.randn(*shape, generator=_gen(device, seed), device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t


def weights(w: Workload, layer: int, proj: int, device="cpu", rows=None) -> torch.Tensor:
    """fp32 W[n, k] ~ N(0, 0.02^2) for one projection of one layer."""
    _, k, n = w.projections[proj]
    t = normal((n, k), seed_of(w.wid, layer, proj, 0), device, WEIGHT_STD)
    return t if rows is None else t[rows]


def activations(w: Workload, layer: int, proj: int, device="cpu", step: int = 0,
                m: int | None = None) -> torch.Tensor:
    """x[m, k] ~ N(0, 1), rounded to the workload's activation dtype."""
    _, k, _ = w.projections[proj]
    m = w.m if m is None else m
    return normal((m, k), seed_of(w.wid, layer, proj, 1, step), device).to(w.x_dtype)


def bits16(t: torch.Tensor):
    """Raw 16-bit words of an fp16/bf16 tensor as a numpy uint16 array (host copy)."""
    assert t.dtype in (torch.float16, torch.bfloat16)
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view("uint16")


# ---------------------------------------------------------------------------
# Activation structures beyond N(0, 1) rows, for accuracy checks of every
# kernel path: what a backbone's activations can look like besides dense
# Gaussian rows.  Only random draws and index placement, no arithmetic of the
# method.
# ---------------------------------------------------------------------------

def onehot_rows(m: int, k: int, seed: int, device="cpu") -> torch.Tensor:
    """fp32 [m, k]: row i has one N(0, 1) entry at a random column, zeros elsewhere."""
    g = _gen("cpu", seed)
    cols = torch.randint(0, k, (m,), generator=g)
    vals = torch.randn(m, generator=g)
    x = torch.zeros((m, k), dtype=torch.float32)
    x[torch.arange(m), cols] = vals
    return x.to(device)


def sparse_rows(m: int, k: int, seed: int, nnz=(4, 8), device="cpu") -> torch.Tensor:
    """fp32 [m, k]: row i has between nnz[0] and nnz[1] N(0, 1) entries at
    distinct random columns, zeros elsewhere."""
    g = _gen("cpu", seed)
    x = torch.zeros((m, k), dtype=torch.float32)
    for i in range(m):
        c = int(torch.randint(nnz[0], nnz[1] + 1, (1,), generator=g))
        cols = torch.randperm(k, generator=g)[:c]
        x[i, cols] = torch.randn(c, generator=g)
    return x.to(device)


def outlier_rows(m: int, k: int, seed: int, channels: int = 4, scale: float = 1000.0,
                 device="cpu") -> torch.Tensor:
    """fp32 [m, k] ~ N(0, 1) with `channels` random columns (the same in every
    row) multiplied by `scale`: the outlier feature channels of a backbone."""
    g = _gen("cpu", seed)
    x = torch.randn((m, k), generator=g)
    cols = torch.randperm(k, generator=g)[:channels]
    x[:, cols] *= scale
    return x.to(device)
