"""Workload definitions: model shapes, prompt layouts and speculative-loop settings.

This module only describes inputs (shapes, seeds, layouts of vision blocks).  It
holds none of the method's arithmetic: position ids, rotations, the forward pass
and the accept/commit rule live in the oracle and, independently, in the HIP
library.

The workloads follow the synthetic stand-ins for the paper's Alpamayo-R1
clips (Sec. 5: prompts dominated by visual tokens, chain-of-causation outputs of
15-20 tokens, greedy verification), sized after a Qwen2.5-VL-7B-class backbone.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    """One decoder stack (target or draft).

    `mrope_section` is (s_T, s_H, s_W) in rotary pairs and must sum to
    head_dim/2 (Sec. 3.3, Eq. rope-3d).  `interleaved` selects the axis
    assignment of Eq. axis-assign.  The draft ignores both (FlatRoPE, Sec. 4.2)
    unless it runs with M-RoPE as the comparison arm of the attention-budget
    readout.
    """
    layers: int
    hidden: int
    q_heads: int
    kv_heads: int
    head_dim: int
    ffn: int
    mrope_section: Tuple[int, int, int] = (16, 24, 24)
    interleaved: bool = False
    rope_base: float = 10000.0
    rms_eps: float = 1e-6


@dataclass(frozen=True)
class VisionBlock:
    """A (t, h, w) patch grid occupying sequence indices [start, start+t*h*w),
    laid out t-major, then h, then w."""
    start: int
    t: int
    h: int
    w: int

    @property
    def ntok(self) -> int:
        return self.t * self.h * self.w


@dataclass(frozen=True)
class SeqLayout:
    """Prompt of `prefix_len` tokens: vision blocks, every other index is text
    (trajectory history / prompt text)."""
    prefix_len: int
    blocks: Tuple[VisionBlock, ...] = ()


@dataclass(frozen=True)
class Workload:
    name: str
    target: ModelShape
    draft: Optional[ModelShape]
    vocab: int
    K: int
    seqs: Tuple[SeqLayout, ...]
    p_accept: Tuple[float, ...]          # per-sequence probability that a synthetic draft token matches the target
    max_new_tokens: int = 20
    stop_token: int = -1
    weight_std: float = 0.02
    gain_std: float = 0.1                 # RMSNorm gains are 1 + gain_std * N(0,1)
    kv_std: float = 1.0                   # synthetic pre-rotation prefix K/V
    seed: int = 0

    @property
    def batch(self) -> int:
        return len(self.seqs)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# ---------------------------------------------------------------------------
# Shapes
# ---------------------------------------------------------------------------

TINY = ModelShape(layers=2, hidden=256, q_heads=4, kv_heads=2, head_dim=64, ffn=688,
                  mrope_section=(8, 12, 12))
TINY_DRAFT = replace(TINY, layers=1)

QWEN7B_LAYER = ModelShape(layers=28, hidden=3584, q_heads=28, kv_heads=4, head_dim=128,
                          ffn=18944, mrope_section=(16, 24, 24))
QWEN7B_DRAFT = replace(QWEN7B_LAYER, layers=2)

# The paper's own target backbone (Sec. 5): 36 decoder layers and 32 attention
# heads, as stated there; the remaining widths (hidden 4096, 8 kv heads, SwiGLU
# 12288, vocabulary 151936) are those of that backbone's public configuration.
# Its rotary axis assignment is the interleaved form of Eq. axis-assign.  The
# draft is one FlatRoPE layer of the same width (the paper's autoregressive draft
# is a single layer).
PAPER_BACKBONE = ModelShape(layers=36, hidden=4096, q_heads=32, kv_heads=8, head_dim=128,
                            ffn=12288, mrope_section=(24, 20, 20), interleaved=True)
PAPER_DRAFT = replace(PAPER_BACKBONE, layers=1, interleaved=False)


def _c1() -> Workload:
    # 1x16x16 vision grid at index 0, then 64 trajectory/text tokens.
    lay = SeqLayout(320, (VisionBlock(0, 1, 16, 16),))
    return Workload("C1-tiny", TINY, TINY_DRAFT, vocab=1024, K=4, seqs=(lay,), p_accept=(0.8,))


def _c2() -> Workload:
    # Two frames, each a 1x48x32 grid, then 256 trajectory/text tokens.  A single
    # target layer; the stand-in head over a 1024-token vocabulary only closes the
    # verify pass with an argmax.
    lay = SeqLayout(3328, (VisionBlock(0, 1, 48, 32), VisionBlock(1536, 1, 48, 32)))
    return Workload("C2-one-layer", replace(QWEN7B_LAYER, layers=1), QWEN7B_DRAFT, vocab=1024, K=8,
                    seqs=(lay,), p_accept=(0.75,))


def _c3() -> Workload:
    # 4x28x32 grid (3584 vision tokens) then 512 trajectory/text tokens.
    lay = SeqLayout(4096, (VisionBlock(0, 4, 28, 32),))
    return Workload("C3-28-layer-verify", QWEN7B_LAYER, QWEN7B_DRAFT, vocab=152064, K=8,
                    seqs=(lay,), p_accept=(0.75,))


def c5_layout(prefix_len: int) -> SeqLayout:
    """Four cameras, each a (2, h_c, 16) grid, placed back to back from index 0;
    h_c is chosen so that vision fills about 85% of the prompt."""
    h_c = max(1, int(round(0.85 * prefix_len / 128)))
    blocks = tuple(VisionBlock(32 * h_c * cam, 2, h_c, 16) for cam in range(4))
    return SeqLayout(prefix_len, blocks)


def _c5(seed: int = 1000) -> Workload:
    import numpy as np
    rng = np.random.default_rng(seed)
    lens = rng.integers(2048, 8193, size=16)
    ps = rng.uniform(0.5, 0.9, size=16)
    seqs = tuple(c5_layout(int(n)) for n in lens)
    return Workload("C5-batched-16", QWEN7B_LAYER, QWEN7B_DRAFT, vocab=152064, K=8, seqs=seqs,
                    p_accept=tuple(float(p) for p in ps), max_new_tokens=20)


def _c6() -> Workload:
    # The paper's verification width: K = 16 proposals (17 verify rows) against
    # its 36-layer backbone, over the 4096-token vision-dominated prompt of C3.
    lay = SeqLayout(4096, (VisionBlock(0, 4, 28, 32),))
    return Workload("C6-paper-backbone-K16", PAPER_BACKBONE, PAPER_DRAFT, vocab=151936, K=16,
                    seqs=(lay,), p_accept=(0.75,))


def get(name: str) -> Workload:
    table = {"C1": _c1, "C2": _c2, "C3": _c3, "C5": _c5, "C6": _c6}
    return table[name]()


def scaled(w: Workload, *, layers: Optional[int] = None, vocab: Optional[int] = None,
           prefix_scale: Optional[float] = None) -> Workload:
    """A reduced copy of a workload (fewer layers, smaller vocabulary or shorter
    prompt) for cases the oracle must finish in seconds."""
    t = w.target if layers is None else replace(w.target, layers=layers)
    seqs = w.seqs
    if prefix_scale is not None:
        new = []
        for s in seqs:
            blocks = tuple(VisionBlock(int(b.start * prefix_scale), b.t, max(1, int(b.h * prefix_scale)), b.w)
                           for b in s.blocks)
            n = max(int(s.prefix_len * prefix_scale), max((b.start + b.ntok for b in blocks), default=0) + 1)
            new.append(SeqLayout(n, blocks))
        seqs = tuple(new)
    return replace(w, target=t, vocab=w.vocab if vocab is None else vocab, seqs=seqs)
