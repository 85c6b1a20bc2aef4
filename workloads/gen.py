"""Seeded synthetic inputs shared by the oracle and the HIP path.

Everything here is input preparation: normal/uniform draws, rounding of the
drawn float32 values to bfloat16 storage, and the draft-token synthesis rule of
the workloads (a draft token equals the target's greedy token with probability
p, otherwise a uniform random token).  No position ids, rotations, forward pass,
argmax or accept/commit rule lives here.

Two sources of weights exist:
  * `HostWeights`   numpy PCG64 per tensor; cheap for small shapes; the bfloat16
                    bits are produced on the host.
  * `DeviceWeights` torch's Philox generator on the GPU, per tensor; used for the
                    7B-class shapes where host generation would take minutes.
                    The oracle reads the same bits back with `get()` (a plain
                    device-to-host copy).
Each test uses one source for both sides, so both see identical bits.
"""
from __future__ import annotations

import hashlib
from typing import Dict, Optional, Tuple

import numpy as np

from .configs import ModelShape, Workload

MODEL_IDS = {"target": 0, "draft": 1, "global": 2}
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
# (w_fuse, w_in: the draft's conditioning on target hidden states, appended so
# that earlier keys keep their streams)
NAME_IDS = {n: i for i, n in enumerate(LAYER_TENSORS + ("final_norm", "embed", "k_prefix", "v_prefix",
                                                        "w_fuse", "w_in"))}


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns.  Inputs are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def tensor_shape(shape: ModelShape, vocab: int, name: str) -> Tuple[int, ...]:
    H, D = shape.hidden, shape.head_dim
    return {
        "attn_norm": (H,), "ffn_norm": (H,), "final_norm": (H,),
        "wq": (shape.q_heads * D, H), "wk": (shape.kv_heads * D, H), "wv": (shape.kv_heads * D, H),
        "wo": (H, shape.q_heads * D),
        "w_gate": (shape.ffn, H), "w_up": (shape.ffn, H), "w_down": (H, shape.ffn),
        "embed": (vocab, H),
        "w_fuse": (H, 3 * H), "w_in": (H, 2 * H),
    }[name]


def _key(seed: int, model: str, layer: int, name: str, extra: int = 0) -> Tuple[int, ...]:
    return (int(seed), MODEL_IDS[model], int(layer) + 1, NAME_IDS[name], int(extra))


def _key_hash63(key: Tuple[int, ...]) -> int:
    h = hashlib.blake2b(repr(key).encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def _is_gain(name: str) -> bool:
    return name.endswith("norm")


class HostWeights:
    """bfloat16 weights generated on the host, one PCG64 stream per tensor."""

    def __init__(self, w: Workload):
        self.w = w
        self._cache: Dict[Tuple, np.ndarray] = {}

    def shape_of(self, model: str) -> ModelShape:
        return self.w.target if model == "target" else self.w.draft

    def get(self, model: str, layer: int, name: str) -> np.ndarray:
        """uint16 bfloat16 bits.  `model` is 'target', 'draft' or 'global'
        (for 'embed'); `layer` is -1 for per-model tensors such as final_norm."""
        key = _key(self.w.seed, model, layer, name)
        if key not in self._cache:
            shp = tensor_shape(self.w.target if model == "global" else self.shape_of(model), self.w.vocab, name)
            rng = np.random.default_rng(list(key))
            z = rng.standard_normal(shp, dtype=np.float32)
            if _is_gain(name):
                z = np.float32(1.0) + np.float32(self.w.gain_std) * z
            else:
                z = np.float32(self.w.weight_std) * z
            self._cache[key] = bf16_bits_from_f32(z)
        return self._cache[key]


class DeviceWeights:
    """bfloat16 weights generated on the GPU with torch's seeded generator."""

    def __init__(self, w: Workload, device: str = "cuda"):
        import torch
        self.w = w
        self.device = device
        self._t: Dict[Tuple, "torch.Tensor"] = {}

    def shape_of(self, model: str) -> ModelShape:
        return self.w.target if model == "target" else self.w.draft

    def tensor(self, model: str, layer: int, name: str):
        import torch
        key = _key(self.w.seed, model, layer, name)
        if key not in self._t:
            shp = tensor_shape(self.w.target if model == "global" else self.shape_of(model), self.w.vocab, name)
            g = torch.Generator(device=self.device)
            g.manual_seed(_key_hash63(key))
            z = torch.randn(shp, generator=g, device=self.device, dtype=torch.float32)
            if _is_gain(name):
                z.mul_(self.w.gain_std).add_(1.0)
            else:
                z.mul_(self.w.weight_std)
            self._t[key] = z.to(torch.bfloat16)
            del z
        return self._t[key]

    def get(self, model: str, layer: int, name: str) -> np.ndarray:
        t = self.tensor(model, layer, name)
        return t.view(__import__("torch").int16).cpu().numpy().view(np.uint16)


def prefix_kv_host(w: Workload, b: int, model: str, layer: int, which: str) -> np.ndarray:
    """Pre-rotation prefix keys or values of sequence b, [prefix_len, kv_heads, head_dim]
    bfloat16 bits, N(0, kv_std^2)."""
    shape = w.target if model == "target" else w.draft
    P = w.seqs[b].prefix_len
    key = _key(w.seed + 1, model, layer, "k_prefix" if which == "k" else "v_prefix", extra=b)
    rng = np.random.default_rng(list(key))
    z = np.float32(w.kv_std) * rng.standard_normal((P, shape.kv_heads, shape.head_dim), dtype=np.float32)
    return bf16_bits_from_f32(z)


def prefix_kv_device(w: Workload, b: int, model: str, layer: int, which: str, device: str = "cuda"):
    import torch
    shape = w.target if model == "target" else w.draft
    P = w.seqs[b].prefix_len
    key = _key(w.seed + 1, model, layer, "k_prefix" if which == "k" else "v_prefix", extra=b)
    g = torch.Generator(device=device)
    g.manual_seed(_key_hash63(key))
    z = torch.randn((P, shape.kv_heads, shape.head_dim), generator=g, device=device, dtype=torch.float32)
    return z.mul_(w.kv_std).to(torch.bfloat16)


def first_pending_token(w: Workload, b: int) -> int:
    """The token at index prefix_len (row 0 of the first verify)."""
    rng = np.random.default_rng([w.seed + 2, b])
    return int(rng.integers(0, w.vocab))


class DraftSynth:
    """Synthetic draft tokens for the verify pass: token j equals the target's
    greedy token at that index with probability p, else a uniform random token.
    The draws come from a seeded per-sequence stream; `greedy` is the target's
    greedy continuation supplied by the caller."""

    def __init__(self, w: Workload, b: int, seed_offset: int = 3):
        self.vocab = w.vocab
        self.p = w.p_accept[b]
        self.rng = np.random.default_rng([w.seed + seed_offset, b])

    def propose(self, greedy: np.ndarray, K: int) -> np.ndarray:
        out = np.empty(K, dtype=np.int32)
        for j in range(K):
            u = self.rng.random()
            r = int(self.rng.integers(0, self.vocab))
            out[j] = int(greedy[j]) if (j < len(greedy) and u < self.p) else r
        return out
