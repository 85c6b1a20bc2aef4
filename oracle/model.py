"""The decoder stack, evaluated on new rows against a KV cache (float64).

The paper treats the target as an unmodified VLA language backbone with 3D
M-RoPE on every attention layer (Sec. 3.3) and the draft as a small transformer
with FlatRoPE (Sec. 4.1-4.2); it does not spell out the block.  The reading used
here is a pre-norm decoder layer:

    a = RMSNorm(x) * g_attn                     (evaluated as ((x * g) W^T) / rms(x))
    q, k, v = a W_q^T, a W_k^T, a W_v^T          (no bias)
    q, k rotated at their token's position      (M-RoPE target / FlatRoPE draft)
    o = softmax(q k^T / sqrt(D)) v              (causal; GQA: q head h reads kv head h // (n_q/n_kv))
    x = x + o W_o^T
    b = RMSNorm(x) * g_ffn
    x = x + (silu(b W_gate^T) * (b W_up^T)) W_down^T

and after the last layer z = (RMSNorm(x) * g_final) E^T with the token embedding
E tied to the LM head.  RMSNorm(x) = x / sqrt(mean(x^2) + eps).

Row i of a call sits at cache slot slots[i] and attends to every slot in
[0, slots[i]] (Eq. verify conditions token j on the committed prefix and on the
proposals before it).
"""
from typing import Callable, Dict, Optional, Sequence

import numpy as np

from . import budget, numerics, rope

ROTARY_MROPE = "mrope"
ROTARY_FLAT = "flat"

_LAYER_NAMES = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q: np.ndarray, kc: np.ndarray, vc: np.ndarray, slots: Sequence[int]) -> np.ndarray:
    """Grouped-query attention over a cache prefix.

    q [M, n_q, D] (rotated), kc/vc [cap, n_kv, D] (keys rotated); row i sees
    cache slots 0..slots[i] (its own slot for causal attention, a later one for
    the rows of a block that see each other).  Returns [M, n_q, D].
    """
    M, nq, D = q.shape
    nkv = kc.shape[1]
    G = nq // nkv
    out = np.empty((M, nq, D), dtype=np.float64)
    scale = 1.0 / np.sqrt(D)
    for i in range(M):
        n_vis = int(slots[i]) + 1
        for h in range(nq):
            kvh = h // G
            s = (kc[:n_vis, kvh, :] @ q[i, h]) * scale
            p = softmax(s)
            out[i, h] = p @ vc[:n_vis, kvh, :]
    return out


class KVCache:
    """Rotated keys and values of one decoder stack for one sequence.

    k[layer], v[layer] are float64 [cap, n_kv, D]; pos3 [3, cap] holds the
    rotary positions of every slot (the draft's are all equal to the slot).
    """

    def __init__(self, layers: int, cap: int, kv_heads: int, head_dim: int, pos3: np.ndarray):
        self.k = [np.zeros((cap, kv_heads, head_dim)) for _ in range(layers)]
        self.v = [np.zeros((cap, kv_heads, head_dim)) for _ in range(layers)]
        self.pos3 = np.asarray(pos3, dtype=np.int64)
        self.cap = cap


class Decoder:
    """A decoder stack reading bfloat16 weights from `provider.get(model, layer, name)`.

    `shape` supplies layers, hidden, q_heads, kv_heads, head_dim, ffn,
    mrope_section, interleaved, rope_base, rms_eps.  `rotary` is ROTARY_MROPE
    for the target or ROTARY_FLAT for the draft.  `mirror` rounds to bfloat16
    where the GPU stores bfloat16 (see numerics.mirror).
    """

    def __init__(self, provider, model: str, shape, vocab: int, rotary: str,
                 mirror: bool = False, cache_weights: bool = True, lm_chunk: int = 16384):
        self.p = provider
        self.model = model
        self.s = shape
        self.vocab = vocab
        self.rotary = rotary
        self.mirror = mirror
        self.cache_weights = cache_weights
        self.lm_chunk = lm_chunk
        self._layers: Dict[int, Dict[str, np.ndarray]] = {}
        self._embed: Optional[np.ndarray] = None
        # attention budget readout (budget.budget): when readout_layer is set,
        # forward() stores the [M, n_q, 4] readout of that layer's attention
        # over slots classified by readout_classes in self.readout
        self.readout_layer: Optional[int] = None
        self.readout_classes: Optional[np.ndarray] = None
        self.readout: Optional[np.ndarray] = None
        # conditioning on another stack's hidden states: input_hook(x, slots)
        # replaces the embedded rows before layer 0; capture_layers names the
        # layers whose output residual rows forward() keeps in self.captured
        self.input_hook: Optional[Callable[[np.ndarray, np.ndarray], np.ndarray]] = None
        self.capture_layers: Sequence[int] = ()
        self.captured: Dict[int, np.ndarray] = {}
        # cross-attention conditioning (Sec. 4.1): layer cross_layer attends,
        # instead of to keys of its own rows, to a context of keys and values
        # that context_kv() computed from another stack's states; row i sees
        # the context slots below both its own slot and cross_len
        self.cross_layer: Optional[int] = None
        self.cross_len: int = 0

    # -- weights -----------------------------------------------------------
    def layer(self, li: int) -> Dict[str, np.ndarray]:
        if li in self._layers:
            return self._layers[li]
        W = {n: numerics.decode(self.p.get(self.model, li, n)) for n in _LAYER_NAMES}
        if self.cache_weights:
            self._layers[li] = W
        return W

    def final_norm(self) -> np.ndarray:
        return numerics.decode(self.p.get(self.model, -1, "final_norm"))

    def embed_bits(self) -> np.ndarray:
        return self.p.get("global", -1, "embed")

    def embed_rows(self, tokens: Sequence[int]) -> np.ndarray:
        return numerics.decode(self.embed_bits()[np.asarray(tokens, dtype=np.int64)])

    def lm_head(self, h: np.ndarray) -> np.ndarray:
        """z = h E^T over the whole vocabulary (tied embedding), float64 [M, V]."""
        E = self.embed_bits()
        if self.cache_weights and self.vocab <= self.lm_chunk:
            if self._embed is None:
                self._embed = numerics.decode(E)
            return h @ self._embed.T
        z = np.empty((h.shape[0], self.vocab))
        for c0 in range(0, self.vocab, self.lm_chunk):
            c1 = min(self.vocab, c0 + self.lm_chunk)
            z[:, c0:c1] = h @ numerics.decode(E[c0:c1]).T
        return z

    def _r(self, x: np.ndarray) -> np.ndarray:
        return numerics.mirror(x) if self.mirror else x

    def _normed(self, x: np.ndarray, g: np.ndarray):
        """RMSNorm(x) * g as the pair (x * g, 1 / sqrt(mean(x^2) + eps)): the
        projection of the normalised rows is (x * g) W^T scaled per row, the
        same product as RMSNorm(x) * g W^T.  In mirror mode x * g is rounded
        to bfloat16, where the GPU stores the projection's input."""
        inv = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + self.s.rms_eps)
        return self._r(x * g), inv

    # -- rotary ------------------------------------------------------------
    def rotate(self, x: np.ndarray, pos3: np.ndarray) -> np.ndarray:
        """x [N, heads, D]; pos3 [3, N] (target) -- the draft uses pos3[0] as m."""
        if self.rotary == ROTARY_MROPE:
            return rope.mrope(x, pos3, self.s.mrope_section, self.s.interleaved, self.s.rope_base)
        return rope.flatrope(x, pos3[0], self.s.rope_base)

    # -- cache -------------------------------------------------------------
    def new_cache(self, cap: int, pos3: np.ndarray) -> KVCache:
        return KVCache(self.s.layers, cap, self.s.kv_heads, self.s.head_dim, pos3)

    def fill_prefix(self, cache: KVCache, layer: int, k_pre_bits: np.ndarray, v_bits: np.ndarray) -> None:
        """Store a prompt's pre-rotation keys (rotated here) and values in slots 0..P-1."""
        P = k_pre_bits.shape[0]
        k = numerics.decode(k_pre_bits)
        v = numerics.decode(v_bits)
        cache.k[layer][:P] = self._r(self.rotate(k, cache.pos3[:, :P]))
        cache.v[layer][:P] = v

    def context_kv(self, cache: KVCache, layer: int, f: np.ndarray, slots: Sequence[int]) -> None:
        """Cross-attention context of `layer` at `slots` (Sec. 4.1: target
        hidden states become the draft's attention keys and values): the rows
        f [N, hidden] go through the layer's attention norm and its W_k, W_v;
        the keys are rotated at each slot's position."""
        s = self.s
        slots = np.asarray(slots, dtype=np.int64)
        N = len(slots)
        W = self.layer(layer)
        a, ia = self._normed(np.asarray(f, dtype=np.float64), W["attn_norm"])
        k = ((a @ W["wk"].T) * ia).reshape(N, s.kv_heads, s.head_dim)
        v = ((a @ W["wv"].T) * ia).reshape(N, s.kv_heads, s.head_dim)
        cache.k[layer][slots] = self._r(self.rotate(k, cache.pos3[:, slots]))
        cache.v[layer][slots] = self._r(v)

    # -- forward -----------------------------------------------------------
    def forward(self, tokens: Sequence[int], slots: Sequence[int], cache: KVCache,
                want_hidden: bool = False, visible: Optional[Sequence[int]] = None):
        """Run the stack on rows (tokens[i] at slots[i]); writes their K/V into the
        cache and returns float64 logits [M, V] (and the final normalised hidden
        rows if want_hidden).  Row i attends to slots 0..visible[i] (default
        slots[i]: causal); every row's K/V of a layer is written before that
        layer's attention, so a row may see later rows of the same call."""
        s = self.s
        M = len(tokens)
        slots = np.asarray(slots, dtype=np.int64)
        vis = slots if visible is None else np.asarray(visible, dtype=np.int64)
        if M == 0:
            return np.zeros((0, self.vocab))
        D, nq, nkv = s.head_dim, s.q_heads, s.kv_heads
        pos = cache.pos3[:, slots]
        x = self.embed_rows(tokens)
        if self.input_hook is not None:
            x = self.input_hook(x, slots)
        self.captured = {}
        for li in range(s.layers):
            W = self.layer(li)
            a, ia = self._normed(x, W["attn_norm"])
            q = ((a @ W["wq"].T) * ia).reshape(M, nq, D)
            q = self._r(self.rotate(q, pos))
            if li == self.cross_layer:
                # the context only: slots before the row's own and before cross_len
                lvis = np.minimum(slots - 1, self.cross_len - 1)
            else:
                k = ((a @ W["wk"].T) * ia).reshape(M, nkv, D)
                v = ((a @ W["wv"].T) * ia).reshape(M, nkv, D)
                cache.k[li][slots] = self._r(self.rotate(k, pos))
                cache.v[li][slots] = self._r(v)
                lvis = vis
            if li == self.readout_layer:
                self.readout = budget.budget(q, cache.k[li], lvis, self.readout_classes)
            o = self._r(attend(q, cache.k[li], cache.v[li], lvis).reshape(M, nq * D))
            x = x + o @ W["wo"].T
            b, ib = self._normed(x, W["ffn_norm"])
            u = self._r(silu((b @ W["w_gate"].T) * ib) * ((b @ W["w_up"].T) * ib))
            x = x + u @ W["w_down"].T
            if li in self.capture_layers:
                self.captured[li] = self._r(x)
        h, ih = self._normed(x, self.final_norm())
        z = self.lm_head(h) * ih
        return (z, h * ih) if want_hidden else z


def greedy_argmax(z: np.ndarray) -> np.ndarray:
    """Per-row argmax; ties go to the lowest index and NaN counts as -inf."""
    zz = np.where(np.isnan(z), -np.inf, z)
    return np.argmax(zz, axis=-1).astype(np.int64)
