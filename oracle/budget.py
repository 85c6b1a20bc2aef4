"""Attention budget readout (Sec. 4.2, "Empirical confirmation", Table attn-budget).

Test infrastructure: the CPU oracle of the readout; only tests, smoke() and the
benchmark's CPU baseline use it.

The paper measures where one attention layer puts its softmax mass, per token
class, and how spread the mass is inside the trajectory-and-text class.  Cache
slots fall into three classes:

  0  visual           a slot inside one of the prompt's vision blocks
  1  trajectory/text  any other prompt slot
  2  generated        a slot after the prompt (committed tokens and the
                      rows of the current pass)

For one query row of one head, with attention probabilities p over the slots
it sees,

  mass_c   = sum of p_k over the visible slots k of class c   (the three sum to 1)
  entropy  = H(q) / ln(n_1), q = p restricted to class 1 and renormalised,
             H(q) = -sum q_k ln q_k, n_1 = visible class-1 slots
             (0 when n_1 <= 1: a single slot carries no spread).

The readout is computed on the attention of one layer during a forward pass
(model.Decoder.readout_layer); values on synthetic weights are not the paper's,
only the definition is.
"""
from typing import Iterable, Sequence, Tuple

import numpy as np

VISUAL, TRAJ_TEXT, GENERATED = 0, 1, 2


def slot_classes(prefix_len: int, blocks: Iterable[Tuple[int, int, int, int]], total_len: int) -> np.ndarray:
    """int8 [total_len]: the class of every slot (blocks are (start, t, h, w))."""
    c = np.full(total_len, GENERATED, dtype=np.int8)
    c[:min(prefix_len, total_len)] = TRAJ_TEXT
    for (s, t, h, w) in blocks:
        c[s:min(s + t * h * w, prefix_len, total_len)] = VISUAL
    return c


def row_budget(p: np.ndarray, classes: np.ndarray) -> np.ndarray:
    """[4] = (mass visual, mass trajectory/text, mass generated, normalised
    entropy within trajectory/text) of one probability vector p over slots
    0..len(p)-1 with the given classes."""
    out = np.zeros(4)
    for c in range(3):
        out[c] = float(np.sum(p[classes == c]))
    sel = p[classes == TRAJ_TEXT]
    n1 = sel.size
    if n1 > 1 and out[TRAJ_TEXT] > 0.0:
        q = sel / out[TRAJ_TEXT]
        nz = q[q > 0.0]
        out[3] = float(-np.sum(nz * np.log(nz)) / np.log(n1))
    return out


def budget(q: np.ndarray, kc: np.ndarray, slots: Sequence[int], classes: np.ndarray) -> np.ndarray:
    """Readout of causal grouped-query attention (the same scores as
    model.attend): q [M, n_q, D] rotated, kc [cap, n_kv, D]; row i sees slots
    0..slots[i].  Returns float64 [M, n_q, 4]."""
    M, nq, D = q.shape
    nkv = kc.shape[1]
    G = nq // nkv
    out = np.zeros((M, nq, 4))
    scale = 1.0 / np.sqrt(D)
    for i in range(M):
        n_vis = int(slots[i]) + 1
        for h in range(nq):
            s = (kc[:n_vis, h // G, :] @ q[i, h]) * scale
            e = np.exp(s - np.max(s))
            out[i, h] = row_budget(e / np.sum(e), classes[:n_vis])
    return out
