"""Per-token rotary positions.

Target (Sec. 3.3, text under Eq. rope-3d; Sec. 4.2, text under Eq. mrope-phase):
each token i carries (p_T(i), p_H(i), p_W(i)).  Text and trajectory-history
tokens collapse all three to the sequence index m = i.  Vision patches carry
frame and grid coordinates.  The paper does not fix the offset of a grid inside
the sequence; the reading used here places a block that starts at sequence
index s with grid (T, H, W), stored t-major then h then w, at
(s + t, s + h, s + w).

Draft (Eq. flatrope-proj; App. A): every token, vision or text, uses its
sequence index m(i) = i on all three axes, so only a 1D index is needed.
"""
from typing import Iterable, Tuple

import numpy as np


def target_positions(total_len: int, blocks: Iterable[Tuple[int, int, int, int]]) -> np.ndarray:
    """int64 array [3, total_len]: rows are (p_T, p_H, p_W).

    `blocks` holds (start, t, h, w) vision grids; every index outside them is text.
    Blocks must lie inside [0, total_len) and must not overlap.
    """
    pos = np.empty((3, total_len), dtype=np.int64)
    idx = np.arange(total_len, dtype=np.int64)
    pos[0] = idx
    pos[1] = idx
    pos[2] = idx
    taken = np.zeros(total_len, dtype=bool)
    for (s, T, H, W) in blocks:
        n = T * H * W
        if s < 0 or s + n > total_len:
            raise ValueError("vision block outside the sequence")
        if taken[s:s + n].any():
            raise ValueError("vision blocks overlap")
        taken[s:s + n] = True
        k = 0
        for t in range(T):
            for h in range(H):
                for w in range(W):
                    pos[0, s + k] = s + t
                    pos[1, s + k] = s + h
                    pos[2, s + k] = s + w
                    k += 1
    return pos


def flat_positions(total_len: int) -> np.ndarray:
    """Eq. flatrope-proj: p_T = p_H = p_W = m(i) = i, as int64 [3, total_len]."""
    idx = np.arange(total_len, dtype=np.int64)
    return np.stack([idx, idx, idx])
