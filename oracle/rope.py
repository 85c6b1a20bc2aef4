"""Rotary position encodings of the target (3D M-RoPE) and the draft (FlatRoPE).

Eq. rope-1d: adjacent dimensions (2d, 2d+1) form pair d; pair d is rotated by
the angle m * omega_d, omega_d = b^(-2d/h), with the 2x2 block
[[cos, -sin], [sin, cos]].

Eq. axis-assign: rotary pair d in [0, D_r) reads the axis a(d) in {T, H, W};
blocked: the first s_T pairs read T, the next s_H read H, the rest read W;
interleaved: a(d) = (T, H, W)[d mod 3].

Eq. mrope-phase: phi_d(i) = theta_d * p_{a(d)}(i), theta_d = 10000^(-2d/D_head).
The per-axis frequency vectors of Eq. rope-3d are read as slices of this single
theta table (the section's pairs keep their global index d).

Eq. flatrope-proj: the draft sets p_T = p_H = p_W = m(i), so its phase is
theta_d * m(i) for every d whatever the axis assignment, i.e. Eq. rope-1d with
the target's theta table.
"""
import numpy as np

AXIS_T, AXIS_H, AXIS_W = 0, 1, 2


def theta(head_dim: int, base: float = 10000.0) -> np.ndarray:
    """theta_d = base^(-2d/head_dim) for d = 0 .. head_dim/2 - 1 (float64)."""
    d = np.arange(head_dim // 2, dtype=np.float64)
    return base ** (-2.0 * d / head_dim)


def axis_assignment(d_rot: int, section=(16, 24, 24), interleaved: bool = False) -> np.ndarray:
    """a(d) for d in [0, d_rot), as an int array of AXIS_T/AXIS_H/AXIS_W."""
    a = np.empty(d_rot, dtype=np.int64)
    if interleaved:
        for d in range(d_rot):
            a[d] = d % 3
        return a
    sT, sH, sW = section
    if sT + sH + sW != d_rot:
        raise ValueError("mrope_section must sum to head_dim/2")
    for d in range(d_rot):
        if d < sT:
            a[d] = AXIS_T
        elif d < sT + sH:
            a[d] = AXIS_H
        else:
            a[d] = AXIS_W
    return a


def phases(pos3: np.ndarray, head_dim: int, section=(16, 24, 24), interleaved: bool = False,
           base: float = 10000.0) -> np.ndarray:
    """phi[n, d] = theta_d * p_{a(d)}(n) for positions pos3 [3, N] -> [N, head_dim/2]."""
    th = theta(head_dim, base)
    a = axis_assignment(head_dim // 2, section, interleaved)
    pos3 = np.asarray(pos3, dtype=np.float64)
    return th[None, :] * pos3[a, :].T


def rotate_pairs(x: np.ndarray, phi: np.ndarray) -> np.ndarray:
    """Rotate adjacent pairs of x [N, heads, D] by phi [N, D/2] (Eq. rope-1d)."""
    x = np.asarray(x, dtype=np.float64)
    xe = x[..., 0::2]
    xo = x[..., 1::2]
    c = np.cos(phi)[:, None, :]
    s = np.sin(phi)[:, None, :]
    out = np.empty_like(x)
    out[..., 0::2] = xe * c - xo * s
    out[..., 1::2] = xe * s + xo * c
    return out


def mrope(x: np.ndarray, pos3: np.ndarray, section=(16, 24, 24), interleaved: bool = False,
          base: float = 10000.0) -> np.ndarray:
    """Eq. rope-3d with the axis assignment of Eq. axis-assign: x [N, heads, D], pos3 [3, N]."""
    return rotate_pairs(x, phases(pos3, x.shape[-1], section, interleaved, base))


def rope1d(x: np.ndarray, m: np.ndarray, base: float = 10000.0) -> np.ndarray:
    """Eq. rope-1d: x [N, heads, D] rotated by the 1D index m [N]."""
    th = theta(x.shape[-1], base)
    phi = th[None, :] * np.asarray(m, dtype=np.float64)[:, None]
    return rotate_pairs(x, phi)


def flatrope(x: np.ndarray, m: np.ndarray, base: float = 10000.0) -> np.ndarray:
    """Eq. flatrope-proj: project (p_T, p_H, p_W) -> m and apply Eq. mrope-phase.
    The axis assignment is irrelevant here; the blocked default is used."""
    m = np.asarray(m, dtype=np.int64)
    pos3 = np.stack([m, m, m])
    D = x.shape[-1]
    return mrope(x, pos3, section=(D // 2, 0, 0), interleaved=False, base=base)
