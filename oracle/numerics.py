"""bfloat16 helpers for the oracle.

`decode` is exact: a bfloat16 value is the float32 whose upper 16 bits are the
stored pattern, and float32 -> float64 is exact.

`mirror` rounds float64 values first to float32 and then to bfloat16 (round to
nearest, ties to even).  The paper fixes no precision; the GPU path stores
normalised activations, rotated q/k/v, attention outputs and SwiGLU outputs in
bfloat16, and the oracle can round at the same points (`mirror=True` on the
model) to tighten parity.  With `mirror=False` (the default) the oracle is the
plain float64 forward pass.
"""
import numpy as np


def decode(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64 values, exactly."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def mirror(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest float32 -> nearest-even bfloat16, returned as float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32)
    nan = np.isnan(f)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)) << np.uint32(16)
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    out[nan] = np.nan
    return out
