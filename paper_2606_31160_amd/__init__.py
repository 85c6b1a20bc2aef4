"""MI355X (gfx950) speculative verify-and-commit for two-reasoner decoding.

The work runs in libspecdec.so (include/spec.h): FlatRoPE draft steps, the 3D
M-RoPE target verify pass, the greedy accept rule and the KV commit/rollback.
`binding` is the ctypes layer with the C names; `harness.Session` opens a
context on a seeded synthetic workload.
"""
from . import binding  # noqa: F401
