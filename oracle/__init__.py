"""CPU oracle for two-reasoner speculative decoding (propose / verify / commit).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It is a plain, slow, obviously
correct float64 numpy implementation of what the GPU path computes, and it
shares no code with the HIP library or its Python binding.

Modules
  numerics   bfloat16 decoding and the optional bfloat16 "mirror" rounding
  positions  per-token (p_T, p_H, p_W) ids of the target and the draft's 1D index
  rope       Eq. rope-1d, Eq. rope-3d, Eq. axis-assign, Eq. mrope-phase, Eq. flatrope-proj
  model      the decoder stack evaluated on new rows against a KV cache
  spec       Eq. stage1 (greedy), Eq. propose, Eq. verify, Eq. accept, Eq. commit
  report     Eq. L-and-speedup and the cost ratio of Sec. 5.1
  budget     the attention-budget readout of Sec. 4.2 (mass per token class,
             entropy within trajectory/text)

Every function with no independent pin says "parity unpinned" in its docstring.
"""
from . import numerics, positions, rope, budget, model, spec, report  # noqa: F401
