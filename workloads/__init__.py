"""Seeded synthetic workloads shared by the oracle, the tests and the benchmark.

Input preparation only: shapes, seeds, vision-grid layouts, random draws and
their rounding to bfloat16 storage.  The method's arithmetic lives elsewhere.
"""
from .configs import ModelShape, VisionBlock, SeqLayout, Workload, get, scaled, c5_layout  # noqa: F401
from .gen import (HostWeights, DeviceWeights, prefix_kv_host, prefix_kv_device,  # noqa: F401
                  first_pending_token, DraftSynth, bf16_bits_from_f32, tensor_shape, LAYER_TENSORS)
