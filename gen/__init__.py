"""Seeded synthetic inputs shaped like video-DiT attention layers.

This package holds only input recipes (random draws and a smooth spatio-temporal
field). It contains none of the sparse-attention method's arithmetic, so both
the CPU oracle's tests and the GPU path can take their inputs from it.
"""
from .synth import smooth_field_qkv, bf16_round  # noqa: F401
from .workloads import WORKLOADS, workload  # noqa: F401
