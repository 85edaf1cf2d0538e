"""Seeded synthetic inputs shared by the oracle, the GPU tests and the benchmark.

This package holds none of the retraining method's arithmetic: it only draws
video-like frames, labels and initial ResNet18 weights from fixed seeds, so
that both sides of every parity check read the same bytes.
"""
from .generator import (  # noqa: F401
    WindowSpec,
    make_window,
    make_frames,
    resnet18_param_spec,
    kaiming_resnet18_weights,
    splitmix64_block,
)
