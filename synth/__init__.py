"""Seeded synthetic inputs shared by the CPU oracle's tests and the GPU path's tests and bench.

This package holds no arithmetic of the reuse method itself: it only draws
weights and renders synthetic video frames.  Both the oracle and the HIP path
consume what it produces; neither imports the other.
"""
from .configs import CONFIGS, ModelConfig, VideoRecipe, get_config  # noqa: F401
from .weights import make_weights, make_blob, pack_weights, weight_layout, round_to_bf16  # noqa: F401
from .video import render_frames, render_frame  # noqa: F401
