"""Model sizes and synthetic-video recipes of the five workloads.

The model sizes follow the standard ViT families the paper names (ViT-L/14 at
224 and 336 px with 257 and 577 tokens, Section 8; CLIP ViT backbones,
Section 7.1).  The video recipes stand in for the paper's evaluation clips
(MSR-VTT, How2QA, NExT-GQA sampled at 2 FPS, Section 7.1), which are not used
here: a smooth periodic background, moving squares, an optional camera pan,
scene cuts and Gaussian pixel noise.
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple

RESTORE_HIDDEN = 128   # hidden width of the restoration MLP (the paper's two-layer MLP, size 128)
DECISION_HIDDEN = 64   # hidden width of the decision MLP (the paper gives none; one per wavefront lane)
DECISION_FEATURES = 6  # its input: similarity s, class-token attention t, one-hot frame type r (4)


@dataclass(frozen=True)
class ModelConfig:
    image_size: int
    patch: int
    depth: int
    width: int
    heads: int
    mlp: int
    dtype: str  # "f32" or "bf16": arithmetic type of the GEMM/attention operands
    restore: bool = False   # per-layer restoration MLP on reused tokens (hidden RESTORE_HIDDEN)
    decision: bool = False  # per-layer learned decision MLP as the gate (hidden DECISION_HIDDEN)
    reorder: bool = False   # I/P/B referencing with past and future references (no weights)

    @property
    def n_patches(self) -> int:
        return (self.image_size // self.patch) ** 2

    @property
    def n_tokens(self) -> int:
        return self.n_patches + 1

    @property
    def head_dim(self) -> int:
        return self.width // self.heads

    def as_dict(self):
        return dict(image_size=self.image_size, patch=self.patch, depth=self.depth,
                    width=self.width, heads=self.heads, mlp=self.mlp, dtype=self.dtype,
                    restore=self.restore, decision=self.decision, reorder=self.reorder)


@dataclass(frozen=True)
class Segment:
    """A span of frames [start, start+length) with its own motion settings."""
    length: int
    n_objects: int
    obj_size: int
    speed: float       # pixels per frame
    pan: float         # background shift, pixels per frame (horizontal)


@dataclass(frozen=True)
class VideoRecipe:
    seed: int
    sigma: float
    segments: Tuple[Segment, ...]      # repeated cyclically
    cut_first: Optional[int] = None    # first scene cut frame (None = no cuts)
    cut_every: Optional[int] = None    # period of scene cuts


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    n_frames: int
    batch_frames: int
    group_size: int
    weight_seed: int
    video: VideoRecipe
    reuse_targets: Tuple[float, ...] = ()
    tau: Optional[float] = None
    notes: str = ""


def _static(n_obj, size, speed, pan=0.0, length=1 << 30):
    return (Segment(length=length, n_objects=n_obj, obj_size=size, speed=speed, pan=pan),)


CONFIGS = {
    # tiny fp32 model: 8 frames of 112 px, patch 16 (50 tokens), depth 4, width 192
    "tiny": Workload(
        name="tiny", model=ModelConfig(112, 16, 4, 192, 3, 768, "f32"),
        n_frames=8, batch_frames=8, group_size=4, weight_seed=1000,
        video=VideoRecipe(seed=2000, sigma=0.01, segments=_static(2, 16, 3.0)),
        tau=0.95),
    # ViT-B/16 (CLIP style): 64 frames of 224 px, 197 tokens
    "vit_b16": Workload(
        name="vit_b16", model=ModelConfig(224, 16, 12, 768, 12, 3072, "bf16"),
        n_frames=64, batch_frames=64, group_size=4, weight_seed=1001,
        video=VideoRecipe(seed=2001, sigma=0.01, segments=_static(4, 32, 3.0)),
        reuse_targets=(0.5,)),
    # ViT-L/14: 256 frames of 224 px, 257 tokens, camera pan 1 px/frame
    "vit_l14": Workload(
        name="vit_l14", model=ModelConfig(224, 14, 24, 1024, 16, 4096, "bf16"),
        n_frames=256, batch_frames=256, group_size=8, weight_seed=1002,
        video=VideoRecipe(seed=2002, sigma=0.02, segments=_static(6, 32, 3.0, pan=1.0)),
        reuse_targets=(0.5, 0.7, 0.9)),
    # ViT-L/14 at 336 px: 1024 frames in batches of 128, 577 tokens, scene cuts mid-group
    "vit_l14_336": Workload(
        name="vit_l14_336", model=ModelConfig(336, 14, 24, 1024, 16, 4096, "bf16"),
        n_frames=1024, batch_frames=128, group_size=8, weight_seed=1003,
        video=VideoRecipe(seed=2003, sigma=0.02, segments=_static(6, 48, 3.0),
                          cut_first=60, cut_every=120),
        reuse_targets=(0.0, 0.3, 0.6, 0.9)),
    # ViT-H/14-class: 7200 frames (1 h at 2 FPS) in batches of 512, head dim 80
    "vit_h14": Workload(
        name="vit_h14", model=ModelConfig(224, 14, 32, 1280, 16, 5120, "bf16"),
        n_frames=7200, batch_frames=512, group_size=8, weight_seed=1004,
        video=VideoRecipe(seed=2004, sigma=0.02, segments=(
            Segment(120, 6, 32, 3.0, 0.0),    # static camera
            Segment(80, 6, 32, 3.0, 1.0),     # slow pan
            Segment(40, 20, 32, 6.0, 0.0),    # burst of motion
        )),
        reuse_targets=(0.6,)),
}


def get_config(name: str) -> Workload:
    return CONFIGS[name]
