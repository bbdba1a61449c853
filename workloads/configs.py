"""The five synthetic workloads the step is checked and measured on.

Shapes follow the paper's setting: video VLM backbones (7B- and 72B-class
decoders with grouped-query attention), frames of 14x14 / 16x16 / 27x27
visual tokens, 512-frame videos sampled at 1 FPS (Results, experimental
setup), and compressed-state budgets B in the paper's sweep range
(Results, Pareto study; Eq. 4 defines the fixed budget B).

Every input is synthetic: the paper's benchmark videos and model weights are
not available, so seeded N(0,1)-like Q/K/V of the same shapes stand in for
them.  The recipe names select the generator in ``workloads.generate``.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    tokens_per_frame: int
    n_frames: int
    capacity: int
    dtype: str  # "f32" or "bf16"
    recipe: str  # "iid", "lowrank", "stress"
    seed: int
    pos_offset: int = 0

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def scale(self) -> float:
        return self.head_dim ** -0.5

    def state_size(self, frame: int) -> int:
        """Number of compressed-state tokens entering frame ``frame`` (0-based)."""
        return min(self.capacity, frame * self.tokens_per_frame)

    @property
    def full_from_frame(self) -> int:
        """First frame index that sees a full state."""
        t = self.tokens_per_frame
        if self.capacity == 0:
            return 0
        return -(-self.capacity // t)

    def with_(self, **kw) -> "WorkloadConfig":
        return replace(self, **kw)


# Seeds: 20260000 + index of the workload in this list.
CONFIGS = {
    # Tiny fp32 single layer: 4 Q / 2 KV heads, d=64, 16 tokens/frame, 8 frames, B=32.
    "tiny_f32": WorkloadConfig("tiny_f32", 1, 4, 2, 64, 16, 8, 32, "f32", "iid", 20260000),
    # 7B-VLM-shaped single layer, bf16: 28 Q / 4 KV heads, d=128, 196 tokens/frame (14x14), 64 frames, B=1024.
    "vlm7b_1layer": WorkloadConfig("vlm7b_1layer", 1, 28, 4, 128, 196, 64, 1024, "bf16", "iid", 20260001),
    # 7B-VLM-shaped 28-layer stack, bf16: 512 frames, B=2048 per layer, independent stream per layer.
    "vlm7b_28layer": WorkloadConfig("vlm7b_28layer", 28, 28, 4, 128, 196, 512, 2048, "bf16", "iid", 20260002),
    # 72B-VLM-shaped 80-layer stack, bf16: 64 Q / 8 KV heads, 256 tokens/frame (16x16), 512 frames, B=4096;
    # keys share a rank-16 component plus noise so scores correlate across frames.
    "vlm72b_80layer": WorkloadConfig("vlm72b_80layer", 80, 64, 8, 128, 256, 512, 4096, "bf16", "lowrank", 20260003),
    # Stress, bf16, 1 layer: 32 Q / 8 KV heads, 729 tokens/frame (27x27), 1024 frames, B=8192;
    # 2% of tokens per frame with 4x key norm, and exact-duplicate key rows (score ties).
    "stress_1layer": WorkloadConfig("stress_1layer", 1, 32, 8, 128, 729, 1024, 8192, "bf16", "stress", 20260004),
}

ORDER = ["tiny_f32", "vlm7b_1layer", "vlm7b_28layer", "vlm72b_80layer", "stress_1layer"]


def get_config(name: str) -> WorkloadConfig:
    return CONFIGS[name]
