"""Workload shapes and value recipes.

Five VLM-shaped prefills (a tiny single-layer case, LLaVA-1.5-7B, LLaVA-NeXT-7B
with five image tiles, a Qwen2-VL-7B-shaped GQA video prefill and a 13B-class
stress case).  Token layout follows the usual VLM prompt order: system text,
then the vision tokens, then the question text.  The paper's own benchmarks
(VQA, captioning and video datasets) are not available; these seeded synthetic
tensors stand in for them, with the shapes of the models the paper evaluates.
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    name: str
    batch: int
    layers: int
    heads_q: int
    heads_kv: int
    head_dim: int
    n_sys: int
    n_vis: int
    n_qst: int
    vis_sigma: float = 0.3          # per-token vision-key noise around the shared mean
    sink: bool = True               # key of token 0 scaled by sink_scale
    sink_scale: float = 4.0
    frames: int = 0                 # >0: vision tokens split into frames with drifting means
    frame_alpha: float = 0.1        # AR(1) innovation weight of the frame-mean random walk
    rhos: Tuple[float, ...] = (0.05,)
    decode_steps: int = 1
    fp32_data: bool = False         # the tiny case is specified in fp32
    tv_gap: float = 0.0             # >0: depth of the text-to-vision logit gap across layers (see gen)

    @property
    def n_tokens(self) -> int:
        return self.n_sys + self.n_vis + self.n_qst

    @property
    def n_text(self) -> int:
        return self.n_sys + self.n_qst

    @property
    def group(self) -> int:
        return self.heads_q // self.heads_kv

    def problem_tuple(self):
        return (self.batch, self.layers, self.heads_q, self.heads_kv, self.head_dim,
                self.n_sys, self.n_vis, self.n_qst)


CONFIGS = {
    # 1 layer, 4 heads, head_dim 64, 8 system + 144 vision + 16 question tokens, fp32.
    "tiny": WorkloadConfig("tiny", 1, 1, 4, 4, 64, 8, 144, 16, vis_sigma=0.3,
                           rhos=(0.10, 0.50, 1.0), decode_steps=1, fp32_data=True),
    # LLaVA-1.5-7B: 32 layers, 32 MHA heads, 35 + 576 + 40 tokens.
    "llava15": WorkloadConfig("llava15", 1, 32, 32, 32, 128, 35, 576, 40, vis_sigma=0.3,
                              rhos=(0.05, 0.10, 0.20), decode_steps=64),
    # LLaVA-NeXT-7B with 5 image tiles: batch 4, 35 + 2880 + 64 tokens.
    "llavanext": WorkloadConfig("llavanext", 4, 32, 32, 32, 128, 35, 2880, 64, vis_sigma=0.25,
                                rhos=(0.05,), decode_steps=128),
    # Qwen2-VL-7B GQA video: 28 layers, 28 query heads over 4 KV heads, 16 frames x 512.
    "qwen2vl_video": WorkloadConfig("qwen2vl_video", 8, 28, 28, 4, 128, 16, 8192, 48,
                                    vis_sigma=0.3, frames=16, frame_alpha=0.1,
                                    rhos=(0.05, 0.10), decode_steps=128),
    # 13B-class stress: 40 layers, 40 heads, batch 16, 35 + 2880 + 256 tokens.
    "stress13b": WorkloadConfig("stress13b", 16, 40, 40, 40, 128, 35, 2880, 256, vis_sigma=0.3,
                                rhos=(0.05,), decode_steps=256),
}

# The model shapes above draw their text queries i.i.d. N(0, 1) (tv_gap 0).  The depth
# profile is a named variant of any of them: question-row queries shifted per layer so that
# shallow layers attend to the image and middle layers hardly at all (see gen), which makes
# TVB's layer budgets spread out over an order of magnitude.
DEPTH_PROFILE_TV_GAP = 6.0


def depth_profile(cfg: "WorkloadConfig", tv_gap: float = DEPTH_PROFILE_TV_GAP) -> "WorkloadConfig":
    """The same workload with the per-layer text-to-vision depth profile (only the question-row
    queries change; keys, values and decode inputs are the same draws)."""
    return dataclasses.replace(cfg, tv_gap=float(tv_gap))


# Ordered as the configs are listed: tiny first, then the four model shapes.
CONFIG_ORDER = ("tiny", "llava15", "llavanext", "qwen2vl_video", "stress13b")


def get_config(name: str) -> WorkloadConfig:
    return CONFIGS[name]


def custom_config(name: str = "custom", *, batch=1, layers=2, heads_q=4, heads_kv=2,
                  head_dim=128, n_sys=5, n_vis=100, n_qst=11, vis_sigma=0.3, sink=True,
                  frames=0, rhos=(0.2,), decode_steps=2, fp32_data=False,
                  frame_alpha=0.1, tv_gap=0.0) -> WorkloadConfig:
    """A small shape for parity tests: spans several kernel tiles with ragged tails."""
    return WorkloadConfig(name, batch, layers, heads_q, heads_kv, head_dim, n_sys, n_vis, n_qst,
                          vis_sigma=vis_sigma, sink=sink, frames=frames, frame_alpha=frame_alpha,
                          rhos=tuple(rhos), decode_steps=decode_steps, fp32_data=fp32_data, tv_gap=tv_gap)


def with_shape(cfg: WorkloadConfig, **changes) -> WorkloadConfig:
    return dataclasses.replace(cfg, **changes)


def frame_size(cfg: WorkloadConfig) -> Optional[int]:
    if cfg.frames <= 0:
        return None
    if cfg.n_vis % cfg.frames != 0:
        raise ValueError("n_vis must split evenly into frames")
    return cfg.n_vis // cfg.frames
