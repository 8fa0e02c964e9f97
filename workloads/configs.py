"""Model shapes and batch recipes for the five measured workloads.

Each workload is a decoder shape (LLaMA-style block: RMSNorm, rotate-half
RoPE, causal multi-head or grouped-query attention, SwiGLU MLP, no biases)
plus a recipe for the inputs the controllers would hand the prefill: per-token
vision scores, a keep budget, and layer / head-group masks.

Shapes follow the backbones the paper evaluates (Sec. 4.1: LLaVA-1.5-7B, and
Sec. 4.4: LLaVA-1.5-13B with 40 layers and a 20-layer prefix), the CLIP
576-token image grid (Sec. 1) and the head-group count G=4 for A=32 heads
(Sec. 3.2, layer-head controller).  Nothing here performs the method's
arithmetic; it only fixes sizes and the laws the generator draws from.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional, Sequence


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    n_groups: int = 4
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    dtype: str = "bf16"          # "f32" or "bf16": weights and hidden inputs

    @property
    def prefix(self) -> int:
        """Layers that always run at full capacity (first half of the stack)."""
        return self.n_layers // 2

    @property
    def qkv_width(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    batch: int
    n_vision: int
    n_text: int
    # keep ratio: one value for every sample, or a set each sample draws from
    keep_ratio: float = 1.0
    keep_choices: Optional[Sequence[float]] = None
    # head-group gating: groups switched off in every executed layer, or a
    # per-sample draw of the number of groups kept
    groups_off: int = 0
    groups_keep_choices: Optional[Sequence[int]] = None
    # layer skipping: fixed count per sample, or a per-sample uniform count
    layers_skipped: int = 0
    layers_skipped_range: Optional[Sequence[int]] = None
    score_law: str = "uniform"   # uniform | lognormal | smooth_crops | smooth_video
    score_grid: Sequence[int] = field(default_factory=tuple)
    score_sigma: float = 2.0
    ffn_coupled: bool = True     # FFN slice j follows head group j
    description: str = ""


def keep_count(ratio: float, n: int) -> int:
    """Integer keep budget for a ratio: nearest integer, halves rounded up."""
    return int(math.floor(ratio * n + 0.5))


TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                  d_ffn=688, n_groups=4, dtype="f32")
LLAVA7B = ModelShape(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
                     head_dim=128, d_ffn=11008, n_groups=4)
GQA7B = ModelShape(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4,
                   head_dim=128, d_ffn=18944, n_groups=4)
LLAVA13B = ModelShape(n_layers=40, d_model=5120, n_heads=40, n_kv_heads=40,
                      head_dim=128, d_ffn=13824, n_groups=4)

WORKLOADS = {
    w.name: w for w in [
        Workload(
            name="tiny_f32", shape=TINY, batch=1, n_vision=64, n_text=16,
            keep_ratio=0.5, groups_off=1, layers_skipped=0,
            score_law="uniform",
            description="2-layer d256 fp32 decoder; keep 32 of 64 vision tokens; "
                        "3 of 4 heads per layer; no skips"),
        Workload(
            name="llava7b_b1_keep25", shape=LLAVA7B, batch=1, n_vision=576, n_text=64,
            keep_ratio=0.25, groups_off=1, layers_skipped=8,
            score_law="lognormal",
            description="LLaVA-1.5-7B-shaped prefill, batch 1, 576+64 tokens, keep 144, "
                        "8 of 32 heads off per layer, 8 of 32 layers skipped, bf16"),
        Workload(
            name="llava7b_b8_ragged", shape=LLAVA7B, batch=8, n_vision=576, n_text=64,
            keep_choices=(1.0, 0.5, 0.25, 0.11), groups_keep_choices=(4, 3, 2),
            layers_skipped_range=(0, 12), score_law="lognormal",
            description="7B shape, batch 8, per-sample keep/head-keep/skip draws, bf16"),
        Workload(
            name="gqa7b_hires_b2", shape=GQA7B, batch=2, n_vision=2880, n_text=128,
            keep_ratio=0.2, groups_off=1, layers_skipped=6,
            score_law="smooth_crops", score_grid=(5, 24, 24), score_sigma=2.0,
            description="GQA 28q/4kv, batch 2, 5 crops x 576 + 128 text, keep 0.2, "
                        "1 of 4 KV groups off, 6 of 28 layers skipped, bf16"),
        Workload(
            name="llava13b_video_b4", shape=LLAVA13B, batch=4, n_vision=3136, n_text=64,
            keep_ratio=0.1, groups_off=2, layers_skipped=10,
            score_law="smooth_video", score_grid=(16, 14, 14), score_sigma=2.0,
            description="13B shape, batch 4, 16x196 video tokens + 64 text, keep 0.1, "
                        "2 of 4 groups off, 10 of 40 layers skipped, bf16"),
    ]
}

HEADLINE = "llava7b_b1_keep25"


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def scaled(w: Workload, *, n_layers: Optional[int] = None, d_model: Optional[int] = None,
           n_heads: Optional[int] = None, n_kv_heads: Optional[int] = None,
           d_ffn: Optional[int] = None, batch: Optional[int] = None,
           n_vision: Optional[int] = None, n_text: Optional[int] = None,
           layers_skipped: Optional[int] = None, name: Optional[str] = None) -> Workload:
    """A smaller copy of a workload with the same recipe (for fast parity runs)."""
    s = w.shape
    shape = ModelShape(
        n_layers=n_layers or s.n_layers, d_model=d_model or s.d_model,
        n_heads=n_heads or s.n_heads, n_kv_heads=n_kv_heads or s.n_kv_heads,
        head_dim=s.head_dim, d_ffn=d_ffn or s.d_ffn, n_groups=s.n_groups,
        rms_eps=s.rms_eps, rope_theta=s.rope_theta, dtype=s.dtype)
    kw = dict(w.__dict__)
    kw.update(shape=shape, name=name or (w.name + "_scaled"))
    if batch is not None:
        kw["batch"] = batch
    if n_vision is not None:
        kw["n_vision"] = n_vision
    if n_text is not None:
        kw["n_text"] = n_text
    if layers_skipped is not None:
        kw["layers_skipped"] = layers_skipped
    return Workload(**kw)
