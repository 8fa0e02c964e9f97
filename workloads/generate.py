"""Seeded draws of every input the prefill consumes.

Every tensor has its own seed derived from (seed, stream, layer, tensor id)
through numpy's SeedSequence, so any subset (one layer's weights, one sample's
scores) can be regenerated alone, on the host or on a GPU.

* small inputs (scores, keep budgets, masks) are drawn with numpy PCG64 on the
  host and are identical everywhere;
* large inputs (hidden states, weights) are drawn with torch's generator on the
  requested device.  Draws on different devices differ, so a test draws once
  and hands the same values to both the GPU path and the oracle.

Laws (recipe stated once for all workloads):
  linear weights  N(0, 0.02^2);  norm gains 1 + N(0, 0.02^2);
  vision / text hidden states N(0, 1);
  compute controller (budget MLP, token-count MLP, gating head): first
  linears N(0, 2/E) with E the encoding width, second linears N(0, 1/H) with
  H the hidden width, their biases N(0, 0.1^2); gating weights
  N(0, gate_std^2 / D); gating biases c = +-(0.5 + spacing * rank) with rank
  a random permutation of the units and the sign + with probability p_on,
  so the bias fixes each unit's on/off decision and every pair of logits
  stays apart by about `spacing`;
  bf16 workloads round every weight and hidden value to bfloat16
  (round-to-nearest-even) -- the oracle sees the same values widened to fp32;
  scores stay fp32.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np
import torch

from .configs import Workload, keep_count

STREAM_SCORES = 1
STREAM_HIDDEN = 2
STREAM_MASKS = 3
STREAM_WEIGHTS = 4
STREAM_CONTROLLER = 5

WEIGHT_NAMES = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def _seed(*parts: int) -> int:
    st = np.random.SeedSequence([int(p) for p in parts]).generate_state(2, np.uint32)
    return (int(st[0]) << 31) ^ int(st[1])


def _np_rng(*parts: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(p) for p in parts])))


def storage_dtype(w: Workload) -> torch.dtype:
    return torch.bfloat16 if w.shape.dtype == "bf16" else torch.float32


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bfloat16 (ties to even), kept as fp32."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


# --------------------------------------------------------------------------- scores
def _smooth(noise: np.ndarray, sigma: float) -> np.ndarray:
    from scipy.ndimage import gaussian_filter
    return gaussian_filter(noise, sigma=sigma, mode="reflect", truncate=4.0)


def draw_scores(w: Workload, seed: int = 0) -> np.ndarray:
    """Vision-token scores, fp32 [B][N] (what the token controller would emit)."""
    out = np.empty((w.batch, w.n_vision), dtype=np.float32)
    for b in range(w.batch):
        rng = _np_rng(seed, STREAM_SCORES, b)
        n = w.n_vision
        if w.score_law == "uniform":
            s = rng.random(n)
        elif w.score_law == "lognormal":
            s = np.exp(rng.standard_normal(n))
        elif w.score_law in ("smooth_crops", "smooth_video"):
            grid = tuple(w.score_grid)
            if int(np.prod(grid)) != n:
                grid = (n,)
            z = rng.standard_normal(grid)
            if w.score_law == "smooth_crops" and len(grid) == 3:
                # each crop is smoothed on its own 2-D grid, crops concatenated
                s = np.concatenate([_smooth(z[c], w.score_sigma).ravel() for c in range(grid[0])])
            else:
                s = _smooth(z, w.score_sigma).ravel()
        else:
            raise ValueError(f"unknown score law {w.score_law}")
        out[b] = s.astype(np.float32)
    return out


# --------------------------------------------------------------------------- masks
def draw_masks(w: Workload, seed: int = 0):
    """Keep budgets and masks as the controllers would hand them over.

    Returns keep int32 [B], layer_mask uint8 [B][L], head_mask uint8 [B][L][A],
    ffn_mask uint8 [B][L][G] (None when the FFN is not coupled to the groups).
    Head group j is the contiguous head range [j*A/G, (j+1)*A/G); skipped
    layers are drawn without replacement from the non-prefix layers [L/2, L).
    """
    s = w.shape
    B, L, A, G = w.batch, s.n_layers, s.n_heads, s.n_groups
    keep = np.zeros(B, dtype=np.int32)
    layer_mask = np.ones((B, L), dtype=np.uint8)
    head_mask = np.ones((B, L, A), dtype=np.uint8)
    group_mask = np.ones((B, L, G), dtype=np.uint8)
    per_group = A // G
    for b in range(B):
        rng = _np_rng(seed, STREAM_MASKS, b)
        ratio = w.keep_ratio if w.keep_choices is None else float(rng.choice(w.keep_choices))
        keep[b] = keep_count(ratio, w.n_vision)
        if w.groups_keep_choices is not None:
            n_off = G - int(rng.choice(w.groups_keep_choices))
        else:
            n_off = w.groups_off
        if w.layers_skipped_range is not None:
            lo, hi = w.layers_skipped_range
            n_skip = int(rng.integers(lo, hi + 1))
        else:
            n_skip = w.layers_skipped
        n_skip = min(n_skip, L - s.prefix)
        if n_skip > 0:
            skipped = rng.choice(np.arange(s.prefix, L), size=n_skip, replace=False)
            layer_mask[b, skipped] = 0
        for l in range(L):
            if n_off > 0:
                off = rng.choice(G, size=n_off, replace=False)
                group_mask[b, l, off] = 0
            for j in range(G):
                head_mask[b, l, j * per_group:(j + 1) * per_group] = group_mask[b, l, j]
    ffn_mask = group_mask if w.ffn_coupled else None
    return keep, layer_mask, head_mask, ffn_mask


# --------------------------------------------------------------------------- tensors
def _randn(shape, seed: int, device, std: float = 1.0, mean: float = 0.0) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t


def draw_hidden(w: Workload, seed: int = 0, device="cpu"):
    """Projected vision tokens [B][N][D] and text embeddings [B][T][D] (storage dtype)."""
    D = w.shape.d_model
    dt = storage_dtype(w)
    vision = _randn((w.batch, w.n_vision, D), _seed(seed, STREAM_HIDDEN, 0), device).to(dt)
    text = _randn((w.batch, w.n_text, D), _seed(seed, STREAM_HIDDEN, 1), device).to(dt)
    return vision, text


def draw_layer_weights(w: Workload, layer: int, seed: int = 0, device="cpu") -> Dict[str, torch.Tensor]:
    """One decoder layer's weights in nn.Linear layout [out][in], storage dtype."""
    s = w.shape
    D, A, KV, d, F = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.d_ffn
    shapes = {
        "attn_norm": (D,), "wq": (A * d, D), "wk": (KV * d, D), "wv": (KV * d, D),
        "wo": (D, A * d), "ffn_norm": (D,), "w_gate": (F, D), "w_up": (F, D), "w_down": (D, F),
    }
    dt = storage_dtype(w)
    out = {}
    for i, name in enumerate(WEIGHT_NAMES):
        sd = _seed(seed, STREAM_WEIGHTS, layer, i)
        if name.endswith("norm"):
            t = _randn(shapes[name], sd, device, std=0.02, mean=1.0)
        else:
            t = _randn(shapes[name], sd, device, std=0.02)
        out[name] = t.to(dt).contiguous()
    return out


@dataclass
class Inputs:
    workload: Workload
    seed: int
    scores: np.ndarray          # f32 [B][N]
    keep: np.ndarray            # i32 [B]
    layer_mask: np.ndarray      # u8 [B][L]
    head_mask: np.ndarray       # u8 [B][L][A]
    ffn_mask: Optional[np.ndarray]  # u8 [B][L][G] or None
    vision: torch.Tensor        # [B][N][D] storage dtype
    text: torch.Tensor          # [B][T][D] storage dtype


def draw_inputs(w: Workload, seed: int = 0, device="cpu") -> Inputs:
    keep, layer_mask, head_mask, ffn_mask = draw_masks(w, seed)
    vision, text = draw_hidden(w, seed, device)
    return Inputs(w, seed, draw_scores(w, seed), keep, layer_mask, head_mask, ffn_mask,
                  vision, text)


def as_f32(t: torch.Tensor) -> np.ndarray:
    """Host fp32 copy of a tensor (bf16 widens exactly)."""
    return t.detach().to("cpu", torch.float32).numpy()


# --------------------------------------------------------------------------- controller
CONTROLLER_NAMES = ("llm_w1", "llm_b1", "llm_w2", "llm_b2", "kap_w1", "kap_b1", "kap_w2",
                    "kap_b2", "gate_w", "gate_b")


@dataclass
class ControllerDraw:
    prefix: int
    units: int
    pe_dim: int
    hidden: int
    pe_scale: float
    pe_base: float
    tensors: Dict[str, torch.Tensor]     # CONTROLLER_NAMES, storage dtype, [out][in]


def draw_controller(w: Workload, seed: int = 0, device="cpu", *, prefix: Optional[int] = None,
                    units: Optional[int] = None, pe_dim: int = 256, hidden: Optional[int] = None,
                    pe_scale: float = 1000.0, pe_base: float = 10000.0, p_on: float = 0.75,
                    spacing: float = 0.1, gate_std: float = 0.002) -> ControllerDraw:
    """Compute-controller parameters of a workload's decoder (law above)."""
    s = w.shape
    P = s.prefix if prefix is None else prefix
    U = s.n_groups if units is None else units
    H = s.d_model if hidden is None else hidden
    D, n = s.d_model, (s.n_layers - P) * U
    dt = storage_dtype(w)
    shapes = {"llm_w1": (H, pe_dim), "llm_b1": (H,), "llm_w2": (D, H), "llm_b2": (D,),
              "kap_w1": (H, pe_dim), "kap_b1": (H,), "kap_w2": (D, H), "kap_b2": (D,),
              "gate_w": (n, D)}
    stds = {"llm_w1": (2.0 / pe_dim) ** 0.5, "kap_w1": (2.0 / pe_dim) ** 0.5,
            "llm_w2": (1.0 / H) ** 0.5, "kap_w2": (1.0 / H) ** 0.5, "gate_w": gate_std / D ** 0.5}
    out = {}
    for i, name in enumerate(CONTROLLER_NAMES[:-1]):
        sd = _seed(seed, STREAM_CONTROLLER, i)
        out[name] = _randn(shapes[name], sd, device, std=stds.get(name, 0.1)).to(dt).contiguous()
    rng = _np_rng(seed, STREAM_CONTROLLER, 99)
    mag = 0.5 + spacing * rng.permutation(n)
    sign = np.where(rng.random(n) < p_on, 1.0, -1.0)
    gb = torch.from_numpy((sign * mag).astype(np.float32))
    out["gate_b"] = gb.to(device=device, dtype=dt).contiguous()
    return ControllerDraw(P, U, pe_dim, H, pe_scale, pe_base, out)
