"""Float32 model of the 16-bit path's rounding points (test infrastructure).

The GPU library computes the decoder layers with float32 accumulation and
rounds a fixed set of intermediate tensors to the 16-bit activation type:
the RMS-normed rows (attention and FFN inputs), Q/K/V after RoPE, the
unnormalised attention probabilities before the probability-value product,
the attention output and the SwiGLU output.  The residual stream stays
float32.  This module recomputes a prefill on the CPU in float32 with any
subset of those points rounded to bf16 or fp16, so that the contribution of
each rounding point to the error against the float64 oracle can be measured
at full depth without a GPU.

It is a model of the kernels' arithmetic, not a second oracle: the tests use
it to locate error sources and to check that the error of the 16-bit path is
what its rounding points explain.  It shares no code with the library or the
oracle (plain torch float32 on the CPU).
"""
from __future__ import annotations

from typing import Callable, Dict, Iterable, List, Optional, Sequence

import numpy as np
import torch

POINTS = ("xn", "qkv", "p", "o", "h")
# "xn" stands for both normed inputs; each can also be named on its own
_SUBPOINTS = {"xn": ("xn_attn", "xn_ffn")}


# "bf16x2": a value carried as two bf16 terms, hi = bf16(x) and
# lo = bf16(x - hi), whose products are summed in float32
_HILO = "bf16x2"


def _round(x: torch.Tensor, dt) -> torch.Tensor:
    if dt is None:
        return x
    if dt == _HILO:
        hi = x.to(torch.bfloat16).to(torch.float32)
        return hi + (x - hi).to(torch.bfloat16).to(torch.float32)
    return x.to(dt).to(torch.float32)


def _rms(x: torch.Tensor, g: torch.Tensor, eps: float) -> torch.Tensor:
    ms = (x * x).mean(dim=-1, keepdim=True)
    return x * torch.rsqrt(ms + eps) * g


def _rope_table(S: int, d: int, theta: float):
    # the library's table: angles in float64, then cos / sin rounded to float32
    r = np.arange(d // 2, dtype=np.float64)
    phi = np.arange(S, dtype=np.float64)[:, None] * (theta ** (-2.0 * r / d))[None, :]
    return (torch.from_numpy(np.cos(phi).astype(np.float32)),
            torch.from_numpy(np.sin(phi).astype(np.float32)))


def _rope(a: torch.Tensor, cs) -> torch.Tensor:
    c, s = cs
    h = a.shape[-1] // 2
    a1, a2 = a[..., :h], a[..., h:]
    return torch.cat([a1 * c - a2 * s, a2 * c + a1 * s], dim=-1)


_DT = {"bf16": torch.bfloat16, "f16": torch.float16, _HILO: _HILO, None: None}


class RoundedPrefill:
    """Runs the decoder layers of one sample's packed sequence in float32 with
    the rounding points `points` (a subset of POINTS) rounded to `act`
    ("bf16", "f16", "bf16x2" or None for none), or with `points` a dict
    giving each rounded point its own type.  Variants share the weights: call `layer`
    with each layer's float32 weights in turn."""

    def __init__(self, shape, x0: np.ndarray, act: Optional[str], points):
        self.shape = shape
        if isinstance(points, dict):
            types = {p: _DT[t] for p, t in points.items()}
        else:
            types = {p: _DT[act] for p in points}
        self.types = {}
        for p, t in types.items():
            for q in _SUBPOINTS.get(p, (p,)):
                self.types[q] = t
        unknown = set(self.types) - set(POINTS) - {"xn_attn", "xn_ffn"}
        if unknown:
            raise ValueError(f"unknown rounding points {sorted(unknown)}")
        self.x = torch.from_numpy(np.ascontiguousarray(x0, dtype=np.float32)).clone()
        self.cs = _rope_table(self.x.shape[0], shape.head_dim, shape.rope_theta)

    def _r(self, t: torch.Tensor, point: str) -> torch.Tensor:
        return _round(t, self.types[point]) if point in self.types else t

    def layer(self, W: Dict[str, torch.Tensor], head_on: Sequence[int],
              ffn_on: Optional[Sequence[int]]) -> None:
        s = self.shape
        A, KV, d, F, G = s.n_heads, s.n_kv_heads, s.head_dim, s.d_ffn, s.n_groups
        rep = A // KV
        x = self.x
        S = x.shape[0]
        heads = [h for h in range(A) if head_on[h]]
        if heads:
            u = self._r(_rms(x, W["attn_norm"], s.rms_eps), "xn_attn")
            kvh = sorted({h // rep for h in heads})
            outs: List[torch.Tensor] = []
            kv = {}
            for g in kvh:
                k = self._r(_rope(u @ W["wk"][g * d:(g + 1) * d].T, self.cs), "qkv")
                v = self._r(u @ W["wv"][g * d:(g + 1) * d].T, "qkv")
                kv[g] = (k, v)
            causal = torch.ones(S, S, dtype=torch.bool).tril()
            for h in heads:
                q = self._r(_rope(u @ W["wq"][h * d:(h + 1) * d].T, self.cs), "qkv")
                k, v = kv[h // rep]
                sc = (q @ k.T) * (1.0 / float(np.sqrt(d)))
                sc = sc.masked_fill(~causal, float("-inf"))
                p = torch.exp(sc - sc.max(dim=1, keepdim=True).values)
                l = p.sum(dim=1, keepdim=True)          # float32 sum of unrounded p
                o = (self._r(p, "p") @ v) / l
                outs.append(self._r(o, "o"))
            o = torch.cat(outs, dim=1)
            cols = torch.cat([torch.arange(h * d, (h + 1) * d) for h in heads])
            x = x + o @ W["wo"][:, cols].T
        if ffn_on is None:
            chans = torch.arange(F)
        else:
            w = F // G
            on = [torch.arange(j * w, (j + 1) * w) for j in range(G) if ffn_on[j]]
            chans = torch.cat(on) if on else torch.zeros(0, dtype=torch.long)
        if chans.numel():
            u = self._r(_rms(x, W["ffn_norm"], s.rms_eps), "xn_ffn")
            g_ = u @ W["w_gate"][chans].T
            e_ = u @ W["w_up"][chans].T
            h = self._r(g_ / (1.0 + torch.exp(-g_)) * e_, "h")
            x = x + h @ W["w_down"][:, chans].T
        self.x = x

    def result(self) -> np.ndarray:
        return self.x.numpy().astype(np.float64)


def normwise_error(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| / max |ref| (the parity metric of the 16-bit path)."""
    return float(np.abs(got - ref).max() / np.abs(ref).max())


def run_variants(shape, layer_weights: Callable[[int], Dict[str, torch.Tensor]], x0: np.ndarray,
                 layer_on: Sequence[int], head_mask, ffn_mask,
                 variants: Dict[str, tuple], reference: Callable[[np.ndarray, dict, int], np.ndarray],
                 report: Optional[Callable[[int, Dict[str, float]], None]] = None) -> Dict[str, float]:
    """Runs every variant (name -> (act, points)) over the executed layers of
    one sample alongside `reference(x, weights, layer)` (the float64 layer the
    variants are compared with) and returns the final normwise errors.
    `report(layer, errors)` is called after every executed layer."""
    models = {n: RoundedPrefill(shape, x0, act, pts) for n, (act, pts) in variants.items()}
    ref = np.asarray(x0, dtype=np.float64)
    errs: Dict[str, float] = {}
    for l in range(shape.n_layers):
        if not layer_on[l]:
            continue
        W = layer_weights(l)
        Wf = {k: v.to(torch.float32) for k, v in W.items()}
        ref = reference(ref, W, l)
        for m in models.values():
            m.layer(Wf, head_mask[l], None if ffn_mask is None else ffn_mask[l])
        errs = {n: normwise_error(m.result(), ref) for n, m in models.items()}
        if report is not None:
            report(l, errs)
    return errs
