"""Shared drivers of the GPU parity tests: run the library through the C ABI
and the CPU oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2607_20357_amd as svl
import workloads as W

FP32_TOL = 1e-4
BF16_TOL = 2e-2


def tol_for(shape) -> float:
    return FP32_TOL if shape.dtype == "f32" else BF16_TOL


def rel_err_per_sample(got: np.ndarray, ref: np.ndarray, cu) -> list:
    """Normwise max relative error per sample: max|g - o| / max|o|."""
    out = []
    for b in range(len(cu) - 1):
        g = got[cu[b]:cu[b + 1]].astype(np.float64)
        o = ref[cu[b]:cu[b + 1]]
        if o.size == 0:
            out.append(0.0)
            continue
        den = np.abs(o).max()
        out.append(float(np.abs(g - o).max() / den) if den > 0 else float(np.abs(g).max()))
    return out


def elementwise_err_per_sample(got: np.ndarray, ref: np.ndarray, cu) -> list:
    """Elementwise diagnostic per sample: max over entries of
    |g - o| / max(|o|, rms(o)), the rms taken over the sample's entries.  It
    sees drift confined to small-magnitude rows or columns (text rows, one
    head's contribution) that the normwise figure averages away."""
    out = []
    for b in range(len(cu) - 1):
        g = got[cu[b]:cu[b + 1]].astype(np.float64)
        o = ref[cu[b]:cu[b + 1]]
        if o.size == 0:
            out.append(0.0)
            continue
        rms = float(np.sqrt(np.mean(o * o)))
        den = np.maximum(np.abs(o), rms if rms > 0 else 1.0)
        out.append(float((np.abs(g - o) / den).max()))
    return out


def host_layer(layer):
    return {k: W.as_f32(v) for k, v in layer.items()}


def gpu_prefill(w, inp, layers, dev="cuda", table=None, compute="f16"):
    cfg = svl.make_config(w.shape, compute=compute)
    B, N = inp.scores.shape
    R = int((np.asarray(inp.keep) + w.n_text).sum())
    scores = torch.from_numpy(np.ascontiguousarray(inp.scores)).to(dev)
    kept = torch.full((B, max(N, 1)), -7, dtype=torch.int32, device=dev)[:, :N].contiguous()
    resid = torch.full((max(R, 1), w.shape.d_model), float("nan"), dtype=torch.float32,
                       device=dev)[:R]
    ws = svl.alloc_workspace(cfg, B, R, dev)
    cu, flops = svl.svl_prefill(cfg, table or layers, inp.keep, scores, inp.vision, inp.text,
                                inp.layer_mask, inp.head_mask, inp.ffn_mask, kept, resid, ws)
    torch.cuda.synchronize()
    return kept.cpu().numpy(), cu, resid.cpu().numpy(), flops


def oracle_prefill(w, inp, layers, samples=None):
    sel = slice(None) if samples is None else list(samples)
    lm = inp.layer_mask[sel]
    deep = w.shape.n_layers >= 16

    def layer(l):
        if deep:
            print(f"  oracle layer {l}", flush=True)   # progress of a long reference run
        return host_layer(layers[l])
    return oracle.prefill(w.shape, layer, inp.scores[sel],
                          np.asarray(inp.keep)[sel], W.as_f32(inp.vision[sel]),
                          W.as_f32(inp.text[sel]), lm, inp.head_mask[sel],
                          None if inp.ffn_mask is None else inp.ffn_mask[sel])


def host_controller(draw):
    """oracle.controller.Controller with the drawn controller's values (fp32 widened)."""
    from oracle.controller import Controller
    t = {k: W.as_f32(v).astype(np.float64) for k, v in draw.tensors.items()}
    return Controller(prefix=draw.prefix, units=draw.units, pe_scale=float(np.float32(draw.pe_scale)),
                      pe_base=float(np.float32(draw.pe_base)), **t)
