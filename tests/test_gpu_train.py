"""GPU parity of the training-time masked decoder (svl_train_step) against
oracle/training.py's masked_train_step, through the C ABI.

Per sample: token and unit masks exact (the decisions compare float32
z + xi with 0 on both sides, and rounding keeps the sign of a sum); the final
hidden states within 1e-4 normwise relative error (the float32 bar); the
gate-logit gradients within TOL_GRAD normwise; each token-logit gradient
within TOL_GRAD of its condition scale: dL/dz_i is the dot product
(dL/dX_0[i] . v_i) y_i (1 - y_i) / tau, whose rounding error is bounded by
the error of dL/dX_0 times sum_d |dL/dX_0[i][d] v_i[d]| y_i (1 - y_i) / tau,
so that scale (from the oracle) divides the difference.  (Gradients of
dropped tokens pass through the RMSNorm of a zero row, which scales them by
eps^(-1/2): they differ from the kept tokens' by orders, and a normwise
measure over all tokens would see only them.)

"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_20357_amd as svl
import workloads as W
from gpu_helpers import host_layer
from oracle import training as ot

pytestmark = pytest.mark.gpu

TOL_HIDDEN = 1e-4
TOL_GRAD = 1e-3


def _normwise(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    if want.size == 0:
        return 0.0
    den = np.abs(want).max()
    return float(np.abs(got - want).max() / den) if den > 0 else float(np.abs(got).max())


def _run(w, seed, prefix, units, tau_tok=0.7, tau_comp=1.3, drop_first=False, noise=True):
    s = w.shape
    B, N, T, D, L = w.batch, w.n_vision, w.n_text, s.d_model, s.n_layers
    S = N + T
    print(f"train {w.name} B={B} N={N} T={T} L={L} P={prefix} U={units} seed={seed}", flush=True)
    cfg = svl.make_config(s)
    vision, text = W.draw_hidden(w, seed, device="cuda")
    layers = [W.draw_layer_weights(w, l, seed, device="cuda") for l in range(L)]
    rng = np.random.default_rng(seed + 101)
    nl = (L - prefix) * units
    z = rng.normal(0.3, 1.5, (B, N)).astype(np.float32)
    if N:
        z[:, 0] = -20.0 if drop_first else 20.0
    g = rng.normal(0.6, 1.5, (B, nl)).astype(np.float32)
    xi = rng.logistic(0, 1, (B, N)).astype(np.float32) if noise else None
    xg = rng.logistic(0, 1, (B, nl)).astype(np.float32) if noise else None
    G = rng.standard_normal((B, S, D)).astype(np.float32)
    t = lambda a: None if a is None else torch.from_numpy(a).cuda()
    prm = svl.svl_train_params(tau_tok, tau_comp, prefix, units)
    ws = svl.alloc_train_workspace(cfg, prm, B, N, T)
    out = svl.svl_train_step(cfg, svl.LayerTable(layers), prm, t(z), t(g), vision, text, t(G), ws,
                             token_noise=t(xi), gate_noise=t(xg))
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}

    hl = [host_layer(l) for l in layers]
    vis, txt = W.as_f32(vision), W.as_f32(text)
    errs = {"hidden": 0.0, "token": 0.0, "gate": 0.0}
    for b in range(B):
        ref = ot.masked_train_step(s, lambda l: hl[l], vis[b], txt[b], z[b].astype(np.float64),
                                   g[b].astype(np.float64), G[b], prefix, units, tau_tok, tau_comp,
                                   xi_tok=None if xi is None else xi[b].astype(np.float64),
                                   xi_gate=None if xg is None else xg[b].astype(np.float64))
        np.testing.assert_array_equal(got["token_mask"][b], ref.token_mask)
        np.testing.assert_array_equal(got["unit_mask"][b], ref.unit_mask)
        errs["hidden"] = max(errs["hidden"], _normwise(got["hidden"][b], ref.hidden))
        v = z[b].astype(np.float64) + (0.0 if xi is None else xi[b].astype(np.float64))
        y = 1.0 / (1.0 + np.exp(-v / tau_tok))
        cond = np.sum(np.abs(ref.grad_x0[:N] * vis[b]), axis=1) * y * (1.0 - y) / tau_tok
        diff = np.abs(got["grad_logits"][b].astype(np.float64) - ref.grad_z)
        errs["token"] = max(errs["token"], float(np.max(diff / cond, initial=0.0)))
        errs["gate"] = max(errs["gate"], _normwise(got["grad_gate"][b], ref.grad_gate))
    print("  " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
    assert errs["hidden"] <= TOL_HIDDEN, errs
    for k in ("token", "gate"):
        assert errs[k] <= TOL_GRAD, (k, errs)
    return got


def _tiny(batch=2):
    return W.scaled(W.get_workload("tiny_f32"), batch=batch, name="tiny_f32_train")


@pytest.mark.parametrize("prefix,units", [(0, 4), (1, 4), (1, 1), (2, 1)])
def test_train_tiny_f32(prefix, units):
    _run(_tiny(), 3, prefix, units)


def test_train_tiny_first_token_dropped_and_no_noise():
    _run(_tiny(), 4, 1, 4, drop_first=True, noise=False)


def test_train_forward_only_matches_the_full_step():
    """Without grad_hidden the call runs the forward alone: same hidden states
    and masks, and no gradient outputs."""
    w = _tiny()
    s = w.shape
    cfg = svl.make_config(s)
    vision, text = W.draw_hidden(w, 5, device="cuda")
    layers = svl.LayerTable([W.draw_layer_weights(w, l, 5, device="cuda") for l in range(2)])
    rng = np.random.default_rng(5)
    z = torch.from_numpy(rng.normal(0, 2, (2, w.n_vision)).astype(np.float32)).cuda()
    g = torch.from_numpy(rng.normal(0, 2, (2, 8)).astype(np.float32)).cuda()
    G = torch.from_numpy(rng.standard_normal((2, w.n_vision + w.n_text, s.d_model))
                         .astype(np.float32)).cuda()
    prm = svl.svl_train_params(0.5, 0.5, 0, 4)
    ws = svl.alloc_train_workspace(cfg, prm, 2, w.n_vision, w.n_text)
    a = svl.svl_train_step(cfg, layers, prm, z, g, vision, text, None, ws)
    b = svl.svl_train_step(cfg, layers, prm, z, g, vision, text, G, ws)
    torch.cuda.synchronize()
    assert "grad_logits" not in a
    assert torch.equal(a["hidden"], b["hidden"])
    assert torch.equal(a["token_mask"], b["token_mask"]) and torch.equal(a["unit_mask"], b["unit_mask"])


@pytest.mark.parametrize("units", [4, 1])
def test_train_scaled_7b_bf16(units):
    w = W.scaled(W.get_workload("llava7b_b1_keep25"), n_layers=3, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, batch=2, n_vision=144, n_text=32,
                 name="llava7b_train_scaled")
    _run(w, 6, 1, units)


def test_train_scaled_gqa_bf16():
    w = W.scaled(W.get_workload("gqa7b_hires_b2"), n_layers=2, d_model=512, n_heads=4,
                 n_kv_heads=2, d_ffn=1024, batch=2, n_vision=160, n_text=48,
                 name="gqa7b_train_scaled")
    _run(w, 7, 0, 4)


def test_train_head_dim_32_gqa():
    """32-dimensional heads (8 query heads over 4 K/V heads, two per group)
    and 130 rows, three 64-row tiles with a ragged last one."""
    base = _tiny()
    shape = dataclasses.replace(base.shape, n_heads=8, n_kv_heads=4, head_dim=32)
    w = dataclasses.replace(base, shape=shape, n_vision=100, n_text=30, name="tiny_hd32_train")
    _run(w, 9, 1, 4)


@pytest.mark.parametrize("n_vision,n_text,prefix", [(0, 40, 1), (60, 0, 1), (40, 24, 2)])
def test_train_edge_shapes(n_vision, n_text, prefix):
    """No vision tokens (no token logits or gradients), no text tokens, and a
    prefix covering every layer (no gate logits or gradients)."""
    w = dataclasses.replace(_tiny(), n_vision=n_vision, n_text=n_text,
                            name=f"tiny_train_n{n_vision}_t{n_text}_p{prefix}")
    got = _run(w, 10, prefix, 4)
    assert got["token_mask"].shape == (2, n_vision)
    assert got["unit_mask"].shape == (2, (w.shape.n_layers - prefix) * 4)


def test_train_headline_width():
    """The headline's width (d_model 4096, 32 heads x 128, FFN 11008; 576 vision
    and 64 text tokens), two layers, the layer-head controller from layer 1."""
    w = W.scaled(W.get_workload("llava7b_b1_keep25"), n_layers=2, name="llava7b_train_width")
    _run(w, 8, 1, 4)
