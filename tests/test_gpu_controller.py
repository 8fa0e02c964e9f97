"""GPU parity of the controlled prefill (svl_prefill_controlled): the compute
controller's budget token, kappa embedding and gating head, the masks it
derives, the budget projection at the prefix boundary and the layers around
it, against oracle/controller.py on the same seeded inputs.

Bars: threshold counts, final keep counts, kept indices, cu_seqlens, masks
and FLOP counts exact; the gating head's term W_h h~ (gate logits minus their
bias) and the hidden states within max relative error 1e-4 (float32) / 2e-2
(bf16).  A unit's on/off decision is taken on float32 logits on the GPU and
float64 ones in the oracle; the controller weights are drawn so that every
logit lies at least 0.5 from 0 and the logits stay apart from each other (the
projection's drop order), and each case asserts those margins on the
oracle's logits before comparing decisions, so that both sides must agree."""
import numpy as np
import pytest
import torch

import paper_2607_20357_amd as svl
import workloads as W
from gpu_helpers import host_controller, host_layer, rel_err_per_sample, tol_for
from oracle import controller as oc

pytestmark = pytest.mark.gpu


def _run(w, seed, prefix, units, budget, shift, pe_dim=64, hidden=128, vocab=0, compute="f16"):
    print(f"controlled {w.name} seed={seed} P={prefix} units={units} b={budget} "
          f"compute={compute}", flush=True)
    dev = "cuda"
    shape = w.shape
    cfg = svl.make_config(shape, compute=compute)
    inp = W.draw_inputs(w, seed, device=dev)
    layers = [W.draw_layer_weights(w, l, seed, device=dev) for l in range(shape.n_layers)]
    draw = W.draw_controller(w, seed, device=dev, prefix=prefix, units=units, pe_dim=pe_dim,
                             hidden=hidden)
    ctrl = svl.Controller(draw.prefix, draw.units, draw.pe_dim, draw.hidden, draw.pe_scale,
                          draw.pe_base, draw.tensors)
    rng = np.random.default_rng(seed + 17)
    B, N, T, D = w.batch, w.n_vision, w.n_text, shape.d_model
    z = (rng.standard_normal((B, N)) + shift).astype(np.float32)
    logits = torch.from_numpy(z).to(dev)
    kept = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    resid = torch.full((B * (N + T + 1), D), float("nan"), dtype=torch.float32, device=dev)
    ws = svl.alloc_controlled_workspace(cfg, ctrl, B, N, T, dev)
    out = svl.svl_prefill_controlled(cfg, svl.LayerTable(layers), ctrl, logits, inp.vision,
                                     inp.text, budget, vocab, kept, resid, ws)
    torch.cuda.synchronize()
    # finite inputs and weights: the call's status word is clear
    assert svl.svl_workspace_status(ws) == 0

    ref = oc.prefill_controlled(shape, lambda l: host_layer(layers[l]), host_controller(draw), z,
                                W.as_f32(inp.vision), W.as_f32(inp.text), budget, vocab)
    # decisions are only comparable away from the threshold and from ties
    lg = ref.logits
    assert np.abs(lg).min() > 0.3, "a gate logit too close to 0 for an exact mask comparison"
    for b in range(B):
        srt = np.sort(lg[b])
        assert srt.size < 2 or np.diff(srt).min() > 1e-2, "two gate logits too close"
    tol = tol_for(shape)
    bias = W.as_f32(draw.tensors["gate_b"]).astype(np.float64)
    term_g = out["gate_logits"].astype(np.float64) - bias
    term_o = lg - bias
    # bar: tol relative to the term, plus 2 float32 ulps of the stored logit
    # (the bias is subtracted from a float32 logit on the host)
    gbar = tol * np.abs(term_o).max() + 2.0 ** -22 * np.abs(lg).max()
    gdiff = np.abs(term_g - term_o).max()
    print(f"  gate term err {gdiff:.2e} (bar {gbar:.2e}); keep {out['keep'].tolist()} of "
          f"{ref.counts.tolist()}", flush=True)
    assert gdiff <= gbar, (gdiff, gbar)

    np.testing.assert_array_equal(out["keep"], ref.keep)
    np.testing.assert_array_equal(out["layer_mask"], ref.layer_mask)
    np.testing.assert_array_equal(out["head_mask"], ref.head_mask)
    np.testing.assert_array_equal(out["ffn_mask"], ref.ffn_mask)
    np.testing.assert_array_equal(out["cu_seqlens"], ref.cu_seqlens)
    np.testing.assert_array_equal(kept.cpu().numpy(), ref.kept_idx)
    R = int(ref.cu_seqlens[-1])
    got = resid[:R].cpu().numpy()
    errs = rel_err_per_sample(got, ref.resid, ref.cu_seqlens)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol, errs
    assert out["flops"]["total"] == ref.flops.total
    for k in ("q", "kv", "o", "attn", "ffn"):
        assert out["flops"][k] == getattr(ref.flops, k), k
    return out, ref


TINY4 = W.scaled(W.get_workload("tiny_f32"), n_layers=4, batch=3, n_vision=40, n_text=6,
                 name="ctrl_tiny_f32")


@pytest.mark.parametrize("budget", [1.0, 0.4])
def test_controlled_tiny_f32_layer_head(budget):
    out, ref = _run(TINY4, 1, prefix=2, units=4, budget=budget, shift=0.2)
    if budget < 1:
        assert np.all(ref.keep < ref.counts)      # tokens left at the prefix boundary


def _raw_masks(w, ref, prefix, units):
    return [oc.masks_from_logits(w.shape, ref.logits[b], prefix, units) for b in range(w.batch)]


def test_controlled_tiny_f32_layer_controller_drops_layers():
    """Layer controller with a budget so small that zero visual tokens do not
    fit: the projection then drops whole dynamic layers."""
    out, ref = _run(TINY4, 2, prefix=1, units=1, budget=0.05, shift=0.5)
    raw = _raw_masks(TINY4, ref, 1, 1)
    assert any(not np.array_equal(ref.layer_mask[b], raw[b][0]) for b in range(TINY4.batch))


def test_controlled_tiny_f32_prefix0_and_group_drops():
    """P = 0 (the controller reads the budget token as embedded) and a budget
    that forces the projection to drop head groups."""
    out, ref = _run(TINY4, 3, prefix=0, units=4, budget=0.05, shift=0.0)
    raw = _raw_masks(TINY4, ref, 0, 4)
    assert any(not np.array_equal(ref.head_mask[b], raw[b][1]) for b in range(TINY4.batch))


def test_controlled_bf16_ragged_batch():
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=8,
                 n_kv_heads=8, d_ffn=1024, batch=4, n_vision=200, n_text=24, name="ctrl_b4")
    out, ref = _run(w, 4, prefix=1, units=4, budget=0.4, shift=-0.2)
    # some samples are trimmed at the prefix boundary, others keep every token
    assert (ref.keep < ref.counts).any() and (ref.keep == ref.counts).any()


def test_controlled_bf16_activations():
    """The ragged batch of the test above with bf16 activations and products
    (the normed rows' low bf16 terms in the QKV and gate/up products)."""
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=8,
                 n_kv_heads=8, d_ffn=1024, batch=4, n_vision=200, n_text=24, name="ctrl_b4_bf16")
    _run(w, 4, prefix=1, units=4, budget=0.4, shift=-0.2, compute="bf16")


def test_controlled_bf16_gqa_layer_controller():
    w = W.scaled(W.get_workload("gqa7b_hires_b2"), n_layers=4, d_model=512, n_heads=8,
                 n_kv_heads=2, d_ffn=1024, n_vision=300, n_text=20, name="ctrl_gqa")
    _run(w, 5, prefix=2, units=1, budget=0.5, shift=0.0)


def test_controlled_headline_full_size():
    """LLaVA-1.5-7B shape, one sample of 576 + 64 tokens, 16 prefix layers,
    encoding width 256 and hidden width 4096, budget 0.25 of C_full."""
    w = W.get_workload("llava7b_b1_keep25")
    out, ref = _run(w, 0, prefix=16, units=4, budget=0.25, shift=-0.6745, pe_dim=256,
                    hidden=4096)
    assert ref.keep[0] < ref.counts[0]


def test_controlled_near_zero_gate_logits_are_self_consistent():
    """Sample 0's gate logits placed within float32 rounding of zero, where the
    library's float32 decisions and the oracle's float64 ones may disagree.
    Whatever the library decides must follow from its own reported float32
    logits by the rule (a unit runs iff its logit > 0, then the budget
    projection with the logits as confidences), and its hidden states must
    equal the oracle's layers run under those decisions (same bar as the
    other cases); the other samples keep ordinary logits and full parity."""
    w = TINY4
    seed, prefix, units, budget = 6, 1, 4, 0.6
    print(f"controlled near-zero gates {w.name} seed={seed}", flush=True)
    shape = w.shape
    cfg = svl.make_config(shape)
    inp = W.draw_inputs(w, seed, device="cuda")
    layers = [W.draw_layer_weights(w, l, seed, device="cuda") for l in range(shape.n_layers)]
    draw = W.draw_controller(w, seed, device="cuda", prefix=prefix, units=units)
    rng = np.random.default_rng(seed + 17)
    B, N, T, D = w.batch, w.n_vision, w.n_text, shape.d_model
    z = (rng.standard_normal((B, N)) + 0.2).astype(np.float32)
    hl = [host_layer(l) for l in layers]
    vis, txt = W.as_f32(inp.vision), W.as_f32(inp.text)
    ref = oc.prefill_controlled(shape, lambda l: hl[l], host_controller(draw), z, vis, txt, budget, 0)
    # new biases: sample 0's float64 logits become 1e-9 of either sign
    bias = W.as_f32(draw.tensors["gate_b"]).astype(np.float64)
    sign = np.where(np.arange(bias.size) % 2 == 0, 1.0, -1.0)
    nb = (bias - ref.logits[0] + 1e-9 * sign).astype(np.float32)
    tensors = dict(draw.tensors)
    tensors["gate_b"] = torch.from_numpy(nb).to(draw.tensors["gate_b"].device).to(
        draw.tensors["gate_b"].dtype)
    ctrl = svl.Controller(draw.prefix, draw.units, draw.pe_dim, draw.hidden, draw.pe_scale,
                          draw.pe_base, tensors)
    logits = torch.from_numpy(z).cuda()
    kept = torch.full((B, N), -7, dtype=torch.int32, device="cuda")
    resid = torch.full((B * (N + T + 1), D), float("nan"), dtype=torch.float32, device="cuda")
    ws = svl.alloc_controlled_workspace(cfg, ctrl, B, N, T, "cuda")
    out = svl.svl_prefill_controlled(cfg, svl.LayerTable(layers), ctrl, logits, inp.vision,
                                     inp.text, budget, 0, kept, resid, ws)
    torch.cuda.synchronize()
    g = out["gate_logits"].astype(np.float64)
    assert np.abs(g[0]).max() < 1e-4, "sample 0's logits should sit at zero"
    for b in range(B):
        k, lo, ho, fo = oc.decide_sample(shape, z[b], g[b], T, budget, 0, prefix, units)
        assert int(out["keep"][b]) == k, b
        np.testing.assert_array_equal(out["layer_mask"][b], lo)
        np.testing.assert_array_equal(out["head_mask"][b], ho)
        np.testing.assert_array_equal(out["ffn_mask"][b], fo)
    kidx, cu, res = oc.finish_controlled(shape, lambda l: hl[l], ref.prefix_resid, z, ref.counts,
                                         out["keep"], out["layer_mask"], out["head_mask"],
                                         out["ffn_mask"], prefix, T)
    np.testing.assert_array_equal(out["cu_seqlens"], cu)
    np.testing.assert_array_equal(kept.cpu().numpy(), kidx)
    errs = rel_err_per_sample(resid[:int(cu[-1])].cpu().numpy(), res, cu)
    print(f"  sample 0 units on: {int(out['head_mask'][0].sum())}; rel err per sample: "
          f"{[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(shape), errs
