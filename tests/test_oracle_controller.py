"""Pins of the compute-controller oracle (CPU only).

Each check ties oracle/controller.py to something outside itself: the
standard normal distribution function of scipy (GELU), torch's float64
linear / GELU layers (the MLPs), scipy's logistic function (kappa and the
sigma > 0.5 rule), closed forms and invariants of the sinusoidal encoding,
brute-force mask expansion, and the already-pinned prefill oracle as the
special cases the controlled prefill reduces to.
"""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
from oracle import budget as ob
from oracle import controller as oc
import workloads as W
from gpu_helpers import host_controller, host_layer

SHAPE_W = W.scaled(W.get_workload("tiny_f32"), n_layers=4, batch=2, n_vision=24, n_text=5,
                   name="ctrl_tiny")


# ============================================================================ encoding
def test_sinusoidal_closed_forms():
    """Width 2 is (sin xs, cos xs); PE(0) alternates 0, 1; the squared norm is
    E/2; the dot product of two encodings depends only on their difference,
    sum_i cos((x - y) s w_i) (the shift property of the Transformer encoding)."""
    for x in (0.0, 0.25, 1.0, 0.7):
        np.testing.assert_allclose(oc.sinusoidal(x, 2, 3.0, 10000.0),
                                   [math.sin(3 * x), math.cos(3 * x)], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(oc.sinusoidal(0.0, 8, 1000.0, 10000.0), [0, 1] * 4)
    rng = np.random.default_rng(0)
    E, s, base = 64, 1000.0, 10000.0
    w = base ** (-2.0 * np.arange(E // 2) / E)
    for _ in range(10):
        x, y = rng.random(2)
        px, py = oc.sinusoidal(x, E, s, base), oc.sinusoidal(y, E, s, base)
        assert abs(px @ px - E / 2) < 1e-12
        assert abs(px @ py - np.sum(np.cos((x - y) * s * w))) < 1e-9
    # entry pairs are ordered by frequency: for a tiny x, sin(x s w_i) ~ x s w_i
    tiny = oc.sinusoidal(1e-9, E, s, base)
    np.testing.assert_allclose(tiny[2::2] / tiny[0:-2:2], base ** (-2.0 / E), rtol=1e-9)


def test_gelu_is_x_times_normal_cdf():
    x = np.linspace(-6, 6, 241)
    np.testing.assert_allclose(oc.gelu(x), x * scipy.stats.norm.cdf(x), rtol=1e-13, atol=1e-15)


def test_mlp_matches_torch_float64():
    rng = np.random.default_rng(1)
    E, H, D = 16, 24, 10
    w1, b1 = rng.normal(size=(H, E)), rng.normal(size=H)
    w2, b2 = rng.normal(size=(D, H)), rng.normal(size=D)
    x = rng.normal(size=E)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    ref = torch.nn.functional.linear(
        torch.nn.functional.gelu(torch.nn.functional.linear(t(x), t(w1), t(b1)), approximate="none"),
        t(w2), t(b2)).numpy()
    np.testing.assert_allclose(oc.mlp(x, w1, b1, w2, b2), ref, rtol=1e-12, atol=1e-12)


def test_kappa_is_mean_logistic():
    rng = np.random.default_rng(2)
    for n in (1, 7, 576):
        z = rng.normal(0, 4, n)
        assert abs(oc.kappa(z) - float(np.mean(scipy.special.expit(z)))) < 1e-14
    z = np.array([np.inf, -np.inf, np.nan, 0.0, 800.0, -800.0])
    assert abs(oc.kappa(z) - (1 + 0 + 0 + 0.5 + 1 + 0) / 6) < 1e-15
    assert oc.kappa(np.zeros(0)) == 0.0


# ============================================================================ gating
@pytest.mark.parametrize("units", [4, 1])
def test_masks_from_logits_brute_force(units):
    """sigma(logit) > 0.5 decides each unit; group j holds heads [jA/G, (j+1)A/G)
    and FFN slice j; a layer runs iff one of its units is on; prefix layers run
    at full capacity (Sec. 3.2)."""
    shape = W.ModelShape(n_layers=6, d_model=64, n_heads=8, n_kv_heads=4, head_dim=8, d_ffn=64,
                         n_groups=4, dtype="f32")
    rng = np.random.default_rng(3)
    P = 2
    for _ in range(30):
        lg = rng.normal(size=(shape.n_layers - P) * units)
        lg[rng.integers(0, lg.size)] = 0.0      # sigma(0) = 0.5 is not > 0.5
        lo, ho, fo = oc.masks_from_logits(shape, lg, P, units)
        on = scipy.special.expit(lg) > 0.5
        for l in range(shape.n_layers):
            for h in range(shape.n_heads):
                want = 1 if l < P else int(on[(l - P) * units + (h // (shape.n_heads // units))])
                assert ho[l, h] == want
            for j in range(shape.n_groups):
                want = 1 if l < P else int(on[(l - P) * units + (j if units > 1 else 0)])
                assert fo[l, j] == want
            assert lo[l] == (1 if l < P else int(ho[l].any()))


def test_gate_logits_read_the_budget_row_plus_kappa_embedding():
    """With a one-hot gating row the logit is one coordinate of h + e_kappa plus
    its bias; with MLP_kappa's second layer zero, exactly h's coordinate."""
    rng = np.random.default_rng(4)
    D, H, E = 12, 6, 8
    h = rng.normal(size=D)
    ctrl = oc.Controller(prefix=0, units=1, pe_scale=1000.0, pe_base=10000.0,
                         llm_w1=np.zeros((H, E)), llm_b1=np.zeros(H), llm_w2=np.zeros((D, H)),
                         llm_b2=np.zeros(D), kap_w1=rng.normal(size=(H, E)), kap_b1=np.zeros(H),
                         kap_w2=np.zeros((D, H)), kap_b2=np.zeros(D),
                         gate_w=np.eye(D)[[3, 7]], gate_b=np.array([0.5, -2.0]))
    np.testing.assert_allclose(oc.gate_logits(ctrl, h, 0.3), [h[3] + 0.5, h[7] - 2.0], atol=1e-15)
    ctrl.kap_b2 = rng.normal(size=D)    # e_kappa = b2 when the hidden layer feeds nothing
    np.testing.assert_allclose(oc.gate_logits(ctrl, h, 0.3),
                               [h[3] + ctrl.kap_b2[3] + 0.5, h[7] + ctrl.kap_b2[7] - 2.0], atol=1e-14)


@pytest.mark.parametrize("budget", [0.6, 0.3, 0.1, 0.03])
def test_projection_with_layer_units(budget):
    """Layer controller: the reduction drops whole layers, lowest logit first
    (ties: the later layer), never a prefix layer, and the result fits."""
    from fractions import Fraction
    shape = W.ModelShape(n_layers=6, d_model=64, n_heads=8, n_kv_heads=8, head_dim=8, d_ffn=128,
                         n_groups=4, dtype="f32")
    rng = np.random.default_rng(int(budget * 100))
    P, T, N = 2, 6, 40
    for _ in range(40):
        z = rng.normal(-0.2, 1, N)
        gl = np.zeros((shape.n_layers, 1))
        gl[P:, 0] = rng.normal(size=shape.n_layers - P)
        lo, ho, fo = oc.masks_from_logits(shape, np.abs(gl[P:, 0]) + 0.1, P, 1)   # all on
        k, lo2, ho2, fo2 = ob.project_sample(shape, z, T, budget, 0, P, lo, ho, fo, gl, units=1)
        dropped = [l for l in range(P, shape.n_layers) if not lo2[l]]
        kept = [l for l in range(P, shape.n_layers) if lo2[l]]
        for l in dropped:
            assert not ho2[l].any() and not fo2[l].any()
        for l in kept:
            assert ho2[l].all() and fo2[l].all()
        key = lambda l: (gl[l, 0], -l)
        if dropped and kept:
            assert max(map(key, dropped)) < min(map(key, kept))
        limit = Fraction(float(np.float32(budget))) * ob.full_cost(shape, N, T, 0)
        a = ob.layer_alphas(shape, lo2, ho2)
        if ob.eq8_cost(shape, T, a, 0) <= limit:
            assert ob.eq8_cost(shape, T + k, a, 0) <= limit


# ============================================================================ controlled prefill
def _case(seed, prefix, units=4, budget=1.0, shift=-0.3, **draw_kw):
    w = SHAPE_W
    inp = W.draw_inputs(w, seed)
    layers = [host_layer(W.draw_layer_weights(w, l, seed)) for l in range(w.shape.n_layers)]
    draw = W.draw_controller(w, seed, prefix=prefix, units=units, pe_dim=16, hidden=32, **draw_kw)
    ctrl = host_controller(draw)
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((w.batch, w.n_vision)) + shift).astype(np.float32)
    vis, txt = W.as_f32(inp.vision), W.as_f32(inp.text)
    res = oc.prefill_controlled(w.shape, lambda l: layers[l], ctrl, z, vis, txt, budget)
    return w, layers, ctrl, z, vis, txt, res


def _text_with_budget_row(txt, ctrl, budget):
    e_b = oc.budget_token(ctrl, budget)
    return np.concatenate([txt, np.broadcast_to(e_b, (txt.shape[0], 1, e_b.size))], axis=1)


@pytest.mark.parametrize("units", [4, 1])
def test_controlled_prefill_without_drops_is_masked_prefill(units):
    """b = 1: no projection, so the controlled prefill is the plain prefill of
    [threshold-kept vision ; text ; budget token] under the controller's masks
    (the prefix layers at full capacity)."""
    w, layers, ctrl, z, vis, txt, res = _case(5, prefix=2, units=units, budget=1.0)
    counts = [ob.threshold_count(z[b]) for b in range(w.batch)]
    np.testing.assert_array_equal(res.keep, counts)
    ref = oracle.prefill(w.shape, lambda l: layers[l], z, np.array(counts),
                         vis, _text_with_budget_row(txt, ctrl, 1.0), res.layer_mask,
                         res.head_mask, res.ffn_mask)
    np.testing.assert_array_equal(res.kept_idx, ref.kept_idx)
    np.testing.assert_array_equal(res.cu_seqlens, ref.cu_seqlens)
    np.testing.assert_allclose(res.resid, ref.resid, rtol=0, atol=1e-12)
    assert res.layer_mask[:, :2].all() and res.head_mask[:, :2].all()
    assert res.flops.total == ref.flops.total
    # the gate logits saw the budget row after the prefix layers
    pre = oracle.prefill(w.shape, lambda l: layers[l], z, np.array(counts), vis,
                         _text_with_budget_row(txt, ctrl, 1.0),
                         np.ones((w.batch, w.shape.n_layers), np.uint8),
                         np.ones((w.batch, w.shape.n_layers, w.shape.n_heads), np.uint8),
                         None, layers=range(2))
    for b in range(w.batch):
        h = pre.resid[pre.cu_seqlens[b + 1] - 1]
        np.testing.assert_allclose(res.logits[b], oc.gate_logits(ctrl, h, oc.kappa(z[b])),
                                   rtol=0, atol=1e-12)


def test_controlled_prefill_prefix0_drops_before_any_layer():
    """P = 0: the projection's discarded tokens leave before the first layer, so
    the result is the plain prefill of the projected keep under the masks."""
    w, layers, ctrl, z, vis, txt, res = _case(6, prefix=0, budget=0.35, shift=0.3)
    counts = np.array([ob.threshold_count(z[b]) for b in range(w.batch)])
    assert np.all(res.keep < counts), "the case must exercise token drops"
    ref = oracle.prefill(w.shape, lambda l: layers[l], z, res.keep, vis,
                         _text_with_budget_row(txt, ctrl, 0.35), res.layer_mask,
                         res.head_mask, res.ffn_mask)
    np.testing.assert_array_equal(res.kept_idx, ref.kept_idx)
    np.testing.assert_array_equal(res.cu_seqlens, ref.cu_seqlens)
    np.testing.assert_allclose(res.resid, ref.resid, rtol=0, atol=1e-12)


def test_controlled_prefill_rows_before_the_first_drop_are_unaffected():
    """0 < P < L with token drops: causal attention and relative RoPE leave the
    rows in front of the first discarded token exactly as the full threshold
    sequence would have them under the same masks."""
    w, layers, ctrl, z, vis, txt, res = _case(7, prefix=2, budget=0.35, shift=0.3)
    counts = np.array([ob.threshold_count(z[b]) for b in range(w.batch)])
    assert np.all(res.keep < counts)
    full = oracle.prefill(w.shape, lambda l: layers[l], z, counts, vis,
                          _text_with_budget_row(txt, ctrl, 0.35), res.layer_mask,
                          res.head_mask, res.ffn_mask)
    checked = 0
    for b in range(w.batch):
        first = oracle.select_topk(z[b], int(counts[b]))
        final = res.kept_idx[b, :res.keep[b]]
        lead = 0
        while lead < final.size and final[lead] == first[lead]:
            lead += 1
        got = res.resid[res.cu_seqlens[b]:res.cu_seqlens[b] + lead]
        want = full.resid[full.cu_seqlens[b]:full.cu_seqlens[b] + lead]
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
        checked += lead
        # and the sequence still ends with the text and budget rows
        assert res.cu_seqlens[b + 1] - res.cu_seqlens[b] == res.keep[b] + w.n_text + 1
    assert checked > 0


def test_controlled_prefill_identity_prefix_equals_plain_prefill_of_projected_keep():
    """0 < P < L with token drops and prefix layers that are the identity on the
    residual stream (their output and down projections zeroed): the sequence
    that enters layer P must be [projected kept vision ; text ; budget row]
    exactly as the plain prefill of the projected keep builds it, so every row
    of the result (kept, text and budget rows alike) equals that prefill under
    the final masks.  This fixes which rows survive the projection at the
    prefix boundary and where the text and budget rows are taken from."""
    P = 2
    w = SHAPE_W
    seed = 11
    inp = W.draw_inputs(w, seed)
    layers = [host_layer(W.draw_layer_weights(w, l, seed)) for l in range(w.shape.n_layers)]
    for l in range(P):
        layers[l] = dict(layers[l])
        layers[l]["wo"] = np.zeros_like(layers[l]["wo"])
        layers[l]["w_down"] = np.zeros_like(layers[l]["w_down"])
    draw = W.draw_controller(w, seed, prefix=P, units=4, pe_dim=16, hidden=32)
    ctrl = host_controller(draw)
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((w.batch, w.n_vision)) + 0.3).astype(np.float32)
    vis, txt = W.as_f32(inp.vision), W.as_f32(inp.text)
    budget = 0.35
    res = oc.prefill_controlled(w.shape, lambda l: layers[l], ctrl, z, vis, txt, budget)
    counts = np.array([ob.threshold_count(z[b]) for b in range(w.batch)])
    assert np.all(res.keep < counts), "the case must exercise token drops"
    assert np.all(res.keep > 0), "the case must keep visual tokens on both sides of a drop"
    # the first discarded token is not the last threshold-kept one, so rows
    # after it (kept vision, then text and budget) change position
    for b in range(w.batch):
        first = oracle.select_topk(z[b], int(counts[b]))
        final = res.kept_idx[b, :res.keep[b]]
        assert not np.array_equal(first[:final.size], final), "a drop ahead of a kept token"
    ref = oracle.prefill(w.shape, lambda l: layers[l], z, res.keep, vis,
                         _text_with_budget_row(txt, ctrl, budget), res.layer_mask,
                         res.head_mask, res.ffn_mask)
    np.testing.assert_array_equal(res.kept_idx, ref.kept_idx)
    np.testing.assert_array_equal(res.cu_seqlens, ref.cu_seqlens)
    np.testing.assert_allclose(res.resid, ref.resid, rtol=0, atol=1e-12)
    # the budget row of each sample is its last row and came through unchanged
    # by the prefix (identity) into the gated layers
    for b in range(w.batch):
        np.testing.assert_allclose(res.prefix_resid[b][-1], oc.budget_token(ctrl, budget),
                                   rtol=0, atol=0)
