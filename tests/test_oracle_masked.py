"""Pins of the training-time masked decoder in the oracle (CPU only).

oracle.training's static-shape forward and its hand-written backward
(Sec. 3.1 Eq. (6) with dropped tokens zeroed, Sec. 3.2 unit masks over head
groups and FFN slices, or one per layer) are tied to things outside them:

  * forward: at binary masks it equals oracle.prefill (itself pinned to HF
    transformers' LlamaModel) run with every token kept on the zeroed input,
    with the heads and FFN slices of the masked-off units gated and, for the
    layer controller, the masked-off layers skipped;
  * backward: torch float64 autograd through HF transformers' LlamaModel, the
    masks applied by hooks on the inputs of the output and down projections
    and the token masks built with the straight-through expression of
    Eq. (6), gives the same hidden states, token-logit and gate-logit
    gradients (HF forms its RoPE angles in float32, hence the 1e-4 bar);
  * backward: central finite differences of the oracle's forward in the
    (real-valued) token and unit masks and in input coordinates, at binary
    and at fractional mask values (1e-6 bar).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import training as ot
from test_oracle_pins import SMALL_GQA, SMALL_MHA, _hf_model, _weights


def _draw(shape, seed, N=12, T=5):
    rng = np.random.default_rng(seed)
    D = shape.d_model
    return rng, rng.standard_normal((N, D)), rng.standard_normal((T, D))


def _inference_masks(shape, M, prefix, units):
    """Head / FFN / layer masks of oracle.prefill equivalent to binary unit masks."""
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    layer_on = np.ones((1, L), np.uint8)
    head_on = np.ones((1, L, A), np.uint8)
    ffn_on = np.ones((1, L, G), np.uint8)
    for l in range(prefix, L):
        row = M[l - prefix]
        if units == 1:
            layer_on[0, l] = int(row[0])
        else:
            assert units == G
            for j in range(units):
                head_on[0, l, j * A // units:(j + 1) * A // units] = int(row[j])
                ffn_on[0, l, j] = int(row[j])
    return layer_on, head_on, ffn_on


@pytest.mark.parametrize("shape", [SMALL_MHA, SMALL_GQA], ids=["mha", "gqa"])
@pytest.mark.parametrize("units_kind", ["groups", "layer"])
def test_forward_at_binary_masks_equals_the_inference_oracle(shape, units_kind):
    W = _weights(shape, 3)
    units = shape.n_groups if units_kind == "groups" else 1
    for seed, prefix in ((1, 0), (2, 1)):
        rng, vision, text = _draw(shape, seed)
        N = vision.shape[0]
        m = (rng.random(N) < 0.6).astype(np.float64)
        M = (rng.random((shape.n_layers - prefix, units)) < 0.6).astype(np.float64)
        hidden, _ = ot.masked_forward(shape, lambda l: W[l], vision, text, m, M, prefix, units)
        layer_on, head_on, ffn_on = _inference_masks(shape, M, prefix, units)
        ref = oracle.prefill(shape, lambda l: W[l], rng.random((1, N)), [N], (vision * m[:, None])[None],
                         text[None], layer_on, head_on, ffn_on)
        np.testing.assert_allclose(hidden, ref.resid, rtol=0, atol=1e-12 * np.abs(ref.resid).max())


def test_all_ones_is_the_dense_prefill_and_zeroing_is_not_discarding():
    shape = SMALL_MHA
    W = _weights(shape, 4)
    rng, vision, text = _draw(shape, 5)
    N = vision.shape[0]
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    ones = np.ones((L, G))
    hidden, _ = ot.masked_forward(shape, lambda l: W[l], vision, text, np.ones(N), ones, 0, G)
    dense = oracle.prefill(shape, lambda l: W[l], rng.random((1, N)), [N], vision[None], text[None],
                       np.ones((1, L), np.uint8), np.ones((1, L, A), np.uint8),
                       np.ones((1, L, G), np.uint8))
    np.testing.assert_allclose(hidden, dense.resid, rtol=0, atol=1e-12 * np.abs(dense.resid).max())
    # dropping the first token by zeroing keeps its row; discarding it removes
    # it, and the text rows differ (the zero key still takes softmax weight)
    m = np.ones(N)
    m[0] = 0.0
    zeroed, _ = ot.masked_forward(shape, lambda l: W[l], vision, text, m, ones, 0, G)
    scores = np.arange(N, 0, -1, dtype=np.float64)[None]
    disc = oracle.prefill(shape, lambda l: W[l], -scores, [N - 1], vision[None], text[None],
                      np.ones((1, L), np.uint8), np.ones((1, L, A), np.uint8),
                      np.ones((1, L, G), np.uint8))
    assert zeroed.shape[0] == N + text.shape[0] and disc.resid.shape[0] == N - 1 + text.shape[0]
    assert np.abs(zeroed[N:] - disc.resid[N - 1:]).max() > 1e-3


def _hf_step(shape, W, vision, text, z, g, xi, xg, tau_tok, tau_comp, prefix, units, G):
    """The same training step through HF LlamaModel with torch float64 autograd."""
    L, A, d, F = shape.n_layers, shape.n_heads, shape.head_dim, shape.d_ffn
    model = _hf_model(shape, W, list(range(L)))
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    gt = torch.tensor(g, dtype=torch.float64, requires_grad=True)

    def ste(logit, noise, tau):
        y = torch.sigmoid((logit + torch.from_numpy(noise)) / tau)
        return (y > 0.5).double() - y.detach() + y

    m = ste(zt, xi, tau_tok)
    M = ste(gt, xg, tau_comp).reshape(L - prefix, units)
    for l in range(prefix, L):
        lay = model.layers[l]
        col = M[l - prefix].repeat_interleave(A * d // units)
        ch = M[l - prefix].repeat_interleave(F // units)
        lay.self_attn.o_proj.register_forward_pre_hook(lambda mod, a, c=col: (a[0] * c,))
        lay.mlp.down_proj.register_forward_pre_hook(lambda mod, a, c=ch: (a[0] * c,))
    x0 = torch.cat([torch.from_numpy(vision) * m[:, None], torch.from_numpy(text)])
    S = x0.shape[0]
    out = model(inputs_embeds=x0[None], position_ids=torch.arange(S)[None]).last_hidden_state[0]
    (out * torch.from_numpy(G)).sum().backward()
    return out.detach().numpy(), zt.grad.numpy(), gt.grad.numpy()


@pytest.mark.parametrize("shape", [SMALL_MHA, SMALL_GQA], ids=["mha", "gqa"])
@pytest.mark.parametrize("units_kind", ["groups", "layer"])
def test_gradients_match_torch_autograd_through_hf_llama(shape, units_kind):
    W = _weights(shape, 6)
    units = shape.n_groups if units_kind == "groups" else 1
    prefix = 1
    rng, vision, text = _draw(shape, 7)
    N, S, D = vision.shape[0], vision.shape[0] + text.shape[0], shape.d_model
    z = rng.normal(0.3, 1.5, N)
    g = rng.normal(0.5, 1.5, (shape.n_layers - prefix) * units)
    xi, xg = rng.logistic(0, 1, N), rng.logistic(0, 1, g.size)
    G = rng.standard_normal((S, D))
    tt, tc = 0.7, 1.3
    res = ot.masked_train_step(shape, lambda l: W[l], vision, text, z, g, G, prefix, units, tt, tc,
                               xi_tok=xi, xi_gate=xg)
    assert 0 < res.token_mask.sum() < N, "the draw should drop some tokens and keep some"
    hid, gz, gg = _hf_step(shape, W, vision, text, z, g, xi, xg, tt, tc, prefix, units, G)
    assert np.abs(res.hidden - hid).max() <= 1e-4 * np.abs(hid).max()
    assert np.abs(res.grad_z - gz).max() <= 1e-4 * np.abs(gz).max()
    assert np.abs(res.grad_gate - gg).max() <= 1e-4 * np.abs(gg).max()
    assert np.abs(gz).max() > 0 and np.abs(gg).max() > 0


def _fd_check(shape, W, prefix, units, m, M, seed):
    rng, vision, text = _draw(shape, seed)
    S, D = vision.shape[0] + text.shape[0], shape.d_model
    G = rng.standard_normal((S, D))
    f = lambda mm, MM, v=vision, t=text: float(np.sum(
        G * ot.masked_forward(shape, lambda l: W[l], v, t, mm, MM, prefix, units)[0]))
    _, caches = ot.masked_forward(shape, lambda l: W[l], vision, text, m, M, prefix, units)
    dx0, dM = ot.masked_backward(shape, lambda l: W[l], caches, units, G)
    N = vision.shape[0]
    dm = np.sum(dx0[:N] * vision, axis=1)
    h = 1e-5
    for i in range(N):
        # a zeroed row's RMSNorm bends on the scale sqrt(eps) / rms(v): a
        # smaller step there keeps the central difference's error below 1e-6
        hi = h if m[i] != 0 else 1e-8
        e = np.zeros(N)
        e[i] = hi
        fd = (f(m + e, M) - f(m - e, M)) / (2 * hi)
        assert abs(fd - dm[i]) <= 1e-6 * max(1.0, abs(fd)), (i, fd, dm[i])
    for l in range(prefix, shape.n_layers):
        for j in range(units):
            E = np.zeros_like(M)
            E[l - prefix, j] = h
            fd = (f(m, M + E) - f(m, M - E)) / (2 * h)
            assert abs(fd - dM[l, j]) <= 1e-6 * max(1.0, abs(fd)), (l, j, fd, dM[l, j])
    # input coordinates: a vision row (scaled by its mask) and a text row
    for (r, c) in ((1, 3), (N + 2, 5)):
        vv, tt = vision.copy(), text.copy()
        if r < N:
            vv[r, c] += h
            fp = f(m, M, vv, tt)
            vv[r, c] -= 2 * h
            fm = f(m, M, vv, tt)
            want = dx0[r, c] * m[r]
        else:
            tt[r - N, c] += h
            fp = f(m, M, vv, tt)
            tt[r - N, c] -= 2 * h
            fm = f(m, M, vv, tt)
            want = dx0[r, c]
        fd = (fp - fm) / (2 * h)
        assert abs(fd - want) <= 1e-6 * max(1.0, abs(fd)), (r, c, fd, want)


@pytest.mark.parametrize("shape", [SMALL_MHA, SMALL_GQA], ids=["mha", "gqa"])
def test_mask_gradients_match_finite_differences(shape):
    W = _weights(shape, 8)
    G = shape.n_groups
    rng = np.random.default_rng(9)
    N = 12
    # binary masks, some off.  Token 0 stays on: a zeroed row at position 0
    # attends only to itself and stays zero through every layer, where each
    # RMSNorm scales its derivative by eps^(-1/2); the derivative there is
    # well defined (the autograd pin covers it) but no step size resolves it.
    m = (rng.random(N) < 0.6).astype(np.float64)
    m[0] = 1.0
    M = (rng.random((shape.n_layers - 1, G)) < 0.6).astype(np.float64)
    _fd_check(shape, W, 1, G, m, M, 10)
    # fractional masks and the layer controller from layer 0
    m = rng.random(N)
    M = rng.random((shape.n_layers, 1))
    _fd_check(shape, W, 0, 1, m, M, 11)


def test_straight_through_factors_and_prefix_rows():
    """grad_z = dL/dm y (1 - y) / tau_tok, grad_gate = dL/dM y (1 - y) / tau_comp on the
    controlled layers only, masks = 1[logit + noise > 0]."""
    shape = SMALL_MHA
    W = _weights(shape, 12)
    rng, vision, text = _draw(shape, 13)
    N, S = vision.shape[0], vision.shape[0] + text.shape[0]
    G = rng.standard_normal((S, shape.d_model))
    z, xi = rng.normal(0, 2, N), rng.logistic(0, 1, N)
    units, P = shape.n_groups, 2
    g, xg = rng.normal(0, 2, (shape.n_layers - P) * units), rng.logistic(0, 1, (shape.n_layers - P) * units)
    r = ot.masked_train_step(shape, lambda l: W[l], vision, text, z, g, G, P, units, 0.5, 2.0,
                             xi_tok=xi, xi_gate=xg)
    y = 1 / (1 + np.exp(-(z + xi) / 0.5))
    np.testing.assert_array_equal(r.token_mask, (z + xi > 0).astype(np.uint8))
    np.testing.assert_allclose(r.grad_z, r.grad_m * y * (1 - y) / 0.5, rtol=1e-13, atol=0)
    yg = 1 / (1 + np.exp(-(g + xg) / 2.0))
    np.testing.assert_array_equal(r.unit_mask, (g + xg > 0).astype(np.uint8))
    np.testing.assert_allclose(r.grad_gate, r.grad_M[P:].reshape(-1) * yg * (1 - yg) / 2.0,
                               rtol=1e-13, atol=0)
    assert r.grad_gate.shape == ((shape.n_layers - P) * units,)
