"""Pins of the training-time budget-term oracle (CPU only).

The oracle's cost is tied to the already-pinned Eq. (8) implementation of
oracle.budget (exact rational arithmetic) at integer counts; its gradient to
torch's float64 autograd of the straight-through expression (Eq. (6)) and to
central finite differences; its masks to scipy's logistic function; and the
loss to the shape of Eq. (9) (zero band, quadratic over, linear under).
"""

import numpy as np
import pytest
import scipy.special
import torch

from oracle import budget as ob
from oracle import training as ot
from workloads import ModelShape

SHAPE = ModelShape(n_layers=6, d_model=64, n_heads=8, n_kv_heads=8, head_dim=8, d_ffn=128,
                   n_groups=4, dtype="f32")
KW = dict(margin=0.1, w_over=2.0, w_under=0.5, lam=0.7, tau_tok=0.8, tau_comp=1.3)


def _case(rng, N=30, P=2, U=4, shift=0.0):
    z = rng.normal(shift, 2.0, N)
    g = rng.normal(0.3, 1.5, (SHAPE.n_layers - P) * U)
    xi = rng.logistic(0, 1, N)
    xg = rng.logistic(0, 1, g.size)
    return z, g, xi, xg


def _torch_term(z, g, T, b, P, U, vocab, xi, xg, margin, w_over, w_under, lam, tau_tok,
                tau_comp):
    """The budget term in torch float64 with the straight-through estimator."""
    D, F, L = SHAPE.d_model, SHAPE.d_ffn, SHAPE.n_layers
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    gt = torch.tensor(g, dtype=torch.float64, requires_grad=True)
    yg = torch.sigmoid((gt + torch.tensor(xg)) / tau_comp)
    M = (yg > 0.5).double() - yg.detach() + yg
    alpha = torch.cat([torch.ones(P, dtype=torch.float64), M.reshape(L - P, U).sum(1) / U])
    S = T + torch.sigmoid(zt).sum()
    cost = alpha.sum() * ((8 * D * D + 6 * D * F) * S + 4 * D * S * S) + 2 * D * vocab * S
    Sf = T + len(z)
    full = L * ((8 * D * D + 6 * D * F) * Sf + 4 * D * Sf * Sf) + 2 * D * vocab * Sf
    r = cost / full
    bb = float(np.float32(b))
    loss = lam * (w_over * torch.relu(r - bb) ** 2 + w_under * torch.relu((bb - margin) - r))
    loss.backward()
    return float(r.detach()), float(loss.detach()), zt.grad.numpy(), gt.grad.numpy()


@pytest.mark.parametrize("units", [4, 1])
@pytest.mark.parametrize("budget", [0.9, 0.5, 0.2])
def test_gradients_match_torch_autograd(units, budget):
    rng = np.random.default_rng(int(budget * 10) + units)
    for vocab in (0, 1000):
        z, g, xi, xg = _case(rng, U=units)
        t = ot.budget_term(SHAPE, z, g, 7, budget, prefix=2, units=units, vocab=vocab,
                           xi_tok=xi, xi_gate=xg, **KW)
        r, loss, gz, gg = _torch_term(z, g, 7, budget, 2, units, vocab, xi, xg, **KW)
        assert abs(t.ratio - r) < 1e-14 and abs(t.loss - loss) < 1e-14
        np.testing.assert_allclose(t.grad_z, gz, rtol=1e-10, atol=1e-18)
        np.testing.assert_allclose(t.grad_gate, gg, rtol=1e-10, atol=1e-18)


def test_cost_equals_eq8_at_integer_counts():
    """With saturated logits (sigma = 0 or 1 exactly in float64) the soft count
    is an integer and the ratio is Eq. (8)'s, computed exactly by oracle.budget."""
    rng = np.random.default_rng(5)
    for _ in range(20):
        N, T, P = 30, 7, 2
        k = int(rng.integers(0, N + 1))
        z = np.where(np.arange(N) < k, 800.0, -800.0)
        g = rng.choice([-50.0, 50.0], (SHAPE.n_layers - P) * 4)
        t = ot.budget_term(SHAPE, z, g, T, 0.5, prefix=P, units=4, vocab=3, **KW)
        assert t.soft_count == k
        layer_on = np.ones(SHAPE.n_layers, np.uint8)
        head_on = np.ones((SHAPE.n_layers, SHAPE.n_heads), np.uint8)
        gm = (g > 0).reshape(-1, 4)
        for i, l in enumerate(range(P, SHAPE.n_layers)):
            for j in range(4):
                head_on[l, 2 * j:2 * j + 2] = gm[i, j]
            layer_on[l] = gm[i].any()
        want = ob.eq8_cost(SHAPE, T + k, ob.layer_alphas(SHAPE, layer_on, head_on), 3) / \
            ob.full_cost(SHAPE, N, T, 3)
        assert abs(t.ratio - float(want)) < 1e-14


def test_token_gradient_matches_finite_differences():
    rng = np.random.default_rng(9)
    z, g, xi, xg = _case(rng, shift=0.5)
    f = lambda zz: ot.budget_term(SHAPE, zz, g, 7, 0.2, prefix=2, units=4, xi_tok=xi,
                                  xi_gate=xg, **KW).loss
    t = ot.budget_term(SHAPE, z, g, 7, 0.2, prefix=2, units=4, xi_tok=xi, xi_gate=xg, **KW)
    assert t.loss > 0
    h = 1e-6
    for i in range(0, z.size, 3):
        e = np.zeros_like(z)
        e[i] = h
        fd = (f(z + e) - f(z - e)) / (2 * h)
        assert abs(fd - t.grad_z[i]) <= 1e-6 * max(1e-12, abs(t.grad_z).max())


def test_loss_shape():
    """Zero inside [b - mu, b]; quadratic above b; linear below b - mu."""
    rng = np.random.default_rng(11)
    z, g, xi, xg = _case(rng)
    t = ot.budget_term(SHAPE, z, g, 7, 1.0, prefix=2, units=4, xi_tok=xi, xi_gate=xg, **KW)
    r = t.ratio
    for b, kind in ((r + 0.05, "band"), (r + KW["margin"] - 1e-9, "band"), (r - 0.1, "over"),
                    (r + KW["margin"] + 0.2, "under")):
        u = ot.budget_term(SHAPE, z, g, 7, b, prefix=2, units=4, xi_tok=xi, xi_gate=xg, **KW)
        bb = float(np.float32(b))
        if kind == "band":
            assert u.loss == 0 and not u.grad_z.any() and not u.grad_gate.any()
        elif kind == "over":
            assert abs(u.loss - KW["lam"] * KW["w_over"] * (r - bb) ** 2) < 1e-14
        else:
            assert abs(u.loss - KW["lam"] * KW["w_under"] * ((bb - KW["margin"]) - r)) < 1e-14
            assert np.all(u.grad_z <= 0)     # more tokens lower an under-use penalty


def test_masks_are_the_logistic_threshold():
    rng = np.random.default_rng(13)
    z, g, xi, xg = _case(rng)
    t = ot.budget_term(SHAPE, z, g, 7, 0.5, prefix=2, units=4, xi_tok=xi, xi_gate=xg, **KW)
    np.testing.assert_array_equal(t.token_mask, scipy.special.expit((z + xi) / KW["tau_tok"]) > 0.5)
    np.testing.assert_array_equal(t.unit_mask, scipy.special.expit((g + xg) / KW["tau_comp"]) > 0.5)
    t0 = ot.budget_term(SHAPE, z, g, 7, 0.5, prefix=2, units=4, **KW)      # no noise
    np.testing.assert_array_equal(t0.token_mask, z > 0)
