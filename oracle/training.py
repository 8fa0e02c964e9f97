"""CPU oracle for the training-time budget term (SmartVL, Sec. 3.1 Eq. (6),
Sec. 3.2, Sec. 3.3 Eq. (8)-(10)).

TEST INFRASTRUCTURE ONLY, like the rest of this package: the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never does.

What is computed, per sample (the controllers' logits in, the budget loss and
its gradient with respect to those logits out):
  * Gumbel-sigmoid decisions (Eq. (6)): y = sigma((z + xi) / tau) with the
    noise xi given; the straight-through mask m = 1[y > 0.5] - sg(y) + y has
    the forward value 1[y > 0.5] and the derivative dy/dz = y (1 - y) / tau.
    Tokens use the token temperature, the compute controller's units the
    compute temperature;
  * the differentiable cost (Eq. (8)) with the soft visual count
    S~ = sum_i sigma(z_i) (noise-free, no temperature), S = T + S~ and the
    layer activity alpha_l = (sum_j M_lj) / U of the straight-through unit
    masks (U = G for the layer-head controller, 1 for the layer controller;
    prefix layers at alpha = 1):
        C^ = sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2] + 2 D V S,
    r = C^ / C_full, C_full at alpha = 1 and S = T + N;
  * the asymmetric loss (Eq. (9), Eq. (10) without L_pred):
        L = lambda (w_over max(0, r - b)^2 + w_under max(0, (b - mu) - r));
  * its gradient: dL/dz_i = dL/dr dr/dS sigma'(z_i) (through S~ only: the
    token masks feed the prediction loss, not the cost) and
    dL/dg_lj = dL/dr dr/dalpha_l (1/U) y_lj (1 - y_lj) / tau_comp.

Readings (listed in the design notes): the noise is an input (the caller
draws it; None means no noise); the loss is per sample (a batch objective
averages them); at r - b = 0 or (b - mu) - r = 0 the hinge's derivative is
taken as 0; the token and unit masks compare the noisy logit with 0
(y > 0.5 iff z + xi > 0 for tau > 0).

Arithmetic: float64 throughout.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np


def sigmoid(x: np.ndarray) -> np.ndarray:
    """Logistic function, evaluated without overflow on either side."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    e = np.exp(x[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def gumbel_sigmoid(logits: np.ndarray, noise: Optional[np.ndarray], tau: float):
    """Eq. (6): the relaxed value y and the straight-through mask's forward
    value m = 1[y > 0.5] (taken as z + xi > 0, the same test for tau > 0)."""
    z = np.asarray(logits, dtype=np.float64)
    v = z if noise is None else z + np.asarray(noise, dtype=np.float64)
    y = sigmoid(v / tau)
    m = (v > 0.0).astype(np.uint8)
    return y, m


@dataclass
class BudgetTerm:
    ratio: float
    loss: float
    token_mask: np.ndarray      # uint8 [N]
    unit_mask: np.ndarray       # uint8 [(L-P) U]
    grad_z: np.ndarray          # [N]
    grad_gate: np.ndarray       # [(L-P) U]
    soft_count: float
    alphas: np.ndarray          # [L]


def budget_term(shape, z, gate_logits, n_text: int, budget: float, margin: float,
                w_over: float, w_under: float, lam: float, tau_tok: float, tau_comp: float,
                prefix: int, units: int, vocab: int = 0, xi_tok=None, xi_gate=None) -> BudgetTerm:
    """The budget term of one sample and its gradient (module docstring)."""
    L, D, F = shape.n_layers, shape.d_model, shape.d_ffn
    z = np.asarray(z, dtype=np.float64)
    N = z.size
    _, m_tok = gumbel_sigmoid(z, xi_tok, tau_tok)
    y_g, m_g = gumbel_sigmoid(np.asarray(gate_logits, np.float64), xi_gate, tau_comp)
    m_g = m_g.reshape(L - prefix, units)
    y_g = y_g.reshape(L - prefix, units)

    sz = sigmoid(z)
    soft = float(sz.sum())
    S = n_text + soft
    alphas = np.ones(L)
    alphas[prefix:] = m_g.sum(axis=1) / units
    c1, c2 = 8.0 * D * D + 6.0 * D * F, 4.0 * D
    per_layer = c1 * S + c2 * S * S
    cost = float(np.sum(alphas) * per_layer + 2.0 * D * vocab * S)
    Sf = float(n_text + N)
    full = L * (c1 * Sf + c2 * Sf * Sf) + 2.0 * D * vocab * Sf
    r = cost / full
    b = float(np.float32(budget))
    over = max(0.0, r - b)
    under = max(0.0, (b - margin) - r)
    loss = lam * (w_over * over * over + w_under * under)

    dldr = lam * (2.0 * w_over * over - (w_under if under > 0.0 else 0.0))
    drds = (float(np.sum(alphas)) * (c1 + 2.0 * c2 * S) + 2.0 * D * vocab) / full
    grad_z = dldr * drds * sz * (1.0 - sz)
    drda = per_layer / full
    grad_gate = dldr * drda * (1.0 / units) * y_g * (1.0 - y_g) / tau_comp
    return BudgetTerm(r, loss, m_tok, m_g.reshape(-1).astype(np.uint8), grad_z,
                      grad_gate.reshape(-1), soft, alphas)
