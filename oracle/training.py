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

And the prediction side of the same training step (Sec. 3.1 Eq. (6) with
zeroing, Sec. 3.2): the decoder run with static shapes under the forward
values of the straight-through masks (dropped vision tokens zeroed, unit
masks scaling head-group attention outputs and FFN slices), and the backward
of that decoder for a given gradient of its final hidden states, down to the
token and gate logits (masked_train_step and the functions above it).  The
backward is written out by hand (RMSNorm, RoPE, causal attention, SwiGLU and
the matrix products); the tests pin it to torch's float64 autograd and to
central finite differences of the forward in the masks.

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


# =========================================================================== masked decoder
# The training-time forward with static shapes and its backward (Sec. 3.1
# Eq. (6): straight-through token masks, dropped tokens zeroed; Sec. 3.2: unit
# masks over head groups and the matching FFN slices, or one mask per layer).
#
# One sample, S = N + T rows: the N vision embeddings, each multiplied by its
# token mask m_i, followed by the T text embeddings, at positions 0..S-1 (the
# sequence keeps its length).  Every layer computes every head and every FFN
# channel; in the controlled layers (l >= P) unit j's mask M_lj multiplies
# the attention output of the heads of group j (before the output projection)
# and the SwiGLU output of FFN slice j (before the down projection).  With one
# unit per layer (the layer controller) the mask multiplies both whole
# branches, so M = 0 makes the layer the identity.  The prefix layers run with
# every mask at 1.
#
# The backward takes an upstream gradient G of the final hidden states (the
# prediction loss is outside: this is dL/dX_L) and returns dL/dX_0, dL/dm and
# dL/dM, treating the masks as real numbers; the straight-through estimator
# then gives dL/dz_i = dL/dm_i y_i (1 - y_i) / tau_tok and
# dL/dg_lj = dL/dM_lj y_lj (1 - y_lj) / tau_comp.


def _heads_of_unit(shape, units: int):
    """Query heads gated by each unit: group j = heads [j A/U, (j+1) A/U)."""
    A = shape.n_heads
    return [list(range(j * A // units, (j + 1) * A // units)) for j in range(units)]


def _chans_of_unit(shape, units: int):
    F = shape.d_ffn
    return [np.arange(j * F // units, (j + 1) * F // units) for j in range(units)]


def rmsnorm_forward(x, gain, eps):
    """y = x r g with r = (mean(x^2) + eps)^(-1/2) per row; returns (y, r)."""
    x = np.asarray(x, np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(gain, np.float64), r


def rmsnorm_backward(x, gain, r, dy):
    """dL/dx of y = x r(x) g: r g dy - x r^3 (sum_k g_k dy_k x_k) / D."""
    x = np.asarray(x, np.float64)
    gdy = dy * np.asarray(gain, np.float64)
    D = x.shape[-1]
    return r * gdy - x * (r ** 3) * np.sum(gdy * x, axis=-1, keepdims=True) / D


def _rope_angles(S, d, theta):
    half = d // 2
    omega = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    phi = np.arange(S, dtype=np.float64)[:, None] * omega[None, :]
    return np.cos(phi), np.sin(phi)


def rope_forward(a, theta):
    """Rotate-half RoPE at positions 0..S-1: pair (r, r + d/2) turned by p omega_r."""
    S, d = a.shape
    c, s = _rope_angles(S, d, theta)
    a1, a2 = a[:, :d // 2], a[:, d // 2:]
    return np.concatenate([a1 * c - a2 * s, a2 * c + a1 * s], axis=1)


def rope_backward(da, theta):
    """The transpose of the rotation (a turn by -p omega_r)."""
    S, d = da.shape
    c, s = _rope_angles(S, d, theta)
    d1, d2 = da[:, :d // 2], da[:, d // 2:]
    return np.concatenate([d1 * c + d2 * s, d2 * c - d1 * s], axis=1)


def attention_forward(q, k, v):
    """Causal softmax attention of one head; returns (out, probabilities)."""
    S, d = q.shape
    s = (q @ k.T) / np.sqrt(d)
    s = np.where(np.triu(np.ones((S, S), dtype=bool), 1), -np.inf, s)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ v, p


def attention_backward(q, k, v, p, do):
    """Gradients of out = P V, P = softmax(q k^T / sqrt(d)) (causal) with
    respect to q, k and v: dV = P^T dO, dP = dO V^T,
    dS = P (dP - rowsum(P dP)), dq = dS k / sqrt(d), dk = dS^T q / sqrt(d)."""
    d = q.shape[1]
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
    return ds @ k / np.sqrt(d), ds.T @ q / np.sqrt(d), dv


def _sigmoid_plain(x):
    return 1.0 / (1.0 + np.exp(-x))


@dataclass
class LayerCache:
    x: np.ndarray       # layer input [S][D]
    r1: np.ndarray      # attention-norm scale per row
    u: np.ndarray       # normed input
    q: list             # per query head, rotated
    k: dict             # per K/V head, rotated
    v: dict
    p: list             # per query head, probabilities
    o: np.ndarray       # attention output, all heads [S][A d], before the masks
    x1: np.ndarray      # after the attention branch
    r2: np.ndarray
    u2: np.ndarray
    a: np.ndarray       # gate projection [S][F]
    e: np.ndarray       # up projection
    h: np.ndarray       # silu(a) e, before the masks
    mask: np.ndarray    # this layer's unit masks [U]


def masked_layer_forward(x, W, shape, mask, units):
    """One LLaMA block with every head and channel computed; unit j's mask
    scales the attention output of its heads and the SwiGLU output of its FFN
    slice."""
    S, D = x.shape
    A, KV, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    rep = A // KV
    col_scale = np.empty(A * d)
    for j, hs in enumerate(_heads_of_unit(shape, units)):
        for h in hs:
            col_scale[h * d:(h + 1) * d] = mask[j]
    ch_scale = np.empty(shape.d_ffn)
    for j, cs in enumerate(_chans_of_unit(shape, units)):
        ch_scale[cs] = mask[j]

    u, r1 = rmsnorm_forward(x, W["attn_norm"], shape.rms_eps)
    wq, wk, wv = (np.asarray(W[n], np.float64) for n in ("wq", "wk", "wv"))
    ks = {g: rope_forward(u @ wk[g * d:(g + 1) * d].T, shape.rope_theta) for g in range(KV)}
    vs = {g: u @ wv[g * d:(g + 1) * d].T for g in range(KV)}
    qs, ps, outs = [], [], []
    for h in range(A):
        qh = rope_forward(u @ wq[h * d:(h + 1) * d].T, shape.rope_theta)
        oh, ph = attention_forward(qh, ks[h // rep], vs[h // rep])
        qs.append(qh)
        ps.append(ph)
        outs.append(oh)
    o = np.concatenate(outs, axis=1)
    x1 = x + (o * col_scale) @ np.asarray(W["wo"], np.float64).T

    u2, r2 = rmsnorm_forward(x1, W["ffn_norm"], shape.rms_eps)
    a = u2 @ np.asarray(W["w_gate"], np.float64).T
    e = u2 @ np.asarray(W["w_up"], np.float64).T
    hh = a * _sigmoid_plain(a) * e
    x2 = x1 + (hh * ch_scale) @ np.asarray(W["w_down"], np.float64).T
    return x2, LayerCache(np.asarray(x, np.float64), r1, u, qs, ks, vs, ps, o, x1, r2, u2, a, e,
                          hh, np.asarray(mask, np.float64))


def masked_layer_backward(c: LayerCache, W, shape, units, dx2):
    """Backward of masked_layer_forward: (dL/dx, dL/dmask [U])."""
    A, KV, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    rep = A // KV
    heads = _heads_of_unit(shape, units)
    chans = _chans_of_unit(shape, units)
    dmask = np.zeros(units)

    # FFN branch: x2 = x1 + (M h) Wd^T
    dhm = dx2 @ np.asarray(W["w_down"], np.float64)          # dL/d(M h)   [S][F]
    dh = np.empty_like(dhm)
    for j, cs in enumerate(chans):
        dmask[j] += np.sum(dhm[:, cs] * c.h[:, cs])
        dh[:, cs] = dhm[:, cs] * c.mask[j]
    sg = _sigmoid_plain(c.a)
    da = dh * c.e * sg * (1.0 + c.a * (1.0 - sg))
    de = dh * c.a * sg
    du2 = da @ np.asarray(W["w_gate"], np.float64) + de @ np.asarray(W["w_up"], np.float64)
    dx1 = dx2 + rmsnorm_backward(c.x1, W["ffn_norm"], c.r2, du2)

    # attention branch: x1 = x + (M o) Wo^T
    dom = dx1 @ np.asarray(W["wo"], np.float64)              # dL/d(M o)   [S][A d]
    du = np.zeros_like(c.u)
    wq, wk, wv = (np.asarray(W[n], np.float64) for n in ("wq", "wk", "wv"))
    dk = {g: np.zeros_like(c.k[g]) for g in range(KV)}
    dv = {g: np.zeros_like(c.v[g]) for g in range(KV)}
    for j, hs in enumerate(heads):
        for h in hs:
            cols = slice(h * d, (h + 1) * d)
            dmask[j] += np.sum(dom[:, cols] * c.o[:, cols])
            dq_h, dk_h, dv_h = attention_backward(c.q[h], c.k[h // rep], c.v[h // rep], c.p[h],
                                                  dom[:, cols] * c.mask[j])
            du += rope_backward(dq_h, shape.rope_theta) @ wq[cols]
            dk[h // rep] += dk_h
            dv[h // rep] += dv_h
    for g in range(KV):
        rows = slice(g * d, (g + 1) * d)
        du += rope_backward(dk[g], shape.rope_theta) @ wk[rows] + dv[g] @ wv[rows]
    dx = dx1 + rmsnorm_backward(c.x, W["attn_norm"], c.r1, du)
    return dx, dmask


def masked_input(vision, text, m_tok):
    """Sec. 3.1 during training: [m_i v_i ; text], the sequence keeps its length."""
    v = np.asarray(vision, np.float64) * np.asarray(m_tok, np.float64)[:, None]
    return np.concatenate([v, np.asarray(text, np.float64)], axis=0)


def masked_forward(shape, layer_weights, vision, text, m_tok, unit_masks, prefix, units):
    """The static-shape forward of one sample.  unit_masks [(L-P)][U] (real
    values allowed); returns (hidden [S][D], per-layer caches)."""
    L = shape.n_layers
    x = masked_input(vision, text, m_tok)
    caches = []
    for l in range(L):
        mask = np.ones(units) if l < prefix else np.asarray(unit_masks[l - prefix], np.float64)
        x, c = masked_layer_forward(x, layer_weights(l), shape, mask, units)
        caches.append(c)
    return x, caches


def masked_backward(shape, layer_weights, caches, units, grad_out):
    """dL/dX_0 [S][D] and dL/dM [L][U] for the upstream gradient grad_out."""
    dx = np.asarray(grad_out, np.float64)
    dM = np.zeros((len(caches), units))
    for l in range(len(caches) - 1, -1, -1):
        dx, dM[l] = masked_layer_backward(caches[l], layer_weights(l), shape, units, dx)
    return dx, dM


@dataclass
class TrainResult:
    hidden: np.ndarray          # [S][D] final hidden states
    token_mask: np.ndarray      # uint8 [N]
    unit_mask: np.ndarray       # uint8 [(L-P) U]
    grad_m: np.ndarray          # dL/dm [N]
    grad_M: np.ndarray          # dL/dM [L][U] (prefix rows: the gradient a mask there would get)
    grad_z: np.ndarray          # dL/dz [N]
    grad_gate: np.ndarray       # dL/dg [(L-P) U]
    grad_x0: np.ndarray         # dL/dX_0 [S][D]


def masked_train_step(shape, layer_weights, vision, text, z, gate_logits, grad_out, prefix,
                      units, tau_tok, tau_comp, xi_tok=None, xi_gate=None) -> TrainResult:
    """Forward under the straight-through masks of Eq. (6) and the gradient of
    L = <grad_out, hidden> with respect to the token and gate logits."""
    y_t, m_t = gumbel_sigmoid(z, xi_tok, tau_tok)
    y_g, m_g = gumbel_sigmoid(gate_logits, xi_gate, tau_comp)
    L = shape.n_layers
    M = m_g.reshape(L - prefix, units).astype(np.float64)
    hidden, caches = masked_forward(shape, layer_weights, vision, text, m_t, M, prefix, units)
    dx0, dM = masked_backward(shape, layer_weights, caches, units, grad_out)
    N = np.asarray(z).size
    dm = np.sum(dx0[:N] * np.asarray(vision, np.float64), axis=1)
    gz = dm * y_t * (1.0 - y_t) / tau_tok
    gg = dM[prefix:].reshape(-1) * y_g * (1.0 - y_g) / tau_comp
    return TrainResult(hidden, m_t, m_g.astype(np.uint8), dm, dM, gz, gg, dx0)
