"""CPU oracle for the LLM-side compute controller and the controlled prefill
(SmartVL inference, Sec. 3.2 and Sec. 3.3 "Inference").

TEST INFRASTRUCTURE ONLY, like the rest of this package: the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never does.

What is computed, per sample:
  * the budget token: the scalar budget b is encoded with the sinusoidal
    encoding PE and mapped by MLP_LLM to a D-vector (Sec. 3.2, "Budget
    encoding and prefix layers"); it is appended at the end of the prompt,
    after the text tokens, and takes part in attention like any other row;
  * the token controller's threshold rule keeps the visual tokens with
    sigma(z_i) > 0.5 (Sec. 3.1); the sequence [kept vision ; text ; budget]
    runs through the P prefix layers at full capacity;
  * kappa = sum_i sigma(z_i) / N, the soft token survival rate; PE(kappa)
    through MLP_kappa is added to the budget token's state after the prefix,
    giving h~ (Eq. (7));
  * the gating head maps h~ to logits W_h h~ + c_h; with the Gumbel noise
    removed, a unit is on iff its logit is > 0 (sigma > 0.5).  Layer-head
    controller (LH): one logit per (dynamic layer, head group), group j
    gating heads [j A/G, (j+1) A/G) and FFN slice j, a layer with every group
    off is skipped.  Layer controller (L): one logit per dynamic layer, the
    layer runs at full capacity or is bypassed (Sec. 3.2);
  * for b < 1 the deterministic budget projection (Sec. 3.3, oracle.budget)
    trims the visual tokens first, then whole units, using the gate logits
    as the confidence order;
  * the layers after the prefix run under those masks on the trimmed
    sequence.

Readings of points the paper leaves open (each listed in the design notes):
  * PE(x) of width E: entry 2i is sin(x s w_i), entry 2i+1 is cos(x s w_i),
    w_i = base^(-2i/E), with a scale s applied to the scalar (the Transformer
    encoding of a position x s);
  * MLP_LLM and MLP_kappa: Linear(E -> H) with bias, GELU (erf form),
    Linear(H -> D) with bias;
  * kappa counts sigma(NaN) as 0; kappa = 0 when there are no visual tokens;
  * h_b^(P) is the budget token's residual-stream row after P layers (no
    norm); the gate logits are laid out [dynamic layer][unit];
  * the projection runs at the prefix boundary, with Eq. (8)'s S = text +
    kept visual tokens (the budget token is not counted), the prefix layers
    at alpha = 1 and the controller's masks on the others; the visual tokens
    it discards leave the sequence there, the remaining rows keep their order
    and RoPE numbers them 0..S'-1 in the layers after the prefix (the
    compressed contiguous sequence of Sec. 3.1);
  * the executed-FLOP counter charges layer matrix products only, as the
    prefill oracle does (the controller's small products are not counted).

Arithmetic: float64 throughout (numpy), inputs widened exactly.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional

import numpy as np

from .budget import project_sample, threshold_count
from .prefill import FlopCounter, decoder_layer, select_topk


@dataclass
class Controller:
    """Compute-controller parameters (float64 arrays, [out][in] layout)."""
    prefix: int
    units: int                  # head groups G (LH controller) or 1 (L controller)
    pe_scale: float
    pe_base: float
    llm_w1: np.ndarray          # [H][E]
    llm_b1: np.ndarray          # [H]
    llm_w2: np.ndarray          # [D][H]
    llm_b2: np.ndarray          # [D]
    kap_w1: np.ndarray
    kap_b1: np.ndarray
    kap_w2: np.ndarray
    kap_b2: np.ndarray
    gate_w: np.ndarray          # [(L-P)*units][D]
    gate_b: np.ndarray          # [(L-P)*units]

    @property
    def pe_dim(self) -> int:
        return int(self.llm_w1.shape[1])


def sinusoidal(x: float, dim: int, scale: float, base: float) -> np.ndarray:
    """PE of a scalar (Sec. 3.1, reused in Sec. 3.2): interleaved sin / cos of
    x * scale at the frequencies base^(-2i/dim)."""
    pos = float(x) * float(scale)
    out = np.empty(dim, dtype=np.float64)
    for i in range(dim // 2):
        w = float(base) ** (-2.0 * i / dim)
        out[2 * i] = math.sin(pos * w)
        out[2 * i + 1] = math.cos(pos * w)
    return out


def gelu(x: np.ndarray) -> np.ndarray:
    """x * Phi(x), Phi the standard normal distribution function (erf form)."""
    x = np.asarray(x, dtype=np.float64)
    erf = np.vectorize(math.erf)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def mlp(x: np.ndarray, w1, b1, w2, b2) -> np.ndarray:
    """Linear -> GELU -> Linear, each linear with its bias."""
    h = gelu(np.asarray(w1, np.float64) @ np.asarray(x, np.float64) + np.asarray(b1, np.float64))
    return np.asarray(w2, np.float64) @ h + np.asarray(b2, np.float64)


def kappa(z: np.ndarray) -> float:
    """Soft token survival rate sum_i sigma(z_i) / N (Eq. (7)); NaN -> 0."""
    z = np.asarray(z, dtype=np.float64).ravel()
    if z.size == 0:
        return 0.0
    total = 0.0
    for v in z:
        if math.isnan(v):
            continue
        if v >= 0:
            total += 1.0 / (1.0 + math.exp(-v))
        else:
            e = math.exp(v)
            total += e / (1.0 + e)
    return total / z.size


def budget_token(ctrl: Controller, budget: float) -> np.ndarray:
    """e_b = MLP_LLM(PE(b)) (Sec. 3.2), b at its float32 value."""
    pe = sinusoidal(float(np.float32(budget)), ctrl.pe_dim, ctrl.pe_scale, ctrl.pe_base)
    return mlp(pe, ctrl.llm_w1, ctrl.llm_b1, ctrl.llm_w2, ctrl.llm_b2)


def gate_logits(ctrl: Controller, h_prefix: np.ndarray, kap: float) -> np.ndarray:
    """W_h (h_b^(P) + MLP_kappa(PE(kappa))) + c_h (Eq. (7) and the gating head)."""
    e_k = mlp(sinusoidal(kap, ctrl.pe_dim, ctrl.pe_scale, ctrl.pe_base),
              ctrl.kap_w1, ctrl.kap_b1, ctrl.kap_w2, ctrl.kap_b2)
    h = np.asarray(h_prefix, np.float64) + e_k
    return np.asarray(ctrl.gate_w, np.float64) @ h + np.asarray(ctrl.gate_b, np.float64)


def masks_from_logits(shape, logits: np.ndarray, prefix: int, units: int):
    """Masks of one sample from its gate logits [(L-P)*units] (Sec. 3.2):
    prefix layers at full capacity; a unit is on iff its logit is > 0."""
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    on = (np.asarray(logits, np.float64).reshape(L - prefix, units) > 0.0)
    layer_on = np.ones(L, dtype=np.uint8)
    head_on = np.ones((L, A), dtype=np.uint8)
    ffn_on = np.ones((L, G), dtype=np.uint8)
    hg = A // G
    for i, l in enumerate(range(prefix, L)):
        if units == 1:
            layer_on[l] = head_on[l, :] = ffn_on[l, :] = 1 if on[i, 0] else 0
        else:
            for j in range(G):
                head_on[l, j * hg:(j + 1) * hg] = ffn_on[l, j] = 1 if on[i, j] else 0
            layer_on[l] = 1 if on[i].any() else 0
    return layer_on, head_on, ffn_on


@dataclass
class ControlledResult:
    kept_idx: np.ndarray        # int32 [B][N]: final kept tokens ascending, rest -1
    cu_seqlens: np.ndarray      # int32 [B+1] of the final sequences (S = keep + T + 1)
    resid: np.ndarray           # float64 [sum S][D]
    keep: np.ndarray            # int32 [B] final visual tokens
    counts: np.ndarray          # int32 [B] threshold counts
    kappa: np.ndarray           # float64 [B]
    logits: np.ndarray          # float64 [B][(L-P)*units]
    layer_mask: np.ndarray      # uint8 [B][L]
    head_mask: np.ndarray       # uint8 [B][L][A]
    ffn_mask: np.ndarray        # uint8 [B][L][G]
    prefix_resid: List[np.ndarray]  # per sample [S1][D] after the prefix layers
    flops: FlopCounter


def prefill_controlled(shape, layer_weights: Callable[[int], Dict[str, np.ndarray]],
                       ctrl: Controller, z: np.ndarray, vision, text, budget: float,
                       vocab: int = 0) -> ControlledResult:
    """The controlled prefill of a batch (Sec. 3.1-3.3 at inference)."""
    z = np.asarray(z)
    B, N = z.shape
    L, A, G, D = shape.n_layers, shape.n_heads, shape.n_groups, shape.d_model
    P, U = ctrl.prefix, ctrl.units
    T = np.asarray(text).shape[1]
    e_b = budget_token(ctrl, budget)
    counter = FlopCounter()

    counts = np.array([threshold_count(z[b]) for b in range(B)], dtype=np.int32)
    kaps = np.array([kappa(z[b]) for b in range(B)])
    seqs = []
    for b in range(B):
        kept = select_topk(z[b], int(counts[b]))
        seqs.append(np.concatenate([np.asarray(vision[b], np.float64)[kept],
                                    np.asarray(text[b], np.float64), e_b[None, :]], axis=0))

    full_heads = np.ones(A, dtype=np.uint8)
    full_ffn = np.ones(G, dtype=np.uint8)
    for l in range(P):
        W = layer_weights(l)
        for b in range(B):
            seqs[b] = decoder_layer(seqs[b], W, shape, full_heads, full_ffn, counter)
    prefix_resid = [s.copy() for s in seqs]

    logits = np.zeros((B, (L - P) * U))
    lm = np.zeros((B, L), np.uint8)
    hm = np.zeros((B, L, A), np.uint8)
    fm = np.zeros((B, L, G), np.uint8)
    keep = np.zeros(B, np.int32)
    for b in range(B):
        logits[b] = gate_logits(ctrl, seqs[b][-1], kaps[b])
        keep[b], lm[b], hm[b], fm[b] = decide_sample(shape, z[b], logits[b], T, budget, vocab, P, U)
    kept_idx, cu, resid = finish_controlled(shape, layer_weights, prefix_resid, z, counts, keep,
                                            lm, hm, fm, P, T, counter)
    return ControlledResult(kept_idx, cu, resid.reshape(-1, D), keep, counts, kaps, logits,
                            lm, hm, fm, prefix_resid, counter)


def decide_sample(shape, z, logits, n_text: int, budget: float, vocab: int, prefix: int,
                  units: int):
    """One sample's decisions from its gate logits: a unit runs iff its logit
    is > 0 (Eq. (7)'s sigma > 0.5), then the budget projection (Sec. 3.3
    "Inference") with the logits as the units' confidences.  Returns
    (keep, layer_on [L], head_on [L][A], ffn_on [L][G])."""
    L = shape.n_layers
    lo, ho, fo = masks_from_logits(shape, logits, prefix, units)
    conf = np.zeros((L, units))
    conf[prefix:] = np.asarray(logits, np.float64).reshape(L - prefix, units)
    return project_sample(shape, z, n_text, budget, vocab, prefix, lo, ho, fo, conf, units=units)


def finish_controlled(shape, layer_weights, prefix_resid, z, counts, keep, lm, hm, fm,
                      prefix: int, n_text: int, counter: Optional[FlopCounter] = None):
    """The controlled prefill after the decisions: each sample's sequence
    after the prefix layers ([threshold-kept vision ; text ; budget token])
    loses the visual tokens the projection discarded (the survivors keep their
    order), then layers P..L-1 run under the masks.  Returns (kept_idx,
    cu_seqlens, resid)."""
    z = np.asarray(z)
    B, N = z.shape
    L, D = shape.n_layers, shape.d_model
    T = n_text
    seqs = [np.array(s, dtype=np.float64, copy=True) for s in prefix_resid]
    kept_idx = np.full((B, N), -1, dtype=np.int32)
    for b in range(B):
        k = int(keep[b])
        first = select_topk(z[b], int(counts[b]))
        final = select_topk(z[b], k)
        kept_idx[b, :k] = final
        if k < counts[b]:
            # the discarded visual tokens leave the sequence at the prefix boundary
            rows = np.concatenate([np.searchsorted(first, final),
                                   counts[b] + np.arange(T + 1)])
            seqs[b] = seqs[b][rows]
    for l in range(prefix, L):
        if not lm[:, l].any():
            continue
        W = layer_weights(l)
        for b in range(B):
            if lm[b, l]:
                seqs[b] = decoder_layer(seqs[b], W, shape, hm[b, l], fm[b, l], counter)
    cu = np.zeros(B + 1, dtype=np.int32)
    for b in range(B):
        cu[b + 1] = cu[b] + seqs[b].shape[0]
    resid = np.concatenate(seqs, axis=0) if seqs else np.zeros((0, D))
    return kept_idx, cu, resid
