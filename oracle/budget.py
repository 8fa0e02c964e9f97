"""CPU oracle for threshold token selection and the deterministic budget
projection (SmartVL inference, Sec. 3.1 and Sec. 3.3 "Inference").

TEST INFRASTRUCTURE ONLY, like the rest of this package: the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never does.

What is computed, per sample b:
  * threshold selection (Sec. 3.1, inference rule): with the Gumbel noise
    removed, visual token i is kept iff sigma(z_i) > 0.5, i.e. iff z_i > 0;
    z_i = 0 and NaN logits are dropped;
  * the estimated prefill cost of Eq. (8) with the discrete sequence length
    S = T + s (T text tokens, s kept visual tokens) and the layer activity
    alpha_l (active query heads / A; 0 for a skipped layer):
        C(s) = sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2] + 2 D V S,
    and C_full, the same with every alpha_l = 1 and s = N;
  * the deterministic budget projection for a budget b < 1 (Sec. 3.3): if the
    threshold set costs more than b * C_full, the lowest-confidence visual
    tokens are discarded first, i.e. the sample keeps the largest s no larger
    than the threshold count with C(s) <= b * C_full (the kept set is then the
    s largest logits, ties to the lower index); only if even s = 0 does not
    fit are layers / heads reduced.

Readings (the paper does not fix these; listed in the design notes):
  * the comparison C(s) <= b * C_full is exact: b is the float32 budget's
    exact binary value and the costs are integers times alpha, compared with
    rational arithmetic;
  * V is the vocabulary size of the LM-head term; V = 0 leaves the term out
    (the reading under which Eq. (8) gives the printed 8.5T full prefill);
  * the layer / head reduction drops whole head groups (heads
    [j A/G, (j+1) A/G) and, with FFN gating, FFN slice j) of layers at or
    after the prefix P, one group at a time: the lowest gate logit first when
    the controller's logits are given (ties: the later layer, then the higher
    group), otherwise the later layer first, then the higher group.  After
    each drop it checks C(0) <= b * C_full; once that holds, the token step
    runs again with the reduced alphas.  A layer whose groups are all dropped
    is skipped (alpha_l = 0).  If dropping every eligible group still leaves
    C(0) > b * C_full, the sample keeps no visual tokens and no eligible group
    (the budget cannot be met);
  * with the layer controller (one gate per layer, units = 1) the unit the
    reduction drops is a whole layer, in the same order (lowest gate logit
    first, ties: the later layer).

Every function below cites the passage it follows.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Optional, Tuple

import numpy as np


def threshold_count(logits: np.ndarray) -> int:
    """Number of visual tokens with sigma(z) > 0.5 (Sec. 3.1: tokens with
    sigma(z_i) <= 0.5 are physically discarded at inference)."""
    z = np.asarray(logits, dtype=np.float64).ravel()
    keep = np.zeros(z.shape, dtype=bool)
    finite_or_inf = ~np.isnan(z)
    keep[finite_or_inf] = z[finite_or_inf] > 0.0
    return int(keep.sum())


def layer_alphas(shape, layer_on: np.ndarray, head_on: np.ndarray) -> list:
    """alpha_l of one sample (Sec. 3.2, layer-head controller): the active
    fraction of the layer's heads, 0 for a skipped layer; exact fractions."""
    A = shape.n_heads
    out = []
    for l in range(shape.n_layers):
        if not layer_on[l]:
            out.append(Fraction(0))
        else:
            out.append(Fraction(int(np.sum(head_on[l] != 0)), A))
    return out


def eq8_cost(shape, S: int, alphas, vocab: int) -> Fraction:
    """Eq. (8) at sequence length S: sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2] + 2 D V S."""
    D, F = shape.d_model, shape.d_ffn
    per_layer = (8 * D * D + 6 * D * F) * S + 4 * D * S * S
    return sum((a * per_layer for a in alphas), Fraction(0)) + 2 * D * vocab * S


def full_cost(shape, n_vision: int, n_text: int, vocab: int) -> Fraction:
    """C_full: every layer at full capacity and every visual token kept."""
    return eq8_cost(shape, n_text + n_vision, [Fraction(1)] * shape.n_layers, vocab)


def _max_tokens(shape, n_text: int, cap: int, alphas, vocab: int, limit: Fraction) -> int:
    """Largest s in [0, cap] with C(T + s) <= limit, or -1 if none (C grows with s)."""
    best = -1
    for s in range(cap + 1):
        if eq8_cost(shape, n_text + s, alphas, vocab) <= limit:
            best = s
        else:
            break
    return best


def project_sample(shape, logits: np.ndarray, n_text: int, budget: float, vocab: int,
                   prefix: int, layer_on: np.ndarray, head_on: np.ndarray,
                   ffn_on: Optional[np.ndarray], gate_logits: Optional[np.ndarray],
                   units: Optional[int] = None
                   ) -> Tuple[int, np.ndarray, np.ndarray, Optional[np.ndarray]]:
    """Threshold selection and the budget projection for one sample (Sec. 3.3).

    units: gates per layer, n_groups (layer-head controller, the default) or
    1 (layer controller: gate_logits [L][1], whole layers are the units).
    Returns (keep count, layer_on, head_on, ffn_on) after the projection; the
    kept tokens are then the `keep` largest logits (select_topk)."""
    N = int(np.asarray(logits).size)
    G, A, L = shape.n_groups, shape.n_heads, shape.n_layers
    layer_on = np.array(layer_on, dtype=np.uint8).copy()
    head_on = np.array(head_on, dtype=np.uint8).copy()
    ffn_on = None if ffn_on is None else np.array(ffn_on, dtype=np.uint8).copy()
    n_pos = threshold_count(logits)
    b = Fraction(float(np.float32(budget)))           # the float32 budget, exactly
    if b >= 1:
        return n_pos, layer_on, head_on, ffn_on
    limit = b * full_cost(shape, N, n_text, vocab)
    alphas = layer_alphas(shape, layer_on, head_on)
    s = _max_tokens(shape, n_text, n_pos, alphas, vocab, limit)
    if s >= 0:
        return s, layer_on, head_on, ffn_on
    # token-level adjustment alone is not enough: drop whole head groups
    # (layer controller: whole layers)
    per_layer = G if units is None else units
    hg = A // per_layer
    order = []
    for l in range(prefix, L):
        if not layer_on[l]:
            continue
        for j in range(per_layer):
            if np.any(head_on[l, j * hg:(j + 1) * hg]):
                conf = float(gate_logits[l, j]) if gate_logits is not None else 0.0
                order.append((conf, -l, -j, l, j))
    order.sort()
    for _, _, _, l, j in order:
        head_on[l, j * hg:(j + 1) * hg] = 0
        if ffn_on is not None:
            if per_layer == 1:
                ffn_on[l, :] = 0
            else:
                ffn_on[l, j] = 0
        if not np.any(head_on[l]):
            layer_on[l] = 0
        alphas = layer_alphas(shape, layer_on, head_on)
        if eq8_cost(shape, n_text, alphas, vocab) <= limit:
            return _max_tokens(shape, n_text, n_pos, alphas, vocab, limit), layer_on, head_on, ffn_on
    return 0, layer_on, head_on, ffn_on


def project_batch(shape, logits: np.ndarray, n_text: int, budget: float, vocab: int,
                  prefix: int, layer_mask: np.ndarray, head_mask: np.ndarray,
                  ffn_mask: Optional[np.ndarray], gate_logits: Optional[np.ndarray] = None):
    """project_sample over a batch: keep [B] and the projected masks."""
    B = logits.shape[0]
    keep = np.zeros(B, dtype=np.int32)
    lm, hm = layer_mask.copy(), head_mask.copy()
    fm = None if ffn_mask is None else ffn_mask.copy()
    for i in range(B):
        k, lo, ho, fo = project_sample(shape, logits[i], n_text, budget, vocab, prefix,
                                       layer_mask[i], head_mask[i],
                                       None if ffn_mask is None else ffn_mask[i],
                                       None if gate_logits is None else gate_logits[i])
        keep[i] = k
        lm[i], hm[i] = lo, ho
        if fm is not None:
            fm[i] = fo
    return keep, lm, hm, fm
