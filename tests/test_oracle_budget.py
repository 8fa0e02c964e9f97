"""Pins of the threshold-selection / budget-projection oracle (CPU only).

Each check ties the oracle to something outside itself: the logistic
function of scipy, the paper's printed full-prefill FLOPs, and the defining
properties of the projection (feasible, maximal, order of the reductions).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

from oracle import budget as ob
from oracle.prefill import select_topk
from workloads import ModelShape

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_figures.json")

TINY = ModelShape(n_layers=6, d_model=64, n_heads=8, n_kv_heads=8, head_dim=8, d_ffn=128,
                  n_groups=4, dtype="f32")


def test_threshold_matches_logistic():
    """sigma(z) > 0.5 (scipy's expit) keeps exactly the tokens the oracle keeps,
    for ordinary values, +-0, +-inf and NaN (Sec. 3.1 inference rule)."""
    rng = np.random.default_rng(0)
    z = np.concatenate([rng.normal(0, 3, 5000), [0.0, -0.0, np.inf, -np.inf, np.nan, 1e-6, -1e-6]])
    for trial in range(20):
        zz = rng.permutation(z)[: rng.integers(1, z.size)]
        with np.errstate(invalid="ignore"):
            want = int(np.sum(scipy.special.expit(zz) > 0.5))
        assert ob.threshold_count(zz) == want
    # below float64's resolution at 0.5, sigma(z) > 0.5 still holds exactly for z > 0
    assert ob.threshold_count(np.array([1e-300, -1e-300])) == 1


def test_eq8_reproduces_printed_full_prefill():
    """Eq. (8) with every alpha = 1, V = 0, S = 576 + 64 gives the printed 8.5T."""
    g = json.load(open(GOLDEN))["full_prefill_flops_llava15_7b"]
    sh = g["shape"]
    shape = ModelShape(n_layers=sh["n_layers"], d_model=sh["d_model"], n_heads=sh["n_heads"],
                       n_kv_heads=sh["n_heads"], head_dim=sh["d_model"] // sh["n_heads"],
                       d_ffn=sh["d_ffn"], n_groups=4, dtype="bf16")
    c = ob.full_cost(shape, sh["image_tokens"], 64, vocab=0)
    assert round(float(c) / 1e12, g["digits"] - 1) == g["value_T"]


def test_eq8_structure():
    """alpha scales the layer terms linearly, the LM term is 2 D V S, and the
    cost grows with S."""
    S = 37
    ones = [Fraction(1)] * TINY.n_layers
    halves = [Fraction(1, 2)] * TINY.n_layers
    c1 = ob.eq8_cost(TINY, S, ones, 0)
    assert ob.eq8_cost(TINY, S, halves, 0) * 2 == c1
    assert ob.eq8_cost(TINY, S, ones, 1000) - c1 == 2 * TINY.d_model * 1000 * S
    assert all(ob.eq8_cost(TINY, s + 1, ones, 50) > ob.eq8_cost(TINY, s, ones, 50) for s in range(60))


def _random_case(rng, B=4, N=40, T=7):
    logits = rng.normal(-0.3, 1.0, (B, N)).astype(np.float32)
    logits[0, :5] = 0.0                       # zeros are dropped
    lm = (rng.random((B, TINY.n_layers)) > 0.2).astype(np.uint8)
    hm = (rng.random((B, TINY.n_layers, TINY.n_heads)) > 0.3).astype(np.uint8)
    fm = (rng.random((B, TINY.n_layers, TINY.n_groups)) > 0.3).astype(np.uint8)
    gl = rng.normal(0, 1, (B, TINY.n_layers, TINY.n_groups)).astype(np.float32)
    return logits, lm, hm, fm, gl, T


@pytest.mark.parametrize("budget", [1.0, 1.5, 0.9, 0.5, 0.3, 0.12, 0.05, 0.01])
def test_projection_properties(budget):
    """The kept count fits the budget and is maximal (Sec. 3.3: drop the
    lowest-confidence tokens first); b >= 1 keeps the threshold set; masks
    change only when even zero visual tokens do not fit."""
    rng = np.random.default_rng(int(budget * 1000))
    for trial in range(6):
        logits, lm, hm, fm, gl, T = _random_case(rng)
        N = logits.shape[1]
        full = ob.full_cost(TINY, N, T, 0)
        limit = Fraction(float(np.float32(budget))) * full
        keep, lm2, hm2, fm2 = ob.project_batch(TINY, logits, T, budget, 0, 2, lm, hm, fm, gl)
        for b in range(logits.shape[0]):
            npos = ob.threshold_count(logits[b])
            assert 0 <= keep[b] <= npos
            a2 = ob.layer_alphas(TINY, lm2[b], hm2[b])
            if budget >= 1:
                assert keep[b] == npos and np.array_equal(hm2[b], hm[b])
                continue
            changed = not np.array_equal(hm2[b], hm[b])
            a1 = ob.layer_alphas(TINY, lm[b], hm[b])
            if not changed:
                assert ob.eq8_cost(TINY, T + keep[b], a1, 0) <= limit
                if keep[b] < npos:
                    assert ob.eq8_cost(TINY, T + keep[b] + 1, a1, 0) > limit
            else:
                # reductions only when zero visual tokens did not fit
                assert ob.eq8_cost(TINY, T, a1, 0) > limit
                # prefix layers (P = 2) untouched; groups dropped whole
                assert np.array_equal(hm2[b, :2], hm[b, :2])
                assert np.all(hm2[b] <= hm[b]) and np.all(fm2[b] <= fm[b])
                if ob.eq8_cost(TINY, T, a2, 0) <= limit:
                    if keep[b] < npos:
                        assert ob.eq8_cost(TINY, T + keep[b] + 1, a2, 0) > limit
                    assert ob.eq8_cost(TINY, T + keep[b], a2, 0) <= limit


def test_projection_drops_lowest_confidence_groups_first():
    """Reduced groups are those with the lowest gate logits (ties: the later
    layer, then the higher group), and no more are dropped than needed."""
    rng = np.random.default_rng(7)
    hg = TINY.n_heads // TINY.n_groups
    checked = 0
    for trial in range(200):
        logits, lm, hm, fm, gl, T = _random_case(rng, B=1)
        lm[:] = 1
        hm[:] = 1
        budget = float(rng.choice([0.02, 0.05, 0.1, 0.2]))
        keep, lm2, hm2, fm2 = ob.project_batch(TINY, logits, T, budget, 0, 2, lm, hm, fm, gl)
        dropped = [(l, j) for l in range(2, TINY.n_layers) for j in range(TINY.n_groups)
                   if hm2[0, l, j * hg] == 0]
        kept = [(l, j) for l in range(2, TINY.n_layers) for j in range(TINY.n_groups)
                if hm2[0, l, j * hg] == 1]
        if not dropped:
            continue
        checked += 1
        key = lambda u: (float(gl[0, u[0], u[1]]), -u[0], -u[1])
        assert max(map(key, dropped)) <= min(map(key, kept), default=(np.inf,))
        limit = Fraction(float(np.float32(budget))) * ob.full_cost(TINY, logits.shape[1], T, 0)
        if kept:     # feasible: restoring the last dropped group would not fit
            last = max(dropped, key=key)
            hm3 = hm2[0].copy()
            hm3[last[0], last[1] * hg:(last[1] + 1) * hg] = 1
            lm3 = lm2[0].copy()
            lm3[last[0]] = 1
            assert ob.eq8_cost(TINY, T, ob.layer_alphas(TINY, lm3, hm3), 0) > limit
        # a layer with every group dropped is skipped
        for l in range(TINY.n_layers):
            if not np.any(hm2[0, l]):
                assert lm2[0, l] == 0
    assert checked > 20


def test_projected_keep_selects_positive_logits():
    """The kept set is the `keep` largest logits, all of them positive."""
    rng = np.random.default_rng(3)
    for trial in range(50):
        logits, lm, hm, fm, gl, T = _random_case(rng, B=1)
        keep, *_ = ob.project_batch(TINY, logits, T, 0.4, 0, 2, lm, hm, fm, gl)
        kept = select_topk(logits[0], int(keep[0]))
        assert np.all(logits[0][kept] > 0)


def test_projection_monotone_in_budget():
    """While the token step alone meets the budget (masks unchanged), a
    larger budget never keeps fewer tokens.  (Once groups are dropped the
    freed budget can hold more tokens, so monotonicity is not claimed there.)"""
    rng = np.random.default_rng(11)
    logits, lm, hm, fm, gl, T = _random_case(rng)
    prev = None
    for budget in np.linspace(0.05, 1.0, 30):
        keep, lm2, hm2, fm2 = ob.project_batch(TINY, logits, T, float(budget), 0, 2, lm, hm, fm, gl)
        same = np.array([np.array_equal(hm2[b], hm[b]) for b in range(len(keep))])
        if prev is not None:
            both = same & prev[1]
            assert np.all(keep[both] >= prev[0][both])
        prev = (keep, same)
