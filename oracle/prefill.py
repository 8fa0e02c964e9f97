"""CPU oracle for the budget-adapted MLLM prefill (SmartVL inference path).

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously-correct
definition that the GPU library is checked against.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never calls it and shares no code with it.

What is computed (paper, Sec. 3 and Sec. 3.3 "Inference"):
  * the token controller's scores pick the vision tokens to keep; the budget
    projection drops the lowest-confidence tokens first, so for an integer
    budget k the kept set is the k highest-scoring tokens;
  * dropped tokens are physically removed and the survivors, followed by the
    text tokens, form a compressed contiguous sequence that RoPE numbers
    0..S-1 with no re-encoding (Sec. 3.1);
  * each decoder layer either runs or is bypassed through its residual
    connection (layer controller, Sec. 3.2); inside a running layer only the
    active heads of the active head groups contribute, and group j also gates
    slice j of the FFN intermediate dimension (layer-head controller, Sec. 3.2);
  * the executed multiply-adds are counted (2 FLOPs each) so that the count can
    be compared with the closed form and with the paper's estimator, Eq. (8).

Arithmetic: every input is widened to float64 and every product, sum and
reduction is done in float64 (numpy; the matrix products are plain BLAS
calls).  No blocking, fusion or reordering beyond the definitions below.

Readings of points the paper leaves open (each listed in the design notes):
  ties in score -> lower index wins; NaN ranks below -inf; -0 == +0;
  kept tokens keep their original order; sequence = [kept vision ; text];
  LLaMA block (pre-RMSNorm, rotate-half RoPE with base theta, causal softmax
  attention with scale 1/sqrt(d), SwiGLU FFN, no biases, no final norm);
  head group j = heads [j*A/G, (j+1)*A/G), FFN slice j = channels
  [j*F/G, (j+1)*F/G); a KV head runs iff one of its query heads is active.

Parity pins: see the oracle tests (HF transformers LLaMA as the dense and
gated special case, brute-force ranking, closed-form FLOPs vs Eq. (8), RoPE
and attention invariants).  Absolute hidden values beyond those pins: parity
unpinned (the paper prints no worked example).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np


# --------------------------------------------------------------------------- FLOP counter
@dataclass
class FlopCounter:
    """Executed FLOPs by component (2 per multiply-add, matrix products only)."""
    q: int = 0
    kv: int = 0
    o: int = 0
    attn: int = 0
    ffn: int = 0

    @property
    def total(self) -> int:
        return self.q + self.kv + self.o + self.attn + self.ffn

    def as_dict(self) -> Dict[str, int]:
        return dict(q=self.q, kv=self.kv, o=self.o, attn=self.attn, ffn=self.ffn,
                    total=self.total)


def _mm(a: np.ndarray, b: np.ndarray, counter: Optional[FlopCounter], part: str) -> np.ndarray:
    """a @ b in float64, counted as 2*m*k*n FLOPs against `part`."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if counter is not None:
        m, k = a.shape
        n = b.shape[1]
        setattr(counter, part, getattr(counter, part) + 2 * m * k * n)
    return a @ b


# --------------------------------------------------------------------------- selection
def select_topk(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k highest scores, returned in ascending index order.

    Sec. 3.3 (budget projection discards the lowest-confidence visual tokens
    first) and Sec. 3.1 (kept tokens form a contiguous sequence in their
    original order).  Ordering: score descending; NaN below every number
    (including -inf); -0 equal to +0; equal scores -> lower index first.
    """
    s = np.asarray(scores, dtype=np.float64).ravel()
    n = s.shape[0]
    if not 0 <= k <= n:
        raise ValueError("keep budget outside [0, N]")
    nan = np.isnan(s)
    value = np.where(nan, 0.0, s) + 0.0      # + 0.0 turns -0 into +0
    idx = np.arange(n)
    # np.lexsort sorts by the last key first: non-NaN first, then larger
    # value first, then lower index first.
    order = np.lexsort((idx, -value, nan))
    return np.sort(order[:k])


def compact(vision: np.ndarray, text: np.ndarray, kept: np.ndarray) -> np.ndarray:
    """[vision[kept] ; text] as one contiguous sequence (Sec. 3.1), float64."""
    v = np.asarray(vision, dtype=np.float64)[np.asarray(kept, dtype=np.int64)]
    t = np.asarray(text, dtype=np.float64)
    return np.concatenate([v, t], axis=0)


# --------------------------------------------------------------------------- block pieces
def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain, row-wise (LLaMA pre-norm)."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope(a: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of rows a [S][d] at the given positions.

    Pair (r, r + d/2) is rotated by angle p * theta**(-2r/d), r < d/2.
    """
    a = np.asarray(a, dtype=np.float64)
    d = a.shape[-1]
    half = d // 2
    r = np.arange(half, dtype=np.float64)
    omega = theta ** (-2.0 * r / d)
    phi = np.asarray(positions, dtype=np.float64)[:, None] * omega[None, :]
    c, s = np.cos(phi), np.sin(phi)
    a1, a2 = a[:, :half], a[:, half:]
    return np.concatenate([a1 * c - a2 * s, a2 * c + a1 * s], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     counter: Optional[FlopCounter] = None) -> np.ndarray:
    """softmax(q k^T / sqrt(d)) v with row i attending to keys 0..i.

    The counter is charged for the causal triangle only (row i uses i+1 keys
    in both products), i.e. what a causal kernel executes.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    S, d = q.shape
    if S == 0:
        return np.zeros((0, v.shape[1]))
    scores = (q @ k.T) / np.sqrt(d)
    future = np.triu(np.ones((S, S), dtype=bool), 1)
    scores = np.where(future, -np.inf, scores)
    scores = scores - scores.max(axis=1, keepdims=True)
    p = np.exp(scores)
    p = p / p.sum(axis=1, keepdims=True)
    if counter is not None:
        counter.attn += 2 * (2 * d * (S * (S + 1) // 2))
    return p @ v


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _channel_index(ffn_on: Optional[Sequence[int]], d_ffn: int, n_groups: int) -> np.ndarray:
    """Active FFN channels: slice j = [j*F/G, (j+1)*F/G) for every active group j."""
    if ffn_on is None:
        return np.arange(d_ffn)
    w = d_ffn // n_groups
    chans = [np.arange(j * w, (j + 1) * w) for j in range(n_groups) if ffn_on[j]]
    return np.concatenate(chans) if chans else np.zeros(0, dtype=np.int64)


def decoder_layer(x: np.ndarray, W: Dict[str, np.ndarray], shape, head_on: Sequence[int],
                  ffn_on: Optional[Sequence[int]], counter: Optional[FlopCounter] = None
                  ) -> np.ndarray:
    """One gated LLaMA block on one sample's sequence x [S][D] (float64).

    head_on[h] in {0,1} for each query head; ffn_on[j] in {0,1} per group, or
    None for an ungated FFN.  Inactive heads and channels are never computed
    and contribute no term (Sec. 3.2, layer-head controller).
    """
    x = np.array(x, dtype=np.float64, copy=True)
    S, D = x.shape
    A, KV, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    rep = A // KV
    pos = np.arange(S)
    heads = [h for h in range(A) if head_on[h]]

    # attention sub-block
    if heads:
        u = rmsnorm(x, W["attn_norm"], shape.rms_eps)
        keys, values = {}, {}
        for g in sorted({h // rep for h in heads}):
            wk = np.asarray(W["wk"][g * d:(g + 1) * d], dtype=np.float64)
            wv = np.asarray(W["wv"][g * d:(g + 1) * d], dtype=np.float64)
            keys[g] = rope(_mm(u, wk.T, counter, "kv"), pos, shape.rope_theta)
            values[g] = _mm(u, wv.T, counter, "kv")
        outs = []
        for h in heads:
            wq = np.asarray(W["wq"][h * d:(h + 1) * d], dtype=np.float64)
            q = rope(_mm(u, wq.T, counter, "q"), pos, shape.rope_theta)
            outs.append(causal_attention(q, keys[h // rep], values[h // rep], counter))
        o = np.concatenate(outs, axis=1)                       # [S][H_a*d]
        cols = np.concatenate([np.arange(h * d, (h + 1) * d) for h in heads])
        wo = np.asarray(W["wo"], dtype=np.float64)[:, cols]    # [D][H_a*d]
        x = x + _mm(o, wo.T, counter, "o")

    # FFN sub-block
    chans = _channel_index(ffn_on, shape.d_ffn, shape.n_groups)
    if chans.size:
        u = rmsnorm(x, W["ffn_norm"], shape.rms_eps)
        wg = np.asarray(W["w_gate"], dtype=np.float64)[chans]
        wu = np.asarray(W["w_up"], dtype=np.float64)[chans]
        g = _mm(u, wg.T, counter, "ffn")
        e = _mm(u, wu.T, counter, "ffn")
        h = silu(g) * e
        wd = np.asarray(W["w_down"], dtype=np.float64)[:, chans]
        x = x + _mm(h, wd.T, counter, "ffn")
    return x


# --------------------------------------------------------------------------- whole path
@dataclass
class PrefillResult:
    kept_idx: np.ndarray        # int32 [B][N]: first keep[b] entries ascending, rest -1
    cu_seqlens: np.ndarray      # int32 [B+1]
    resid: np.ndarray           # float64 [sum S_b][D], packed in sample order
    flops: FlopCounter = field(default_factory=FlopCounter)


def select_and_compact(scores, keep, vision, text):
    """Token selection and packing for a batch (kept indices, cu_seqlens, packed rows)."""
    scores = np.asarray(scores)
    B, N = scores.shape
    kept_idx = np.full((B, N), -1, dtype=np.int32)
    seqs: List[np.ndarray] = []
    cu = np.zeros(B + 1, dtype=np.int32)
    for b in range(B):
        kept = select_topk(scores[b], int(keep[b]))
        kept_idx[b, :kept.size] = kept
        seqs.append(compact(vision[b], text[b], kept))
        cu[b + 1] = cu[b] + seqs[-1].shape[0]
    return kept_idx, cu, seqs


def prefill(shape, layer_weights: Callable[[int], Dict[str, np.ndarray]], scores, keep,
            vision, text, layer_mask, head_mask, ffn_mask=None,
            layers: Optional[Sequence[int]] = None) -> PrefillResult:
    """Budget-adapted prefill of a batch (Eq. (1) with the masks given).

    layer_weights(l) returns layer l's weights (lets callers stream layers);
    layer_mask [B][L], head_mask [B][L][A], ffn_mask [B][L][G] or None.
    A layer with layer_mask 0 is the identity for that sample.
    """
    kept_idx, cu, seqs = select_and_compact(scores, keep, vision, text)
    counter = FlopCounter()
    B = len(seqs)
    for l in (range(shape.n_layers) if layers is None else layers):
        if not any(layer_mask[b][l] for b in range(B)):
            continue
        W = layer_weights(l)
        for b in range(B):
            if layer_mask[b][l]:
                seqs[b] = decoder_layer(seqs[b], W, shape, head_mask[b][l],
                                        None if ffn_mask is None else ffn_mask[b][l], counter)
    D = shape.d_model
    resid = np.concatenate(seqs, axis=0) if seqs else np.zeros((0, D))
    return PrefillResult(kept_idx, cu, resid.reshape(-1, D), counter)
