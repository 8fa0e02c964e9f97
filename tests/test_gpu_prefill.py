"""GPU parity of the whole budget-adapted prefill (svl_prefill) and of one
layer (svl_layer_forward) against the CPU oracle.

Bars: kept indices and cu_seqlens bit-exact; FLOP count exact; hidden
states within max relative error (per sample, max|gpu - oracle| / max|oracle|)
1e-4 for float32 workloads and 2e-2 for bf16 workloads (oracle in float64)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20357_amd as svl
import workloads as W
import os

from gpu_helpers import (elementwise_err_per_sample, gpu_prefill, host_layer, oracle_prefill,
                         rel_err_per_sample, tol_for)

pytestmark = pytest.mark.gpu


def _check_prefill(w, seed=0, samples_for_oracle=None, compute="f16"):
    print(f"prefill {w.name} seed={seed} compute={compute}", flush=True)
    inp = W.draw_inputs(w, seed, device="cuda")
    layers = [W.draw_layer_weights(w, l, seed, device="cuda") for l in range(w.shape.n_layers)]
    kept, cu, resid, flops = gpu_prefill(w, inp, layers, compute=compute)
    ref = oracle_prefill(w, inp, layers, samples_for_oracle)
    samples = list(range(w.batch)) if samples_for_oracle is None else list(samples_for_oracle)
    for j, b in enumerate(samples):
        np.testing.assert_array_equal(kept[b], ref.kept_idx[j])
        assert cu[b + 1] - cu[b] == ref.cu_seqlens[j + 1] - ref.cu_seqlens[j]
    rows = np.concatenate([np.arange(cu[b], cu[b + 1]) for b in samples])
    errs = rel_err_per_sample(resid[rows], ref.resid, ref.cu_seqlens)
    elem = elementwise_err_per_sample(resid[rows], ref.resid, ref.cu_seqlens)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    print(f"  elementwise err per sample: {[f'{e:.2e}' for e in elem]}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs
    if samples_for_oracle is None:
        assert flops["total"] == ref.flops.total
        for k in ("q", "kv", "o", "attn", "ffn"):
            assert flops[k] == getattr(ref.flops, k), k
    return errs


def test_prefill_tiny_f32():
    _check_prefill(W.get_workload("tiny_f32"))


def test_prefill_tiny_f32_other_seeds():
    for seed in (1, 2):
        _check_prefill(W.get_workload("tiny_f32"), seed)


def test_prefill_llava7b_headline_full_size():
    """The benchmarked workload at its real shape: 32 layers, d 4096, keep 144."""
    _check_prefill(W.get_workload("llava7b_b1_keep25"))


def test_prefill_llava7b_headline_bf16_full_size():
    """The benchmarked workload at its real shape with bf16 activations and
    bf16 MFMA products (svl_compute SVL_COMPUTE_BF16), against the 2e-2 bar.
    The normed rows enter the QKV and gate/up products as two bf16 terms
    (hi and lo): with every point rounded to a single bf16 the error was
    2.23e-2 after the 24 executed layers, and the float32 rounding model
    (tests/rounding_model.py) gives 1.34e-2 with the two terms."""
    _check_prefill(W.get_workload("llava7b_b1_keep25"), compute="bf16")


_SLOW = pytest.mark.skipif(os.environ.get("SVL_SLOW_PARITY") != "1",
                           reason="full-depth oracle takes minutes: set SVL_SLOW_PARITY=1")


@pytest.mark.slow
@_SLOW
@pytest.mark.parametrize("name", ["llava7b_b8_ragged", "gqa7b_hires_b2", "llava13b_video_b4"])
def test_prefill_full_depth_real_shape(name):
    """The batched workloads end to end at their real depth, width, batch and
    masks (seed 0): every sample against the float64 oracle."""
    _check_prefill(W.get_workload(name))


def test_prefill_scaled_ragged_batch():
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=6, d_model=1024, n_heads=8,
                 n_kv_heads=8, d_ffn=2816, name="ragged_b8_small")
    _check_prefill(w)


def test_prefill_scaled_gqa():
    w = W.scaled(W.get_workload("gqa7b_hires_b2"), n_layers=4, d_model=1024, n_heads=8,
                 n_kv_heads=4, d_ffn=2048, layers_skipped=1, name="gqa_small")
    _check_prefill(w)


def test_prefill_scaled_video():
    w = W.scaled(W.get_workload("llava13b_video_b4"), n_layers=4, d_model=1024, n_heads=8,
                 n_kv_heads=8, d_ffn=2048, layers_skipped=1, name="video_small")
    _check_prefill(w)


def _layer_case(shape, seqlens, layer_on, head_mask, ffn_mask, seed=3, compute="f16"):
    dev = "cuda"
    cfg = svl.make_config(shape, compute=compute)
    R = int(np.sum(seqlens))
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    g = torch.Generator(device=dev).manual_seed(seed)
    x0 = torch.randn(R, shape.d_model, generator=g, device=dev)
    wl = W.Workload(name="layer", shape=shape, batch=len(seqlens), n_vision=0, n_text=0)
    weights = W.draw_layer_weights(wl, 0, seed, device=dev)
    resid = x0.clone()
    ws = svl.alloc_workspace(cfg, len(seqlens), R, dev)
    svl.svl_layer_forward(cfg, 0, weights, cu, layer_on, head_mask, ffn_mask, resid, ws)
    torch.cuda.synchronize()
    got = resid.cpu().numpy()
    x = x0.cpu().numpy().astype(np.float64)
    Wh = host_layer(weights)
    ref = np.empty_like(x)
    for b in range(len(seqlens)):
        rows = slice(cu[b], cu[b + 1])
        if layer_on[b]:
            ref[rows] = oracle.decoder_layer(x[rows], Wh, shape, head_mask[b],
                                             None if ffn_mask is None else ffn_mask[b])
        else:
            ref[rows] = x[rows]
            # a bypassed sample's rows are not touched at all
            np.testing.assert_array_equal(got[rows], x0.cpu().numpy()[rows])
    elem = elementwise_err_per_sample(got, ref, cu)
    print(f"  elementwise err per sample: {[f'{e:.2e}' for e in elem]}", flush=True)
    return rel_err_per_sample(got, ref, cu)


@pytest.mark.parametrize("dtype,compute", [("f32", "f16"), ("bf16", "f16"), ("bf16", "bf16")])
def test_layer_masks_and_edges(dtype, compute):
    """Per-head masks (not only whole groups), FFN coupled / ungated / all
    off, a bypassed sample, an empty sample and a one-row sample; both
    activation types of bf16-stored weights."""
    hd = 64
    shape = W.ModelShape(n_layers=1, d_model=512, n_heads=8, n_kv_heads=4, head_dim=hd,
                         d_ffn=1024, n_groups=4, dtype=dtype)
    seqlens = np.array([70, 0, 1, 129, 200], np.int32)
    B = len(seqlens)
    rng = np.random.default_rng(0)
    head_mask = (rng.random((B, 8)) > 0.4).astype(np.uint8)
    head_mask[3] = 0                 # attention block off entirely
    head_mask[4] = 1
    ffn_mask = (rng.random((B, 4)) > 0.4).astype(np.uint8)
    ffn_mask[4] = 0                  # FFN block off entirely
    layer_on = np.array([1, 1, 1, 1, 0], np.uint8)
    tol = tol_for(shape)
    for fm in (ffn_mask, None):
        print(f"layer edges dtype={dtype} compute={compute} "
              f"ffn={'coupled' if fm is not None else 'ungated'}", flush=True)
        errs = _layer_case(shape, seqlens, layer_on, head_mask, fm, compute=compute)
        print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
        assert max(errs) <= tol, errs


@pytest.mark.parametrize("name,compute", [("llava7b_b1_keep25", "f16"), ("llava7b_b1_keep25", "bf16"),
                                          ("llava7b_b8_ragged", "f16"), ("llava7b_b8_ragged", "bf16"),
                                          ("gqa7b_hires_b2", "f16"),
                                          ("llava13b_video_b4", "f16")])
def test_layer_full_size(name, compute):
    """One decoder layer at each workload's real width, sequence lengths and
    masks (first non-prefix layer of the seed-0 draw).  The batched workloads'
    output / down projections have more tiles than CUs and run as 4-wave
    tiles."""
    w = W.get_workload(name)
    keep, lm, hm, fm = W.draw_masks(w, 0)
    l = w.shape.prefix
    seqlens = (keep + w.n_text).astype(np.int32)
    print(f"layer full size {name} compute={compute} seqlens={seqlens.tolist()}", flush=True)
    errs = _layer_case(w.shape, seqlens, lm[:, l], hm[:, l], None if fm is None else fm[:, l],
                       compute=compute)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


@pytest.mark.parametrize("compute", ["f16", "bf16"])
def test_layer_row_block_counts(compute):
    """Single-tile samples of 64 to 208 rows (4 to 13 row blocks, odd block
    counts and counts just past a multiple of 64) with K chunk lists of 1 to
    9 chunks (one active head of 64 columns up to d_model 576, including a
    K that is not a multiple of the 4-chunk weight stage)."""
    rng = np.random.default_rng(5)
    for D, A, seqlens in ((512, 8, [80, 144, 208, 65, 129, 193]),
                          (576, 9, [70, 64, 81, 128, 145, 192, 200]),
                          (1024, 16, [208, 140, 75])):
        G = 4 if A % 4 == 0 else 3
        shape = W.ModelShape(n_layers=1, d_model=D, n_heads=A, n_kv_heads=A, head_dim=64,
                             d_ffn=G * 256, n_groups=G, dtype="bf16")
        B = len(seqlens)
        head_mask = (rng.random((B, A)) > 0.5).astype(np.uint8)
        head_mask[0] = 0
        head_mask[0, 1] = 1              # one active head: a one-chunk output projection
        head_mask[1] = 1
        ffn_mask = (rng.random((B, G)) > 0.3).astype(np.uint8)
        ffn_mask[:, 0] = 1
        print(f"row block counts d_model {D} compute={compute} rows {seqlens}", flush=True)
        errs = _layer_case(shape, np.array(seqlens, np.int32), np.ones(B, np.uint8), head_mask,
                           ffn_mask, compute=compute)
        print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
        assert max(errs) <= tol_for(shape), errs


@pytest.mark.parametrize("split,compute", [(2, "f16"), (3, "f16"), (2, "bf16")])
def test_layer_forced_paired_split(split, compute, monkeypatch):
    """The split-K QKV and gate/up path (float32 slices, then the finish
    kernels: RoPE or SwiGLU after the ordered sum), which the planner uses
    only when forced: the per-head-mask edge case and the headline layer."""
    monkeypatch.setenv("SVL_PAIRED_SPLIT", str(split))
    shape = W.ModelShape(n_layers=1, d_model=512, n_heads=8, n_kv_heads=4, head_dim=64,
                         d_ffn=1024, n_groups=4, dtype="bf16")
    seqlens = np.array([70, 0, 1, 129, 200], np.int32)
    rng = np.random.default_rng(1)
    head_mask = (rng.random((5, 8)) > 0.4).astype(np.uint8)
    ffn_mask = (rng.random((5, 4)) > 0.4).astype(np.uint8)
    layer_on = np.array([1, 1, 1, 1, 1], np.uint8)
    print(f"forced split {split} compute={compute}: edge case", flush=True)
    errs = _layer_case(shape, seqlens, layer_on, head_mask, ffn_mask, compute=compute)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(shape), errs
    w = W.get_workload("llava7b_b1_keep25")
    keep, lm, hm, fm = W.draw_masks(w, 0)
    l = w.shape.prefix
    print(f"forced split {split} compute={compute}: headline layer", flush=True)
    errs = _layer_case(w.shape, (keep + w.n_text).astype(np.int32), lm[:, l], hm[:, l], fm[:, l],
                       compute=compute)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


@pytest.mark.parametrize("compute", ["f16", "bf16"])
def test_norm_row_groups(compute, monkeypatch):
    """The 8-row-group residual norm (taken by launches of 1024+ rows), forced
    onto small launches: ragged segments whose lengths are not multiples of 8,
    split-K partial slices to add (the output and down projections split at
    these row counts), a final add-only launch, and row widths in registers of
    2, 16 and 20 float4 per lane (d_model 512, 4096, 5120)."""
    monkeypatch.setenv("SVL_NORM8_MIN_ROWS", "0")
    rng = np.random.default_rng(3)
    for D, A, seqlens in ((512, 8, [70, 0, 1, 129, 200]), (5120, 8, [37, 250])):
        shape = W.ModelShape(n_layers=1, d_model=D, n_heads=A, n_kv_heads=A // 2, head_dim=64,
                             d_ffn=1024, n_groups=4, dtype="bf16")
        B = len(seqlens)
        head_mask = (rng.random((B, A)) > 0.3).astype(np.uint8)
        ffn_mask = (rng.random((B, 4)) > 0.3).astype(np.uint8)
        print(f"row-group norm: d_model {D}, rows {seqlens}, compute={compute}", flush=True)
        errs = _layer_case(shape, np.array(seqlens, np.int32), np.ones(B, np.uint8), head_mask,
                           ffn_mask, compute=compute)
        print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
        assert max(errs) <= tol_for(shape), errs
    w = W.get_workload("llava7b_b1_keep25")
    keep, lm, hm, fm = W.draw_masks(w, 0)
    l = w.shape.prefix
    print(f"row-group norm: headline layer, compute={compute}", flush=True)
    errs = _layer_case(w.shape, (keep + w.n_text).astype(np.int32), lm[:, l], hm[:, l], fm[:, l],
                       compute=compute)
    print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_threshold_budget_prefill():
    """Threshold selection and the budget projection feeding the prefill
    (Sec. 3.1, Sec. 3.3): GPU threshold counts, the library's projection and
    the prefill on the projected keep counts and masks, against the oracle's
    projection and prefill; kept indices exact, hidden states within the
    tolerance."""
    import dataclasses
    from oracle import budget as obudget
    cases = (("tiny_f32", None, (0.5, 0.08)),
             ("llava7b_b8_ragged", dict(n_layers=4, d_model=512, n_heads=8, n_kv_heads=8,
                                        d_ffn=1024, name="thr"), (0.4, 0.1)))
    bound = reduced = 0
    for name, scale, budgets in cases:
        w = W.get_workload(name)
        if scale:
            w = W.scaled(w, **scale)
        inp = W.draw_inputs(w, 5, device="cuda")
        layers = [W.draw_layer_weights(w, l, 5, device="cuda") for l in range(w.shape.n_layers)]
        B, N = inp.scores.shape
        rng = np.random.default_rng(5)
        logits = (rng.standard_normal((B, N)) - 0.3).astype(np.float32)
        logits[0, :3] = 0.0
        logits[-1, 5] = np.nan
        ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
        counts = svl.svl_count_positive(torch.from_numpy(logits).cuda(), ws)
        np.testing.assert_array_equal(counts, [obudget.threshold_count(logits[b]) for b in range(B)])
        cfg = svl.make_config(w.shape)
        P = w.shape.n_layers // 2
        for budget in budgets:
            keep, lm, hm, fm = svl.svl_budget_project(cfg, counts, N, w.n_text, budget, 0, P,
                                                      inp.layer_mask, inp.head_mask, inp.ffn_mask)
            wk, wlm, whm, wfm = obudget.project_batch(w.shape, logits, w.n_text, budget, 0, P,
                                                      inp.layer_mask, inp.head_mask, inp.ffn_mask)
            np.testing.assert_array_equal(keep, wk)
            np.testing.assert_array_equal(hm, whm)
            bound += int(np.any(keep < counts))
            reduced += int(not np.array_equal(hm, inp.head_mask))
            inp2 = dataclasses.replace(inp, scores=logits, keep=keep, layer_mask=lm, head_mask=hm,
                                       ffn_mask=fm)
            print(f"{name} budget {budget}: counts {counts.tolist()} keep {keep.tolist()}", flush=True)
            kept, cu, got, _ = gpu_prefill(w, inp2, layers)
            ref = oracle_prefill(w, inp2, layers)
            np.testing.assert_array_equal(kept, ref.kept_idx)
            np.testing.assert_array_equal(cu, ref.cu_seqlens)
            errs = rel_err_per_sample(got, ref.resid, cu)
            print(f"  rel err per sample: {[f'{e:.2e}' for e in errs]}", flush=True)
            assert max(errs) <= tol_for(w.shape), errs
    assert bound > 0 and reduced > 0


def test_prefill_deterministic_and_flops():
    w = W.get_workload("llava7b_b8_ragged")
    w = W.scaled(w, n_layers=3, d_model=512, n_heads=4, n_kv_heads=4, d_ffn=1024, name="det")
    inp = W.draw_inputs(w, 4, device="cuda")
    layers = [W.draw_layer_weights(w, l, 4, device="cuda") for l in range(w.shape.n_layers)]
    a = gpu_prefill(w, inp, layers)
    b = gpu_prefill(w, inp, layers)
    np.testing.assert_array_equal(a[2], b[2])
    cfg = svl.make_config(w.shape)
    f = svl.svl_count_flops(cfg, inp.keep + w.n_text, inp.layer_mask, inp.head_mask, inp.ffn_mask)
    assert f == a[3]


def test_prefill_edge_batches():
    """keep = 0, keep = N, no text tokens, every layer skipped for a sample,
    all heads and FFN slices off in a layer (alpha = 0)."""
    base = W.Workload(name="edges", shape=W.ModelShape(n_layers=3, d_model=256, n_heads=4,
                                                        n_kv_heads=2, head_dim=64, d_ffn=512,
                                                        n_groups=2, dtype="bf16"),
                      batch=4, n_vision=40, n_text=0, keep_ratio=0.5)
    for T in (0, 5):
        w = W.Workload(**{**base.__dict__, "n_text": T})
        inp = W.draw_inputs(w, 1, device="cuda")
        inp.keep[:] = [0, 40, 13, 1]
        inp.layer_mask[2, :] = 0
        inp.head_mask[1, 1, :] = 0
        inp.ffn_mask[1, 1, :] = 0
        layers = [W.draw_layer_weights(w, l, 1, device="cuda") for l in range(3)]
        print(f"edge batch T={T} keep={inp.keep.tolist()}", flush=True)
        kept, cu, resid, flops = gpu_prefill(w, inp, layers)
        ref = oracle_prefill(w, inp, layers)
        np.testing.assert_array_equal(kept, ref.kept_idx)
        np.testing.assert_array_equal(cu, ref.cu_seqlens)
        errs = rel_err_per_sample(resid, ref.resid, cu)
        assert max(errs) <= tol_for(w.shape), errs
        # the sample that skips every layer is its packed input, exactly
        rows = slice(cu[2], cu[3])
        np.testing.assert_array_equal(resid[rows], ref.resid[rows].astype(np.float32))
        assert flops["total"] == ref.flops.total


def test_gated_weights_are_never_read():
    """NaN in every weight row / column of inactive heads and FFN slices, and
    in every weight of a layer no sample runs, leaves the output bit-identical."""
    w = W.scaled(W.get_workload("llava7b_b1_keep25"), n_layers=4, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, layers_skipped=1, name="poison")
    inp = W.draw_inputs(w, 2, device="cuda")
    layers = [W.draw_layer_weights(w, l, 2, device="cuda") for l in range(4)]
    clean = gpu_prefill(w, inp, layers)[2]
    d, F, G = w.shape.head_dim, w.shape.d_ffn, w.shape.n_groups
    poisoned = []
    for l, lw in enumerate(layers):
        lw = {k: v.clone() for k, v in lw.items()}
        if not inp.layer_mask[0, l]:
            for v in lw.values():
                v.fill_(float("nan"))
        else:
            for h in range(w.shape.n_heads):
                if not inp.head_mask[0, l, h]:
                    for n in ("wq", "wk", "wv"):
                        lw[n][h * d:(h + 1) * d] = float("nan")
                    lw["wo"][:, h * d:(h + 1) * d] = float("nan")
            for j in range(G):
                if not inp.ffn_mask[0, l, j]:
                    sl = slice(j * F // G, (j + 1) * F // G)
                    lw["w_gate"][sl] = float("nan")
                    lw["w_up"][sl] = float("nan")
                    lw["w_down"][:, sl] = float("nan")
        poisoned.append(lw)
    got = gpu_prefill(w, inp, poisoned)[2]
    np.testing.assert_array_equal(got, clean)
