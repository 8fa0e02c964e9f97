"""GPU parity of decode on the pruned and gated KV cache.

A decode step runs the masked decoder on one new token per sample at the
next position, attending to the cached keys / values; its output must equal
the last row of the oracle's prefill over the sequence extended by that
token (causal attention), so the oracle here is the prefill oracle on the
extended text.  The prefill that fills the cache must also give exactly the
plain prefill's result."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20357_amd as svl
import workloads as W
from gpu_helpers import gpu_prefill, host_layer, tol_for

pytestmark = pytest.mark.gpu


def _row_err(g, o):
    g = np.asarray(g, np.float64)
    den = np.abs(o).max()
    return float(np.abs(g - o).max() / den) if den > 0 else float(np.abs(g).max())


def _decode_case(w, seed, steps, extra=3, compute="f16"):
    dev = "cuda"
    shape = w.shape
    cfg = svl.make_config(shape, compute=compute)
    inp = W.draw_inputs(w, seed, device=dev)
    layers = [W.draw_layer_weights(w, l, seed, device=dev) for l in range(shape.n_layers)]
    table = svl.LayerTable(layers)
    B, N = inp.scores.shape
    T, D = w.n_text, shape.d_model
    seq = (np.asarray(inp.keep) + T).astype(np.int32)
    R = int(seq.sum())
    max_len = int(seq.max()) + steps + extra
    cache = svl.alloc_kv_cache(cfg, B, max_len, dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    scores = torch.from_numpy(np.ascontiguousarray(inp.scores)).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, D), dtype=torch.float32, device=dev)
    cu = svl.svl_prefill_cache(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                               inp.head_mask, inp.ffn_mask, kept, resid, cache, max_len, ws)
    torch.cuda.synchronize()
    # finite inputs and weights: the call's status word is clear
    assert svl.svl_workspace_status(ws) == 0
    # the cache writes leave the prefill itself unchanged
    _, cu2, plain, _ = gpu_prefill(w, inp, layers, table=table, compute=compute)
    np.testing.assert_array_equal(cu, cu2)
    np.testing.assert_array_equal(resid.cpu().numpy(), plain)

    g = torch.Generator(device=dev).manual_seed(seed + 100)
    new = torch.randn(steps, B, D, generator=g, device=dev).to(torch.bfloat16).to(torch.float32)
    dws = svl.alloc_decode_workspace(cfg, B, max_len, dev)
    cache_len = seq.copy()
    outs = []
    for t in range(steps):
        x = new[t].clone()
        svl.svl_decode_step(cfg, table, x, cache_len, inp.layer_mask, inp.head_mask,
                            inp.ffn_mask, cache, max_len, dws)
        torch.cuda.synchronize()
        outs.append(x.cpu().numpy())
        cache_len += 1

    # oracle: the prefill over the text extended by the new tokens
    text_ext = np.concatenate([W.as_f32(inp.text), new.permute(1, 0, 2).cpu().numpy()], axis=1)
    ref = oracle.prefill(shape, lambda l: host_layer(layers[l]), inp.scores, np.asarray(inp.keep),
                         W.as_f32(inp.vision), text_ext, inp.layer_mask, inp.head_mask,
                         inp.ffn_mask)
    errs = []
    for t in range(steps):
        for b in range(B):
            row = ref.cu_seqlens[b] + seq[b] + t
            errs.append(_row_err(outs[t][b], ref.resid[row]))
    return errs


def test_decode_ragged_batch():
    """8 samples with their own keep counts, head groups and skipped layers,
    three decode steps each."""
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, name="dec8")
    errs = _decode_case(w, 7, steps=3)
    print(f"max rel err over rows: {max(errs):.2e}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_decode_ragged_batch_bf16():
    """The ragged batch with bf16 activations: a bf16 cache and bf16 products
    (the cache-filling prefill carries the normed rows' low bf16 terms into
    its QKV and gate/up products, the decode steps the high terms only)."""
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, name="dec8_bf16")
    errs = _decode_case(w, 7, steps=3, compute="bf16")
    print(f"max rel err over rows: {max(errs):.2e}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_decode_gqa():
    """Grouped K/V heads (2 query heads per K/V head) with whole K/V groups off."""
    w = W.scaled(W.get_workload("gqa7b_hires_b2"), n_layers=3, d_model=512, n_heads=4,
                 n_kv_heads=2, d_ffn=1024, n_vision=160, n_text=24, name="decgqa")
    errs = _decode_case(w, 8, steps=2)
    print(f"max rel err over rows: {max(errs):.2e}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_decode_batch_past_eight_uses():
    """A batch of 11 samples: the shared row-vector launches split each
    weight block's samples into groups of at most 8 (8 + 3), with heads of
    64 columns (one K chunk per head), grouped K/V heads and per-sample head
    groups, FFN slices and skipped layers."""
    import dataclasses
    base = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=3, d_model=512,
                    d_ffn=1024, batch=11, n_vision=96, n_text=16, name="dec11")
    w = dataclasses.replace(base, shape=dataclasses.replace(base.shape, n_heads=8, n_kv_heads=4,
                                                            head_dim=64))
    errs = _decode_case(w, 9, steps=2)
    print(f"max rel err over rows: {max(errs):.2e}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_decode_headline_full_size():
    """The headline shape (32 layers, d 4096, one sample, 144 + 64 tokens),
    two decode steps."""
    w = W.get_workload("llava7b_b1_keep25")
    errs = _decode_case(w, 0, steps=2)
    print(f"rel err per row: {[f'{e:.2e}' for e in errs]}", flush=True)
    assert max(errs) <= tol_for(w.shape), errs


def test_decode_rejects_bad_arguments():
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=2, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, batch=2, name="decbad")
    cfg = svl.make_config(w.shape)
    layers = [W.draw_layer_weights(w, l, 0, device="cuda") for l in range(2)]
    max_len = 32
    cache = svl.alloc_kv_cache(cfg, 2, max_len)
    dws = svl.alloc_decode_workspace(cfg, 2, max_len)
    x = torch.zeros(2, 512, device="cuda")
    lm = np.ones((2, 2), np.uint8)
    hm = np.ones((2, 2, 4), np.uint8)
    for cl in ([max_len, 0], [-1, 0]):
        with pytest.raises(svl.SvlError):
            svl.svl_decode_step(cfg, layers, x, np.array(cl, np.int32), lm, hm, None, cache,
                                max_len, dws)
    with pytest.raises(svl.SvlError):
        svl.svl_decode_step(cfg, layers, x, np.zeros(2, np.int32), lm, hm, None, cache,
                            max_len, dws[:100])
