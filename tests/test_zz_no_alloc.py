"""GPU check of the allocation-free decode step (svl_decode_step_noalloc).

It runs the same kernels as svl_decode_step on the library's own device
scratch instead of a caller workspace, so on the same inputs its outputs (the
new rows' residuals and the K / V rows it appends to the cache) must equal
svl_decode_step's exactly.  Two calls in a row share the scratch: the second
uses a smaller batch and a shorter cache, and must not see the first call's
leftovers."""
import numpy as np
import pytest
import torch

import paper_2607_20357_amd as svl
import workloads as W

pytestmark = pytest.mark.gpu


def _setup(w, seed, max_len):
    dev = "cuda"
    cfg = svl.make_config(w.shape)
    inp = W.draw_inputs(w, seed, device=dev)
    layers = [W.draw_layer_weights(w, l, seed, device=dev) for l in range(w.shape.n_layers)]
    table = svl.LayerTable(layers)
    B, N = inp.scores.shape
    D = w.shape.d_model
    seq = (np.asarray(inp.keep) + w.n_text).astype(np.int32)
    R = int(seq.sum())
    cache = svl.alloc_kv_cache(cfg, B, max_len, dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    scores = torch.from_numpy(np.ascontiguousarray(inp.scores)).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, D), dtype=torch.float32, device=dev)
    svl.svl_prefill_cache(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                          inp.head_mask, inp.ffn_mask, kept, resid, cache, max_len, ws)
    torch.cuda.synchronize()
    return cfg, inp, table, seq, cache


def _compare_one_step(w, seed, max_len):
    cfg, inp, table, seq, cache = _setup(w, seed, max_len)
    B, D = w.batch, w.shape.d_model
    g = torch.Generator(device="cuda").manual_seed(seed + 1)
    x0 = torch.randn(B, D, generator=g, device="cuda").to(torch.bfloat16).to(torch.float32)
    cache_ref = cache.clone()
    x_ref = x0.clone()
    dws = svl.alloc_decode_workspace(cfg, B, max_len)
    svl.svl_decode_step(cfg, table, x_ref, seq, inp.layer_mask, inp.head_mask, inp.ffn_mask,
                        cache_ref, max_len, dws)
    x_na = x0.clone()
    svl.svl_decode_step_noalloc(cfg, table, x_na, seq, inp.layer_mask, inp.head_mask,
                                inp.ffn_mask, cache, max_len)
    torch.cuda.synchronize()
    got, want = x_na.cpu().numpy(), x_ref.cpu().numpy()
    assert np.isfinite(want).all()
    print(f"{w.name}: batch {B}, max_len {max_len}, max |diff| "
          f"{np.abs(got - want).max():.3e}", flush=True)
    np.testing.assert_array_equal(got, want)
    assert torch.equal(cache, cache_ref), "appended K / V rows differ"


def test_noalloc_decode_matches_decode_step_twice():
    base = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=4,
                    n_kv_heads=4, d_ffn=1024, name="na8")
    _compare_one_step(base, 21, max_len=700)
    # second call: a smaller batch and a shorter cache on the same scratch
    small = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=4, d_model=512, n_heads=4,
                     n_kv_heads=4, d_ffn=1024, batch=3, n_vision=200, name="na3")
    _compare_one_step(small, 22, max_len=300)


def test_noalloc_decode_headline_shape():
    """The headline's full 7B shape, one sample (the serving case)."""
    _compare_one_step(W.get_workload("llava7b_b1_keep25"), 0, max_len=256)


def test_noalloc_decode_rejects_shapes_past_its_scratch():
    w = W.get_workload("llava7b_b1_keep25")
    cfg = svl.make_config(w.shape)
    layers = [W.draw_layer_weights(w, 0, 0, device="cuda")] * w.shape.n_layers
    B, max_len = 64, 64
    need = svl.binding.load_library().svl_decode_workspace_bytes(
        svl.binding.ctypes.byref(cfg), B, max_len)
    assert need > svl.binding.SVL_NOALLOC_SCRATCH_BYTES
    cache = torch.empty(svl.svl_kv_cache_bytes(cfg, B, max_len), dtype=torch.uint8, device="cuda")
    x = torch.zeros(B, w.shape.d_model, device="cuda")
    with pytest.raises(svl.SvlError, match="allocation-free scratch"):
        svl.svl_decode_step_noalloc(cfg, layers, x, np.zeros(B, np.int32),
                                    np.ones((B, w.shape.n_layers), np.uint8),
                                    np.ones((B, w.shape.n_layers, w.shape.n_heads), np.uint8),
                                    None, cache, max_len)
