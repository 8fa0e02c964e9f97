"""GPU check of the prefill status word (svl_workspace_status).

The prefill clears the word at its end and sets it to SVL_STATUS_NONFINITE
when an output value is inf or NaN (with fp16 activations, a value past
fp16's range becomes inf and reaches the output rows).  The cases here keep
non-finite values away from the matrix-product and attention kernels: the
non-finite value is an input row that no layer processes (every layer
skipped, so only the gather and the status scan read it), or a dropped vision
token, which no kernel reads at all."""
import numpy as np
import pytest
import torch

import paper_2607_20357_amd as svl
import workloads as W
from gpu_helpers import oracle_prefill, rel_err_per_sample

pytestmark = pytest.mark.gpu


def _case(batch):
    w = W.scaled(W.get_workload("llava7b_b8_ragged"), n_layers=2, d_model=512, n_heads=4,
                 n_kv_heads=4, d_ffn=1024, batch=batch, name=f"status_b{batch}")
    inp = W.draw_inputs(w, 3, device="cuda")
    layers = [W.draw_layer_weights(w, l, 3, device="cuda") for l in range(2)]
    return w, inp, layers


def _run(w, inp, layers, ws=None):
    print(f"status case {w.name}", flush=True)
    cfg = svl.make_config(w.shape)
    B, N = inp.scores.shape
    R = int((np.asarray(inp.keep) + w.n_text).sum())
    scores = torch.from_numpy(np.ascontiguousarray(inp.scores)).cuda()
    kept = torch.empty((B, N), dtype=torch.int32, device="cuda")
    resid = torch.empty((R, w.shape.d_model), dtype=torch.float32, device="cuda")
    if ws is None:
        ws = svl.alloc_workspace(cfg, B, R, "cuda")
    cu, _ = svl.svl_prefill(cfg, layers, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                            inp.head_mask, inp.ffn_mask, kept, resid, ws)
    return svl.svl_workspace_status(ws), resid.cpu().numpy(), ws, kept.cpu().numpy()


def test_status_clear_for_ordinary_inputs():
    w, inp, layers = _case(batch=3)
    status, got, _, _ = _run(w, inp, layers)
    assert status == 0
    ref = oracle_prefill(w, inp, layers)
    assert max(rel_err_per_sample(got, ref.resid, ref.cu_seqlens)) <= 2e-2


def test_status_set_by_an_inf_output_row_and_cleared_by_the_next_call():
    w, inp, layers = _case(batch=2)
    # sample 1 skips every layer, so its rows are its inputs; its last text
    # row holds +inf (bf16): the output holds it and the word is set
    inp.layer_mask[1, :] = 0
    text = inp.text.clone()
    text[1, -1, 5] = float("inf")
    bad = W.Inputs(inp.workload, inp.seed, inp.scores, inp.keep, inp.layer_mask, inp.head_mask,
                   inp.ffn_mask, inp.vision, text)
    status, got, ws, _ = _run(w, bad, layers)
    print(f"  inf row: status {status}", flush=True)
    assert status == svl.SVL_STATUS_NONFINITE
    assert np.isinf(got).sum() == 1
    # the same workspace, finite inputs: cleared
    status2, got2, _, _ = _run(w, inp, layers, ws=ws)
    assert status2 == 0 and np.isfinite(got2).all()


def test_status_clear_when_a_dropped_token_is_nan():
    w, inp, layers = _case(batch=2)
    keep = np.asarray(inp.keep)
    assert keep[0] < w.n_vision, "the draw should drop tokens of sample 0"
    # the lowest-scoring token of sample 0 is dropped: it is never read
    lowest = int(np.argmin(inp.scores[0]))
    vision = inp.vision.clone()
    vision[0, lowest, :] = float("nan")
    bad = W.Inputs(inp.workload, inp.seed, inp.scores, inp.keep, inp.layer_mask, inp.head_mask,
                   inp.ffn_mask, vision, inp.text)
    status, got, _, kept = _run(w, bad, layers)
    assert lowest not in kept[0][:keep[0]]
    assert status == 0 and np.isfinite(got).all()
