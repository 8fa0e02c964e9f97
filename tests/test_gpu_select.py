"""GPU parity of token selection and packing (svl_select_tokens): bit-exact
against the oracle's ranking (score descending, NaN lowest, -0 == +0, ties
to the lower index; kept indices ascending) and exact packed rows."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_20357_amd as svl
import workloads as W

pytestmark = pytest.mark.gpu


def _scores(kind, B, N, rng):
    if kind == "lognormal":
        return np.exp(rng.standard_normal((B, N))).astype(np.float32)
    if kind == "uniform":
        return rng.random((B, N)).astype(np.float32)
    if kind == "ties":
        return (rng.integers(0, 5, (B, N)) * 0.25).astype(np.float32)
    if kind == "constant":
        return np.full((B, N), 0.5, np.float32)
    if kind == "special":
        pool = np.array([np.nan, -np.inf, np.inf, -0.0, 0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-45],
                        np.float32)
        return pool[rng.integers(0, len(pool), (B, N))]
    if kind == "negative":
        return (-np.exp(rng.standard_normal((B, N)))).astype(np.float32)
    raise ValueError(kind)


def _run(cfg, keep, scores, vision, text):
    dev = "cuda"
    B, N = scores.shape
    T = text.shape[1]
    R = int(np.sum(keep) + B * T)
    s = torch.from_numpy(scores).to(dev)
    kept = torch.full((B, N), -7, dtype=torch.int32, device=dev)
    resid = torch.full((max(R, 1), cfg.d_model), float("nan"), dtype=torch.float32, device=dev)[:R]
    ws = svl.alloc_workspace(cfg, B, R, dev)
    cu = svl.svl_select_tokens(cfg, keep, s, vision, text, kept, resid, ws)
    torch.cuda.synchronize()
    return kept.cpu().numpy(), cu, resid.cpu().numpy()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_select_and_gather_exact(dtype):
    rng = np.random.default_rng(11)
    D = 64
    cfg = svl.make_config(n_layers=1, d_model=D, n_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64,
                          n_groups=1, dtype=dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cases = 0
    for N in [1, 7, 64, 255, 256, 257, 576, 1000, 3136]:
        for kind in ["lognormal", "ties", "special", "constant", "negative", "uniform"]:
            B = 3
            T = int(rng.integers(0, 5))
            scores = _scores(kind, B, N, rng)
            keep = np.array([0, N, int(rng.integers(0, N + 1))], np.int32)
            if N > 2:
                keep[0] = 1
                keep[1] = N - 1
            print(f"select case N={N} kind={kind} keep={keep.tolist()} T={T}", flush=True)
            vision = torch.randn(B, N, D).to(tdt).cuda()
            text = torch.randn(B, max(T, 0), D).to(tdt).cuda()
            kept, cu, resid = _run(cfg, keep, scores, vision, text)
            ref_idx, ref_cu, seqs = oracle.select_and_compact(
                scores, keep, W.as_f32(vision), W.as_f32(text))
            np.testing.assert_array_equal(kept, ref_idx, err_msg=f"N={N} {kind}")
            np.testing.assert_array_equal(cu, ref_cu)
            if resid.shape[0]:
                np.testing.assert_array_equal(resid, np.concatenate(seqs).astype(np.float32))
            cases += 1
    assert cases > 0


def test_select_workload_scores_exact():
    """Selection on every workload's score law at its real shape."""
    for name, w in W.WORKLOADS.items():
        scores = W.draw_scores(w, 0)
        keep, *_ = W.draw_masks(w, 0)
        cfg = svl.make_config(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64,
                              d_ffn=64, n_groups=1, dtype="bf16")
        B, N = scores.shape
        vision = torch.zeros(B, N, 64, dtype=torch.bfloat16, device="cuda")
        text = torch.zeros(B, w.n_text, 64, dtype=torch.bfloat16, device="cuda")
        print(f"workload scores {name}", flush=True)
        kept, cu, _ = _run(cfg, keep, scores, vision, text)
        for b in range(B):
            ref = oracle.select_topk(scores[b], keep[b])
            np.testing.assert_array_equal(kept[b, :keep[b]], ref, err_msg=name)
            assert (kept[b, keep[b]:] == -1).all()


def test_dropped_rows_are_not_read():
    """NaN in every dropped vision row leaves the packed rows unchanged."""
    rng = np.random.default_rng(5)
    B, N, T, D = 2, 300, 3, 128
    cfg = svl.make_config(n_layers=1, d_model=D, n_heads=1, n_kv_heads=1, head_dim=128, d_ffn=64,
                          n_groups=1, dtype="bf16")
    scores = _scores("lognormal", B, N, rng)
    keep = np.array([77, 150], np.int32)
    vision = torch.randn(B, N, D).to(torch.bfloat16)
    for b in range(B):
        drop = np.setdiff1d(np.arange(N), oracle.select_topk(scores[b], keep[b]))
        vision[b, drop] = float("nan")
    text = torch.randn(B, T, D).to(torch.bfloat16)
    kept, cu, resid = _run(cfg, keep, scores, vision.cuda(), text.cuda())
    assert np.isfinite(resid).all()


def test_count_positive_exact():
    """Threshold counts (sigma(z) > 0.5, i.e. z > 0) on the GPU equal the
    oracle's, including zeros, -0, NaN, +-inf and ragged lengths."""
    from oracle import budget as obudget
    rng = np.random.default_rng(21)
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    for N in [1, 7, 255, 256, 257, 576, 3136]:
        for kind in ["special", "lognormal", "negative", "ties"]:
            B = 5
            z = _scores(kind, B, N, rng)
            if kind == "ties":
                z = z - 0.5                 # values in {-0.5, -0.25, 0, 0.25, 0.5}
            got = svl.svl_count_positive(torch.from_numpy(z).cuda(), ws)
            want = np.array([obudget.threshold_count(z[b]) for b in range(B)])
            np.testing.assert_array_equal(got, want)
