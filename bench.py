"""Benchmark of the budget-adapted prefill on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one svl_prefill call over one batch of seeded synthetic inputs
already resident in HBM: top-k selection and packing of the vision tokens,
then every decoder layer under the layer / head / FFN masks.  The default
workload is the LLaVA-1.5-7B-shaped batch-1 prefill with keep ratio 0.25
(576 vision + 64 text tokens, 144 kept; 8 of 32 heads and the matching FFN
slice off per layer; 8 of 32 layers skipped; bf16 weights and activations,
float32 accumulation and residual).

Prints one JSON line.  `value` is effective prefill tokens/s = B*(N+T) per
step time (tokens the prefill stands for, before pruning).  The `roofline`
object covers the dominant kernel (the gate/up GEMM), timed with HIP events
recorded by the library on the launch stream in a second pass of the same
steps; `cpu_baseline` times the CPU oracle on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 vector, published


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default=None)
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--compute", choices=("f16", "bf16"), default="f16",
                   help="activation / matrix-input type of the 16-bit path (fp16 or bf16 MFMA)")
    p.add_argument("--no-bf16-line", action="store_true",
                   help="skip the extra prefill timings of the default run: the headline "
                        "with bf16 activations and the compute-bound ragged batch of 8 (the "
                        "counter runs skip them, so only the headline's GEMMs are counted)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-train-line", action="store_true",
                   help="skip the training-step timing (svl_train_step) of the default run")
    p.add_argument("--train", action="store_true",
                   help="time only the training step of the masked decoder at the workload's "
                        "shape (one JSON line)")
    p.add_argument("--cpu-layers", type=int, default=0,
                   help="executed layers the CPU-baseline sample runs (0: all of them, no "
                        "extrapolation; the headline's 24 take about 20 s on 16 host threads)")
    p.add_argument("--traffic-from", default=None,
                   help="directory holding fetch/ and write/ rocprofv3 --pmc FETCH_SIZE / "
                        "WRITE_SIZE runs of `bench.py --copy-calibration`: write the gate/up "
                        "traffic summary and exit")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run one plain device copy of COPY_BYTES (the known-size kernel "
                        "that scales the FETCH_SIZE / WRITE_SIZE counters of a --pmc run)")
    p.add_argument("--threshold-budget", type=float, default=None, metavar="B",
                   help="instead of the integer keep budget: threshold selection (logits > 0) "
                        "and the budget projection to B * C_full inside each step, on the "
                        "headline shapes and masks with logits N(0,1) - 0.674 (a quarter of "
                        "the tokens positive)")
    p.add_argument("--controller", type=float, default=None, metavar="B",
                   help="instead of the given keep budget and masks: the controlled prefill "
                        "(threshold selection on logits N(0,1) - 0.674, the budget token, "
                        "P = L/2 prefix layers, the compute controller's masks, the budget "
                        "projection to B * C_full at the prefix boundary) with seeded "
                        "controller weights (encoding width 256, hidden width d_model)")
    p.add_argument("--decode", type=int, default=None, metavar="N",
                   help="instead of the prefill step: N timed decode steps on the pruned and "
                        "gated KV cache the workload's prefill leaves (one new token per sample "
                        "per step)")
    p.add_argument("--library-gemms", action="store_true",
                   help="instead of the step benchmark: torch's matmul (the vendor BLAS) "
                        "at the headline's four GEMM shapes, in fp16 and bf16, "
                        "next to this library's per-launch times of the same GEMMs; one JSON "
                        "line")
    p.add_argument("--memory-sweep", action="store_true",
                   help="instead of the step benchmark: HBM rate of the memory-bound kernels "
                        "(select, gather, residual norm) on the headline per-row structure "
                        "with the batch raised to 64 and 256, next to a device copy; one JSON "
                        "line per batch")
    return p.parse_args()


COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gate_up_traffic.json")
# the gate/up kernel's source and the headers it includes
GEMM_SOURCE = [os.path.join(ROOT, "paper_2607_20357_amd", "csrc", n)
               for n in ("gemm_mfma.hip", "device_util.h", "svl_internal.h", "plan_types.h")]
GEMM_SOURCE.append(os.path.join(ROOT, "include", "svl.h"))


def source_hash(paths, read=None):
    """sha256 of the files' code with C / C++ comments and whitespace removed,
    so that edits to their documentation leave it unchanged (the files hold
    no string literal with a comment marker in it)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for path in paths:
        if read is None:
            with open(path) as f:
                text = f.read()
        else:
            text = read(path)
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def write_traffic(run_dir):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the gate/up GEMM, each
    scaled by counter / true bytes of the COPY_BYTES calibration copy (the
    dispatch whose WRITE_SIZE is largest), into TRAFFIC_FILE."""
    import collections
    import csv

    def per_dispatch(path, counter):
        vals, names = collections.defaultdict(float), {}
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                d = int(r["Dispatch_Id"])
                vals[d] += float(r["Counter_Value"])
                names[d] = r["Kernel_Name"]
        return vals, names

    out = {"gemm_source_sha256": source_hash(GEMM_SOURCE), "copy_bytes": COPY_BYTES}
    for kind, sub in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        path = os.path.join(run_dir, kind, "p_counter_collection.csv")
        vals, names = per_dispatch(path, sub)
        copies = [d for d, n in names.items() if "elementwise" in n or "copy" in n.lower()]
        if kind == "write":
            cal = max(copies, key=lambda d: vals[d])
            cal_kib_write = vals[cal]
        else:
            # the copy dispatch is the one right before the first prefill kernel
            first = min(d for d, n in names.items() if "svl::" in n)
            cal = max(d for d in copies if d < first)
        factor = COPY_BYTES / (vals[cal] * 1024.0)
        gu = [vals[d] for d, n in names.items() if "gemm_mfma_kernel<2," in n]
        out[f"{kind}_kib_per_dispatch_raw"] = sum(gu) / len(gu)
        out[f"{kind}_calibration_factor"] = factor
        out[f"{kind}_bytes_per_launch"] = sum(gu) / len(gu) * 1024.0 * factor
        out[f"{kind}_dispatches"] = len(gu)
        out[f"{kind}_counter"] = sub
    out["command"] = ("rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE TCP_TCC_READ_REQ_sum) "
                      "-d <dir> -o p --output-format csv -- python3 -u bench.py --workload "
                      "llava7b_b1_keep25 --steps 2 --warmup 1 --no-cpu-baseline --no-bf16-line "
                      "--no-train-line --copy-calibration")
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def measured_traffic():
    """HBM bytes per gate/up launch from the committed counter runs, or None
    when there are none or the GEMM source changed since they were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_source_sha256") != source_hash(GEMM_SOURCE):
        return None
    return t


def gemm_bytes(shape, seqlens, layer_mask, head_mask, ffn_mask):
    """Algorithmic HBM bytes of each GEMM class over one step: the weights of
    the union of the samples' active heads / K-V heads / FFN slices (each
    weight block read once; the headline has one sample), the activation
    operand and the output, bf16 (2 B) activations / weights and float32
    residual read-modify-write for the output / down projections."""
    D, A, KV, d, F, G = (shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                         shape.d_ffn, shape.n_groups)
    rep = A // KV
    out = {"qkv": 0, "o": 0, "gu": 0, "down": 0}
    launches = {"qkv": 0, "o": 0, "gu": 0, "down": 0}
    B, L = layer_mask.shape
    for l in range(L):
        rows_a = rows_f = 0
        act_qkv = act_o = act_gu = act_down = 0
        heads = np.zeros(A, bool)
        kvs = np.zeros(KV, bool)
        chans = np.zeros(G, bool)
        for b in range(B):
            if not layer_mask[b, l] or seqlens[b] == 0:
                continue
            hm = head_mask[b, l].astype(bool)
            H = int(hm.sum())
            kv = np.array([hm[g * rep:(g + 1) * rep].any() for g in range(KV)])
            fm = np.ones(G, bool) if ffn_mask is None else ffn_mask[b, l].astype(bool)
            C = int(fm.sum()) * (F // G)
            S = int(seqlens[b])
            if H:
                rows_a += S
                heads |= hm
                kvs |= kv
                act_qkv += S * D * 2 + S * (H + 2 * int(kv.sum())) * d * 2
                act_o += S * H * d * 2 + S * D * 8
            if C:
                rows_f += S
                chans |= fm
                act_gu += S * D * 2 + S * C * 2
                act_down += S * C * 2 + S * D * 8
        if rows_a:
            out["qkv"] += (int(heads.sum()) + 2 * int(kvs.sum())) * d * D * 2 + act_qkv
            out["o"] += D * int(heads.sum()) * d * 2 + act_o
            launches["qkv"] += 1
            launches["o"] += 1
        if rows_f:
            cu = int(chans.sum()) * (F // G)
            out["gu"] += 2 * cu * D * 2 + act_gu
            out["down"] += D * cu * 2 + act_down
            launches["gu"] += 1
            launches["down"] += 1
    return out, launches


def cpu_baseline(w, inp, layers, n_exec_layers):
    """The CPU oracle on the first `n_exec_layers` executed layers (0: all) of the same
    inputs (selection and packing included); the rate is scaled to the whole
    prefill by the executed-layer count."""
    import oracle
    import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        nproc = os.cpu_count()
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    B = w.batch
    executed = [l for l in range(w.shape.n_layers) if inp.layer_mask[:, l].any()]
    sample = executed[:n_exec_layers] if n_exec_layers > 0 else executed
    host = {}
    for l in sample:
        host[l] = {k: W.as_f32(v) for k, v in layers[l].items()}
    vis, txt = W.as_f32(inp.vision), W.as_f32(inp.text)
    t0 = time.perf_counter()
    oracle.prefill(w.shape, lambda l: host[l], inp.scores, inp.keep, vis, txt, inp.layer_mask,
                   inp.head_mask, inp.ffn_mask, layers=sample)
    dt = time.perf_counter() - t0
    est = dt * len(executed) / max(1, len(sample))
    tokens = B * (w.n_vision + w.n_text)
    return {"value": tokens / est, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "nproc": int(nproc), "os_cpu_count": os.cpu_count(), "blas_threads": int(threads),
            "cpu_model": model,
            "layers_timed": len(sample), "layers_executed": len(executed),
            "seconds_timed": round(dt, 2),
            "sample": f"{len(sample)} of {len(executed)} executed layers (float64 numpy oracle, "
                      f"selection and packing included), {dt:.1f} s on {threads} BLAS threads "
                      f"({nproc} usable cores, {model}), rate scaled by "
                      f"{len(executed)}/{len(sample)}"}


def eq8_flops(shape, seqlens, layer_mask, head_mask, n_vision, n_text):
    """The paper's estimator, Eq. (8), with V = 0 (no LM head): per sample,
    sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2], alpha_l = active query heads
    / A (0 for a skipped layer), S the sample's executed sequence length; and
    the same at full capacity (every alpha_l = 1, S = N + T).  Reported next
    to the executed (causal) count for comparison with the paper's figures."""
    D, F, A, L = shape.d_model, shape.d_ffn, shape.n_heads, shape.n_layers
    per_s = lambda S: (8 * D * D + 6 * D * F) * S + 4 * D * S * S
    pruned = 0.0
    for b, S in enumerate(seqlens):
        for l in range(L):
            if layer_mask[b][l]:
                pruned += float(np.sum(head_mask[b][l])) / A * per_s(int(S))
    full = len(seqlens) * L * per_s(n_vision + n_text)
    return int(round(pruned)), int(full)


def memory_sweep(args):
    """Select, gather and residual-norm launches of the headline per-row
    structure (576 vision + 64 text tokens, keep 144, d_model 4096) with the
    batch raised until the gather and norm working sets pass 1 GB (4x the
    last-level cache).  Rates are algorithmic bytes / launch time (HIP events
    the library records on the launch stream), next to a 1 GiB device-to-device
    copy on the same GPU.  At these row counts the output and down projections
    need no split-K, so each norm launch moves exactly rows*D*(4 in + 2 out)
    bytes plus the gain."""
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W

    dev = torch.device("cuda:0")
    reps = max(5, args.steps // 5)
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * COPY_BYTES / (e0.elapsed_time(e1) / reps * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    head = W.get_workload(W.HEADLINE)
    for B in (64, 256):
        w = W.scaled(head, batch=B, name=f"{head.name}_b{B}")
        shape = w.shape
        inp = W.draw_inputs(w, args.seed, device=dev)
        cfg = svl.make_config(shape)
        k = int(inp.keep[0])
        R = int((inp.keep + w.n_text).sum())
        scores = torch.from_numpy(inp.scores).to(dev)
        kept = torch.empty((B, w.n_vision), dtype=torch.int32, device=dev)
        resid = torch.empty((R, shape.d_model), dtype=torch.float32, device=dev)
        ws = svl.alloc_workspace(cfg, B, R, dev)
        weights = W.draw_layer_weights(w, 0, args.seed, device=dev)
        stream = torch.cuda.current_stream()
        cu = svl.svl_select_tokens(cfg, inp.keep, scores, inp.vision, inp.text, kept, resid, ws,
                                   stream=stream)
        lon = np.ones(B, np.uint8)
        fm = None if inp.ffn_mask is None else inp.ffn_mask[:, 0]
        svl.svl_layer_forward(cfg, 0, weights, cu, lon, inp.head_mask[:, 0], fm, resid, ws,
                              stream=stream)
        torch.cuda.synchronize()
        svl.svl_timing_enable(True)
        for _ in range(reps):
            svl.svl_select_tokens(cfg, inp.keep, scores, inp.vision, inp.text, kept, resid, ws,
                                  stream=stream)
            svl.svl_layer_forward(cfg, 0, weights, cu, lon, inp.head_mask[:, 0], fm, resid, ws,
                                  stream=stream)
        torch.cuda.synchronize()
        svl.svl_timing_enable(False)
        t = {c: svl.svl_timing_read(c) for c in ("select", "gather", "rmsnorm")}
        D, N, T = shape.d_model, w.n_vision, w.n_text
        algo = {"select": B * N * 4 + B * k * 4,
                "gather": B * (k + T) * D * (2 + 4),
                "rmsnorm": R * D * (4 + 2) + D * 2}
        line = {"memory_sweep": True, "batch": B, "rows": R, "d_model": D,
                "copy_gbs": round(copy_gbs, 1), "hbm_peak_gbs": HBM_PEAK_GBS}
        for c, (ms, n) in t.items():
            avg_ms = ms / max(1, n)
            gbs = algo[c] / (avg_ms * 1e-3) / 1e9
            line[c] = {"bytes_per_launch": algo[c], "avg_launch_ms": round(avg_ms, 5),
                       "launches": n, "gbs": round(gbs, 1),
                       "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
                       "frac_of_copy": round(gbs / copy_gbs, 4)}
        print(json.dumps(line), flush=True)
        del inp, scores, kept, resid, ws, weights
        torch.cuda.empty_cache()


def library_gemms(args):
    """The headline's GEMM shapes (kept rows x active output columns x active
    reduction width) through torch's matmul, which dispatches to the vendor
    BLAS, fp16 and bf16, weights rotated over 8 copies so none is
    cache-resident, 40 calls replayed from one captured graph; next to this
    library's per-launch GEMM times over the same headline prefill (HIP
    events the library records).  The library's
    launches also apply RoPE / SwiGLU / the split-K partial store."""
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W

    dev = torch.device("cuda:0")
    w = W.get_workload(W.HEADLINE)
    shape = w.shape
    inp = W.draw_inputs(w, args.seed, device=dev)
    l = next(l for l in range(shape.n_layers) if inp.layer_mask[0, l])
    H = int(inp.head_mask[0, l].sum())
    C = shape.d_ffn if inp.ffn_mask is None else int(inp.ffn_mask[0, l].sum()) * (shape.d_ffn // shape.n_groups)
    M = int(inp.keep[0]) + w.n_text
    D, d = shape.d_model, shape.head_dim
    shapes = {"gemm_qkv": (M, 3 * H * d, D), "gemm_o": (M, D, H * d),
              "gemm_gate_up": (M, 2 * C, D), "gemm_down": (M, D, C)}
    layers = [W.draw_layer_weights(w, k, args.seed, device=dev) for k in range(shape.n_layers)]
    table = svl.LayerTable(layers)
    cfg = svl.make_config(shape)
    B, N = inp.scores.shape
    R = int((np.asarray(inp.keep) + w.n_text).sum())
    scores = torch.from_numpy(inp.scores).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, D), dtype=torch.float32, device=dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    stream = torch.cuda.current_stream()

    def step():
        svl.svl_prefill(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                        inp.head_mask, inp.ffn_mask, kept, resid, ws, stream=stream,
                        want_flops=False)
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    svl.svl_timing_enable(True)
    for _ in range(10):
        step()
    torch.cuda.synchronize()
    svl.svl_timing_enable(False)
    del layers, table, ws
    torch.cuda.empty_cache()
    out = {"library_gemms": True, "workload": w.name, "rows": M}
    for k, (m, n, kk) in shapes.items():
        ms, cnt = svl.svl_timing_read(k)
        ours = 1e3 * ms / max(1, cnt)
        line = {"m": m, "n": n, "k": kk, "svl_us": round(ours, 1)}
        for dt, tag in ((torch.float16, "blas_f16_us"), (torch.bfloat16, "blas_bf16_us")):
            x = torch.randn(m, kk, device=dev, dtype=dt)
            wts = [torch.randn(n, kk, device=dev, dtype=dt) * 0.02 for _ in range(8)]
            ys = [torch.nn.functional.linear(x, wts[i]) for i in range(8)]
            torch.cuda.synchronize()
            # 40 calls captured in one graph: a short call's host launch time
            # would otherwise leave the GPU idle between kernels and be timed
            graph = torch.cuda.CUDAGraph()
            reps = 40
            with torch.cuda.graph(graph):
                for i in range(reps):
                    torch.mm(x, wts[i % 8].t(), out=ys[i % 8])
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            graph.replay()
            torch.cuda.synchronize()
            e0.record()
            for _ in range(2):
                graph.replay()
            e1.record()
            torch.cuda.synchronize()
            line[tag] = round(e0.elapsed_time(e1) / (2 * reps) * 1e3, 1)
            del x, wts, ys, graph
            torch.cuda.empty_cache()
        out[k] = line
    print(json.dumps(out), flush=True)


def decode_bench(args):
    """Decode on the pruned and gated KV cache: the workload's prefill fills
    the cache (untimed), then each step feeds one new token per sample (seeded
    hidden states, bf16-rounded) through every layer under the sample's masks.
    The step's HBM bytes are the active weights it streams (the GEMM classes
    at one row per sample) plus the cached K / V it reads."""
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W

    dev = torch.device("cuda:0")
    w = W.get_workload(args.workload or W.HEADLINE)
    shape = w.shape
    print(f"# decode after workload {w.name}: {w.description}", file=sys.stderr, flush=True)
    inp = W.draw_inputs(w, args.seed, device=dev)
    layers = [W.draw_layer_weights(w, l, args.seed, device=dev) for l in range(shape.n_layers)]
    table = svl.LayerTable(layers)
    cfg = svl.make_config(shape)
    B, N = inp.scores.shape
    D, KV, d = shape.d_model, shape.n_kv_heads, shape.head_dim
    seq = (np.asarray(inp.keep) + w.n_text).astype(np.int32)
    R = int(seq.sum())
    K, Wm = args.decode, args.warmup
    total = Wm + 2 * K
    max_len = int(seq.max()) + total + 1
    cache = svl.alloc_kv_cache(cfg, B, max_len, dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    scores = torch.from_numpy(inp.scores).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, D), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    svl.svl_prefill_cache(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                          inp.head_mask, inp.ffn_mask, kept, resid, cache, max_len, ws,
                          stream=stream)
    dws = svl.alloc_decode_workspace(cfg, B, max_len, dev)
    g = torch.Generator(device=dev).manual_seed(args.seed + 100)
    xs = torch.randn(total, B, D, generator=g, device=dev).to(torch.bfloat16).to(torch.float32)
    x = torch.empty((B, D), dtype=torch.float32, device=dev)
    cache_len = seq.copy()
    lens_timed = []

    def step(i):
        x.copy_(xs[i])
        svl.svl_decode_step(cfg, table, x, cache_len, inp.layer_mask, inp.head_mask, inp.ffn_mask,
                            cache, max_len, dws, stream=stream)
        cache_len[:] += 1

    for i in range(Wm):
        step(i)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    evs[0].record(stream)
    for i in range(K):
        lens_timed.append(cache_len.copy())
        step(Wm + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / K
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(K)])
    svl.svl_timing_enable(True)
    for i in range(K):
        step(Wm + K + i)
    torch.cuda.synchronize()
    svl.svl_timing_enable(False)
    ktime = {k: svl.svl_timing_read(k) for k in svl.KCLASS}
    per_kernel = {k: {"ms_per_step": v[0] / K, "launches_per_step": v[1] / K}
                  for k, v in ktime.items() if v[1]}

    bytes_, launches = gemm_bytes(shape, np.ones(B, np.int64), inp.layer_mask, inp.head_mask,
                                  inp.ffn_mask)
    rep = shape.n_heads // KV
    kv_bytes = 0.0
    mean_len = np.mean(np.array(lens_timed), axis=0) + 1          # keys per sample incl. the new one
    for l in range(shape.n_layers):
        for b in range(B):
            if not inp.layer_mask[b, l]:
                continue
            hm = inp.head_mask[b, l]
            kact = sum(int(hm[k * rep:(k + 1) * rep].any()) for k in range(KV))
            kv_bytes += kact * mean_len[b] * d * 2 * 2
    step_bytes = sum(bytes_.values()) + kv_bytes
    gu_ms, gu_n = ktime["gemm_gate_up"]
    gu_avg_ms = gu_ms / max(1, gu_n)
    gu_bytes = bytes_["gu"] / max(1, launches["gu"])
    result = {
        "metric": "decode tokens/s on the pruned and gated KV cache, 7B-shaped",
        "value": round(B / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms, 4),
        "ms_per_step_p10_p50_p90": [round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if shape.dtype == "bf16" else "f32",
        "storage_dtype": shape.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}_decode", "batch": B, "prefill_rows": [int(v) for v in seq],
                   "cached_positions_mean": [round(float(v), 1) for v in mean_len],
                   "layers_executed_per_sample": [int(v) for v in inp.layer_mask.sum(1)],
                   "parallelism": "none (1 GPU)"},
        "step_hbm_bytes": int(step_bytes),
        "step_hbm_gbs": round(step_bytes / (ms * 1e-3) / 1e9, 1),
        "step_hbm_frac": round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "per_kernel": per_kernel,
        "roofline": {
            "kernel": ("gemv_kernel<EPI_SWIGLU> (gate/up row-vector products + SwiGLU, one row per "
                       "sample)" if B == 1 else
                       "gemv_mfma_shared_kernel<EPI_SWIGLU> (gate/up: each weight block once for "
                       "every sample using it, MFMA over the samples' rows, + SwiGLU)"),
            "bound": "hbm", "achieved": round(gu_bytes / (gu_avg_ms * 1e-3) / 1e9, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gu_bytes / (gu_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": None, "avg_launch_ms": round(gu_avg_ms, 5),
            "algorithmic_bytes_per_launch": int(gu_bytes),
        },
    }
    print(json.dumps(result))


def train_flops(shape, B, S):
    """FLOPs the training step executes (2 per multiply-add): the forward, the
    forward again during the backward (without the down projection), the
    data-gradient products and the attention backward (seven S x S x d
    products per head against the forward's two)."""
    D, A, KV, d, F, L = (shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                         shape.d_ffn, shape.n_layers)
    M = B * S
    gemm = 2 * M * (D * (A + 2 * KV) * d + A * d * D + 3 * D * F)
    attn = 2 * A * d * S * (S + 1) * B
    per_layer = 3 * gemm - 2 * M * D * F + 2 * attn + 3.5 * attn
    return int(L * per_layer)


def train_line(w, seed, dev, steps=2, warmup=1):
    """Times svl_train_step (forward + backward to the token and gate logits)
    at the workload's shape: prefix L/2, one unit per head group."""
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W
    shape = w.shape
    B, N, T = w.batch, w.n_vision, w.n_text
    S = N + T
    P, U = shape.n_layers // 2, shape.n_groups
    cfg = svl.make_config(shape)
    vision, text = W.draw_hidden(w, seed, device=dev)
    table = svl.LayerTable([W.draw_layer_weights(w, l, seed, device=dev)
                            for l in range(shape.n_layers)])
    rng = np.random.default_rng([seed, 11])
    z = torch.from_numpy(rng.normal(-0.7, 1.5, (B, N)).astype(np.float32)).to(dev)
    g = torch.from_numpy(rng.normal(0.6, 1.5, (B, (shape.n_layers - P) * U)).astype(np.float32)).to(dev)
    xi = torch.from_numpy(rng.logistic(0, 1, (B, N)).astype(np.float32)).to(dev)
    xg = torch.from_numpy(rng.logistic(0, 1, tuple(g.shape)).astype(np.float32)).to(dev)
    G = torch.from_numpy(rng.standard_normal((B, S, shape.d_model)).astype(np.float32)).to(dev)
    prm = svl.svl_train_params(0.7, 1.3, P, U)
    ws = svl.alloc_train_workspace(cfg, prm, B, N, T, dev)
    stream = torch.cuda.current_stream()

    def step():
        svl.svl_train_step(cfg, table, prm, z, g, vision, text, G, ws, token_noise=xi,
                           gate_noise=xg, stream=stream)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    fl = train_flops(shape, B, S)
    tf = fl / (ms * 1e-3) / 1e12
    print(f"# training step: {ms:.2f} ms", file=sys.stderr, flush=True)
    return {"what": "svl_train_step: static-shape forward under straight-through masks + "
                    "backward to the token and gate logits, float32",
            "workload": w.name, "batch": B, "seq_len": S, "prefix": P, "units": U,
            "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 3),
            "tokens_per_s": round(B * S / (ms * 1e-3), 1),
            "executed_flops_per_step": fl, "executed_tflops": round(tf, 2),
            "fp32_peak_tflops": FP32_PEAK_TFLOPS, "frac_fp32_peak": round(tf / FP32_PEAK_TFLOPS, 4)}


COMPUTE_BOUND = "llava7b_b8_ragged"


def compute_bound_line(headline, table, compute: str, seed: int, dev, steps: int = 5,
                       warmup: int = 2) -> dict:
    """GEMM MFMA fraction of the compute-bound ragged batch of 8 (same 7B shape,
    so the headline's weights, which depend only on shape and seed, serve it
    unchanged): executed GEMM FLOPs over the GEMM launches' event time at the
    dense peak."""
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W

    w = W.get_workload(COMPUTE_BOUND)
    if w.shape != headline.shape:
        return {"workload": COMPUTE_BOUND, "skipped": "shape differs from the headline's"}
    inp = W.draw_inputs(w, seed, device=dev)
    cfg = svl.make_config(w.shape, compute=compute)
    B, N = inp.scores.shape
    seqlens = (inp.keep + w.n_text).astype(np.int64)
    R = int(seqlens.sum())
    scores = torch.from_numpy(inp.scores).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, w.shape.d_model), dtype=torch.float32, device=dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    stream = torch.cuda.current_stream()

    def step():
        svl.svl_prefill(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                        inp.head_mask, inp.ffn_mask, kept, resid, ws, stream=stream,
                        want_flops=False)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    svl.svl_timing_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    svl.svl_timing_enable(False)
    ktime = {k: svl.svl_timing_read(k) for k in svl.KCLASS}
    flops = svl.svl_count_flops(cfg, seqlens, inp.layer_mask, inp.head_mask, inp.ffn_mask)
    gemm_flops = flops["q"] + flops["kv"] + flops["o"] + flops["ffn"]
    gemm_ms = sum(ktime[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")) / steps
    return {"workload": COMPUTE_BOUND, "batch": B, "kept_tokens": R, "ms_per_step": round(ms, 3),
            "gemm_ms_per_step": round(gemm_ms, 3),
            "mfma_util_gemm_pct": round(100 * gemm_flops / (gemm_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 2),
            "mfma_util_prefill_pct": round(100 * flops["total"] / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 2)}


def main():
    args = parse()
    if args.train:
        import torch

        import workloads as W
        if args.gpus != 1 or not torch.cuda.is_available():
            raise SystemExit("bench.py --train runs on one GPU")
        w = W.get_workload(args.workload or W.HEADLINE)
        print(json.dumps(train_line(w, args.seed, torch.device("cuda:0"), steps=args.steps,
                                    warmup=args.warmup)))
        return
    if args.traffic_from:
        write_traffic(args.traffic_from)
        return
    if args.library_gemms:
        library_gemms(args)
        return
    if args.memory_sweep:
        memory_sweep(args)
        return
    if args.decode is not None:
        if args.gpus != 1:
            print(json.dumps({"error": "this build runs on one GPU"}))
            sys.exit(2)
        decode_bench(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; multi-GPU runs are not part of "
                                   "it (samples would shard data-parallel, see DESIGN.md)"}))
        sys.exit(2)
    import torch

    import paper_2607_20357_amd as svl
    import workloads as W

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    w = W.get_workload(args.workload or W.HEADLINE)
    shape = w.shape
    print(f"# workload {w.name}: {w.description}", file=sys.stderr, flush=True)
    inp = W.draw_inputs(w, args.seed, device=dev)
    layers = [W.draw_layer_weights(w, l, args.seed, device=dev) for l in range(shape.n_layers)]
    table = svl.LayerTable(layers)
    cfg = svl.make_config(shape, compute=args.compute)
    B, N = inp.scores.shape
    seqlens = (inp.keep + w.n_text).astype(np.int64)
    R = int(seqlens.sum())
    scores = torch.from_numpy(inp.scores).to(dev)
    kept = torch.empty((B, N), dtype=torch.int32, device=dev)
    resid = torch.empty((R, shape.d_model), dtype=torch.float32, device=dev)
    ws = svl.alloc_workspace(cfg, B, R, dev)
    stream = torch.cuda.current_stream()

    keep_run, lm_run, hm_run, fm_run = inp.keep, inp.layer_mask, inp.head_mask, inp.ffn_mask
    if args.threshold_budget is not None:
        # logits of the token controller (seeded; a quarter positive) and the
        # projection's cost terms: no LM head (V = 0), prefix P = L / 2
        rng = np.random.default_rng([args.seed, 7])
        logits_np = (rng.standard_normal((B, N)) - 0.6745).astype(np.float32)
        scores = torch.from_numpy(logits_np).to(dev)
        count_ws = torch.empty(max(256, 4 * B), dtype=torch.uint8, device=dev)
        prefix = shape.n_layers // 2
        # the count kernel runs on a stream of its own (default priority): its
        # sync waits for the count alone, so the host projects and plans the
        # next step while the previous step's prefill still runs on `stream`
        count_stream = torch.cuda.Stream(device=dev)

        def project():
            counts = svl.svl_count_positive(scores, count_ws, stream=count_stream)
            return counts, svl.svl_budget_project(cfg, counts, N, w.n_text, args.threshold_budget,
                                                  0, prefix, inp.layer_mask, inp.head_mask,
                                                  inp.ffn_mask)

        counts0, (keep_run, lm_run, hm_run, fm_run) = project()
        seqlens = (np.asarray(keep_run) + w.n_text).astype(np.int64)
        R = int(seqlens.sum())
        resid = torch.empty((R, shape.d_model), dtype=torch.float32, device=dev)
        ws = svl.alloc_workspace(cfg, B, R, dev)

        def step():
            _, (k, lm, hm, fm) = project()
            svl.svl_prefill(cfg, table, k, scores, inp.vision, inp.text, lm, hm, fm, kept, resid,
                            ws, stream=stream, want_flops=False)
    elif args.controller is not None:
        rng = np.random.default_rng([args.seed, 7])
        logits_np = (rng.standard_normal((B, N)) - 0.6745).astype(np.float32)
        scores = torch.from_numpy(logits_np).to(dev)
        draw = W.draw_controller(w, args.seed, device=dev, prefix=shape.n_layers // 2)
        ctrl = svl.Controller(draw.prefix, draw.units, draw.pe_dim, draw.hidden, draw.pe_scale,
                              draw.pe_base, draw.tensors)
        resid = torch.empty((B * (N + w.n_text + 1), shape.d_model), dtype=torch.float32,
                            device=dev)
        ws = svl.alloc_controlled_workspace(cfg, ctrl, B, N, w.n_text, dev)
        state = {}

        def step():
            state["out"] = svl.svl_prefill_controlled(cfg, table, ctrl, scores, inp.vision,
                                                      inp.text, args.controller, 0, kept, resid,
                                                      ws, stream=stream)
    else:
        def step():
            svl.svl_prefill(cfg, table, inp.keep, scores, inp.vision, inp.text, inp.layer_mask,
                            inp.head_mask, inp.ffn_mask, kept, resid, ws, stream=stream,
                            want_flops=False)

    if args.copy_calibration:
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # one event after each step (recording an event adds no GPU work)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t_wall = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    print(f"# timed {args.steps} steps: {ms:.4f} ms/step (wall {1e3 * t_wall / args.steps:.4f})",
          file=sys.stderr, flush=True)

    bf16_line = None
    if (not args.no_bf16_line and args.compute == "f16" and shape.dtype == "bf16"
            and args.threshold_budget is None and args.controller is None):
        # the same step with bf16 activations and bf16 MFMA products
        cfg16, ws16 = cfg, ws
        cfg = svl.make_config(shape, compute="bf16")
        # bf16 activations add a plane of the normed rows' low bf16 parts
        ws = svl.alloc_workspace(cfg, B, R, dev)
        for _ in range(max(1, args.warmup)):
            step()
        torch.cuda.synchronize()
        eb0, eb1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        eb0.record(stream)
        for _ in range(args.steps):
            step()
        eb1.record(stream)
        torch.cuda.synchronize()
        ms_b = eb0.elapsed_time(eb1) / args.steps
        tok = B * (w.n_vision + w.n_text)
        bf16_line = {"compute": "bf16 activations, bf16 MFMA", "ms_per_step": round(ms_b, 4),
                     "value": round(tok / (ms_b * 1e-3), 1), "unit": "tokens/s"}
        cfg, ws = cfg16, ws16
        print(f"# bf16 compute: {ms_b:.4f} ms/step", file=sys.stderr, flush=True)

    # second pass, same steps, every launch bracketed by HIP events on `stream`
    svl.svl_timing_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    svl.svl_timing_enable(False)
    ktime = {k: svl.svl_timing_read(k) for k in svl.KCLASS}

    if args.controller is not None:
        # two phases: the prefix layers at the threshold lengths, the others at
        # the projected ones
        out = state["out"]
        P = shape.n_layers // 2
        counts0 = (logits_np > 0).sum(1)
        keep_run, lm_run, hm_run, fm_run = out["keep"], out["layer_mask"], out["head_mask"], out["ffn_mask"]
        seq1 = (counts0 + w.n_text + 1).astype(np.int64)
        seqlens = (np.asarray(keep_run) + w.n_text + 1).astype(np.int64)
        R = int(seqlens.sum())
        lm1 = np.zeros_like(lm_run)
        lm1[:, :P] = 1
        lm2 = lm_run.copy()
        lm2[:, :P] = 0
        flops = out["flops"]
        b1, n1 = gemm_bytes(shape, seq1, lm1, hm_run, fm_run)
        b2, n2 = gemm_bytes(shape, seqlens, lm2, hm_run, fm_run)
        bytes_ = {k: b1[k] + b2[k] for k in b1}
        launches = {k: n1[k] + n2[k] for k in n1}
    else:
        flops = svl.svl_count_flops(cfg, seqlens, lm_run, hm_run, fm_run)
        bytes_, launches = gemm_bytes(shape, seqlens, lm_run, hm_run, fm_run)
    gemm_flops = flops["q"] + flops["kv"] + flops["o"] + flops["ffn"]
    gemm_bytes_total = sum(bytes_.values())
    gemm_t_mfma = gemm_flops / (BF16_PEAK_TFLOPS * 1e12)
    gemm_floor = max(gemm_t_mfma, gemm_bytes_total / (HBM_PEAK_GBS * 1e9))
    eq8 = eq8_flops(shape, seqlens, lm_run, hm_run, w.n_vision, w.n_text)
    gemm_ms = sum(ktime[k][0] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")) / args.steps
    attn_ms = ktime["attention"][0] / args.steps
    tokens = B * (w.n_vision + w.n_text)
    value = tokens / (ms * 1e-3)

    default_mode = args.threshold_budget is None and args.controller is None
    traffic = measured_traffic() if w.name == W.HEADLINE and default_mode else None
    gu_ms, gu_n = ktime["gemm_gate_up"]
    gu_avg_ms = gu_ms / max(1, gu_n)
    gu_bytes_per_launch = bytes_["gu"] / max(1, launches["gu"])
    achieved = gu_bytes_per_launch / (gu_avg_ms * 1e-3) / 1e9
    per_kernel = {k: {"ms_per_step": v[0] / args.steps, "launches_per_step": v[1] / args.steps}
                  for k, v in ktime.items() if v[1]}

    if args.controller is not None:
        metric = (f"effective prefill tokens/s, 7B-shaped, compute controller after "
                  f"{shape.n_layers // 2} prefix layers + threshold selection + budget "
                  f"projection to {args.controller} of C_full")
        workload = f"{w.name}_controller_b{args.controller}"
    elif args.threshold_budget is not None:
        metric = (f"effective prefill tokens/s, 7B-shaped, threshold selection + budget "
                  f"projection to {args.threshold_budget} of C_full")
        workload = f"{w.name}_threshold_b{args.threshold_budget}"
    else:
        metric = "effective prefill tokens/s + MFMA util (% peak), 7B-shaped, keep 0.25"
        workload = w.name
    result = {
        "metric": metric,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_p10_p50_p90": [round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("f16" if args.compute == "f16" else "bf16") if shape.dtype == "bf16" else "f32",
        "storage_dtype": shape.dtype,
        "data": "synthetic",
        "config": {"workload": workload,
                   "batch": B, "n_vision": w.n_vision, "n_text": w.n_text,
                   "keep": [int(k) for k in keep_run], "kept_tokens": R,
                   "layers_executed_per_sample": [int(x) for x in np.asarray(lm_run).sum(1)],
                   "n_layers": shape.n_layers, "d_model": shape.d_model,
                   "heads": shape.n_heads, "kv_heads": shape.n_kv_heads,
                   "d_ffn": shape.d_ffn, "parallelism": "none (1 GPU)"},
        "kept_tokens_per_s": round(R / (ms * 1e-3), 1),
        "executed_tflops": round(flops["total"] / (ms * 1e-3) / 1e12, 2),
        "executed_flops_per_step": flops["total"],
        "eq8_flops_per_step": eq8[0],
        "eq8_flops_full_capacity": eq8[1],
        "eq8_note": "the paper's estimator, Eq. (8), V = 0: non-causal 4 D S^2 and alpha on "
                    "every projection (the executed count is the causal closed form)",
        "mfma_util_gemm_pct": round(100 * gemm_flops / (gemm_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 2),
        "mfma_util_attn_pct": round(100 * flops["attn"] / (attn_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 3)
        if attn_ms > 0 else None,
        "mfma_util_prefill_pct": round(100 * flops["total"] / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 2),
        "gemm_ms_per_step": round(gemm_ms, 4),
        # the GEMMs' floor is the larger of their MFMA time at the dense peak
        # and their algorithmic bytes at 8 TB/s; the ceiling of the MFMA
        # fraction is that MFMA time over the floor (HBM-bound launches
        # cannot reach 100 %), the roofline fraction the floor over the
        # measured GEMM time
        "mfma_util_gemm_ceiling_pct": round(100 * gemm_t_mfma / gemm_floor, 2),
        "gemm_roofline_frac": round(gemm_floor / (gemm_ms * 1e-3), 4),
        "gemm_algorithmic_bytes_per_step": int(gemm_bytes_total),
        "per_kernel": per_kernel,
        "roofline": {
            "kernel": "gemm_mfma_kernel<EPI_SWIGLU> (gate/up projection + SwiGLU)",
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": (traffic["fetch_bytes_per_launch"] + traffic["write_bytes_per_launch"])
            if traffic else None,
            "avg_launch_ms": round(gu_avg_ms, 5),
            "algorithmic_bytes_per_launch": int(gu_bytes_per_launch),
            "traffic_source": os.path.relpath(TRAFFIC_FILE, ROOT) if traffic else None,
        },
    }
    if args.threshold_budget is not None:
        result["threshold"] = {"positive_logits": [int(c) for c in counts0], "budget": args.threshold_budget,
                               "vocab_term": 0, "prefix_layers": shape.n_layers // 2,
                               "groups_dropped_by_projection":
                                   int(np.sum(np.asarray(inp.head_mask) != np.asarray(hm_run)) //
                                       (shape.n_heads // shape.n_groups)),
                               "step": "count kernel (own stream) + host sync + projection + "
                                       "prefill; the next step's count, projection and "
                                       "planning overlap this step's prefill"}
    if args.controller is not None:
        result["controller"] = {
            "positive_logits": [int(c) for c in counts0], "budget": args.controller,
            "vocab_term": 0, "prefix_layers": shape.n_layers // 2, "units": "head groups",
            "gate_logits_positive": int((out["gate_logits"] > 0).sum()),
            "gate_logits": int(out["gate_logits"].size),
            "layers_skipped": int((lm_run == 0).sum()),
            "step": "stats kernel + sync + prefix layers + controller head + sync + projection "
                    "+ row compaction + remaining layers"}
    if bf16_line is not None:
        result["bf16_compute"] = bf16_line
    if not args.no_bf16_line and default_mode and w.name == W.HEADLINE:
        # the compute-bound counterpart of the headline's MFMA fraction
        result["compute_bound"] = compute_bound_line(w, table, args.compute, args.seed, dev)
    if not args.no_train_line and default_mode and w.name == W.HEADLINE:
        result["train_step"] = train_line(w, args.seed, dev)
    if not args.no_cpu_baseline and default_mode:
        result["cpu_baseline"] = cpu_baseline(w, inp, layers, args.cpu_layers)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
