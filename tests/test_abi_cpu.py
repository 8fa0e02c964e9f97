"""Host-side checks of libsvl (no GPU needed): the library loads and exports
every function include/svl.h declares, the closed-form FLOP count equals the
oracle's executed count, and invalid arguments are rejected before anything
is enqueued (every case below fails a host-side check, so no device pointer
is ever touched)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2607_20357_amd as svl
from paper_2607_20357_amd import binding
from workloads import ModelShape, WORKLOADS, draw_masks

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "svl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(svl_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = svl.load_library()
    names = _declared_functions()
    assert "svl_prefill" in names and "svl_layer_forward" in names and "svl_select_tokens" in names
    for n in names:
        assert hasattr(lib, n), n
    assert svl.svl_abi_version() == 1


def _rand_case(shape, B, rng):
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    seq = rng.integers(0, 40, B)
    lm = (rng.random((B, L)) > 0.3).astype(np.uint8)
    hm = (rng.random((B, L, A)) > 0.4).astype(np.uint8)
    fm = (rng.random((B, L, G)) > 0.4).astype(np.uint8)
    return seq, lm, hm, fm


@pytest.mark.parametrize("kv", [4, 2, 1])
def test_count_flops_equals_oracle_counter(kv):
    shape = ModelShape(n_layers=3, d_model=32, n_heads=4, n_kv_heads=kv, head_dim=8, d_ffn=48,
                       n_groups=4, dtype="f32")
    rng = np.random.default_rng(kv)
    cfg = svl.make_config(shape)
    for trial in range(4):
        B = 3
        seq, lm, hm, fm = _rand_case(shape, B, rng)
        W = [dict(attn_norm=np.ones(32), ffn_norm=np.ones(32),
                  wq=rng.standard_normal((32, 32)), wk=rng.standard_normal((8 * kv, 32)),
                  wv=rng.standard_normal((8 * kv, 32)), wo=rng.standard_normal((32, 32)),
                  w_gate=rng.standard_normal((48, 32)), w_up=rng.standard_normal((48, 32)),
                  w_down=rng.standard_normal((32, 48))) for _ in range(3)]
        for ffn in (fm, None):
            counter = oracle.FlopCounter()
            for b in range(B):
                x = rng.standard_normal((int(seq[b]), 32))
                for l in range(3):
                    if lm[b, l]:
                        x = oracle.decoder_layer(x, W[l], shape, hm[b, l],
                                                 None if ffn is None else ffn[b, l], counter)
            got = svl.svl_count_flops(cfg, seq, lm, hm, ffn)
            assert got == counter.as_dict()


def test_count_flops_workloads():
    """The headline workload's executed count; the others are at least
    internally consistent (sum of parts)."""
    w = WORKLOADS["llava7b_b1_keep25"]
    keep, lm, hm, fm = draw_masks(w, 0)
    f = svl.svl_count_flops(svl.make_config(w.shape), keep + w.n_text, lm, hm, fm)
    assert f["total"] == 1_521_795_465_216
    for w in WORKLOADS.values():
        keep, lm, hm, fm = draw_masks(w, 0)
        f = svl.svl_count_flops(svl.make_config(w.shape), keep + w.n_text, lm, hm, fm)
        assert f["total"] == f["q"] + f["kv"] + f["o"] + f["attn"] + f["ffn"]


def _call_prefill(cfg, keep, n_vision=8, n_text=2, lm=None, hm=None, fm=None, ws_bytes=1 << 40,
                  ptr=16 * 4096):
    """Calls svl_prefill with fake (never dereferenced) device pointers."""
    lib = svl.load_library()
    B = len(keep)
    kp = np.asarray(keep, np.int32)
    batch = binding.svl_batch(B, n_vision, n_text, kp.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    lm = np.ones((B, L), np.uint8) if lm is None else lm
    hm = np.ones((B, L, A), np.uint8) if hm is None else hm
    fake = binding.svl_layer_weights(*([ptr] * 9))
    table = (binding.svl_layer_weights * L)(*([fake] * L))
    cu = np.zeros(B + 1, np.int32)
    P = ctypes.c_void_p
    st = lib.svl_prefill(ctypes.byref(cfg), table, ctypes.byref(batch), P(ptr), P(ptr), P(ptr),
                         lm.ctypes.data_as(P), hm.ctypes.data_as(P),
                         None if fm is None else fm.ctypes.data_as(P), P(ptr), P(ptr),
                         cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), None, P(ptr),
                         ctypes.c_size_t(ws_bytes), None)
    return st, lib.svl_last_error().decode()


def _cfg(**kw):
    base = dict(n_layers=2, d_model=128, n_heads=4, n_kv_heads=2, head_dim=64, d_ffn=256,
                n_groups=2, dtype="bf16")
    base.update(kw)
    return svl.make_config(**base)


def test_validation_errors():
    st, msg = _call_prefill(_cfg(), [3, 9])           # keep > n_vision
    assert st == 3 and "keep[1]" in msg
    st, _ = _call_prefill(_cfg(), [-1])
    assert st == 3
    st, _ = _call_prefill(_cfg(n_heads=3, n_kv_heads=2), [2])
    assert st == 2
    st, _ = _call_prefill(_cfg(head_dim=63), [2])
    assert st == 2
    st, _ = _call_prefill(_cfg(d_ffn=250), [2])        # not divisible by groups
    assert st == 2
    st, _ = _call_prefill(_cfg(d_ffn=2 * 96), [2])     # bf16 slice not a multiple of 64
    assert st == 2
    st, _ = _call_prefill(_cfg(dtype=7), [2])
    assert st == 5
    bad = np.ones((1, 2, 4), np.uint8)
    bad[0, 1, 2] = 2
    st, msg = _call_prefill(_cfg(), [2], hm=bad)
    assert st == 3 and "head_mask" in msg
    st, msg = _call_prefill(_cfg(), [2], ws_bytes=100)
    assert st == 4
    st, _ = _call_prefill(_cfg(), [2], ptr=16 * 4096 + 4)   # misaligned
    assert st == 7
    lib = svl.load_library()
    assert lib.svl_prefill(None, None, None, None, None, None, None, None, None, None, None,
                           None, None, None, 0, None) == 1


def test_workspace_bytes_monotone():
    cfg = _cfg()
    a = svl.svl_workspace_bytes(cfg, 1, 10)
    b = svl.svl_workspace_bytes(cfg, 1, 1000)
    c = svl.svl_workspace_bytes(cfg, 4, 1000)
    assert 0 < a < b <= c
    assert svl.load_library().svl_workspace_bytes(None, 1, 1) == 0


# --------------------------------------------------------------------------- budget projection
from oracle import budget as obudget  # noqa: E402

BUDGET_SHAPES = [
    ModelShape(n_layers=6, d_model=64, n_heads=8, n_kv_heads=8, head_dim=8, d_ffn=128,
               n_groups=4, dtype="f32"),
    ModelShape(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
               d_ffn=11008, n_groups=4, dtype="bf16"),
    ModelShape(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
               d_ffn=18944, n_groups=4, dtype="bf16"),
]


@pytest.mark.parametrize("si", range(len(BUDGET_SHAPES)))
def test_budget_projection_matches_oracle(si):
    """svl_budget_project (host code of the library) against the oracle:
    identical keep counts and projected masks, for budgets from 0.002 to 1.2,
    with and without FFN gating and gate logits, vocab 0 and 32000."""
    shape = BUDGET_SHAPES[si]
    cfg = svl.make_config(shape)
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    rng = np.random.default_rng(si)
    n_vision, n_text, B = (40, 7, 5) if si == 0 else (576, 64, 3)
    reduced = 0
    for trial in range(24):
        counts = rng.integers(0, n_vision + 1, B).astype(np.int32)
        counts[0] = n_vision
        lm = (rng.random((B, L)) > 0.2).astype(np.uint8)
        hm = (rng.random((B, L, A)) > 0.25).astype(np.uint8)
        fm = (rng.random((B, L, G)) > 0.25).astype(np.uint8) if trial % 2 else None
        gl = rng.normal(0, 1, (B, L, G)).astype(np.float32) if trial % 3 else None
        budget = float(rng.choice([1.2, 1.0, 0.9, 0.5, 0.25, 0.12, 0.05, 0.02, 0.008, 0.002]))
        vocab = 32000 if trial % 4 == 1 else 0
        prefix = int(rng.integers(0, L // 2 + 1))
        keep, lm2, hm2, fm2 = svl.svl_budget_project(cfg, counts, n_vision, n_text, budget, vocab,
                                                     prefix, lm, hm, fm, gl)
        # the oracle takes logits; any logits with these threshold counts will do
        logits = np.full((B, n_vision), -1.0, np.float32)
        for b in range(B):
            logits[b, :counts[b]] = 1.0
        wk, wlm, whm, wfm = obudget.project_batch(shape, logits, n_text, budget, vocab, prefix,
                                                  lm, hm, fm, gl)
        np.testing.assert_array_equal(keep, wk)
        np.testing.assert_array_equal(lm2, wlm)
        np.testing.assert_array_equal(hm2, whm)
        if fm is not None:
            np.testing.assert_array_equal(fm2, wfm)
        reduced += int(not np.array_equal(hm2, hm))
    assert reduced > 0          # the layer / head step was exercised


def test_budget_projection_rejects_bad_arguments():
    shape = BUDGET_SHAPES[0]
    cfg = svl.make_config(shape)
    L, A, G = shape.n_layers, shape.n_heads, shape.n_groups
    lm, hm = np.ones((1, L), np.uint8), np.ones((1, L, A), np.uint8)
    ok = dict(counts=[3], n_vision=10, n_text=2, budget=0.5, vocab=0, prefix=0,
              layer_mask=lm, head_mask=hm)
    svl.svl_budget_project(cfg, **ok)
    for bad in (dict(budget=float("nan")), dict(budget=0.0), dict(budget=-1.0),
                dict(budget=float("inf")), dict(vocab=-1), dict(prefix=L + 1), dict(counts=[11]),
                dict(counts=[-1]), dict(head_mask=np.full((1, L, A), 2, np.uint8)),
                dict(gate_logits=np.full((1, L, G), np.nan, np.float32))):
        with pytest.raises(svl.SvlError):
            svl.svl_budget_project(cfg, **{**ok, **bad})


# --------------------------------------------------------------------------- controlled prefill
def _fake_controller(**kw):
    base = dict(prefix=1, units=2, pe_dim=16, hidden=32, pe_scale=1000.0, pe_base=10000.0)
    base.update({k: v for k, v in kw.items() if k in base})
    ptrs = [kw.get(n, 16 * 4096 * (i + 1)) for i, n in enumerate(binding.CONTROLLER_FIELDS)]
    return binding.svl_controller(base["prefix"], base["units"], base["pe_dim"], base["hidden"],
                                  base["pe_scale"], base["pe_base"], *ptrs)


def _call_controlled(cfg, ctrl, B=2, N=8, T=3, budget=0.5, ws_bytes=None):
    lib = svl.load_library()
    L = cfg.n_layers
    layers = (binding.svl_layer_weights * L)(
        *[binding.svl_layer_weights(*[16 * 4096 * (j + 20)] * 9) for j in range(L)])
    n = lib.svl_controlled_workspace_bytes(ctypes.byref(cfg), ctypes.byref(ctrl), B, N, T)
    ws_bytes = (n - 1 if n else 1 << 20) if ws_bytes is None else ws_bytes
    host = [np.zeros(s, t) for s, t in (((B + 1,), np.int32), ((B,), np.int32),
                                         ((B, L), np.uint8), ((B, L, cfg.n_heads), np.uint8),
                                         ((B, L, cfg.n_groups), np.uint8))]
    vp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    dev = 16 * 4096 * 100
    st = lib.svl_prefill_controlled(ctypes.byref(cfg), layers, ctypes.byref(ctrl), B, N, T,
                                    ctypes.c_float(budget), ctypes.c_int64(0), dev, dev, dev, dev,
                                    dev, *[vp(h) for h in host], None, None, dev, ws_bytes, None)
    return st, lib.svl_last_error().decode()


def test_controlled_prefill_rejects_bad_arguments():
    """Every case fails a host-side check before the first launch (a workspace
    one byte short of svl_controlled_workspace_bytes is the last check)."""
    cfg = _cfg()
    st, msg = _call_controlled(cfg, _fake_controller())
    assert st == 4, msg
    cases = [(dict(prefix=2), 3), (dict(prefix=-1), 3), (dict(units=3), 3), (dict(pe_dim=12), 2),
             (dict(hidden=0), 2), (dict(pe_base=0.0), 3), (dict(pe_scale=float("inf")), 3),
             (dict(llm_w2=None), 1), (dict(gate_b=None), 1), (dict(kap_w1=16 * 4096 + 8), 7)]
    for kw, want in cases:
        st, msg = _call_controlled(cfg, _fake_controller(**kw))
        assert st == want, (kw, st, msg)
    for budget in (float("nan"), 0.0, -0.5, float("inf")):
        st, _ = _call_controlled(cfg, _fake_controller(), budget=budget)
        assert st == 3
    st, _ = _call_controlled(cfg, _fake_controller(), B=0)
    assert st == 2


def test_controlled_workspace_covers_the_prefill_workspace():
    cfg = _cfg()
    lib = svl.load_library()
    ctrl = _fake_controller()
    for B, N, T in ((1, 8, 3), (3, 100, 20), (2, 0, 5)):
        n = lib.svl_controlled_workspace_bytes(ctypes.byref(cfg), ctypes.byref(ctrl), B, N, T)
        assert n >= svl.svl_workspace_bytes(cfg, B, B * (N + T + 1)) + 4 * B * (N + T + 1) * 128
    assert lib.svl_controlled_workspace_bytes(ctypes.byref(cfg), ctypes.byref(
        _fake_controller(units=3)), 1, 8, 3) == 0


def test_budget_loss_rejects_bad_arguments():
    """Host-side checks of svl_budget_loss (no launch happens in these cases)."""
    cfg = _cfg()
    lib = svl.load_library()
    dev = 16 * 4096 * 100

    def call(B=2, N=8, T=3, **kw):
        base = dict(budget=0.5, margin=0.1, w_over=1.0, w_under=1.0, lambda_t=1.0, tau_tok=1.0,
                    tau_comp=1.0, prefix=1, units=2, vocab=0)
        base.update(kw)
        prm = binding.svl_budget_loss_params(*base.values())
        st = lib.svl_budget_loss(ctypes.byref(cfg), ctypes.byref(prm), B, N, T, dev, None, dev,
                                 None, dev, dev, dev, dev, dev, dev, None)
        return st
    for kw, want in ((dict(budget=float("nan")), 3), (dict(budget=0.0), 3), (dict(tau_tok=0.0), 3),
                     (dict(tau_comp=-1.0), 3), (dict(margin=-0.1), 3), (dict(w_over=float("inf")), 3),
                     (dict(lambda_t=-1.0), 3), (dict(prefix=2), 3), (dict(units=3), 3),
                     (dict(vocab=-5), 3), (dict(B=0), 2), (dict(N=0, T=0), 2)):
        assert call(**kw) == want, kw
    assert lib.svl_budget_loss(ctypes.byref(cfg), None, 1, 1, 1, dev, None, dev, None, dev, dev,
                               dev, dev, dev, dev, None) == 1


# ============================================================================ binding checks
# The binding checks every tensor's dtype and size against the configuration
# and the batch before a pointer reaches the library: a short buffer or a
# wrong element type would otherwise let a kernel read or write past the
# allocation.  These run on CPU tensors: every case must fail on its shape or
# dtype check, which comes before the device check, and a correct set of
# tensors gets as far as the device check ("must be a GPU tensor").
import torch  # noqa: E402

_BSHAPE = ModelShape(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=64, d_ffn=256,
                     n_groups=4, dtype="bf16")


def _bind_case(dtype=torch.bfloat16):
    cfg = svl.make_config(_BSHAPE)
    B, N, T, D = 2, 12, 3, _BSHAPE.d_model
    keep = np.array([5, 12], np.int32)
    R = int(keep.sum()) + B * T
    layers = []
    for _ in range(_BSHAPE.n_layers):
        w = {n: torch.zeros(shp, dtype=dtype) for n, shp in binding._weight_shapes(cfg).items()}
        layers.append(w)
    L, A, G = _BSHAPE.n_layers, _BSHAPE.n_heads, _BSHAPE.n_groups
    args = dict(cfg=cfg, layers=layers, keep=keep,
                scores=torch.zeros((B, N), dtype=torch.float32),
                vision=torch.zeros((B, N, D), dtype=dtype), text=torch.zeros((B, T, D), dtype=dtype),
                layer_mask=np.ones((B, L), np.uint8), head_mask=np.ones((B, L, A), np.uint8),
                ffn_mask=np.ones((B, L, G), np.uint8),
                kept_idx=torch.zeros((B, N), dtype=torch.int32),
                resid=torch.zeros((R, D), dtype=torch.float32),
                ws=torch.zeros(64, dtype=torch.uint8))
    return args


def _prefill(**a):
    return svl.svl_prefill(a["cfg"], a["layers"], a["keep"], a["scores"], a["vision"], a["text"],
                           a["layer_mask"], a["head_mask"], a["ffn_mask"], a["kept_idx"],
                           a["resid"], a["ws"])


def test_binding_prefill_accepts_consistent_tensors_up_to_the_device_check():
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        _prefill(**_bind_case())


@pytest.mark.parametrize("change, match", [
    (lambda a: a.update(resid=a["resid"][:-1]), "resid holds"),
    (lambda a: a.update(resid=a["resid"].to(torch.float64)), "resid has dtype"),
    (lambda a: a.update(vision=a["vision"][:, :-1]), "vision has shape"),
    (lambda a: a.update(text=a["text"].float()), "text has dtype"),
    (lambda a: a.update(scores=a["scores"].double()), "scores has dtype"),
    (lambda a: a.update(kept_idx=a["kept_idx"].long()), "kept_idx has dtype"),
    (lambda a: a.update(kept_idx=a["kept_idx"][:1]), "kept_idx holds"),
    (lambda a: a["layers"][1].update(w_down=a["layers"][1]["w_down"].t()), "layer 1.w_down has shape"),
    (lambda a: a["layers"][0].update(wq=a["layers"][0]["wq"].float()), "layer 0.wq has dtype"),
    (lambda a: a["layers"][0].update(wk=a["layers"][0]["wq"]), "layer 0.wk has shape"),
    (lambda a: a["layers"][0].pop("ffn_norm"), "ffn_norm is missing"),
    (lambda a: a.update(layers=a["layers"][:1]), "1 layers given"),
    (lambda a: a.update(head_mask=a["head_mask"][:, :, :2]), "head_mask has shape"),
    (lambda a: a.update(layer_mask=a["layer_mask"][:1]), "layer_mask has shape"),
    (lambda a: a.update(ffn_mask=a["ffn_mask"][..., :3]), "ffn_mask has shape"),
    (lambda a: a.update(keep=np.array([5, 13], np.int32)), "keep values"),
    (lambda a: a.update(keep=np.array([5], np.int32)), "keep has shape"),
])
def test_binding_prefill_rejects_mismatched_tensors(change, match):
    a = _bind_case()
    change(a)
    with pytest.raises(ValueError, match=match):
        _prefill(**a)


def test_binding_select_layer_decode_reject_mismatched_tensors():
    a = _bind_case()
    cfg, D = a["cfg"], _BSHAPE.d_model
    # selection: resid one row short
    with pytest.raises(ValueError, match="resid holds"):
        svl.svl_select_tokens(cfg, a["keep"], a["scores"], a["vision"], a["text"], a["kept_idx"],
                              a["resid"][:-1], a["ws"])
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        svl.svl_select_tokens(cfg, a["keep"], a["scores"], a["vision"], a["text"], a["kept_idx"],
                              a["resid"], a["ws"])
    # one layer: resid shorter than cu_seqlens[-1] rows, wrong weight dtype, mask shapes
    cu = np.array([0, 8, 23], np.int32)
    ok = dict(cfg=cfg, layer=0, weights=a["layers"][0], cu_seqlens=cu,
              layer_on=np.ones(2, np.uint8), head_mask=np.ones((2, 4), np.uint8),
              ffn_mask=np.ones((2, 4), np.uint8), resid=torch.zeros((23, D)), ws=a["ws"])
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        svl.svl_layer_forward(**ok)
    for bad, match in ((dict(resid=torch.zeros((22, D))), "resid holds"),
                       (dict(head_mask=np.ones((2, 3), np.uint8)), "head_mask has shape"),
                       (dict(layer_on=np.ones(3, np.uint8)), "layer_on has shape"),
                       (dict(weights={**a["layers"][0], "wo": a["layers"][0]["wo"].float()}),
                        "wo has dtype")):
        with pytest.raises(ValueError, match=match):
            svl.svl_layer_forward(**{**ok, **bad})
    # decode: x not [B][D] float32, cache_len of the wrong length
    x = torch.zeros((2, D))
    dec = dict(cfg=cfg, layers=a["layers"], x=x, cache_len=np.array([3, 4], np.int32),
               layer_mask=a["layer_mask"], head_mask=a["head_mask"], ffn_mask=a["ffn_mask"],
               kv_cache=torch.zeros(svl.svl_kv_cache_bytes(cfg, 2, 16), dtype=torch.uint8),
               max_len=16, ws=a["ws"])
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        svl.svl_decode_step(**dec)
    for bad, match in ((dict(x=torch.zeros((2, D), dtype=torch.float64)), "x has dtype"),
                       (dict(cache_len=np.array([3], np.int32)), "cache_len has shape"),
                       (dict(kv_cache=torch.zeros(100, dtype=torch.uint8)), "kv_cache holds")):
        with pytest.raises(ValueError, match=match):
            svl.svl_decode_step(**{**dec, **bad})


def test_noalloc_decode_rejects_shapes_past_its_scratch_on_the_host():
    """svl_decode_step_noalloc checks its decode workspace against the
    library's scratch size before anything else touches the GPU (fake,
    never dereferenced device pointers)."""
    lib = svl.load_library()
    cfg = svl.make_config(n_layers=2, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                          d_ffn=11008, n_groups=4, dtype="bf16")
    P = ctypes.c_void_p
    ptr = 16 * 4096
    fake = binding.svl_layer_weights(*([ptr] * 9))
    table = (binding.svl_layer_weights * 2)(fake, fake)
    for B, max_len, fits in ((64, 64, False), (1, 40000, None)):
        need = lib.svl_decode_workspace_bytes(ctypes.byref(cfg), B, max_len)
        if fits is False:
            assert need > binding.SVL_NOALLOC_SCRATCH_BYTES
        cl = np.zeros(B, np.int32)
        lm = np.ones((B, 2), np.uint8)
        hm = np.ones((B, 2, 32), np.uint8)
        st = lib.svl_decode_step_noalloc(ctypes.byref(cfg), table, B, P(ptr), cl.ctypes.data_as(P),
                                         lm.ctypes.data_as(P), hm.ctypes.data_as(P), None, P(ptr),
                                         max_len, None)
        msg = lib.svl_last_error().decode()
        if fits is False:
            assert st == 4 and "allocation-free scratch" in msg, msg
        else:
            assert st == 2 and "max_len" in msg, msg      # max_len past 32768


def test_train_step_rejects_bad_arguments():
    """Host-side checks of svl_train_step and svl_train_workspace_bytes (every
    case is rejected before a launch)."""
    cfg = svl.make_config(WORKLOADS["tiny_f32"].shape)
    lib = svl.load_library()
    dev = 16 * 4096 * 100
    L = cfg.n_layers
    table = (binding.svl_layer_weights * L)(*[binding.svl_layer_weights(*([dev] * 9))] * L)

    def prm(**kw):
        base = dict(tau_tok=0.7, tau_comp=1.3, prefix=1, units=4)
        base.update(kw)
        return binding.svl_train_params(*base.values())

    def call(p=None, B=2, N=8, T=3, ws_bytes=None, **ptr):
        p = p or prm()
        n = lib.svl_train_workspace_bytes(ctypes.byref(cfg), ctypes.byref(p), B, N, T)
        args = dict(logits=dev, tnoise=None, glog=dev, gnoise=None, vision=dev, text=dev,
                    grad=dev, hidden=dev, tmask=dev, umask=dev, gl=dev, gg=dev, ws=dev)
        args.update(ptr)
        return lib.svl_train_step(ctypes.byref(cfg), table, ctypes.byref(p), B, N, T,
                                  args["logits"], args["tnoise"], args["glog"], args["gnoise"],
                                  args["vision"], args["text"], args["grad"], args["hidden"],
                                  args["tmask"], args["umask"], args["gl"], args["gg"], args["ws"],
                                  (n - 1) if ws_bytes is None else ws_bytes, None)

    # the workspace one byte short is the last check: every other case fails earlier
    assert call() == 4
    for p, want in ((prm(tau_tok=0.0), 3), (prm(tau_comp=float("nan")), 3), (prm(prefix=-1), 3),
                    (prm(prefix=L + 1), 3), (prm(units=0), 3), (prm(units=3), 2)):
        assert call(p) == want
        assert lib.svl_train_workspace_bytes(ctypes.byref(cfg), ctypes.byref(p), 2, 8, 3) == 0
    assert call(B=0) == 2 and call(N=0, T=0) == 2 and call(B=70000) == 2
    assert call(hidden=None) == 1 and call(logits=None) == 1 and call(text=None) == 1
    assert call(glog=None) == 1 and call(gl=None) == 1 and call(gg=None) == 1
    assert call(ws=None) == 1 and call(vision=dev + 4) == 7 and call(ws=dev + 8) == 7
    # without grad_hidden the gradient outputs are not needed; N = 0 needs no token arrays;
    # P = L controls no layer and needs no gate arrays (the workspace check still fails last)
    assert call(grad=None, gl=None, gg=None) == 4
    assert call(N=0, logits=None, vision=None, tmask=None, gl=None) == 4
    assert call(prm(prefix=L), glog=None, umask=None, gg=None) == 4
    bad = svl.make_config(WORKLOADS["tiny_f32"].shape)
    bad.head_dim = 16
    assert lib.svl_train_workspace_bytes(ctypes.byref(bad), ctypes.byref(prm()), 2, 8, 3) == 0
    sizes = [lib.svl_train_workspace_bytes(ctypes.byref(cfg), ctypes.byref(prm()), b, 8, 3)
             for b in (1, 2, 4)]
    assert sizes[0] < sizes[1] < sizes[2]


def test_workspace_status_rejects_bad_arguments():
    """Host-side checks of svl_workspace_status (no copy is issued)."""
    lib = svl.load_library()
    dev = 16 * 4096 * 100
    out = ctypes.c_uint32(7)
    assert lib.svl_workspace_status(None, 4096, ctypes.byref(out), None) == 1
    assert lib.svl_workspace_status(dev, 4096, None, None) == 1
    assert lib.svl_workspace_status(dev + 4, 4096, ctypes.byref(out), None) == 7
    assert lib.svl_workspace_status(dev, 255, ctypes.byref(out), None) == 4
    assert out.value == 7


def test_every_workspace_layout_reserves_the_status_word():
    """svl_workspace_bytes grows by the 256 bytes that hold the status word at
    the end of the buffer, for every workload shape."""
    for name, w in WORKLOADS.items():
        cfg = svl.make_config(w.shape)
        n = svl.svl_workspace_bytes(cfg, w.batch, w.batch * (w.n_vision + w.n_text))
        assert n >= 256 and n % 256 == 0, name
