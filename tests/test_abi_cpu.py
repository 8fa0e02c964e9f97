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
