"""Python binding of libsvl (ctypes): argument marshalling only.

Every step of the prefill runs in the library's HIP kernels; this module
only turns torch tensors into device pointers, numpy arrays into host
pointers, and status codes into exceptions.  There is no fallback: if the
library is not built or a tensor is not on the GPU, the call fails.

Function names follow the C ABI (include/svl.h).
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsvl.so")

SVL_F32, SVL_BF16 = 0, 1
SVL_COMPUTE_F16, SVL_COMPUTE_BF16 = 0, 1
KCLASS = {"select": 0, "gather": 1, "rmsnorm": 2, "gemm_qkv": 3, "attention": 4, "gemm_o": 5,
          "gemm_gate_up": 6, "gemm_down": 7, "rope_table": 8, "finish": 9, "kv_append": 10,
          "controller": 11}
STATUS = {0: "SVL_OK", 1: "SVL_E_NULL", 2: "SVL_E_SHAPE", 3: "SVL_E_VALUE", 4: "SVL_E_WORKSPACE",
          5: "SVL_E_DTYPE", 6: "SVL_E_HIP", 7: "SVL_E_ALIGN"}
WEIGHT_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
CONTROLLER_FIELDS = ("llm_w1", "llm_b1", "llm_w2", "llm_b2", "kap_w1", "kap_b1", "kap_w2",
                     "kap_b2", "gate_w", "gate_b")


class SvlError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class svl_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("n_groups", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("compute", ctypes.c_int32)]


class svl_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


class svl_batch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_vision", ctypes.c_int32),
                ("n_text", ctypes.c_int32), ("keep", ctypes.POINTER(ctypes.c_int32))]


class svl_controller(ctypes.Structure):
    _fields_ = [("prefix", ctypes.c_int32), ("units", ctypes.c_int32), ("pe_dim", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("pe_scale", ctypes.c_float),
                ("pe_base", ctypes.c_float)] + [(n, ctypes.c_void_p) for n in CONTROLLER_FIELDS]


class svl_budget_loss_params(ctypes.Structure):
    _fields_ = [("budget", ctypes.c_float), ("margin", ctypes.c_float),
                ("w_over", ctypes.c_float), ("w_under", ctypes.c_float),
                ("lambda_t", ctypes.c_float), ("tau_tok", ctypes.c_float),
                ("tau_comp", ctypes.c_float), ("prefix", ctypes.c_int32),
                ("units", ctypes.c_int32), ("vocab", ctypes.c_int64)]


class svl_flops(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in ("q", "kv", "o", "attn", "ffn", "total")]

    def as_dict(self) -> Dict[str, int]:
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libsvl.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, u64, sz = ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    cfgp = ctypes.POINTER(svl_config)
    lib.svl_select_tokens.argtypes = [cfgp, ctypes.POINTER(svl_batch), P, P, P, P, P,
                                      ctypes.POINTER(i32), P, sz, P]
    lib.svl_layer_forward.argtypes = [cfgp, i32, ctypes.POINTER(svl_layer_weights), i32,
                                      ctypes.POINTER(i32), P, P, P, P, P, sz, P]
    lib.svl_prefill.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights), ctypes.POINTER(svl_batch),
                                P, P, P, P, P, P, P, P, ctypes.POINTER(i32),
                                ctypes.POINTER(svl_flops), P, sz, P]
    lib.svl_count_positive.argtypes = [i32, i32, P, P, P, sz, P]
    lib.svl_prefill_cache.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights), ctypes.POINTER(svl_batch),
                                      P, P, P, P, P, P, P, P, ctypes.POINTER(i32), P, i32, P, sz, P]
    lib.svl_decode_step.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights), i32, P, P, P, P, P, P,
                                    i32, P, sz, P]
    lib.svl_kv_cache_bytes.argtypes = [cfgp, i32, i32]
    lib.svl_kv_cache_bytes.restype = sz
    lib.svl_decode_workspace_bytes.argtypes = [cfgp, i32, i32]
    lib.svl_decode_workspace_bytes.restype = sz
    lib.svl_budget_project.argtypes = [cfgp, i32, i32, i32, P, ctypes.c_float, ctypes.c_int64,
                                       i32, P, P, P, P, P]
    lib.svl_controlled_workspace_bytes.argtypes = [cfgp, ctypes.POINTER(svl_controller), i32, i32,
                                                   i32]
    lib.svl_controlled_workspace_bytes.restype = sz
    lib.svl_prefill_controlled.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights),
                                           ctypes.POINTER(svl_controller), i32, i32, i32,
                                           ctypes.c_float, ctypes.c_int64, P, P, P, P, P, P, P,
                                           P, P, P, P, ctypes.POINTER(svl_flops), P, sz, P]
    lib.svl_budget_loss.argtypes = [cfgp, ctypes.POINTER(svl_budget_loss_params), i32, i32, i32,
                                    P, P, P, P, P, P, P, P, P, P, P]
    lib.svl_workspace_bytes.argtypes = [cfgp, i32, i32]
    lib.svl_workspace_bytes.restype = sz
    lib.svl_count_flops.argtypes = [cfgp, i32, ctypes.POINTER(i32), P, P, P,
                                    ctypes.POINTER(svl_flops)]
    lib.svl_last_error.restype = ctypes.c_char_p
    lib.svl_abi_version.restype = i32
    lib.svl_timing_enable.argtypes = [i32]
    lib.svl_timing_read.argtypes = [i32, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    for f in ("svl_select_tokens", "svl_layer_forward", "svl_prefill", "svl_count_flops",
              "svl_timing_enable", "svl_timing_read", "svl_count_positive", "svl_budget_project",
              "svl_prefill_cache", "svl_decode_step", "svl_prefill_controlled",
              "svl_budget_loss"):
        getattr(lib, f).restype = i32
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        raise SvlError(status, load_library().svl_last_error().decode())


# ------------------------------------------------------------------ marshalling helpers
def make_config(shape=None, **kw) -> svl_config:
    """svl_config from an object with the decoder-shape attributes (or keywords).

    compute: "f16" (default) or "bf16", the activation / matrix-input type of
    bf16-stored workloads."""
    get = (lambda n, d=None: kw.get(n, getattr(shape, n, d))) if shape is not None else kw.get
    dtype = get("dtype", "bf16")
    if isinstance(dtype, str):
        dtype = SVL_BF16 if dtype == "bf16" else SVL_F32
    compute = kw.get("compute", "f16")
    if isinstance(compute, str):
        compute = SVL_COMPUTE_BF16 if compute == "bf16" else SVL_COMPUTE_F16
    return svl_config(int(get("n_layers")), int(get("d_model")), int(get("n_heads")),
                      int(get("n_kv_heads")), int(get("head_dim")), int(get("d_ffn")),
                      int(get("n_groups", 4)), float(get("rms_eps", 1e-6)),
                      float(get("rope_theta", 10000.0)), int(dtype), int(compute))


def _dev(t: Optional[torch.Tensor], name: str) -> int:
    """Device pointer of a GPU tensor; an empty tensor passes NULL (the library
    checks whether the argument may be empty)."""
    if t is None:
        raise ValueError(f"{name} is required")
    if t.numel() == 0:
        return 0
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (no CPU path exists)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _host_u8(a, name: str):
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.uint8))
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def _host_i32(a):
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        stream = stream.cuda_stream
    return ctypes.c_void_p(int(stream))


def layer_weights(w: Dict[str, torch.Tensor]) -> svl_layer_weights:
    return svl_layer_weights(*[_dev(w[n], n) for n in WEIGHT_FIELDS])


# ------------------------------------------------------------------ entry points
def svl_abi_version() -> int:
    return int(load_library().svl_abi_version())


def svl_workspace_bytes(cfg: svl_config, batch: int, total_rows: int) -> int:
    n = load_library().svl_workspace_bytes(ctypes.byref(cfg), int(batch), int(total_rows))
    if n == 0:
        raise SvlError(2, "svl_workspace_bytes: invalid configuration")
    return int(n)


def alloc_workspace(cfg: svl_config, batch: int, total_rows: int, device="cuda") -> torch.Tensor:
    """Caller-owned workspace (torch provides the device memory)."""
    return torch.empty(svl_workspace_bytes(cfg, batch, total_rows), dtype=torch.uint8, device=device)


def svl_count_flops(cfg: svl_config, seqlens, layer_mask, head_mask, ffn_mask=None) -> Dict[str, int]:
    sq, sqp = _host_i32(seqlens)
    lm, lmp = _host_u8(layer_mask, "layer_mask")
    hm, hmp = _host_u8(head_mask, "head_mask")
    fm, fmp = (None, None) if ffn_mask is None else _host_u8(ffn_mask, "ffn_mask")
    out = svl_flops()
    _check(load_library().svl_count_flops(ctypes.byref(cfg), int(sq.shape[0]), sqp, lmp, hmp, fmp,
                                          ctypes.byref(out)))
    return out.as_dict()


def svl_count_positive(logits: torch.Tensor, ws: torch.Tensor, stream=None) -> np.ndarray:
    """Threshold counts (logits > 0 per sample), host int32 [B]; synchronises the stream."""
    B, N = logits.shape
    counts = np.zeros(B, dtype=np.int32)
    _check(load_library().svl_count_positive(int(B), int(N), _dev(logits, "logits"),
                                             counts.ctypes.data_as(ctypes.c_void_p),
                                             _dev(ws, "ws"), ws.numel(), _stream(stream)))
    return counts


def svl_budget_project(cfg: svl_config, counts, n_vision: int, n_text: int, budget: float,
                       vocab: int, prefix: int, layer_mask, head_mask, ffn_mask=None,
                       gate_logits=None):
    """Budget projection (host only): returns (keep [B], layer_mask, head_mask, ffn_mask)
    after the projection; the inputs are not modified."""
    cnt, cntp = _host_i32(counts)
    B = int(cnt.shape[0])
    lm = np.array(layer_mask, dtype=np.uint8, copy=True, order="C")
    hm = np.array(head_mask, dtype=np.uint8, copy=True, order="C")
    fm = None if ffn_mask is None else np.array(ffn_mask, dtype=np.uint8, copy=True, order="C")
    gl = None if gate_logits is None else np.ascontiguousarray(np.asarray(gate_logits, dtype=np.float32))
    keep = np.zeros(B, dtype=np.int32)
    vp = lambda a: None if a is None else a.ctypes.data_as(ctypes.c_void_p)
    _check(load_library().svl_budget_project(
        ctypes.byref(cfg), B, int(n_vision), int(n_text), cntp, ctypes.c_float(budget),
        ctypes.c_int64(int(vocab)), int(prefix), vp(lm), vp(hm), vp(fm), vp(gl),
        keep.ctypes.data_as(ctypes.c_void_p)))
    return keep, lm, hm, fm


def svl_select_tokens(cfg: svl_config, keep, scores: torch.Tensor, vision: torch.Tensor,
                      text: torch.Tensor, kept_idx: torch.Tensor, resid: torch.Tensor,
                      ws: torch.Tensor, stream=None) -> np.ndarray:
    """Top-k selection and packing; returns cu_seqlens (host int32 [B+1])."""
    kp, kpp = _host_i32(keep)
    B, N = scores.shape
    batch = svl_batch(int(B), int(N), int(text.shape[1]), kpp)
    cu = np.zeros(B + 1, dtype=np.int32)
    _check(load_library().svl_select_tokens(
        ctypes.byref(cfg), ctypes.byref(batch), _dev(scores, "scores"), _dev(vision, "vision"),
        _dev(text, "text"), _dev(kept_idx, "kept_idx"), _dev(resid, "resid"),
        cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), _dev(ws, "ws"), ws.numel(),
        _stream(stream)))
    return cu


def svl_layer_forward(cfg: svl_config, layer: int, weights: Dict[str, torch.Tensor], cu_seqlens,
                      layer_on, head_mask, ffn_mask, resid: torch.Tensor, ws: torch.Tensor,
                      stream=None) -> None:
    cu, cup = _host_i32(cu_seqlens)
    lo, lop = _host_u8(layer_on, "layer_on")
    hm, hmp = _host_u8(head_mask, "head_mask")
    fm, fmp = (None, None) if ffn_mask is None else _host_u8(ffn_mask, "ffn_mask")
    w = layer_weights(weights)
    _check(load_library().svl_layer_forward(
        ctypes.byref(cfg), int(layer), ctypes.byref(w), int(cu.shape[0] - 1), cup, lop, hmp, fmp,
        _dev(resid, "resid"), _dev(ws, "ws"), ws.numel(), _stream(stream)))


class LayerTable:
    """Host array of svl_layer_weights for svl_prefill (built once, reused)."""

    def __init__(self, layers: Sequence[Dict[str, torch.Tensor]]):
        self.layers = list(layers)         # keeps the tensors alive
        self.array = (svl_layer_weights * len(self.layers))(*[layer_weights(w) for w in self.layers])


def svl_prefill(cfg: svl_config, layers, keep, scores: torch.Tensor, vision: torch.Tensor,
                text: torch.Tensor, layer_mask, head_mask, ffn_mask, kept_idx: torch.Tensor,
                resid: torch.Tensor, ws: torch.Tensor, stream=None, want_flops: bool = True):
    """The whole budget-adapted prefill; returns (cu_seqlens, flops dict or None).

    `layers` is a LayerTable or a list of per-layer weight dicts."""
    table = layers if isinstance(layers, LayerTable) else LayerTable(layers)
    kp, kpp = _host_i32(keep)
    B, N = scores.shape
    batch = svl_batch(int(B), int(N), int(text.shape[1]), kpp)
    lm, lmp = _host_u8(layer_mask, "layer_mask")
    hm, hmp = _host_u8(head_mask, "head_mask")
    fm, fmp = (None, None) if ffn_mask is None else _host_u8(ffn_mask, "ffn_mask")
    cu = np.zeros(B + 1, dtype=np.int32)
    fl = svl_flops()
    _check(load_library().svl_prefill(
        ctypes.byref(cfg), table.array, ctypes.byref(batch), _dev(scores, "scores"),
        _dev(vision, "vision"), _dev(text, "text"), lmp, hmp, fmp, _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        ctypes.byref(fl) if want_flops else None, _dev(ws, "ws"), ws.numel(), _stream(stream)))
    return cu, (fl.as_dict() if want_flops else None)


def svl_kv_cache_bytes(cfg: svl_config, batch: int, max_len: int) -> int:
    return int(load_library().svl_kv_cache_bytes(ctypes.byref(cfg), int(batch), int(max_len)))


def alloc_kv_cache(cfg: svl_config, batch: int, max_len: int, device="cuda") -> torch.Tensor:
    """Caller-owned KV cache (torch provides the device memory)."""
    n = svl_kv_cache_bytes(cfg, batch, max_len)
    if n == 0:
        raise SvlError(2, "bad KV cache shape")
    return torch.empty(n, dtype=torch.uint8, device=device)


def alloc_decode_workspace(cfg: svl_config, batch: int, max_len: int, device="cuda") -> torch.Tensor:
    n = int(load_library().svl_decode_workspace_bytes(ctypes.byref(cfg), int(batch), int(max_len)))
    if n == 0:
        raise SvlError(2, "bad decode workspace shape")
    return torch.empty(n, dtype=torch.uint8, device=device)


def svl_prefill_cache(cfg: svl_config, layers, keep, scores: torch.Tensor, vision: torch.Tensor,
                      text: torch.Tensor, layer_mask, head_mask, ffn_mask, kept_idx: torch.Tensor,
                      resid: torch.Tensor, kv_cache: torch.Tensor, max_len: int, ws: torch.Tensor,
                      stream=None) -> np.ndarray:
    """The prefill that also fills the KV cache; returns cu_seqlens."""
    table = layers if isinstance(layers, LayerTable) else LayerTable(layers)
    kp, kpp = _host_i32(keep)
    B, N = scores.shape
    batch = svl_batch(int(B), int(N), int(text.shape[1]), kpp)
    lm, lmp = _host_u8(layer_mask, "layer_mask")
    hm, hmp = _host_u8(head_mask, "head_mask")
    fm, fmp = (None, None) if ffn_mask is None else _host_u8(ffn_mask, "ffn_mask")
    cu = np.zeros(B + 1, dtype=np.int32)
    _check(load_library().svl_prefill_cache(
        ctypes.byref(cfg), table.array, ctypes.byref(batch), _dev(scores, "scores"),
        _dev(vision, "vision"), _dev(text, "text"), lmp, hmp, fmp, _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        _dev(kv_cache, "kv_cache"), int(max_len), _dev(ws, "ws"), ws.numel(), _stream(stream)))
    return cu


def svl_decode_step(cfg: svl_config, layers, x: torch.Tensor, cache_len, layer_mask, head_mask,
                    ffn_mask, kv_cache: torch.Tensor, max_len: int, ws: torch.Tensor,
                    stream=None) -> None:
    """One decode step, x [B][D] float32 updated in place; the caller advances cache_len."""
    table = layers if isinstance(layers, LayerTable) else LayerTable(layers)
    cl, clp = _host_i32(cache_len)
    lm, lmp = _host_u8(layer_mask, "layer_mask")
    hm, hmp = _host_u8(head_mask, "head_mask")
    fm, fmp = (None, None) if ffn_mask is None else _host_u8(ffn_mask, "ffn_mask")
    _check(load_library().svl_decode_step(
        ctypes.byref(cfg), table.array, int(x.shape[0]), _dev(x, "x"),
        clp, lmp, hmp, fmp, _dev(kv_cache, "kv_cache"), int(max_len), _dev(ws, "ws"), ws.numel(),
        _stream(stream)))


def svl_timing_enable(on: bool) -> None:
    _check(load_library().svl_timing_enable(1 if on else 0))


def svl_timing_read(kernel_class: str):
    """(total ms, launches) recorded for a kernel class since the last read."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(load_library().svl_timing_read(KCLASS[kernel_class], ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)


class Controller:
    """Compute-controller parameters as an svl_controller (keeps the tensors alive).

    tensors: CONTROLLER_FIELDS -> GPU tensors in the storage dtype."""

    def __init__(self, prefix: int, units: int, pe_dim: int, hidden: int, pe_scale: float,
                 pe_base: float, tensors: Dict[str, torch.Tensor]):
        self.tensors = dict(tensors)
        self.struct = svl_controller(int(prefix), int(units), int(pe_dim), int(hidden),
                                     float(pe_scale), float(pe_base),
                                     *[_dev(self.tensors[n], n) for n in CONTROLLER_FIELDS])


def svl_controlled_workspace_bytes(cfg: svl_config, ctrl: Controller, batch: int, n_vision: int,
                                   n_text: int) -> int:
    n = load_library().svl_controlled_workspace_bytes(ctypes.byref(cfg), ctypes.byref(ctrl.struct),
                                                      int(batch), int(n_vision), int(n_text))
    if n == 0:
        raise SvlError(2, "svl_controlled_workspace_bytes: invalid arguments")
    return int(n)


def alloc_controlled_workspace(cfg: svl_config, ctrl: Controller, batch: int, n_vision: int,
                               n_text: int, device="cuda") -> torch.Tensor:
    return torch.empty(svl_controlled_workspace_bytes(cfg, ctrl, batch, n_vision, n_text),
                       dtype=torch.uint8, device=device)


def svl_prefill_controlled(cfg: svl_config, layers, ctrl: Controller, logits: torch.Tensor,
                           vision: torch.Tensor, text: torch.Tensor, budget: float, vocab: int,
                           kept_idx: torch.Tensor, resid: torch.Tensor, ws: torch.Tensor,
                           stream=None, want_flops: bool = True) -> Dict[str, object]:
    """The controlled prefill (synchronises the stream twice).  resid needs room
    for B (N + T + 1) rows.  Returns the host outputs: cu_seqlens, keep,
    layer_mask, head_mask, ffn_mask, gate_logits and flops."""
    table = layers if isinstance(layers, LayerTable) else LayerTable(layers)
    B, N = logits.shape
    T = int(text.shape[1])
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    nl = (L - ctrl.struct.prefix) * ctrl.struct.units
    out = {"cu_seqlens": np.zeros(B + 1, np.int32), "keep": np.zeros(B, np.int32),
           "layer_mask": np.zeros((B, L), np.uint8), "head_mask": np.zeros((B, L, A), np.uint8),
           "ffn_mask": np.zeros((B, L, G), np.uint8),
           "gate_logits": np.zeros((B, max(nl, 0)), np.float32)}
    vp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    fl = svl_flops()
    _check(load_library().svl_prefill_controlled(
        ctypes.byref(cfg), table.array, ctypes.byref(ctrl.struct), int(B), int(N), T,
        ctypes.c_float(budget), ctypes.c_int64(int(vocab)), _dev(logits, "logits"),
        _dev(vision, "vision"), _dev(text, "text"), _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), vp(out["cu_seqlens"]), vp(out["keep"]), vp(out["layer_mask"]),
        vp(out["head_mask"]), vp(out["ffn_mask"]), vp(out["gate_logits"]),
        ctypes.byref(fl) if want_flops else None, _dev(ws, "ws"), ws.numel(), _stream(stream)))
    out["flops"] = fl.as_dict() if want_flops else None
    return out


def svl_budget_loss(cfg: svl_config, params: svl_budget_loss_params, logits: torch.Tensor,
                    gate_logits: torch.Tensor, n_text: int, token_noise=None, gate_noise=None,
                    stream=None) -> Dict[str, torch.Tensor]:
    """Training-time budget term on the GPU; returns device tensors token_mask,
    unit_mask, ratio, loss, grad_logits, grad_gate (enqueued on the stream)."""
    B, N = logits.shape
    nl = gate_logits.shape[1]
    dev = logits.device
    out = {"token_mask": torch.empty((B, N), dtype=torch.uint8, device=dev),
           "unit_mask": torch.empty((B, nl), dtype=torch.uint8, device=dev),
           "ratio": torch.empty(B, dtype=torch.float32, device=dev),
           "loss": torch.empty(B, dtype=torch.float32, device=dev),
           "grad_logits": torch.empty((B, N), dtype=torch.float32, device=dev),
           "grad_gate": torch.empty((B, nl), dtype=torch.float32, device=dev)}
    opt = lambda t, n: None if t is None else _dev(t, n)
    _check(load_library().svl_budget_loss(
        ctypes.byref(cfg), ctypes.byref(params), int(B), int(N), int(n_text),
        _dev(logits, "logits"), opt(token_noise, "token_noise"), _dev(gate_logits, "gate_logits"),
        opt(gate_noise, "gate_noise"), _dev(out["token_mask"], "token_mask"),
        _dev(out["unit_mask"], "unit_mask"), _dev(out["ratio"], "ratio"), _dev(out["loss"], "loss"),
        _dev(out["grad_logits"], "grad_logits"), _dev(out["grad_gate"], "grad_gate"),
        _stream(stream)))
    return out
