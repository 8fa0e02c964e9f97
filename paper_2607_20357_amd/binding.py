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
SVL_NOALLOC_SCRATCH_BYTES = 64 << 20   # include/svl.h
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


class svl_train_params(ctypes.Structure):
    _fields_ = [("tau_tok", ctypes.c_float), ("tau_comp", ctypes.c_float),
                ("prefix", ctypes.c_int32), ("units", ctypes.c_int32)]


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
    lib.svl_decode_step_noalloc.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights), i32, P, P, P,
                                            P, P, P, i32, P]
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
    lib.svl_train_workspace_bytes.argtypes = [cfgp, ctypes.POINTER(svl_train_params), i32, i32, i32]
    lib.svl_train_workspace_bytes.restype = sz
    lib.svl_train_step.argtypes = [cfgp, ctypes.POINTER(svl_layer_weights),
                                   ctypes.POINTER(svl_train_params), i32, i32, i32, P, P, P, P, P,
                                   P, P, P, P, P, P, P, P, sz, P]
    lib.svl_workspace_status.argtypes = [P, sz, ctypes.POINTER(ctypes.c_uint32), P]
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
              "svl_prefill_cache", "svl_decode_step", "svl_decode_step_noalloc",
              "svl_prefill_controlled",
              "svl_budget_loss", "svl_train_step", "svl_workspace_status"):
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
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} is on {t.device}, the library launches on "
                         f"cuda:{torch.cuda.current_device()}")
    return t.data_ptr()


# ------------------------------------------------------------------ tensor checks
# The C ABI takes plain pointers, so it cannot see a tensor's size or type:
# a short buffer or a wrong element type would make a kernel read or write
# past the allocation.  Every entry point below therefore checks each
# tensor's dtype and element count against the configuration and the batch
# before anything is passed to the library (and before the device check, so
# the host tests can exercise these checks without a GPU).
def storage_dtype(cfg: svl_config) -> torch.dtype:
    """Torch dtype of weights and hidden inputs for a configuration."""
    return torch.bfloat16 if cfg.dtype == SVL_BF16 else torch.float32


def _expect(t: Optional[torch.Tensor], name: str, dtype: torch.dtype, numel: int,
            shape: Optional[tuple] = None) -> None:
    """t must have `dtype` and at least `numel` elements (exactly `shape` if given)."""
    if t is None:
        if numel > 0:
            raise ValueError(f"{name} is required")
        return
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs at least {numel}")


def _weight_shapes(cfg: svl_config) -> Dict[str, tuple]:
    D, A, KV, d, F = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ffn
    return {"attn_norm": (D,), "wq": (A * d, D), "wk": (KV * d, D), "wv": (KV * d, D),
            "wo": (D, A * d), "ffn_norm": (D,), "w_gate": (F, D), "w_up": (F, D),
            "w_down": (D, F)}


def check_layer_weights(cfg: svl_config, w: Dict[str, torch.Tensor], what: str = "layer") -> None:
    """Every weight tensor has the configuration's storage dtype and its exact shape."""
    dt = storage_dtype(cfg)
    for n, shp in _weight_shapes(cfg).items():
        if n not in w:
            raise ValueError(f"{what}: weight {n} is missing")
        _expect(w[n], f"{what}.{n}", dt, int(np.prod(shp)), shp)


def _check_hidden(cfg: svl_config, B: int, N: int, T: int, scores, vision, text,
                  kept_idx, score_name: str = "scores") -> None:
    D = cfg.d_model
    dt = storage_dtype(cfg)
    _expect(scores, score_name, torch.float32, B * N, (B, N))
    _expect(vision, "vision", dt, B * N * D, (B, N, D))
    _expect(text, "text", dt, B * T * D, (B, T, D))
    _expect(kept_idx, "kept_idx", torch.int32, B * N)


def _check_table(cfg: svl_config, table: "LayerTable") -> None:
    if len(table.layers) != cfg.n_layers:
        raise ValueError(f"{len(table.layers)} layers given, the configuration has {cfg.n_layers}")
    if table.cfg_checked is not None and table.cfg_checked == _cfg_key(cfg):
        return
    for l, w in enumerate(table.layers):
        check_layer_weights(cfg, w, f"layer {l}")
    table.cfg_checked = _cfg_key(cfg)


def _table(cfg: svl_config, layers) -> "LayerTable":
    """A checked LayerTable from a LayerTable or a list of per-layer weight dicts
    (the dicts are checked before any device pointer is taken)."""
    if not isinstance(layers, LayerTable):
        layers = list(layers)
        if len(layers) != cfg.n_layers:
            raise ValueError(f"{len(layers)} layers given, the configuration has {cfg.n_layers}")
        for l, w in enumerate(layers):
            check_layer_weights(cfg, w, f"layer {l}")
        table = LayerTable(layers)
        table.cfg_checked = _cfg_key(cfg)
        return table
    _check_table(cfg, layers)
    return layers


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _cfg_key(cfg: svl_config) -> tuple:
    return tuple(getattr(cfg, n) for n, _ in cfg._fields_)


def _batch_dims(scores: torch.Tensor, text: torch.Tensor, score_name: str = "scores"):
    """(B, N, T) from scores [B][N] and text [B][T][D]."""
    if not isinstance(scores, torch.Tensor) or scores.dim() != 2:
        raise ValueError(f"{score_name} must be a [B][N] tensor")
    if not isinstance(text, torch.Tensor) or text.dim() != 3:
        raise ValueError("text must be a [B][T][D] tensor")
    return int(scores.shape[0]), int(scores.shape[1]), int(text.shape[1])


def _check_keep(kp: np.ndarray, B: int, N: int) -> int:
    if kp.shape != (B,):
        raise ValueError(f"keep has shape {kp.shape}, expected ({B},)")
    if np.any(kp < 0) or np.any(kp > N):
        raise ValueError(f"keep values must lie in [0, {N}]")
    return int(kp.sum())


def _host_mask(a, name: str, shape: tuple):
    arr, ptr = _host_u8(a, name)
    if arr.shape != tuple(shape):
        raise ValueError(f"{name} has shape {arr.shape}, expected {tuple(shape)}")
    return arr, ptr


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


SVL_STATUS_NONFINITE = 1


def svl_workspace_status(ws: torch.Tensor, stream=None) -> int:
    """Status word of the last svl_prefill / svl_prefill_cache /
    svl_prefill_controlled on `ws`
    (SVL_STATUS_NONFINITE: an output value was inf or NaN); synchronises the
    stream."""
    out = ctypes.c_uint32(0)
    _check(load_library().svl_workspace_status(_dev(ws, "ws"), _nbytes(ws), ctypes.byref(out),
                                               _stream(stream)))
    return int(out.value)


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
    if not isinstance(logits, torch.Tensor) or logits.dim() != 2:
        raise ValueError("logits must be a [B][N] tensor")
    B, N = logits.shape
    _expect(logits, "logits", torch.float32, B * N)
    counts = np.zeros(B, dtype=np.int32)
    _check(load_library().svl_count_positive(int(B), int(N), _dev(logits, "logits"),
                                             counts.ctypes.data_as(ctypes.c_void_p),
                                             _dev(ws, "ws"), _nbytes(ws), _stream(stream)))
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
    B, N, T = _batch_dims(scores, text)
    R = _check_keep(kp, B, N) + B * T
    _check_hidden(cfg, B, N, T, scores, vision, text, kept_idx)
    _expect(resid, "resid", torch.float32, R * cfg.d_model)
    batch = svl_batch(int(B), int(N), int(T), kpp)
    cu = np.zeros(B + 1, dtype=np.int32)
    _check(load_library().svl_select_tokens(
        ctypes.byref(cfg), ctypes.byref(batch), _dev(scores, "scores"), _dev(vision, "vision"),
        _dev(text, "text"), _dev(kept_idx, "kept_idx"), _dev(resid, "resid"),
        cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), _dev(ws, "ws"), _nbytes(ws),
        _stream(stream)))
    return cu


def svl_layer_forward(cfg: svl_config, layer: int, weights: Dict[str, torch.Tensor], cu_seqlens,
                      layer_on, head_mask, ffn_mask, resid: torch.Tensor, ws: torch.Tensor,
                      stream=None) -> None:
    cu, cup = _host_i32(cu_seqlens)
    if cu.ndim != 1 or cu.shape[0] < 2:
        raise ValueError("cu_seqlens must be a host array of batch + 1 entries")
    B = int(cu.shape[0] - 1)
    lo, lop = _host_mask(layer_on, "layer_on", (B,))
    hm, hmp = _host_mask(head_mask, "head_mask", (B, cfg.n_heads))
    fm, fmp = (None, None) if ffn_mask is None else _host_mask(ffn_mask, "ffn_mask",
                                                                (B, cfg.n_groups))
    check_layer_weights(cfg, weights)
    _expect(resid, "resid", torch.float32, int(cu[-1]) * cfg.d_model)
    w = layer_weights(weights)
    _check(load_library().svl_layer_forward(
        ctypes.byref(cfg), int(layer), ctypes.byref(w), int(cu.shape[0] - 1), cup, lop, hmp, fmp,
        _dev(resid, "resid"), _dev(ws, "ws"), _nbytes(ws), _stream(stream)))


class LayerTable:
    """Host array of svl_layer_weights for svl_prefill (built once, reused).

    The weights' shapes and dtypes are checked against the configuration of
    the first call that uses the table (and again if the configuration
    changes)."""

    def __init__(self, layers: Sequence[Dict[str, torch.Tensor]]):
        self.layers = list(layers)         # keeps the tensors alive
        self.cfg_checked = None
        self.array = (svl_layer_weights * len(self.layers))(*[layer_weights(w) for w in self.layers])


def svl_prefill(cfg: svl_config, layers, keep, scores: torch.Tensor, vision: torch.Tensor,
                text: torch.Tensor, layer_mask, head_mask, ffn_mask, kept_idx: torch.Tensor,
                resid: torch.Tensor, ws: torch.Tensor, stream=None, want_flops: bool = True):
    """The whole budget-adapted prefill; returns (cu_seqlens, flops dict or None).

    `layers` is a LayerTable or a list of per-layer weight dicts."""
    kp, kpp = _host_i32(keep)
    B, N, T = _batch_dims(scores, text)
    R = _check_keep(kp, B, N) + B * T
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    _check_hidden(cfg, B, N, T, scores, vision, text, kept_idx)
    _expect(resid, "resid", torch.float32, R * cfg.d_model)
    batch = svl_batch(int(B), int(N), int(T), kpp)
    lm, lmp = _host_mask(layer_mask, "layer_mask", (B, L))
    hm, hmp = _host_mask(head_mask, "head_mask", (B, L, A))
    fm, fmp = (None, None) if ffn_mask is None else _host_mask(ffn_mask, "ffn_mask", (B, L, G))
    cu = np.zeros(B + 1, dtype=np.int32)
    fl = svl_flops()
    table = _table(cfg, layers)
    _check(load_library().svl_prefill(
        ctypes.byref(cfg), table.array, ctypes.byref(batch), _dev(scores, "scores"),
        _dev(vision, "vision"), _dev(text, "text"), lmp, hmp, fmp, _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        ctypes.byref(fl) if want_flops else None, _dev(ws, "ws"), _nbytes(ws), _stream(stream)))
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
    kp, kpp = _host_i32(keep)
    B, N, T = _batch_dims(scores, text)
    R = _check_keep(kp, B, N) + B * T
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    _check_hidden(cfg, B, N, T, scores, vision, text, kept_idx)
    _expect(resid, "resid", torch.float32, R * cfg.d_model)
    _expect(kv_cache, "kv_cache", torch.uint8, svl_kv_cache_bytes(cfg, B, max_len))
    batch = svl_batch(int(B), int(N), int(T), kpp)
    lm, lmp = _host_mask(layer_mask, "layer_mask", (B, L))
    hm, hmp = _host_mask(head_mask, "head_mask", (B, L, A))
    fm, fmp = (None, None) if ffn_mask is None else _host_mask(ffn_mask, "ffn_mask", (B, L, G))
    cu = np.zeros(B + 1, dtype=np.int32)
    table = _table(cfg, layers)
    _check(load_library().svl_prefill_cache(
        ctypes.byref(cfg), table.array, ctypes.byref(batch), _dev(scores, "scores"),
        _dev(vision, "vision"), _dev(text, "text"), lmp, hmp, fmp, _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        _dev(kv_cache, "kv_cache"), int(max_len), _dev(ws, "ws"), _nbytes(ws), _stream(stream)))
    return cu


def svl_decode_step(cfg: svl_config, layers, x: torch.Tensor, cache_len, layer_mask, head_mask,
                    ffn_mask, kv_cache: torch.Tensor, max_len: int, ws: torch.Tensor,
                    stream=None) -> None:
    """One decode step, x [B][D] float32 updated in place; the caller advances cache_len."""
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("x must be a [B][D] tensor")
    B = int(x.shape[0])
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    _expect(x, "x", torch.float32, B * cfg.d_model, (B, cfg.d_model))
    _expect(kv_cache, "kv_cache", torch.uint8, svl_kv_cache_bytes(cfg, B, max_len))
    cl, clp = _host_i32(cache_len)
    if cl.shape != (B,):
        raise ValueError(f"cache_len has shape {cl.shape}, expected ({B},)")
    lm, lmp = _host_mask(layer_mask, "layer_mask", (B, L))
    hm, hmp = _host_mask(head_mask, "head_mask", (B, L, A))
    fm, fmp = (None, None) if ffn_mask is None else _host_mask(ffn_mask, "ffn_mask", (B, L, G))
    table = _table(cfg, layers)
    _check(load_library().svl_decode_step(
        ctypes.byref(cfg), table.array, int(x.shape[0]), _dev(x, "x"),
        clp, lmp, hmp, fmp, _dev(kv_cache, "kv_cache"), int(max_len), _dev(ws, "ws"), _nbytes(ws),
        _stream(stream)))


def svl_decode_step_noalloc(cfg: svl_config, layers, x: torch.Tensor, cache_len, layer_mask,
                            head_mask, ffn_mask, kv_cache: torch.Tensor, max_len: int,
                            stream=None) -> None:
    """svl_decode_step on the library's own device scratch (no workspace
    argument; the library allocates nothing).  Calls on one GPU share that
    scratch, so overlapping calls must be serialised by the caller."""
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("x must be a [B][D] tensor")
    B = int(x.shape[0])
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    _expect(x, "x", torch.float32, B * cfg.d_model, (B, cfg.d_model))
    _expect(kv_cache, "kv_cache", torch.uint8, svl_kv_cache_bytes(cfg, B, max_len))
    cl, clp = _host_i32(cache_len)
    if cl.shape != (B,):
        raise ValueError(f"cache_len has shape {cl.shape}, expected ({B},)")
    lm, lmp = _host_mask(layer_mask, "layer_mask", (B, L))
    hm, hmp = _host_mask(head_mask, "head_mask", (B, L, A))
    fm, fmp = (None, None) if ffn_mask is None else _host_mask(ffn_mask, "ffn_mask", (B, L, G))
    table = _table(cfg, layers)
    _check(load_library().svl_decode_step_noalloc(
        ctypes.byref(cfg), table.array, B, _dev(x, "x"), clp, lmp, hmp, fmp,
        _dev(kv_cache, "kv_cache"), int(max_len), _stream(stream)))


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

    def check(self, cfg: svl_config) -> None:
        """The parameters' dtypes and shapes against the configuration."""
        E, H, D = self.struct.pe_dim, self.struct.hidden, cfg.d_model
        n = (cfg.n_layers - self.struct.prefix) * self.struct.units
        shapes = {"llm_w1": (H, E), "llm_b1": (H,), "llm_w2": (D, H), "llm_b2": (D,),
                  "kap_w1": (H, E), "kap_b1": (H,), "kap_w2": (D, H), "kap_b2": (D,),
                  "gate_w": (max(n, 0), D), "gate_b": (max(n, 0),)}
        dt = storage_dtype(cfg)
        for name, shp in shapes.items():
            _expect(self.tensors.get(name), f"controller.{name}", dt, int(np.prod(shp)), shp)


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
    B, N, T = _batch_dims(logits, text, "logits")
    L, A, G = cfg.n_layers, cfg.n_heads, cfg.n_groups
    _check_hidden(cfg, B, N, T, logits, vision, text, kept_idx, "logits")
    _expect(resid, "resid", torch.float32, B * (N + T + 1) * cfg.d_model)
    ctrl.check(cfg)
    nl = (L - ctrl.struct.prefix) * ctrl.struct.units
    out = {"cu_seqlens": np.zeros(B + 1, np.int32), "keep": np.zeros(B, np.int32),
           "layer_mask": np.zeros((B, L), np.uint8), "head_mask": np.zeros((B, L, A), np.uint8),
           "ffn_mask": np.zeros((B, L, G), np.uint8),
           "gate_logits": np.zeros((B, max(nl, 0)), np.float32)}
    vp = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    fl = svl_flops()
    table = _table(cfg, layers)
    _check(load_library().svl_prefill_controlled(
        ctypes.byref(cfg), table.array, ctypes.byref(ctrl.struct), int(B), int(N), T,
        ctypes.c_float(budget), ctypes.c_int64(int(vocab)), _dev(logits, "logits"),
        _dev(vision, "vision"), _dev(text, "text"), _dev(kept_idx, "kept_idx"),
        _dev(resid, "resid"), vp(out["cu_seqlens"]), vp(out["keep"]), vp(out["layer_mask"]),
        vp(out["head_mask"]), vp(out["ffn_mask"]), vp(out["gate_logits"]),
        ctypes.byref(fl) if want_flops else None, _dev(ws, "ws"), _nbytes(ws), _stream(stream)))
    out["flops"] = fl.as_dict() if want_flops else None
    return out


def svl_budget_loss(cfg: svl_config, params: svl_budget_loss_params, logits: torch.Tensor,
                    gate_logits: torch.Tensor, n_text: int, token_noise=None, gate_noise=None,
                    stream=None) -> Dict[str, torch.Tensor]:
    """Training-time budget term on the GPU; returns device tensors token_mask,
    unit_mask, ratio, loss, grad_logits, grad_gate (enqueued on the stream)."""
    if not isinstance(logits, torch.Tensor) or logits.dim() != 2:
        raise ValueError("logits must be a [B][N] tensor")
    if not isinstance(gate_logits, torch.Tensor) or gate_logits.dim() != 2:
        raise ValueError("gate_logits must be a [B][units] tensor")
    B, N = logits.shape
    nl = gate_logits.shape[1]
    _expect(logits, "logits", torch.float32, B * N)
    _expect(gate_logits, "gate_logits", torch.float32, B * nl, (B, nl))
    if token_noise is not None:
        _expect(token_noise, "token_noise", torch.float32, B * N, (B, N))
    if gate_noise is not None:
        _expect(gate_noise, "gate_noise", torch.float32, B * nl, (B, nl))
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


def svl_train_workspace_bytes(cfg: svl_config, params: svl_train_params, batch: int,
                              n_vision: int, n_text: int) -> int:
    n = load_library().svl_train_workspace_bytes(ctypes.byref(cfg), ctypes.byref(params),
                                                 int(batch), int(n_vision), int(n_text))
    if n == 0:
        raise SvlError(2, "svl_train_workspace_bytes: " + load_library().svl_last_error().decode())
    return int(n)


def alloc_train_workspace(cfg: svl_config, params: svl_train_params, batch: int, n_vision: int,
                          n_text: int, device="cuda") -> torch.Tensor:
    n = svl_train_workspace_bytes(cfg, params, batch, n_vision, n_text)
    return torch.empty(n, dtype=torch.uint8, device=device)


def svl_train_step(cfg: svl_config, layers, params: svl_train_params, logits: torch.Tensor,
                   gate_logits: Optional[torch.Tensor], vision: torch.Tensor, text: torch.Tensor,
                   grad_hidden: Optional[torch.Tensor], ws: torch.Tensor, token_noise=None,
                   gate_noise=None, stream=None) -> Dict[str, torch.Tensor]:
    """Training step of the masked decoder (svl_train_step in svl.h).  Returns
    device tensors hidden [B][S][D], token_mask, unit_mask and, with
    grad_hidden, grad_logits [B][N] and grad_gate [B][(L-P) U]."""
    if not isinstance(logits, torch.Tensor) or logits.dim() != 2:
        raise ValueError("logits must be a [B][N] tensor")
    if not isinstance(text, torch.Tensor) or text.dim() != 3:
        raise ValueError("text must be a [B][T][D] tensor")
    B, N = logits.shape
    T = text.shape[1]
    S, D = N + T, cfg.d_model
    nl = (cfg.n_layers - params.prefix) * params.units
    dt = storage_dtype(cfg)
    _expect(logits, "logits", torch.float32, B * N, (B, N))
    _expect(vision, "vision", dt, B * N * D, (B, N, D))
    _expect(text, "text", dt, B * T * D, (B, T, D))
    if token_noise is not None:
        _expect(token_noise, "token_noise", torch.float32, B * N, (B, N))
    if nl > 0:
        _expect(gate_logits, "gate_logits", torch.float32, B * nl, (B, nl))
        if gate_noise is not None:
            _expect(gate_noise, "gate_noise", torch.float32, B * nl, (B, nl))
    if grad_hidden is not None:
        _expect(grad_hidden, "grad_hidden", torch.float32, B * S * D, (B, S, D))
    table = _table(cfg, layers)
    dev = logits.device
    out = {"hidden": torch.empty((B, S, D), dtype=torch.float32, device=dev),
           "token_mask": torch.empty((B, N), dtype=torch.uint8, device=dev),
           "unit_mask": torch.empty((B, nl), dtype=torch.uint8, device=dev)}
    if grad_hidden is not None:
        out["grad_logits"] = torch.empty((B, N), dtype=torch.float32, device=dev)
        out["grad_gate"] = torch.empty((B, nl), dtype=torch.float32, device=dev)
    opt = lambda t, n: None if t is None or t.numel() == 0 else _dev(t, n)
    _check(load_library().svl_train_step(
        ctypes.byref(cfg), table.array, ctypes.byref(params), int(B), int(N), int(T),
        opt(logits, "logits"), opt(token_noise, "token_noise"),
        None if nl == 0 else _dev(gate_logits, "gate_logits"),
        None if nl == 0 else opt(gate_noise, "gate_noise"), opt(vision, "vision"),
        opt(text, "text"), opt(grad_hidden, "grad_hidden"), _dev(out["hidden"], "hidden"),
        opt(out["token_mask"], "token_mask"), opt(out["unit_mask"], "unit_mask"),
        opt(out.get("grad_logits"), "grad_logits"), opt(out.get("grad_gate"), "grad_gate"),
        _dev(ws, "ws"), _nbytes(ws), _stream(stream)))
    return out
