"""Thin Python binding of the Block-GTQ C ABI (include/blockgtq.h).

Argument marshalling only: every step of the path runs in libblockgtq.so.
PyTorch provides device memory (tensors) and the stream.  The binding raises
if the library is missing or a call returns an error; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libblockgtq.so")

BGTQ_FP32, BGTQ_BF16 = 0, 1
HEAD_DIM = 128
N_BLOCKS = 64
MAX_GROUPS = 8

EXPORTED = [
    "blockgtq_last_error", "blockgtq_energy_scores", "blockgtq_allocate", "blockgtq_codebook",
    "blockgtq_layout_bytes", "blockgtq_cache_bytes", "blockgtq_workspace_bytes",
    "blockgtq_layout_init", "blockgtq_quantize_append", "blockgtq_decode_attn",
    "blockgtq_decode_attn_fp16", "blockgtq_prefill_workspace_bytes", "blockgtq_prefill_attn",
    "blockgtq_window_bytes", "blockgtq_window_append", "blockgtq_protected_workspace_bytes",
    "blockgtq_decode_attn_protected", "blockgtq_rope_step_workspace_bytes", "blockgtq_rope_decode_step",
    "blockgtq_read_probe", "blockgtq_decode_attn_noalloc",
]


class BlockGTQError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"blockgtq error {code}: {msg}")
        self.code = code


class _Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "batch", "n_kv_heads", "group", "head_dim", "capacity",
        "k_budget", "v_bits", "in_dtype")]


class _Cache(ctypes.Structure):
    _fields_ = [("k_codes", ctypes.c_void_p), ("k_norms", ctypes.c_void_p),
                ("v_codes", ctypes.c_void_p), ("v_norms", ctypes.c_void_p)]


_lib_handle = None


def lib():
    """Load libblockgtq.so (built by paper_2606_24033_amd.build.build())."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        L.blockgtq_last_error.restype = ctypes.c_char_p
        P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        PSZ = ctypes.POINTER(ctypes.c_size_t)
        sig = {
            "blockgtq_energy_scores": [P, P, I32, I32, I32, P],
            "blockgtq_allocate": [P, I32, I32, I32, I32, I32, P],
            "blockgtq_codebook": [I32, P, P],
            "blockgtq_layout_bytes": [P, PSZ],
            "blockgtq_cache_bytes": [P, PSZ, PSZ, PSZ, PSZ],
            "blockgtq_workspace_bytes": [P, I32, I32, I32, PSZ],
            "blockgtq_layout_init": [P, P, P, P, P, P],
            "blockgtq_quantize_append": [P, P, I32, P, P, I32, P, P, P],
            "blockgtq_decode_attn": [P, P, I32, P, P, I32, P, P, P, SZ, I32, P],
            "blockgtq_decode_attn_fp16": [P, I32, P, P, I32, P, P, P, P, SZ, I32, P],
            "blockgtq_prefill_workspace_bytes": [P, I32, PSZ],
            "blockgtq_prefill_attn": [P, P, I32, P, I32, P, I32, P, P, P, SZ, P],
            "blockgtq_window_bytes": [P, I32, I32, PSZ],
            "blockgtq_window_append": [P, I32, P, P, I32, P, I32, I32, P, P],
            "blockgtq_protected_workspace_bytes": [P, I32, I32, I32, PSZ],
            "blockgtq_decode_attn_protected": [P, P, I32, P, P, I32, P, P, I32, I32, P, P, SZ, I32, P],
            "blockgtq_rope_step_workspace_bytes": [P, I32, I32, PSZ],
            "blockgtq_rope_decode_step": [P, P, ctypes.c_double, P, P, P, P, I32, P, P, P, SZ, I32, P],
            "blockgtq_read_probe": [P, SZ, P, P],
            "blockgtq_decode_attn_noalloc": [P, P, I32, P, P, I32, P, P, I32, P],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        _lib_handle = L
    return _lib_handle


def _check(rc):
    if rc != 0:
        raise BlockGTQError(rc, lib().blockgtq_last_error().decode())


def _ptr(a):
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data_as(ctypes.c_void_p)
    return ctypes.c_void_p(a.data_ptr())


@dataclass
class Config:
    n_layers: int
    batch: int
    n_kv_heads: int
    group: int
    capacity: int
    k_budget: int
    v_bits: int
    in_dtype: int = BGTQ_BF16
    head_dim: int = HEAD_DIM

    def c(self):
        return _Config(self.n_layers, self.batch, self.n_kv_heads, self.group, self.head_dim,
                       self.capacity, self.k_budget, self.v_bits, self.in_dtype)

    @property
    def n_q_heads(self):
        return self.n_kv_heads * self.group

    @property
    def k_words(self):
        return (2 * self.k_budget + 31) // 32


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ----------------------------------------------------------------- host calls

def blockgtq_energy_scores(q_cal: np.ndarray, k_cal: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q_cal, dtype=np.float32)
    k = np.ascontiguousarray(k_cal, dtype=np.float32)
    n, g, d = q.shape
    out = np.zeros(d // 2, dtype=np.float64)
    _check(lib().blockgtq_energy_scores(_ptr(q), _ptr(k), n, g, d, _ptr(out)))
    return out


def blockgtq_allocate(scores: np.ndarray, budget: int, b_min: int = 1, b_max: int = 8) -> np.ndarray:
    s = np.ascontiguousarray(np.atleast_2d(scores), dtype=np.float64)
    out = np.zeros(s.shape, dtype=np.uint8)
    _check(lib().blockgtq_allocate(_ptr(s), s.shape[0], s.shape[1], budget, b_min, b_max, _ptr(out)))
    return out


def blockgtq_codebook(b: int):
    c16 = np.zeros(1 << b, dtype=np.uint16)
    thr = np.zeros((1 << b) - 1, dtype=np.float32)
    _check(lib().blockgtq_codebook(b, _ptr(c16), _ptr(thr)))
    return c16.view(np.float16), thr


def cache_bytes(cfg: Config):
    vals = [ctypes.c_size_t() for _ in range(4)]
    _check(lib().blockgtq_cache_bytes(ctypes.byref(cfg.c()), *[ctypes.byref(v) for v in vals]))
    return [v.value for v in vals]


def workspace_bytes(cfg: Config, n_layers_in_call: int, n_splits: int, max_ctx: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().blockgtq_workspace_bytes(ctypes.byref(cfg.c()), n_layers_in_call, n_splits, max_ctx,
                                          ctypes.byref(v)))
    return v.value


# ---------------------------------------------------------------- device state

class Layout:
    """Device layout blob (rotations, codebooks, per-head grouping tables)."""

    def __init__(self, cfg: Config, k_bits: np.ndarray, rot_k_flat: np.ndarray, rot_v: np.ndarray,
                 device="cuda", stream=None):
        import torch
        n = ctypes.c_size_t()
        _check(lib().blockgtq_layout_bytes(ctypes.byref(cfg.c()), ctypes.byref(n)))
        self.blob = torch.empty(n.value, dtype=torch.uint8, device=device)
        bits = np.ascontiguousarray(k_bits, dtype=np.uint8).reshape(cfg.n_layers * cfg.n_kv_heads, N_BLOCKS)
        rk = np.ascontiguousarray(rot_k_flat, dtype=np.float32)
        rv = np.ascontiguousarray(rot_v, dtype=np.float32)
        _check(lib().blockgtq_layout_init(ctypes.byref(cfg.c()), _ptr(bits), _ptr(rk), _ptr(rv),
                                          _ptr(self.blob), _stream(stream)))
        self.k_bits = bits


class Cache:
    """The packed cache (zero-filled torch tensors in the documented layout)."""

    def __init__(self, cfg: Config, device="cuda"):
        import torch
        L, B, H, C = cfg.n_layers, cfg.batch, cfg.n_kv_heads, cfg.capacity
        self.k_codes = torch.zeros((L, B, H, C, cfg.k_words), dtype=torch.int32, device=device)
        self.k_norms = torch.zeros((L, B, H, C * MAX_GROUPS), dtype=torch.float16, device=device)
        self.v_codes = torch.zeros((L, B, H, C // 32, HEAD_DIM, cfg.v_bits), dtype=torch.int32, device=device)
        self.v_norms = torch.zeros((L, B, H, C), dtype=torch.float16, device=device)

    def c(self):
        return _Cache(self.k_codes.data_ptr(), self.k_norms.data_ptr(), self.v_codes.data_ptr(),
                      self.v_norms.data_ptr())

    def nbytes_used(self, cfg: Config, n_groups_per_row: np.ndarray, tokens: int) -> int:
        """Bytes of codes and norms for `tokens` rows of every (layer, seq, head)."""
        per_row = cfg.k_words * 4 + HEAD_DIM * cfg.v_bits // 8 + 2
        rows = cfg.batch * tokens
        return int(rows * (per_row * cfg.n_layers * cfg.n_kv_heads + 2 * int(np.sum(n_groups_per_row))))


def _check_dev(t, dtype=None):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("device tensors must be contiguous CUDA tensors")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"expected {dtype}, got {t.dtype}")


def _in_dtype(cfg):
    import torch
    return torch.bfloat16 if cfg.in_dtype == BGTQ_BF16 else torch.float32


def blockgtq_quantize_append(cfg: Config, layout: Layout, layer: int, k, v, write_pos, cache: Cache,
                             stream=None, host_write_pos=None):
    """Append n_new rows per sequence.  k, v: [batch, n_new, H_kv, 128] (or with a
    leading layer dim for layer == -1).  write_pos: int32 device tensor [batch].
    host_write_pos (optional list) lets the binding check the capacity bound."""
    import torch
    for t in (k, v):
        _check_dev(t, _in_dtype(cfg))
    _check_dev(write_pos, torch.int32)
    n_new = k.shape[-3]
    if host_write_pos is not None and max(host_write_pos) + n_new > cfg.capacity:
        raise BlockGTQError(-3, "append beyond capacity")
    _check(lib().blockgtq_quantize_append(ctypes.byref(cfg.c()), _ptr(layout.blob), layer, _ptr(k), _ptr(v),
                                          n_new, _ptr(write_pos), ctypes.byref(cache.c()), _stream(stream)))


def blockgtq_decode_attn(cfg: Config, layout: Layout, layer: int, q, ctx_len, max_ctx: int, cache: Cache,
                         out=None, workspace=None, n_splits: int = 0, stream=None):
    import torch
    _check_dev(q, _in_dtype(cfg))
    _check_dev(ctx_len, torch.int32)
    n_lc = cfg.n_layers if layer < 0 else 1
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.zeros(workspace_bytes(cfg, n_lc, n_splits, max_ctx), dtype=torch.uint8, device=q.device)
    _check(lib().blockgtq_decode_attn(ctypes.byref(cfg.c()), _ptr(layout.blob), layer, _ptr(q), _ptr(ctx_len),
                                      max_ctx, ctypes.byref(cache.c()), _ptr(out), _ptr(workspace),
                                      workspace.numel(), n_splits, _stream(stream)))
    return out


def blockgtq_decode_attn_noalloc(cfg: Config, layout: Layout, layer: int, q, ctx_len, max_ctx: int, cache: Cache,
                                 out, n_splits: int = 0, stream=None):
    """blockgtq_decode_attn with its workspace in the library's static device
    array (no allocation in the call; `out` is the caller's)."""
    import torch
    _check_dev(q, _in_dtype(cfg))
    _check_dev(ctx_len, torch.int32)
    _check_dev(out, torch.float32)
    _check(lib().blockgtq_decode_attn_noalloc(ctypes.byref(cfg.c()), _ptr(layout.blob), layer, _ptr(q),
                                              _ptr(ctx_len), max_ctx, ctypes.byref(cache.c()), _ptr(out), n_splits,
                                              _stream(stream)))
    return out


def blockgtq_decode_attn_fp16(cfg: Config, layer: int, q, ctx_len, max_ctx: int, k16, v16, out=None,
                              workspace=None, n_splits: int = 0, stream=None):
    import torch
    _check_dev(q, _in_dtype(cfg))
    _check_dev(ctx_len, torch.int32)
    _check_dev(k16, torch.float16)
    _check_dev(v16, torch.float16)
    n_lc = cfg.n_layers if layer < 0 else 1
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.zeros(workspace_bytes(cfg, n_lc, n_splits, max_ctx), dtype=torch.uint8, device=q.device)
    _check(lib().blockgtq_decode_attn_fp16(ctypes.byref(cfg.c()), layer, _ptr(q), _ptr(ctx_len), max_ctx,
                                           _ptr(k16), _ptr(v16), _ptr(out), _ptr(workspace), workspace.numel(),
                                           n_splits, _stream(stream)))
    return out


def prefill_workspace_bytes(cfg: Config, n_q: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().blockgtq_prefill_workspace_bytes(ctypes.byref(cfg.c()), n_q, ctypes.byref(v)))
    return v.value


def blockgtq_prefill_attn(cfg: Config, layout: Layout, layer: int, q, q_pos0, max_pos: int, cache: Cache,
                          out=None, workspace=None, stream=None):
    """Causal prefill attention of one layer.  q: [batch, n_q, Hq, 128] in the
    config's input dtype; q_pos0: int32 device tensor [batch] (position of
    query 0 of each sequence); max_pos: host bound of q_pos0 + n_q - 1."""
    import torch
    _check_dev(q, _in_dtype(cfg))
    _check_dev(q_pos0, torch.int32)
    n_q = q.shape[1]
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.empty(max(prefill_workspace_bytes(cfg, n_q), 1), dtype=torch.uint8, device=q.device)
    _check(lib().blockgtq_prefill_attn(ctypes.byref(cfg.c()), _ptr(layout.blob), layer, _ptr(q), n_q, _ptr(q_pos0),
                                       max_pos, ctypes.byref(cache.c()), _ptr(out), _ptr(workspace),
                                       workspace.numel(), _stream(stream)))
    return out


# ---------------------------------------------------------------- protected fp16 window

def window_bytes(cfg: Config, n_sink: int, n_recent: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().blockgtq_window_bytes(ctypes.byref(cfg.c()), n_sink, n_recent, ctypes.byref(v)))
    return v.value


def protected_workspace_bytes(cfg: Config, n_layers_in_call: int, n_splits: int, max_ctx: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().blockgtq_protected_workspace_bytes(ctypes.byref(cfg.c()), n_layers_in_call, n_splits, max_ctx,
                                                    ctypes.byref(v)))
    return v.value


def blockgtq_window_append(cfg: Config, layer: int, k, v, write_pos, n_sink: int, n_recent: int, window,
                           stream=None):
    """fp16 copies of appended rows into the window (same k, v, write_pos as
    blockgtq_quantize_append).  window: fp16 device tensor of window_bytes."""
    import torch
    for t in (k, v):
        _check_dev(t, _in_dtype(cfg))
    _check_dev(write_pos, torch.int32)
    _check_dev(window, torch.float16)
    if window.numel() * 2 < window_bytes(cfg, n_sink, n_recent):
        raise BlockGTQError(-1, "window tensor too small")
    _check(lib().blockgtq_window_append(ctypes.byref(cfg.c()), layer, _ptr(k), _ptr(v), k.shape[-3], _ptr(write_pos),
                                        n_sink, n_recent, _ptr(window), _stream(stream)))


def blockgtq_decode_attn_protected(cfg: Config, layout: Layout, layer: int, q, ctx_len, max_ctx: int, cache: Cache,
                                   window, n_sink: int, n_recent: int, out=None, workspace=None, n_splits: int = 0,
                                   stream=None):
    import torch
    _check_dev(q, _in_dtype(cfg))
    _check_dev(ctx_len, torch.int32)
    _check_dev(window, torch.float16)
    if window.numel() * 2 < window_bytes(cfg, n_sink, n_recent):
        raise BlockGTQError(-1, "window tensor too small")
    n_lc = cfg.n_layers if layer < 0 else 1
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = torch.zeros(protected_workspace_bytes(cfg, n_lc, n_splits, max_ctx), dtype=torch.uint8,
                                device=q.device)
    _check(lib().blockgtq_decode_attn_protected(ctypes.byref(cfg.c()), _ptr(layout.blob), layer, _ptr(q),
                                                _ptr(ctx_len), max_ctx, ctypes.byref(cache.c()), _ptr(window),
                                                n_sink, n_recent, _ptr(out), _ptr(workspace), workspace.numel(),
                                                n_splits, _stream(stream)))
    return out


# ---------------------------------------------------------------- decode step from pre-RoPE inputs

def rope_step_workspace_bytes(cfg: Config, max_ctx: int, n_splits: int = 0) -> int:
    v = ctypes.c_size_t()
    _check(lib().blockgtq_rope_step_workspace_bytes(ctypes.byref(cfg.c()), max_ctx, n_splits, ctypes.byref(v)))
    return v.value


def blockgtq_rope_decode_step(cfg: Config, layout: Layout, rope_base: float, q_pre, k_pre, v, pos, max_ctx: int,
                              cache: Cache, out=None, workspace=None, n_splits: int = 0, stream=None):
    """One all-layer decode step from pre-RoPE q [L, B, Hq, 128] and k, v
    [L, B, 1, H_kv, 128] (in_dtype) at device positions pos (int32 [B])."""
    import torch
    for t in (q_pre, k_pre, v):
        _check_dev(t, _in_dtype(cfg))
    _check_dev(pos, torch.int32)
    if out is None:
        out = torch.empty(q_pre.shape, dtype=torch.float32, device=q_pre.device)
    if workspace is None:
        workspace = torch.zeros(rope_step_workspace_bytes(cfg, max_ctx, n_splits), dtype=torch.uint8,
                                device=q_pre.device)
    _check(lib().blockgtq_rope_decode_step(ctypes.byref(cfg.c()), _ptr(layout.blob), float(rope_base), _ptr(q_pre),
                                           _ptr(k_pre), _ptr(v), _ptr(pos), max_ctx, ctypes.byref(cache.c()),
                                           _ptr(out), _ptr(workspace), workspace.numel(), n_splits,
                                           _stream(stream)))
    return out


def blockgtq_read_probe(src, sink, stream=None):
    """Stream-read every byte of the device tensor `src` (measurement helper)."""
    _check_dev(src)
    _check(lib().blockgtq_read_probe(_ptr(src), src.numel() * src.element_size(), _ptr(sink), _stream(stream)))

