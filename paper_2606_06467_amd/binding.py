"""Thin Python binding of libclsa (include/clsa.h): argument marshalling only.

Every function here has the name of the C entry point it wraps and takes
torch tensors that already live on the GPU; it passes their device pointers,
the shape struct and a HIP stream to the library, and raises ``ClsaError`` when
the library returns an error status.  No step of the path runs in Python, and
there is no fallback: if ``libclsa.so`` is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libclsa.so")

CLSA_OK = 0
CLSA_ERR_INVALID_ARG = -1
CLSA_ERR_UNSUPPORTED = -2
CLSA_ERR_WORKSPACE = -3
CLSA_ERR_HIP = -4
CLSA_ERR_SCRATCH_LIMIT = -5
CLSA_NOALLOC_SCRATCH_BYTES = 32 << 20

CLSA_OP_INDEX = 0
CLSA_OP_TOPK = 1
CLSA_OP_ATTN = 2
CLSA_OP_DECODE = 3
CLSA_OP_DENSE = 4
CLSA_OP_KD_TARGET = 5
CLSA_OP_KD_LOSS = 6


class ClsaError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {clsa_status_string(status)} ({status})")
        self.status = status


class ClsaShape(ctypes.Structure):
    """Mirror of ``clsa_shape``."""
    _fields_ = [("batch", ctypes.c_int32), ("n_q", ctypes.c_int32),
                ("idx_heads", ctypes.c_int32), ("idx_dim", ctypes.c_int32),
                ("q_heads", ctypes.c_int32), ("kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]


def make_shape(batch: int, n_q: int, max_len: int, top_k: int, *, idx_heads: int = 4,
               idx_dim: int = 64, q_heads: int = 32, kv_heads: int = 8, head_dim: int = 128,
               page_size: int = 0, max_pages: int = 0, causal: bool = False,
               softmax_scale: Optional[float] = None) -> ClsaShape:
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(head_dim)
    return ClsaShape(batch, n_q, idx_heads, idx_dim, q_heads, kv_heads, head_dim, max_len,
                     page_size, max_pages, top_k, int(bool(causal)), softmax_scale)


_lib_handle = None


def lib() -> ctypes.CDLL:
    """The loaded libclsa.so (raises if it has not been built)."""
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    P, SP = ctypes.c_void_p, ctypes.POINTER(ClsaShape)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "clsa_workspace_bytes": (sz, [SP, i32, i32]),
        "clsa_index_scores": (i32, [SP, P, P, P, P, P, P, P]),
        "clsa_topk": (i32, [SP, P, P, P, P, P, P, sz, P]),
        "clsa_sparse_attn": (i32, [SP, P, P, P, P, P, P, P, P, P, sz, P]),
        "clsa_decode_step": (i32, [SP, P, P, P, P, P, P, P, i32, P, P, P, P, P, P, sz, P]),
        "clsa_decode_step_noalloc": (i32, [SP, P, P, P, P, P, P, P, i32, P, P, P, P, P, P]),
        "clsa_decode_step_grouped": (i32, [SP, P, i64, P, i64, P, P, P, P, P, i32, i32, P, P, P,
                                           P, P, P, sz, P]),
        "clsa_dense_attn": (i32, [SP, P, P, P, P, P, P, P, P, P, sz, P]),
        "clsa_project_append": (i32, [SP, i32, P, P, P, P, P, P, P, P, P]),
        "clsa_kd_target": (i32, [SP, i32, P, P, P, P, P, P, P, P, sz, P]),
        "clsa_kd_loss": (i32, [SP, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "clsa_status_string": (ctypes.c_char_p, [i32]),
        "clsa_set_phase_events": (i32, [ctypes.POINTER(P), i32]),
        "clsa_get_device_error": (i32, [ctypes.POINTER(ctypes.c_uint32)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    _lib_handle = L
    return L


def _ptr(t: Optional[torch.Tensor], name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(status: int, where: str) -> None:
    if status != CLSA_OK:
        raise ClsaError(status, where)


def clsa_status_string(status: int) -> str:
    return lib().clsa_status_string(int(status)).decode()


def clsa_workspace_bytes(shape: ClsaShape, op: int, n_layers: int = 0) -> int:
    return int(lib().clsa_workspace_bytes(ctypes.byref(shape), int(op), int(n_layers)))


def clsa_index_scores(shape, q_idx, k_idx, page_table, seq_lens, q_pos, scores, stream=None):
    _check(lib().clsa_index_scores(ctypes.byref(shape), _ptr(q_idx, "q_idx"), _ptr(k_idx, "k_idx"),
                                   _ptr(page_table, "page_table"), _ptr(seq_lens, "seq_lens"),
                                   _ptr(q_pos, "q_pos"), _ptr(scores, "scores"), _stream(stream)),
           "clsa_index_scores")


def clsa_topk(shape, scores, seq_lens, q_pos, idx, n_sel, ws=None, stream=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_topk(ctypes.byref(shape), _ptr(scores, "scores"), _ptr(seq_lens, "seq_lens"),
                           _ptr(q_pos, "q_pos"), _ptr(idx, "idx"), _ptr(n_sel, "n_sel"),
                           _ptr(ws, "ws"), wsb, _stream(stream)), "clsa_topk")


def clsa_sparse_attn(shape, q, k_cache, v_cache, page_table, idx, n_sel, out, lse=None, ws=None,
                     stream=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_sparse_attn(ctypes.byref(shape), _ptr(q, "q"), _ptr(k_cache, "k_cache"),
                                  _ptr(v_cache, "v_cache"), _ptr(page_table, "page_table"),
                                  _ptr(idx, "idx"), _ptr(n_sel, "n_sel"), _ptr(out, "out"),
                                  _ptr(lse, "lse"), _ptr(ws, "ws"), wsb, _stream(stream)),
           "clsa_sparse_attn")


def clsa_decode_step(shape, q_idx, k_idx, k_cache, v_cache, page_table, seq_lens, q_pos,
                     q_layers, out_layers, lse_layers, idx, n_sel, ws, stream=None):
    n_layers = 0 if q_layers is None else int(q_layers.shape[0])
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_decode_step(ctypes.byref(shape), _ptr(q_idx, "q_idx"), _ptr(k_idx, "k_idx"),
                                  _ptr(k_cache, "k_cache"), _ptr(v_cache, "v_cache"),
                                  _ptr(page_table, "page_table"), _ptr(seq_lens, "seq_lens"),
                                  _ptr(q_pos, "q_pos"), n_layers, _ptr(q_layers, "q_layers"),
                                  _ptr(out_layers, "out_layers"), _ptr(lse_layers, "lse_layers"),
                                  _ptr(idx, "idx"), _ptr(n_sel, "n_sel"), _ptr(ws, "ws"), wsb,
                                  _stream(stream)), "clsa_decode_step")


def clsa_decode_step_noalloc(shape, q_idx, k_idx, k_cache, v_cache, page_table, seq_lens, q_pos,
                             q_layers, out_layers, lse_layers, idx, n_sel, stream=None):
    """clsa_decode_step on the library's fixed per-device scratch (no workspace)."""
    n_layers = 0 if q_layers is None else int(q_layers.shape[0])
    _check(lib().clsa_decode_step_noalloc(
        ctypes.byref(shape), _ptr(q_idx, "q_idx"), _ptr(k_idx, "k_idx"), _ptr(k_cache, "k_cache"),
        _ptr(v_cache, "v_cache"), _ptr(page_table, "page_table"), _ptr(seq_lens, "seq_lens"),
        _ptr(q_pos, "q_pos"), n_layers, _ptr(q_layers, "q_layers"), _ptr(out_layers, "out_layers"),
        _ptr(lse_layers, "lse_layers"), _ptr(idx, "idx"), _ptr(n_sel, "n_sel"), _stream(stream)),
        "clsa_decode_step_noalloc")


def clsa_decode_step_grouped(shape, q_idx, q_idx_group_stride, k_idx, k_idx_group_stride,
                             k_cache, v_cache, page_table, seq_lens, q_pos, group, q_layers,
                             out_layers, lse_layers, idx, n_sel, ws, stream=None):
    """Strides in bf16 elements between the index queries / keys of consecutive sets."""
    n_layers = 0 if q_layers is None else int(q_layers.shape[0])
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_decode_step_grouped(
        ctypes.byref(shape), _ptr(q_idx, "q_idx"), int(q_idx_group_stride), _ptr(k_idx, "k_idx"),
        int(k_idx_group_stride), _ptr(k_cache, "k_cache"), _ptr(v_cache, "v_cache"),
        _ptr(page_table, "page_table"), _ptr(seq_lens, "seq_lens"), _ptr(q_pos, "q_pos"),
        n_layers, int(group), _ptr(q_layers, "q_layers"), _ptr(out_layers, "out_layers"),
        _ptr(lse_layers, "lse_layers"), _ptr(idx, "idx"), _ptr(n_sel, "n_sel"), _ptr(ws, "ws"),
        wsb, _stream(stream)), "clsa_decode_step_grouped")


def clsa_dense_attn(shape, q, k_cache, v_cache, page_table, seq_lens, q_pos, out, lse=None,
                    ws=None, stream=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_dense_attn(ctypes.byref(shape), _ptr(q, "q"), _ptr(k_cache, "k_cache"),
                                 _ptr(v_cache, "v_cache"), _ptr(page_table, "page_table"),
                                 _ptr(seq_lens, "seq_lens"), _ptr(q_pos, "q_pos"),
                                 _ptr(out, "out"), _ptr(lse, "lse"), _ptr(ws, "ws"), wsb,
                                 _stream(stream)), "clsa_dense_attn")


def clsa_project_append(shape, d_model, h, w, pos, page_table, q_idx, k_idx, k_cache, v_cache,
                        stream=None):
    _check(lib().clsa_project_append(ctypes.byref(shape), int(d_model), _ptr(h, "h"), _ptr(w, "w"),
                                     _ptr(pos, "pos"), _ptr(page_table, "page_table"),
                                     _ptr(q_idx, "q_idx"), _ptr(k_idx, "k_idx"),
                                     _ptr(k_cache, "k_cache"), _ptr(v_cache, "v_cache"),
                                     _stream(stream)), "clsa_project_append")


def clsa_kd_target(shape, n_layers, q_layers, k_cache, page_table, seq_lens, q_pos, abar,
                   ws=None, stream=None, lse_layers=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_kd_target(ctypes.byref(shape), int(n_layers), _ptr(q_layers, "q_layers"),
                                _ptr(k_cache, "k_cache"), _ptr(page_table, "page_table"),
                                _ptr(seq_lens, "seq_lens"), _ptr(q_pos, "q_pos"),
                                _ptr(lse_layers, "lse_layers"), _ptr(abar, "abar"),
                                _ptr(ws, "ws"), wsb, _stream(stream)), "clsa_kd_target")


def clsa_kd_loss(shape, abar, q_idx, k_idx, page_table, seq_lens, q_pos, loss, dq_idx, dk_idx,
                 ws=None, stream=None):
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().clsa_kd_loss(ctypes.byref(shape), _ptr(abar, "abar"), _ptr(q_idx, "q_idx"),
                              _ptr(k_idx, "k_idx"), _ptr(page_table, "page_table"),
                              _ptr(seq_lens, "seq_lens"), _ptr(q_pos, "q_pos"),
                              _ptr(loss, "loss"), _ptr(dq_idx, "dq_idx"), _ptr(dk_idx, "dk_idx"),
                              _ptr(ws, "ws"), wsb, _stream(stream)), "clsa_kd_loss")


CLSA_DEVERR_SEQ_LEN = 1
CLSA_DEVERR_N_SEL = 2


def clsa_get_device_error() -> int:
    """Device error bits (CLSA_DEVERR_*) raised since the last call on the
    current device, cleared by the call.  Synchronises the device."""
    v = ctypes.c_uint32(0)
    _check(lib().clsa_get_device_error(ctypes.byref(v)), "clsa_get_device_error")
    return int(v.value)


def clsa_set_phase_events(events: Optional[Sequence[int]]) -> None:
    """events: 4 + 2m raw hipEvent_t handles (ints): the four phase marks, then a
    (before, after) pair around the attention kernel of each of the first m
    layers; None switches the hook off."""
    if not events:
        _check(lib().clsa_set_phase_events(None, 0), "clsa_set_phase_events")
        return
    arr = (ctypes.c_void_p * len(events))(*[ctypes.c_void_p(int(e)) for e in events])
    _check(lib().clsa_set_phase_events(arr, len(events)), "clsa_set_phase_events")


def workspace(shape: ClsaShape, op: int, n_layers: int = 0, device="cuda") -> Optional[torch.Tensor]:
    """A device byte tensor large enough for ``op`` (None if none is needed)."""
    n = clsa_workspace_bytes(shape, op, n_layers)
    if n == 0:
        return None
    return torch.empty(n, dtype=torch.uint8, device=device)


HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence


class HipEvents:
    """Raw HIP events (libamdhip64) for timing work on a given stream.

    ``timing_only`` events skip the system-scope fence that an event record
    otherwise performs (a cache write-back and invalidate, which both costs time
    and slows the work after it); read them only after the device has been
    synchronised."""

    def __init__(self, n: int, timing_only: bool = False):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                      ctypes.c_uint]
        self._hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                  ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.handles = []
        for _ in range(n):
            h = ctypes.c_void_p()
            flags = HIP_EVENT_DISABLE_SYSTEM_FENCE if timing_only else 0
            if self._hip.hipEventCreateWithFlags(ctypes.byref(h), flags) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.handles.append(h.value)

    def record(self, i: int, stream=None) -> None:
        if self._hip.hipEventRecord(ctypes.c_void_p(self.handles[i]), _stream(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, i: int, j: int) -> float:
        self._hip.hipEventSynchronize(ctypes.c_void_p(self.handles[j]))
        ms = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(self.handles[i]),
                                         ctypes.c_void_p(self.handles[j])) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def close(self) -> None:
        for h in self.handles:
            self._hip.hipEventDestroy(ctypes.c_void_p(h))
        self.handles = []


def bf16_from_bits(bits, device="cuda") -> torch.Tensor:
    """A bfloat16 device tensor holding the given uint16 bit patterns (numpy array)."""
    import numpy as np
    arr = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(device)


def bits_from_bf16(t: torch.Tensor):
    """uint16 numpy bit patterns of a bfloat16 tensor."""
    import numpy as np
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
