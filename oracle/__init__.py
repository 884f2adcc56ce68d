"""Python access to the CPU oracle (``clsa_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py``; the product package never imports it.
It does not import the product package either.

``build()`` compiles the C oracle with gcc (plain -O2, no fast-math) into
``oracle/liboracle.so``; the wrappers below take numpy arrays (bfloat16 as
uint16 bits) and return numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "clsa_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build() -> str:
    """Compile the oracle (always) and return the path of the shared library."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-fno-fast-math", "-Wall",
           "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q", ctypes.c_int32),
                ("idx_heads", ctypes.c_int32), ("idx_dim", ctypes.c_int32),
                ("q_heads", ctypes.c_int32), ("kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("softmax_scale", ctypes.c_double)]


def shape(batch, n_q, max_len, top_k, *, idx_heads=4, idx_dim=64, q_heads=32, kv_heads=8,
          head_dim=128, page_size=0, max_pages=0, causal=False, softmax_scale=None) -> Shape:
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(head_dim)
    return Shape(batch, n_q, idx_heads, idx_dim, q_heads, kv_heads, head_dim, max_len,
                 page_size, max_pages, top_k, int(bool(causal)), float(softmax_scale))


def shape_of(w, **over) -> Shape:
    """Oracle shape for a ``Workload`` (sizes only; no inputs)."""
    kw = dict(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k,
              idx_heads=w.idx_heads, idx_dim=w.idx_dim, q_heads=w.q_heads,
              kv_heads=w.kv_heads, head_dim=w.head_dim, page_size=w.page_size,
              max_pages=w.max_pages, causal=w.causal, softmax_scale=w.softmax_scale)
    kw.update(over)
    return shape(**kw)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    SP = ctypes.POINTER(Shape)
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    lib.oracle_get_threads.argtypes = []
    lib.oracle_get_threads.restype = ctypes.c_int
    lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_double.restype = ctypes.c_double
    lib.oracle_valid_len.argtypes = [SP, P, P, ctypes.c_int, ctypes.c_int]
    lib.oracle_valid_len.restype = ctypes.c_int
    lib.oracle_index_scores.argtypes = [SP, P, P, P, P, P, P]
    lib.oracle_topk.argtypes = [SP, P, P, P, P, P]
    lib.oracle_sparse_attn.argtypes = [SP, P, P, P, P, P, P, P, P]
    lib.oracle_decode_step.argtypes = [SP, P, P, P, P, P, P, P, ctypes.c_int, P, P, P, P, P, P]
    lib.oracle_project.argtypes = [SP, ctypes.c_int, P, P, ctypes.c_int, P, P, P, P]
    lib.oracle_kd_target.argtypes = [SP, ctypes.c_int, P, P, P, P, P, P]
    lib.oracle_kd_loss.argtypes = [SP, P, P, P, P, P, P, P, P, P]
    for f in ("oracle_index_scores", "oracle_topk", "oracle_sparse_attn", "oracle_decode_step",
              "oracle_project", "oracle_kd_target", "oracle_kd_loss"):
        getattr(lib, f).restype = None
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def set_threads(n: int) -> None:
    """Host threads for the row / head loops (results do not depend on it)."""
    _load().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


def bf16_to_double(h: int) -> float:
    return _load().oracle_bf16_to_double(int(h))


def index_scores(sh: Shape, q_idx, k_idx, seq_lens, q_pos=None, page_table=None,
                 fill=np.nan) -> np.ndarray:
    """fp64 scores [B, T, max_len] (Eq. 3); positions outside the valid prefix hold ``fill``."""
    lib = _load()
    q_idx, k_idx = _c(q_idx, np.uint16), _c(k_idx, np.uint16)
    seq_lens, q_pos, page_table = _c(seq_lens, np.int32), _c(q_pos, np.int32), _c(page_table, np.int32)
    out = np.full((sh.batch, sh.n_q, sh.max_len), fill, dtype=np.float64)
    lib.oracle_index_scores(ctypes.byref(sh), _p(q_idx), _p(k_idx), _p(page_table), _p(seq_lens),
                            _p(q_pos), _p(out))
    return out


def topk(sh: Shape, scores_f32, seq_lens, q_pos=None):
    """(idx [B,T,k] int32 ascending with -1 padding, n_sel [B,T] int32) from float32 scores."""
    lib = _load()
    scores_f32 = _c(scores_f32, np.float32)
    assert scores_f32.size == sh.batch * sh.n_q * sh.max_len
    seq_lens, q_pos = _c(seq_lens, np.int32), _c(q_pos, np.int32)
    idx = np.empty((sh.batch, sh.n_q, sh.top_k), dtype=np.int32)
    n_sel = np.empty((sh.batch, sh.n_q), dtype=np.int32)
    lib.oracle_topk(ctypes.byref(sh), _p(scores_f32), _p(seq_lens), _p(q_pos), _p(idx), _p(n_sel))
    return idx, n_sel


def sparse_attn(sh: Shape, q, k_cache, v_cache, idx, n_sel, page_table=None):
    """(out [B,T,Hq,D] fp64, lse [B,T,Hq] fp64) for one layer (Eq. 4)."""
    lib = _load()
    q, k_cache, v_cache = _c(q, np.uint16), _c(k_cache, np.uint16), _c(v_cache, np.uint16)
    idx, n_sel, page_table = _c(idx, np.int32), _c(n_sel, np.int32), _c(page_table, np.int32)
    assert idx.shape[-1] == sh.top_k
    out = np.empty((sh.batch, sh.n_q, sh.q_heads, sh.head_dim), dtype=np.float64)
    lse = np.empty((sh.batch, sh.n_q, sh.q_heads), dtype=np.float64)
    lib.oracle_sparse_attn(ctypes.byref(sh), _p(q), _p(k_cache), _p(v_cache), _p(page_table),
                           _p(idx), _p(n_sel), _p(out), _p(lse))
    return out, lse


def project(sh: Shape, h, w, pos, page_table=None):
    """Eq. 2 for new tokens: (out [rows, n_out] fp64 = h w^T, dest [rows] int64 cache
    row of each token, -1 outside [0, max_len)); h [rows, d_model], w [n_out, d_model]
    as bf16 bits."""
    lib = _load()
    h, w = _c(h, np.uint16), _c(w, np.uint16)
    pos, page_table = _c(pos, np.int32), _c(page_table, np.int32)
    rows = sh.batch * sh.n_q
    d_model = h.shape[-1]
    n_out = w.shape[0]
    assert h.size == rows * d_model and w.shape[1] == d_model and pos.size == rows
    out = np.empty((rows, n_out), dtype=np.float64)
    dest = np.empty(rows, dtype=np.int64)
    lib.oracle_project(ctypes.byref(sh), int(d_model), _p(h), _p(w), int(n_out), _p(pos),
                       _p(page_table), _p(out), _p(dest))
    return out, dest


def kd_target(sh: Shape, q_layers, k_cache, seq_lens, q_pos=None, page_table=None,
              fill=np.nan) -> np.ndarray:
    """Eq. 5 target abar [B, T, max_len] fp64 (invalid positions hold ``fill``)."""
    lib = _load()
    q_layers, k_cache = _c(q_layers, np.uint16), _c(k_cache, np.uint16)
    seq_lens, q_pos, page_table = _c(seq_lens, np.int32), _c(q_pos, np.int32), _c(page_table, np.int32)
    n_layers = q_layers.shape[0]
    out = np.full((sh.batch, sh.n_q, sh.max_len), fill, dtype=np.float64)
    lib.oracle_kd_target(ctypes.byref(sh), int(n_layers), _p(q_layers), _p(k_cache), _p(page_table),
                         _p(seq_lens), _p(q_pos), _p(out))
    return out


def kd_loss(sh: Shape, abar, q_idx, k_idx, seq_lens, q_pos=None, page_table=None):
    """Eq. 6: (loss, dq_idx [B,T,256] fp64, dk_idx fp64 shaped like k_idx; rows never
    written hold nan)."""
    lib = _load()
    abar = np.ascontiguousarray(abar, dtype=np.float64)
    q_idx, k_idx = _c(q_idx, np.uint16), _c(k_idx, np.uint16)
    seq_lens, q_pos, page_table = _c(seq_lens, np.int32), _c(q_pos, np.int32), _c(page_table, np.int32)
    loss = np.zeros(1, dtype=np.float64)
    dq = np.empty(q_idx.shape, dtype=np.float64)
    dk = np.full(k_idx.shape, np.nan, dtype=np.float64)
    lib.oracle_kd_loss(ctypes.byref(sh), _p(abar), _p(q_idx), _p(k_idx), _p(page_table),
                       _p(seq_lens), _p(q_pos), _p(loss), _p(dq), _p(dk))
    return float(loss[0]), dq, dk


def decode_step(sh: Shape, q_idx, k_idx, k_cache, v_cache, seq_lens, q_layers, q_pos=None,
                page_table=None):
    """The whole step: dict with scores (fp64), idx, n_sel, out [L,...] fp64, lse [L,...]."""
    lib = _load()
    q_idx, k_idx = _c(q_idx, np.uint16), _c(k_idx, np.uint16)
    k_cache, v_cache, q_layers = _c(k_cache, np.uint16), _c(v_cache, np.uint16), _c(q_layers, np.uint16)
    seq_lens, q_pos, page_table = _c(seq_lens, np.int32), _c(q_pos, np.int32), _c(page_table, np.int32)
    L = q_layers.shape[0]
    scores = np.empty((sh.batch, sh.n_q, sh.max_len), dtype=np.float64)
    idx = np.empty((sh.batch, sh.n_q, sh.top_k), dtype=np.int32)
    n_sel = np.empty((sh.batch, sh.n_q), dtype=np.int32)
    out = np.empty((L, sh.batch, sh.n_q, sh.q_heads, sh.head_dim), dtype=np.float64)
    lse = np.empty((L, sh.batch, sh.n_q, sh.q_heads), dtype=np.float64)
    lib.oracle_decode_step(ctypes.byref(sh), _p(q_idx), _p(k_idx), _p(k_cache), _p(v_cache),
                           _p(page_table), _p(seq_lens), _p(q_pos), L, _p(q_layers), _p(out),
                           _p(lse), _p(idx), _p(n_sel), _p(scores))
    return dict(scores=scores, idx=idx, n_sel=n_sel, out=out, lse=lse)


def valid_lens(sh: Shape, seq_lens, q_pos=None) -> np.ndarray:
    """[B, T] number of valid keys per query row."""
    lib = _load()
    seq_lens, q_pos = _c(seq_lens, np.int32), _c(q_pos, np.int32)
    v = np.empty((sh.batch, sh.n_q), dtype=np.int32)
    for b in range(sh.batch):
        for t in range(sh.n_q):
            v[b, t] = lib.oracle_valid_len(ctypes.byref(sh), _p(seq_lens), _p(q_pos), b, t)
    return v


def kth_gap(scores64: np.ndarray, n_valid: np.ndarray, k: int) -> np.ndarray:
    """Relative gap (s_(k) - s_(k+1)) / max(|s_(k)|, 1e-30) per row of fp64 scores.

    Rows with n_valid <= k (nothing excluded) get +inf.  A row whose gap is
    below 1e-5 is in the tie band: its top-k set may legitimately depend on the
    rounding order of the score sums."""
    rows = scores64.reshape(-1, scores64.shape[-1])
    nv = np.asarray(n_valid).reshape(-1)
    gap = np.full(rows.shape[0], np.inf)
    for r in range(rows.shape[0]):
        n = int(nv[r])
        if n <= k:
            continue
        part = -np.partition(-rows[r, :n], (k - 1, k))
        sk, sk1 = part[k - 1], part[k]
        gap[r] = (sk - sk1) / max(abs(sk), 1e-30)
    return gap.reshape(np.asarray(n_valid).shape)
