"""Seeded synthetic inputs for the CLSA decode path.

This module only draws random numbers and lays them out in memory; it holds none
of the method's arithmetic (no scoring, no selection, no attention).  Both the
GPU path's tests/benchmark and the CPU oracle are fed the same bytes produced
here, so the two sides never share any code beyond this generator.

Recipe (the same for every workload):
  * numpy ``PCG64``; a workload seed ``1000*workload_id + stream`` names one
    stream per tensor; each stream is cut into 2**20-element chunks seeded by
    ``SeedSequence(seed).spawn`` so that generation can run on several threads
    and still give the same bits on every machine;
  * ``standard_normal(float32)`` times a scale, rounded to bfloat16 with
    round-to-nearest-even on the float32 bit pattern;
  * index queries / index keys ~ N(0,1)/8, K, V and per-layer queries ~ N(0,1);
  * planted structure (128K decode): 64 distinct positions per sequence whose
    index key gets ``+3 * (1/8) * q_hat`` (q_hat = the sequence's index query
    as a unit 256-vector), i.e. +3 standard deviations of the score, then
    re-rounded to bfloat16;
  * ragged lengths ~ U{lo..hi}; paged caches hold 64-token pages whose physical
    order is a seeded random permutation.

Stream numbers: 1 q_idx, 2 k_idx, 3 K, 4 V, 5 planted positions, 6 lengths,
7 page permutation, 100+l the layer-l query.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional

import numpy as np

_CHUNK = 1 << 20


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round a float32 array to bfloat16 (nearest, ties to even); return uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint32, copy=True)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = (u >> 16) & 1
    r += 0x7FFF
    u += r
    u >>= 16
    out = u.astype(np.uint16)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bits to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    """``shape`` draws of N(0,1)*scale rounded to bfloat16, as uint16 bits."""
    n = int(np.prod(shape, dtype=np.int64))
    out = np.empty(n, dtype=np.uint16)
    if n == 0:
        return out.reshape(shape)
    nch = (n + _CHUNK - 1) // _CHUNK
    seqs = np.random.SeedSequence(seed).spawn(nch)
    sc = np.float32(scale)

    def work(i: int) -> None:
        g = np.random.Generator(np.random.PCG64(seqs[i]))
        lo = i * _CHUNK
        hi = min(n, lo + _CHUNK)
        a = g.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            a *= sc
        u = a.view(np.uint32)
        r = (u >> 16) & 1
        r += 0x7FFF
        u += r
        u >>= 16
        out[lo:hi] = u

    if nch == 1:
        work(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nch)))
    return out.reshape(shape)


@dataclasses.dataclass
class Workload:
    """Sizes of one synthetic workload (names follow the paper's notation)."""
    name: str
    wid: int                 # workload id, used for seeds
    batch: int               # B
    lens: List[int]          # n per sequence (cache length incl. the current token)
    top_k: int               # k
    n_layers: int            # L cross-decoder layers sharing one index set
    n_q: int = 1             # T query tokens per sequence (1 = decode)
    idx_heads: int = 4
    idx_dim: int = 64
    q_heads: int = 32
    kv_heads: int = 8
    head_dim: int = 128
    page_size: int = 0       # 0 = contiguous caches
    causal: bool = False
    planted: int = 0         # planted aligned index keys per sequence
    q_pos0: Optional[List[int]] = None  # absolute position of the first query row per sequence

    @property
    def max_len(self) -> int:
        m = max(self.lens) if self.lens else 0
        if self.page_size:
            m = (m + self.page_size - 1) // self.page_size * self.page_size
        return max(m, self.page_size or 1)

    @property
    def max_pages(self) -> int:
        return self.max_len // self.page_size if self.page_size else 0

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


def _lens_uniform(seed: int, batch: int, lo: int, hi: int) -> List[int]:
    g = np.random.Generator(np.random.PCG64(seed))
    return [int(x) for x in g.integers(lo, hi + 1, size=batch)]


def workload(name: str) -> Workload:
    """The five named workloads of the long-context decode/prefill study, and the
    training-side distillation workload."""
    if name == "decode_b1_n4k":
        return Workload(name, 1, 1, [4096], 512, 4)
    if name == "decode_b8_n32k":
        return Workload(name, 2, 8, [32768] * 8, 2048, 16)
    if name == "decode_b4_n128k_planted":
        return Workload(name, 3, 4, [131072] * 4, 2048, 16, planted=64)
    if name == "prefill_t8k_n128k":
        return Workload(name, 4, 1, [131072], 2048, 16, n_q=8192, causal=True,
                        q_pos0=[122880])
    if name == "decode_b32_ragged_paged":
        return Workload(name, 5, 32, _lens_uniform(5006, 32, 16384, 65536), 2048, 24,
                        page_size=64)
    if name == "kd_train_t32k":
        # training side (Section 2.2): one 32,768-token sequence, every token a
        # causal query row, the target averaged over L = 16 layers x 32 heads
        return Workload(name, 6, 1, [32768], 2048, 16, n_q=32768, causal=True, q_pos0=[0])
    raise KeyError(name)


WORKLOADS = ["decode_b1_n4k", "decode_b8_n32k", "decode_b4_n128k_planted",
             "prefill_t8k_n128k", "decode_b32_ragged_paged"]
# The distillation workload (not a decode-step configuration).
KD_WORKLOADS = ["kd_train_t32k"]


def page_table_for(w: Workload, seed: int) -> np.ndarray:
    """[B, max_pages] int32 physical page of each logical page; unused slots hold -1.

    Physical pages are a seeded random permutation of 0..P-1, P = sum ceil(len/page)."""
    ps = w.page_size
    need = [(n + ps - 1) // ps for n in w.lens]
    total = int(sum(need))
    perm = np.random.Generator(np.random.PCG64(seed)).permutation(total).astype(np.int32)
    pt = np.full((w.batch, w.max_pages), -1, dtype=np.int32)
    off = 0
    for b, c in enumerate(need):
        pt[b, :c] = perm[off:off + c]
        off += c
    return pt


def make_inputs(w: Workload, layers: Optional[List[int]] = None, seed_base: Optional[int] = None,
                index_only: bool = False) -> Dict[str, np.ndarray]:
    """Host arrays for workload ``w``.

    Returns uint16 bfloat16 bits for ``q_idx [B,T,Hi,Di]``, ``k_idx``, ``k_cache``,
    ``v_cache`` (contiguous ``[B,max_len,H,D]`` or paged ``[P,page,H,D]``),
    ``q_layers [L,B,T,Hq,D]`` and int32 ``seq_lens [B]``, ``q_pos [B,T]`` (or
    None), ``page_table [B,max_pages]`` (or None).  ``layers`` restricts which
    layer queries are generated (default: all ``n_layers``); ``index_only`` skips
    K, V and the layer queries (they are then None)."""
    base = 1000 * w.wid if seed_base is None else seed_base
    B, T = w.batch, w.n_q
    out: Dict[str, np.ndarray] = {}
    out["q_idx"] = normal_bf16(base + 1, (B, T, w.idx_heads, w.idx_dim), 1.0 / 8.0)
    if w.page_size:
        pt = page_table_for(w, base + 7)
        P = int((pt >= 0).sum())
        rows_shape = (P, w.page_size)
        out["page_table"] = pt
    else:
        rows_shape = (B, w.max_len)
        out["page_table"] = None
    out["k_idx"] = normal_bf16(base + 2, rows_shape + (w.idx_heads, w.idx_dim), 1.0 / 8.0)
    if w.planted:
        _plant(w, out, base + 5)
    if index_only:
        out["k_cache"] = out["v_cache"] = out["q_layers"] = None
    else:
        out["k_cache"] = normal_bf16(base + 3, rows_shape + (w.kv_heads, w.head_dim), 1.0)
        out["v_cache"] = normal_bf16(base + 4, rows_shape + (w.kv_heads, w.head_dim), 1.0)
        ls = list(range(w.n_layers)) if layers is None else list(layers)
        ql = np.empty((len(ls), B, T, w.q_heads, w.head_dim), dtype=np.uint16)
        for i, l in enumerate(ls):
            ql[i] = normal_bf16(base + 100 + l, (B, T, w.q_heads, w.head_dim), 1.0)
        out["q_layers"] = ql
    out["seq_lens"] = np.asarray(w.lens, dtype=np.int32)
    if w.causal:
        p0 = w.q_pos0 if w.q_pos0 is not None else [n - T for n in w.lens]
        out["q_pos"] = (np.asarray(p0, dtype=np.int32)[:, None]
                        + np.arange(T, dtype=np.int32)[None, :]).astype(np.int32)
    else:
        out["q_pos"] = None
    return out


def _token_row(w: Workload, pt: Optional[np.ndarray], b: int, j: int):
    if pt is None:
        return (b, j)
    return (int(pt[b, j // w.page_size]), j % w.page_size)


def _plant(w: Workload, arrs: Dict[str, np.ndarray], seed: int) -> None:
    """Add +3*(1/8)*q_hat to the index keys of ``w.planted`` distinct positions per sequence."""
    g = np.random.Generator(np.random.PCG64(seed))
    kid = arrs["k_idx"]
    pt = arrs["page_table"]
    for b in range(w.batch):
        q = f32_from_bf16_bits(arrs["q_idx"][b, 0]).astype(np.float64).reshape(-1)
        nrm = float(np.sqrt((q * q).sum()))
        if nrm == 0.0:
            continue
        qhat = (q / nrm).reshape(w.idx_heads, w.idx_dim)
        pos = g.choice(w.lens[b], size=min(w.planted, w.lens[b]), replace=False)
        for j in pos:
            r = _token_row(w, pt, b, int(j))
            row = f32_from_bf16_bits(kid[r]).astype(np.float64)
            kid[r] = bf16_bits_from_f32((row + 3.0 * (1.0 / 8.0) * qhat).astype(np.float32))


def planted_positions(w: Workload, seed_base: Optional[int] = None) -> np.ndarray:
    """The planted positions [B, planted] that ``make_inputs`` used (same seed stream)."""
    base = 1000 * w.wid if seed_base is None else seed_base
    g = np.random.Generator(np.random.PCG64(base + 5))
    return np.stack([g.choice(w.lens[b], size=min(w.planted, w.lens[b]), replace=False)
                     for b in range(w.batch)])


def small_workload(name: str = "small", *, batch: int = 2, lens=(300, 777), top_k: int = 64,
                   n_layers: int = 2, n_q: int = 1, page_size: int = 0, causal: bool = False,
                   q_pos0=None, q_heads: int = 32, kv_heads: int = 8, wid: int = 900) -> Workload:
    """A small workload that the oracle finishes in well under a second."""
    return Workload(name, wid, batch, list(lens), top_k, n_layers, n_q=n_q, q_heads=q_heads,
                    kv_heads=kv_heads, page_size=page_size, causal=causal,
                    q_pos0=None if q_pos0 is None else list(q_pos0))


def random_scores(seed: int, rows: int, n: int, *, ties: float = 0.0, levels: int = 0
                  ) -> np.ndarray:
    """float32 score rows [rows, n] ~ N(0, 0.25^2) for stand-alone top-k tests.

    ``levels`` > 0 quantises the scores onto that many distinct values (many exact
    ties); ``ties`` in (0,1] copies that fraction of entries from a random other
    entry of the same row (scattered exact ties)."""
    g = np.random.Generator(np.random.PCG64(seed))
    s = (g.standard_normal((rows, n), dtype=np.float32) * np.float32(0.25))
    if levels:
        s = np.round(s * levels) / np.float32(levels)
        s = s.astype(np.float32)
    if ties > 0 and n > 1:
        m = g.random((rows, n)) < ties
        src = g.integers(0, n, size=(rows, n))
        r = np.arange(rows)[:, None].repeat(n, 1)
        s[m] = s[r[m], src[m]]
    return np.ascontiguousarray(s, dtype=np.float32)
