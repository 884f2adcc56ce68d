"""Helpers for the GPU parity tests: move seeded inputs to the device, run the
library through its binding, and compare with the oracle.

Nothing here feeds a GPU result into the oracle: the oracle only ever sees the
generator's arrays."""
from __future__ import annotations

import os
import sys
import numpy as np

import oracle as orc
from paper_2606_06467_amd import inputs

# The oracle's results do not depend on its thread count (tests/test_oracle_threads.py);
# threads only shorten the full-size parity cases.
try:
    _CPUS = len(os.sched_getaffinity(0))
except (AttributeError, OSError):
    _CPUS = os.cpu_count() or 1
orc.set_threads(max(1, min(16, _CPUS)))

# Tolerances for bf16 inputs against the fp64 oracle (attention outputs).
ATTN_MAX_ABS = 2e-2
ATTN_MEAN_ABS = 2e-3
LSE_MAX_ABS = 1e-3
# Relative k-th / (k+1)-th score gap below which a row's set may depend on rounding order.
TIE_BAND = 1e-5
U32 = 2.0 ** -24


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x):
    import torch
    from paper_2606_06467_amd import binding as B
    d = {}
    for k, v in x.items():
        if v is None:
            d[k] = None
        elif v.dtype == np.uint16:
            d[k] = B.bf16_from_bits(v)
        else:
            d[k] = torch.from_numpy(np.ascontiguousarray(v)).cuda()
    return d


def shape_of(w, **over):
    from paper_2606_06467_amd import binding as B
    kw = dict(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k, idx_heads=w.idx_heads,
              idx_dim=w.idx_dim, q_heads=w.q_heads, kv_heads=w.kv_heads, head_dim=w.head_dim,
              page_size=w.page_size, max_pages=w.max_pages, causal=w.causal)
    kw.update(over)
    return B.make_shape(**kw)


def higham_bound(w, x) -> np.ndarray:
    """gamma_256 * sum_i |q_i k_i| per (b, t, j): a bound on any fp32 summation order."""
    B, T = w.batch, w.n_q
    q = np.abs(inputs.f32_from_bf16_bits(x["q_idx"]).astype(np.float64)).reshape(B, T, -1)
    kk = np.abs(inputs.f32_from_bf16_bits(x["k_idx"]).astype(np.float64))
    d = q.shape[-1]
    gamma = d * U32 / (1 - d * U32)
    out = np.zeros((B, T, w.max_len))
    for b in range(B):
        if w.page_size:
            pt = x["page_table"][b]
            n = w.lens[b]
            pages = pt[: (n + w.page_size - 1) // w.page_size]
            kb = kk[pages].reshape(-1, d)[:n]
        else:
            kb = kk[b, : w.lens[b]].reshape(-1, d)
        out[b, :, : kb.shape[0]] = q[b] @ kb.T
    return gamma * out + 1e-30


def check_index_sets(w, sh_orc, scores64, gpu_idx, gpu_nsel, seq_lens, q_pos=None, ref=None,
                     bound=None):
    """Compare GPU index sets with the oracle's.

    Rows outside the tie band must match exactly; rows inside it must hold a valid
    top-k of the exact scores (every kept score >= every dropped score, up to the
    score error bound).  Returns (rows, in_band, in_band_differing)."""
    s32 = scores64.astype(np.float32)
    if ref is None:
        ref = orc.topk(sh_orc, s32, seq_lens, q_pos)
    oidx, onsel = ref
    nvalid = orc.valid_lens(sh_orc, seq_lens, q_pos)
    gap = orc.kth_gap(scores64, nvalid, w.top_k)
    np.testing.assert_array_equal(gpu_nsel, onsel)
    rows = gap.size
    in_band = 0
    differ = 0
    for r in np.ndindex(gap.shape):
        same = np.array_equal(gpu_idx[r], oidx[r])
        if gap[r] < TIE_BAND:
            in_band += 1
            if not same:
                differ += 1
                n = int(nvalid[r])
                m = int(gpu_nsel[r])
                sel = gpu_idx[r][:m]
                assert np.all(np.diff(sel) > 0) and sel.min() >= 0 and sel.max() < n
                assert np.all(gpu_idx[r][m:] == -1)
                mask = np.zeros(n, bool)
                mask[sel] = True
                s = scores64[r][:n]
                tol = 2 * (bound[r][:n].max() if bound is not None else 1e-6)
                assert s[mask].min() >= s[~mask].max() - tol, r
        else:
            assert same, f"row {r} outside the tie band (gap {gap[r]:.3g}) differs"
    return rows, in_band, differ


def compare_attn(out_gpu_bf16, lse_gpu, out_ref, lse_ref, mask_rows=None, what=""):
    """bf16 GPU output vs fp64 oracle output; optional boolean mask of rows to compare."""
    o = inputs.f32_from_bf16_bits(out_gpu_bf16).astype(np.float64)
    if mask_rows is not None:
        o, out_ref = o[mask_rows], out_ref[mask_rows]
        if lse_gpu is not None:
            lse_gpu, lse_ref = lse_gpu[mask_rows], lse_ref[mask_rows]
    err = np.abs(o - out_ref)
    mx, mean = float(err.max(initial=0.0)), float(err.mean()) if err.size else 0.0
    log(f"  attn {what}: max|d|={mx:.3e} mean|d|={mean:.3e} over {err.size} values")
    assert np.isfinite(o).all()
    assert mx <= ATTN_MAX_ABS, (what, mx)
    assert mean <= ATTN_MEAN_ABS, (what, mean)
    if lse_gpu is not None:
        fin = np.isfinite(lse_ref)
        assert np.array_equal(fin, np.isfinite(lse_gpu))
        if fin.any():
            d = float(np.abs(lse_gpu[fin] - lse_ref[fin]).max())
            assert d <= LSE_MAX_ABS, (what, d)
        assert np.all(lse_gpu[~fin] == -np.inf)
