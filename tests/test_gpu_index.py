"""GPU parity of clsa_index_scores (Eq. 3) against the fp64 oracle.

Every valid score must lie within Higham's bound gamma_256 * sum|q_i k_i| of the
exact value (any fp32 summation order satisfies it); positions outside the valid
prefix must not be written."""
import numpy as np
import pytest

import oracle as orc
from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _run(w, x):
    import torch
    from paper_2606_06467_amd import binding as B
    d = U.to_dev(x)
    sc = torch.full((w.batch, w.n_q, w.max_len), float("nan"), device="cuda")
    B.clsa_index_scores(U.shape_of(w), d["q_idx"], d["k_idx"], d["page_table"], d["seq_lens"],
                        d["q_pos"], sc)
    torch.cuda.synchronize()
    return sc.cpu().numpy()


def _check(w, x, got):
    ref = orc.index_scores(orc.shape_of(w), x["q_idx"], x["k_idx"], x["seq_lens"], x["q_pos"],
                           x["page_table"])
    bound = U.higham_bound(w, x)
    valid = ~np.isnan(ref)
    assert np.array_equal(valid, ~np.isnan(got)), "written positions differ from the valid set"
    err = np.abs(got[valid] - ref[valid])
    assert np.all(err <= bound[valid]), float((err / bound[valid]).max())
    U.log(f"  index {w.name}: {valid.sum()} scores, max err {err.max(initial=0):.3e}, "
          f"max err/bound {(err / bound[valid]).max(initial=0):.3f}")


# one or two short rows take fewer tiles per workgroup (1 or 2) so that the grid
# still covers the chip
@pytest.mark.parametrize("lens", [(300, 777), (1, 128), (0, 129), (4096, 4095), (65531,), (40000, 3)])
def test_contiguous_small(lens):
    w = inputs.small_workload(batch=len(lens), lens=lens, n_layers=1, wid=61)
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


@pytest.mark.parametrize("page", [16, 64, 256])
def test_paged_ragged(page):
    w = inputs.small_workload(batch=3, lens=(1000, 64, 2500), page_size=page, n_layers=1, wid=62)
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


def test_causal_rows():
    w = inputs.small_workload(batch=2, lens=(600, 900), n_q=7, causal=True, q_pos0=(300, 895),
                              n_layers=1, wid=63)
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


def test_full_size_128k_planted():
    w = inputs.workload("decode_b4_n128k_planted")
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


def test_full_size_ragged_paged():
    w = inputs.workload("decode_b32_ragged_paged")
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


# Many query rows per sequence: the scores come from the matrix-core kernel.
@pytest.mark.parametrize("batch,lens,n_q,causal,q_pos0,page", [
    (1, (6000,), 64, True, (5936,), 0),             # one chunk, causal, aligned rows
    (2, (3001, 2500), 37, True, (2964, 100), 0),    # ragged query block, unaligned rows
    (2, (4000, 1500), 150, False, None, 64),        # two query blocks, paged
    (1, (2049,), 32, False, None, 0),               # smallest row count on this path
    (3, (1100, 17, 2200), 45, True, (1055, 0, 900), 16),  # short causal rows, small pages
])
def test_many_rows_matrix_cores(batch, lens, n_q, causal, q_pos0, page):
    w = inputs.small_workload(batch=batch, lens=lens, n_q=n_q, causal=causal, q_pos0=q_pos0,
                              page_size=page, n_layers=1, wid=64)
    x = inputs.make_inputs(w, index_only=True)
    _check(w, x, _run(w, x))


def test_full_size_prefill_sampled_rows():
    """The 8192 x 131072 causal block of the chunked-prefill workload, checked on
    sampled rows (block edges, the first and last rows, seeded random rows)."""
    import dataclasses
    import torch
    from paper_2606_06467_amd import binding as B
    w = inputs.workload("prefill_t8k_n128k")
    x = inputs.make_inputs(w, index_only=True)
    d = U.to_dev(x)
    sc = torch.full((w.batch, w.n_q, w.max_len), float("nan"), device="cuda")
    B.clsa_index_scores(U.shape_of(w), d["q_idx"], d["k_idx"], d["page_table"], d["seq_lens"],
                        d["q_pos"], sc)
    torch.cuda.synchronize()
    g = np.random.default_rng(6401)
    rows = sorted(set([0, 1, 15, 16, 31, 32, 127, 128, 4095, 4096, 8190, 8191]
                      + [int(r) for r in g.choice(w.n_q, 12, replace=False)]))
    got = sc[:, rows].cpu().numpy()
    del sc
    ws = dataclasses.replace(w, n_q=len(rows))
    xs = dict(x, q_idx=np.ascontiguousarray(x["q_idx"][:, rows]),
              q_pos=np.ascontiguousarray(x["q_pos"][:, rows]))
    _check(ws, xs, got)
