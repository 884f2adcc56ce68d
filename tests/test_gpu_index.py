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


@pytest.mark.parametrize("lens", [(300, 777), (1, 128), (0, 129), (4096, 4095)])
def test_contiguous_small(lens):
    w = inputs.small_workload(lens=lens, n_layers=1, wid=61)
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
