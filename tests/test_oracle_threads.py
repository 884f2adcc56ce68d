"""The oracle's host threads change nothing: a step, and the distillation
target, computed with 1 and with several threads are bit-identical (every work
item writes only its own outputs with the same arithmetic)."""
import numpy as np
import pytest

from paper_2606_06467_amd import inputs


def _step(orc, w, x, threads):
    orc.set_threads(threads)
    try:
        return orc.decode_step(orc.shape_of(w), x["q_idx"], x["k_idx"], x["k_cache"],
                               x["v_cache"], x["seq_lens"], x["q_layers"], x["q_pos"],
                               x["page_table"])
    finally:
        orc.set_threads(1)


@pytest.mark.parametrize("case", ["ragged", "paged", "causal"])
def test_threaded_step_is_bit_identical(orc, case):
    if case == "ragged":
        w = inputs.small_workload(batch=3, lens=(9000, 100, 4500), top_k=512, n_layers=2, wid=71)
    elif case == "paged":
        w = inputs.small_workload(batch=2, lens=(5000, 3000), top_k=256, n_layers=2,
                                  page_size=64, wid=72)
    else:
        w = inputs.small_workload(batch=1, lens=(5000,), n_q=9, causal=True, q_pos0=(4991,),
                                  top_k=1024, n_layers=1, wid=73)
    x = inputs.make_inputs(w)
    one = _step(orc, w, x, 1)
    assert orc.get_threads() == 1
    for t in (3, 8):
        many = _step(orc, w, x, t)
        for key in ("scores", "idx", "n_sel", "out", "lse"):
            a, b = one[key], many[key]
            if a.dtype.kind == "f":
                fin = np.isfinite(a)
                assert np.array_equal(fin, np.isfinite(b)), key
                assert np.array_equal(a[fin], b[fin]), (key, t)   # scores beyond the valid prefix are untouched
            else:
                assert np.array_equal(a, b), (key, t)


def test_threaded_distillation_target_is_bit_identical(orc):
    w = inputs.small_workload(batch=1, lens=(300,), n_q=40, causal=True, q_pos0=(260,),
                              n_layers=2, wid=74)
    x = inputs.make_inputs(w)
    sh = orc.shape_of(w)
    ref = orc.kd_target(sh, x["q_layers"], x["k_cache"], x["seq_lens"], x["q_pos"], fill=0.0)
    orc.set_threads(6)
    try:
        got = orc.kd_target(sh, x["q_layers"], x["k_cache"], x["seq_lens"], x["q_pos"], fill=0.0)
    finally:
        orc.set_threads(1)
    assert np.array_equal(ref, got)
