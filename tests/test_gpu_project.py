"""GPU parity of clsa_project_append (Eq. 2 for new tokens, with their K / V /
index-key cache writes) against the fp64 oracle.

Tolerance: the GPU sums in fp32 (error within gamma_d * sum|h_i w_i|, Higham)
and rounds to bf16 (half an ulp, 2^-9 relative); the test allows one bf16 ulp
(2^-8 relative) plus twice the summation bound.  Cache rows that no new token
maps to must be left exactly as they were."""
import numpy as np
import pytest

import oracle as orc
from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _case(w, d_model, pos, seed, what):
    import torch
    from paper_2606_06467_amd import binding as B
    rows = w.batch * w.n_q
    kvw = w.kv_heads * w.head_dim
    n_feat = 512 + 2 * kvw
    h = inputs.normal_bf16(seed, (rows, d_model), 1.0)
    wt = inputs.normal_bf16(seed + 1, (n_feat, d_model), 0.02)
    x = inputs.make_inputs(w, layers=[0])
    d = U.to_dev(x)
    q_idx = torch.full((rows, 256), float("nan"), dtype=torch.bfloat16, device="cuda")
    pos_d = torch.from_numpy(np.asarray(pos, np.int32)).cuda()
    B.clsa_project_append(U.shape_of(w), d_model, B.bf16_from_bits(h), B.bf16_from_bits(wt),
                          pos_d, d["page_table"], q_idx, d["k_idx"], d["k_cache"], d["v_cache"])
    torch.cuda.synchronize()
    got_q = B.bits_from_bf16(q_idx)
    caches = {n: B.bits_from_bf16(d[n]) for n in ("k_idx", "k_cache", "v_cache")}

    ref, dest = orc.project(orc.shape_of(w), h, wt, np.asarray(pos, np.int32), x["page_table"])
    hf = np.abs(inputs.f32_from_bf16_bits(h).astype(np.float64))
    wf = np.abs(inputs.f32_from_bf16_bits(wt).astype(np.float64))
    gamma = d_model * U.U32 / (1 - d_model * U.U32)
    tol = np.abs(ref) * 2.0 ** -8 + 2 * gamma * (hf @ wf.T) + 1e-30

    def check(got_bits, r, c0, c1, name):
        g = inputs.f32_from_bf16_bits(got_bits).astype(np.float64)
        err = np.abs(g - ref[r, c0:c1])
        assert np.all(err <= tol[r, c0:c1]), (name, r, float((err / tol[r, c0:c1]).max()))

    for r in range(rows):
        check(got_q[r], r, 0, 256, "q_idx")
    widths = {"k_idx": 256, "k_cache": kvw, "v_cache": kvw}
    flat = {n: c.reshape(-1, widths[n]) for n, c in caches.items()}      # one row per token
    orig = {n: x[n].reshape(-1, widths[n]) for n in caches}
    untouched = {n: np.ones(flat[n].shape[0], bool) for n in caches}
    for r in range(rows):
        if dest[r] < 0:
            continue
        check(flat["k_idx"][dest[r]], r, 256, 512, "k_idx")
        check(flat["k_cache"][dest[r]], r, 512, 512 + kvw, "k")
        check(flat["v_cache"][dest[r]], r, 512 + kvw, 512 + 2 * kvw, "v")
        for n in untouched:
            untouched[n][dest[r]] = False
    for n in caches:
        np.testing.assert_array_equal(flat[n][untouched[n]], orig[n][untouched[n]])
    U.log(f"  project {what}: {rows} rows, {int((dest >= 0).sum())} cache rows written")


def test_decode_rows_appended_at_the_end():
    w = inputs.small_workload(batch=4, lens=(300, 777, 1, 64), n_layers=1, wid=101)
    _case(w, 2560, [299, 776, 0, 63], 11, "decode d=2560")


@pytest.mark.parametrize("d_model", [512, 1024, 3072, 4096])
def test_model_widths(d_model):
    w = inputs.small_workload(batch=2, lens=(100, 200), n_layers=1, wid=102)
    _case(w, d_model, [50, 199], 12, f"d={d_model}")


def test_paged_ragged_and_out_of_range_positions():
    # max_len is 2560 (2500 rounded up to whole pages): 2560 is past the end
    w = inputs.small_workload(batch=3, lens=(1000, 64, 2500), page_size=64, n_layers=1, wid=103)
    _case(w, 2560, [999, -1, 2560], 13, "paged, positions -1 and max_len not written")


def test_gqa_five_to_one():
    w = inputs.small_workload(batch=2, lens=(400, 400), q_heads=20, kv_heads=4, n_layers=1,
                              wid=104)
    _case(w, 2560, [10, 399], 14, "Hq=20 Hkv=4")


def test_many_rows_chunk():
    """A chunk of new tokens per sequence (the many-rows kernel)."""
    w = inputs.small_workload(batch=2, lens=(600, 700), n_q=100, causal=True,
                              q_pos0=(500, 600), n_layers=1, wid=105)
    pos = np.concatenate([np.arange(500, 600), np.arange(600, 700)]).astype(np.int32)
    _case(w, 1024, pos, 15, "200 rows")


def test_many_rows_tiles_ragged_paged():
    """The tiled kernel: 600 rows (four 128-row tiles and a tail of 88), paged
    caches, d_model 2560; every 50th position past the cache and one negative,
    so those rows write their index query only."""
    T = 300
    w = inputs.small_workload(batch=2, lens=(2000, 2400), n_q=T, causal=True,
                              q_pos0=(1700, 2100), page_size=64, n_layers=1, wid=106)
    pos = np.concatenate([np.arange(1700, 2000), np.arange(2100, 2400)]).astype(np.int32)
    pos[::50] = w.max_len
    pos[7] = -1
    _case(w, 2560, pos, 16, "600 rows, tiles + tail, paged")
