"""GPU parity of clsa_dense_attn (Eq. 1 with GQA over every valid key) against
the fp64 oracle evaluated on the full index set (every valid position)."""
import numpy as np
import pytest

import oracle as orc
from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _full_sets(w, seq_lens, q_pos):
    """All valid positions of every row (the oracle's dense attention)."""
    sh = orc.shape_of(w, top_k=w.max_len)
    n = orc.valid_lens(sh, seq_lens, q_pos)
    idx = np.full((w.batch, w.n_q, w.max_len), -1, np.int32)
    for b in range(w.batch):
        for t in range(w.n_q):
            idx[b, t, :n[b, t]] = np.arange(n[b, t], dtype=np.int32)
    return sh, idx, n.astype(np.int32)


def _case(w, what):
    import torch
    from paper_2606_06467_amd import binding as B
    x = inputs.make_inputs(w, layers=[0])
    d = U.to_dev(x)
    q = B.bf16_from_bits(x["q_layers"][0])
    out = torch.full(q.shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full(q.shape[:-1], float("nan"), device="cuda")
    sh = U.shape_of(w)
    ws = B.workspace(sh, B.CLSA_OP_DENSE)
    B.clsa_dense_attn(sh, q, d["k_cache"], d["v_cache"], d["page_table"], d["seq_lens"],
                      d["q_pos"], out, lse, ws)
    torch.cuda.synchronize()
    osh, idx, n = _full_sets(w, x["seq_lens"], x["q_pos"])
    ref_o, ref_l = orc.sparse_attn(osh, x["q_layers"][0], x["k_cache"], x["v_cache"], idx, n,
                                   x["page_table"])
    U.compare_attn(B.bits_from_bf16(out), lse.cpu().numpy().astype(np.float64), ref_o, ref_l,
                   what=what)


@pytest.mark.parametrize("qh,kvh", [(32, 8), (8, 8), (20, 4), (64, 8)])
def test_gqa_groups(qh, kvh):
    w = inputs.small_workload(batch=2, lens=(3000, 1700), q_heads=qh, kv_heads=kvh, n_layers=1,
                              wid=71)
    _case(w, f"dense Hq={qh} Hkv={kvh}")


def test_paged_ragged_with_empty_sequence():
    w = inputs.small_workload(batch=3, lens=(2500, 0, 700), page_size=64, n_layers=1, wid=72)
    _case(w, "dense paged, one empty sequence")


def test_causal_rows():
    w = inputs.small_workload(batch=2, lens=(1500, 900), n_q=5, causal=True, q_pos0=(1400, 0),
                              n_layers=1, wid=73)
    _case(w, "dense causal rows")


@pytest.mark.parametrize("qh,kvh,nq,ps", [(8, 8, 520, 0), (32, 8, 520, 64), (20, 4, 1030, 0)])
def test_many_rows_split_by_key_range(qh, kvh, nq, ps):
    """Dense attention over 4096+ (row, KV head) units (the one-wave chunked-prefill
    form with its rotated chunk order), split by key range: groups of 1, 4 and 5
    heads, contiguous and paged caches."""
    w = inputs.small_workload(batch=1, lens=(1500,), n_q=nq, causal=True, q_pos0=(1500 - nq,),
                              q_heads=qh, kv_heads=kvh, page_size=ps, n_layers=1, wid=75)
    _case(w, f"dense {nq} causal rows Hq={qh} Hkv={kvh} page={ps}")


def test_many_splits_one_row():
    """One long row: the most splits the merge supports."""
    w = inputs.small_workload(batch=1, lens=(20000,), n_layers=1, wid=74)
    _case(w, "dense 20000 keys")


def test_full_size_128k():
    w = inputs.workload("decode_b4_n128k_planted")
    _case(w, "dense decode_b4_n128k_planted")
