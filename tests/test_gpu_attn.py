"""GPU parity of clsa_sparse_attn (Eq. 4) against the fp64 oracle on the same
index sets (made by the oracle or by the seeded generator, never by the GPU)."""
import numpy as np
import pytest

import oracle as orc
from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _random_sets(seed, rows_shape, lens, k, nsel_override=None):
    g = np.random.default_rng(seed)
    B, T = rows_shape
    idx = np.full((B, T, k), -1, np.int32)
    ns = np.zeros((B, T), np.int32)
    for b in range(B):
        for t in range(T):
            m = min(k, lens[b])
            if nsel_override is not None and nsel_override.get((b, t)) is not None:
                m = nsel_override[(b, t)]
            idx[b, t, :m] = np.sort(g.choice(lens[b], size=m, replace=False))
            ns[b, t] = m
    return idx, ns


def _run(w, x, q, idx, ns, with_lse=True):
    import torch
    from paper_2606_06467_amd import binding as B
    d = U.to_dev(x)
    sh = U.shape_of(w)
    qd = B.bf16_from_bits(q)
    out = torch.full(qd.shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full(qd.shape[:-1], float("nan"), device="cuda") if with_lse else None
    ws = B.workspace(sh, B.CLSA_OP_ATTN)
    B.clsa_sparse_attn(sh, qd, d["k_cache"], d["v_cache"], d["page_table"],
                       torch.from_numpy(idx).cuda(), torch.from_numpy(ns).cuda(), out, lse, ws)
    torch.cuda.synchronize()
    return B.bits_from_bf16(out), (lse.cpu().numpy().astype(np.float64) if with_lse else None)


def _case(w, seed, nsel_override=None, with_lse=True, what=""):
    x = inputs.make_inputs(w, layers=[0])
    idx, ns = _random_sets(seed, (w.batch, w.n_q), w.lens, w.top_k, nsel_override)
    q = x["q_layers"][0]
    out, lse = _run(w, x, q, idx, ns, with_lse)
    ref_o, ref_l = orc.sparse_attn(orc.shape_of(w), q, x["k_cache"], x["v_cache"], idx, ns,
                                   x["page_table"])
    U.compare_attn(out, lse, ref_o, ref_l, what=what)


@pytest.mark.parametrize("qh,kvh", [(32, 8), (8, 8), (16, 8), (20, 4), (64, 8)])
def test_gqa_groups(qh, kvh):
    w = inputs.small_workload(batch=2, lens=(3000, 1700), top_k=512, q_heads=qh, kv_heads=kvh,
                              n_layers=1, wid=81)
    _case(w, 1, what=f"Hq={qh} Hkv={kvh}")


@pytest.mark.parametrize("k", [1, 63, 64, 65, 2048, 8192])
def test_split_counts(k):
    w = inputs.small_workload(batch=1, lens=(9000,), top_k=k, n_layers=1, wid=82)
    _case(w, 2, what=f"k={k}")


def test_partial_and_empty_sets():
    w = inputs.small_workload(batch=3, lens=(5000, 5000, 5000), top_k=1024, n_layers=1, wid=83)
    _case(w, 3, nsel_override={(0, 0): 0, (1, 0): 37}, what="n_sel 0 / 37 / 1024")


def test_single_split_many_rows():
    """Enough rows that each (row, KV head) gets one workgroup and no merge."""
    w = inputs.small_workload(batch=1, lens=(4000,), n_q=300, causal=True, q_pos0=(3700,),
                              top_k=256, n_layers=1, wid=84)
    _case(w, 4, what="300 rows, one split each")


def test_many_rows_split_by_key_range():
    """Over 4096 (row, KV head) units: each index list is cut into stretches that
    are issued stretch by stretch over all rows, then merged."""
    w = inputs.small_workload(batch=1, lens=(4000,), n_q=520, causal=True, q_pos0=(3480,),
                              top_k=512, q_heads=8, kv_heads=8, n_layers=1, wid=87)
    _case(w, 5, what="520 rows x 8 KV heads, split by key range")


@pytest.mark.parametrize("qh,kvh,nq,k,ps", [(16, 4, 1030, 256, 0), (16, 2, 2050, 128, 64),
                                            (20, 4, 1030, 320, 64), (16, 8, 600, 512, 64)])
def test_matrix_core_logits_form(qh, kvh, nq, k, ps):
    """Over 4096 (row, KV head) units the chunked-prefill form runs (one wave per
    workgroup, rotated chunk order, logits and weighted V on the matrix cores,
    per-wave softmax states): groups of 4, 8, 5 and 2 heads, one split (k = 128)
    and several, contiguous and paged, ragged counts (0, 1, 37, 63, 65) that
    leave splits shorter than the chunk they would start from."""
    w = inputs.small_workload(batch=1, lens=(4000,), n_q=nq, causal=True, q_pos0=(4000 - nq,),
                              top_k=k, q_heads=qh, kv_heads=kvh, page_size=ps, n_layers=1,
                              wid=88)
    _case(w, 9, nsel_override={(0, 3): 37, (0, 5): 1, (0, 7): 0, (0, 8): 63, (0, 9): 65},
          what=f"matrix-core form Hq={qh} Hkv={kvh} rows={nq} k={k} page={ps}")


def test_paged():
    w = inputs.small_workload(batch=3, lens=(3000, 64, 5000), top_k=512, page_size=64, n_layers=1,
                              wid=85)
    _case(w, 5, what="paged")


def test_without_lse():
    w = inputs.small_workload(batch=2, lens=(3000, 1700), top_k=512, n_layers=1, wid=86)
    _case(w, 6, with_lse=False, what="no lse")


@pytest.mark.parametrize("case", range(10))
def test_many_unit_shape_sweep(case):
    """Seeded shapes over 4096 (row, KV head) units, where the kernel runs one
    wave per workgroup and walks each workgroup's chunks in a rotated order:
    KV heads 2, 4 or 8, groups of 1, 2, 4, 5 or 8 query heads, contiguous or
    paged caches, top-k values that are not multiples of the 16-token chunk,
    sequences shorter than k, and some rows' counts overridden (0, 1, a
    random count) so that splits end inside a chunk or hold fewer chunks than
    the one they would start from."""
    g = np.random.default_rng(9100 + case)
    kvh = (2, 4, 8)[case % 3]
    grp = (1, 2, 4, 5, 8)[case % 5]
    k = int(g.integers(17, 700))
    batch = int(g.choice([1, 2]))
    nq = -(-4096 // (kvh * batch)) + int(g.integers(0, 64))
    lens = tuple(int(v) for v in g.integers(max(k // 2, 8), 5000, size=batch))
    ps = int(g.choice([0, 64]))
    w = inputs.small_workload(batch=batch, lens=lens, n_q=nq, top_k=k, q_heads=kvh * grp,
                              kv_heads=kvh, page_size=ps, n_layers=1, wid=90 + case)
    over = {}
    for t in g.choice(nq, size=6, replace=False):
        b = int(g.integers(0, batch))
        over[(b, int(t))] = int(g.choice([0, 1, int(g.integers(0, min(k, lens[b]) + 1))]))
    what = (f"sweep {case}: B={batch} rows={nq} Hkv={kvh} G={grp} k={k} lens={lens} "
            f"page={ps}")
    U.log("  " + what)
    _case(w, 40 + case, nsel_override=over, what=what)
