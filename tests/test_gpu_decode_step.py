"""GPU parity of the whole step (clsa_decode_step) against the oracle: one index
pass, one top-k, L layers sharing that index set.

Index sets: rows whose exact k-th / (k+1)-th score gap is at least 1e-5 relative
must match the oracle exactly; rows inside that tie band must hold a valid top-k
(counted and printed).  Attention outputs are compared on every row whose set
matches: max |d| <= 2e-2, mean |d| <= 2e-3 against the fp64 oracle."""
import dataclasses

import numpy as np
import pytest

import oracle as orc
from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _gpu_step(w, x, n_layers, ws_fill=None):
    """One step through clsa_decode_step; ws_fill: a byte the workspace is
    filled with first (None: whatever the allocator hands out)."""
    import torch
    from paper_2606_06467_amd import binding as B
    d = U.to_dev(x)
    sh = U.shape_of(w)
    L = n_layers
    out = torch.full((L, w.batch, w.n_q, w.q_heads, w.head_dim), float("nan"),
                     dtype=torch.bfloat16, device="cuda")
    lse = torch.full((L, w.batch, w.n_q, w.q_heads), float("nan"), device="cuda")
    idx = torch.full((w.batch, w.n_q, w.top_k), -7, dtype=torch.int32, device="cuda")
    ns = torch.full((w.batch, w.n_q), -7, dtype=torch.int32, device="cuda")
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L)
    if ws is not None and ws_fill is not None:
        ws.fill_(ws_fill)
    B.clsa_decode_step(sh, d["q_idx"], d["k_idx"], d["k_cache"], d["v_cache"], d["page_table"],
                       d["seq_lens"], d["q_pos"], d["q_layers"], out, lse, idx, ns, ws)
    torch.cuda.synchronize()
    return (B.bits_from_bf16(out), lse.cpu().numpy().astype(np.float64), idx.cpu().numpy(),
            ns.cpu().numpy())


def _check_step(w, x, check_layers, what):
    L = x["q_layers"].shape[0]
    out, lse, gidx, gns = _gpu_step(w, x, L)
    sh = orc.shape_of(w)
    scores = orc.index_scores(sh, x["q_idx"], x["k_idx"], x["seq_lens"], x["q_pos"],
                              x["page_table"])
    oidx, ons = orc.topk(sh, scores.astype(np.float32), x["seq_lens"], x["q_pos"])
    rows, in_band, differ = U.check_index_sets(w, sh, scores, gidx, gns, x["seq_lens"],
                                               x["q_pos"], ref=(oidx, ons),
                                               bound=U.higham_bound(w, x))
    U.log(f"  step {what}: {rows} rows, {in_band} in the tie band, {differ} of them differ, "
          f"0 differ outside it")
    same = np.array([[np.array_equal(gidx[b, t], oidx[b, t]) for t in range(w.n_q)]
                     for b in range(w.batch)])
    for l in check_layers:
        ro, rl = orc.sparse_attn(sh, x["q_layers"][l], x["k_cache"], x["v_cache"], oidx, ons,
                                 x["page_table"])
        U.compare_attn(out[l], lse[l], ro, rl, mask_rows=same, what=f"{what} layer {l}")
    return gidx, gns, out


def test_decode_b1_n4k_all_layers():
    w = inputs.workload("decode_b1_n4k")
    x = inputs.make_inputs(w)
    _check_step(w, x, range(w.n_layers), w.name)


def test_small_ragged_with_short_rows():
    w = inputs.small_workload(batch=4, lens=(5000, 100, 0, 2049), top_k=2048, n_layers=3, wid=91)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(3), "ragged small")


@pytest.mark.parametrize("q_heads,kv_heads,page_size", [(8, 8, 0), (16, 8, 0), (40, 8, 0),
                                                    (64, 8, 0), (32, 4, 0), (40, 8, 64)])
def test_step_group_sizes_in_kernel_merge(q_heads, kv_heads, page_size):
    """Every GQA group size through the step, whose attention merges its splits
    inside the kernel (the last split of each (row, KV head) to arrive): one
    wave per query head for G <= 4, several heads per wave for G = 5 and 8;
    rows with every split holding tokens next to rows whose short index sets
    fill only some of the splits, and an empty row; every layer compared."""
    # paged caches take at most 8 splits (the in-kernel merge) from 128 (row, KV
    # head) units on: 16 sequences; (32, 4) plans 16 splits and merges in a
    # second launch
    lens = (9000, 700, 0, 5000) if page_size == 0 else (
        9000, 700, 0, 5000, 3100, 8100, 1024, 1025, 6000, 2047, 4500, 7777, 300, 9999, 2600, 5100)
    w = inputs.small_workload(batch=len(lens), lens=lens, top_k=1024, n_layers=2,
                              q_heads=q_heads, kv_heads=kv_heads, page_size=page_size, wid=97)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(w.n_layers), f"group {q_heads // kv_heads} kv {kv_heads} page {page_size}")


def test_single_layer_gathers_from_the_cache():
    """With one layer the step attends straight from the cache (no compact copy)."""
    w = inputs.small_workload(batch=3, lens=(9000, 2500, 4000), top_k=1024, n_layers=1, wid=94)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(1), "one layer")
    wp = inputs.small_workload(batch=2, lens=(9000, 2500), top_k=1024, n_layers=1, page_size=64,
                               wid=95)
    _check_step(wp, inputs.make_inputs(wp), range(1), "one layer paged")


def test_small_paged():
    w = inputs.small_workload(batch=3, lens=(7000, 3000, 64), top_k=1024, page_size=64, n_layers=2,
                              wid=92)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(2), "paged small")


def test_chunked_prefill_small():
    w = inputs.small_workload(batch=1, lens=(6000,), n_q=64, causal=True, q_pos0=(5936,),
                              top_k=512, n_layers=2, wid=93)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(2), "prefill 64 rows")


def test_deterministic_bits():
    w = inputs.workload("decode_b1_n4k")
    x = inputs.make_inputs(w)
    a = _gpu_step(w, x, w.n_layers)
    b = _gpu_step(w, x, w.n_layers)
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("kind", ["prefill", "decode"])
def test_workspace_contents_do_not_matter(kind):
    """The workspace carries nothing from one call to the next: filled with one
    bits (NaN scores, counts and counters at their maximum) or with zero bits
    before the step, it gives the same bits as a freshly allocated one.  prefill:
    600 causal rows through the two-pass top-k (forty rows with a zero index
    query finish the slow way) and the many-unit attention with its in-kernel
    merge; decode: four long rows through the coarse histogram and the wide
    top-k."""
    if kind == "prefill":
        w = inputs.small_workload(batch=2, lens=(20000, 20000), n_q=300, causal=True,
                                  q_pos0=(19700, 19700), top_k=256, n_layers=2, wid=87)
        x = inputs.make_inputs(w)
        x["q_idx"][0, :40] = 0
        assert w.batch * w.n_q > 128 and w.batch * w.n_q * w.kv_heads >= 4096
    else:
        w = inputs.small_workload(batch=4, lens=(60000, 45000, 30001, 52000), top_k=2048,
                                  n_layers=2, wid=88)
        x = inputs.make_inputs(w)
    ref = _gpu_step(w, x, w.n_layers)
    for fill in (0xFF, 0x00):
        U.log(f"  {kind}: workspace filled with {fill:#04x}")
        got = _gpu_step(w, x, w.n_layers, ws_fill=fill)
        for u, v in zip(ref, got):
            np.testing.assert_array_equal(u, v)


def test_full_decode_b4_n128k_planted():
    w = inputs.workload("decode_b4_n128k_planted")
    x = inputs.make_inputs(w)
    gidx, gns, _ = _check_step(w, x, range(w.n_layers), w.name)
    pos = inputs.planted_positions(w)
    frac = np.mean([np.isin(pos[b], gidx[b, 0]).mean() for b in range(w.batch)])
    U.log(f"  planted positions selected: {frac:.3f}")
    assert frac > 0.5


def test_tie_band_statistics_128k_planted_many_seeds():
    """Index sets of the 128K planted step over 16 input seeds (64 rows; the index
    pass and the top-k of clsa_decode_step, with no layers): every row outside
    the tie band matches the oracle exactly; the rows inside it are counted and,
    where they differ, checked to hold a valid top-k of the exact scores."""
    import torch
    from paper_2606_06467_amd import binding as B
    w = inputs.workload("decode_b4_n128k_planted")
    sh, shg = orc.shape_of(w), U.shape_of(w)
    ws = B.workspace(shg, B.CLSA_OP_DECODE, 0)
    tot = np.zeros(3, np.int64)
    for s in range(16):
        x = inputs.make_inputs(w, seed_base=1000 * w.wid + 30000 * (s + 1), index_only=True)
        d = U.to_dev(x)
        idx = torch.full((w.batch, w.n_q, w.top_k), -7, dtype=torch.int32, device="cuda")
        ns = torch.full((w.batch, w.n_q), -7, dtype=torch.int32, device="cuda")
        B.clsa_decode_step(shg, d["q_idx"], d["k_idx"], None, None, d["page_table"],
                           d["seq_lens"], d["q_pos"], None, None, None, idx, ns, ws)
        torch.cuda.synchronize()
        scores = orc.index_scores(sh, x["q_idx"], x["k_idx"], x["seq_lens"], x["q_pos"],
                                  x["page_table"])
        tot += U.check_index_sets(w, sh, scores, idx.cpu().numpy(), ns.cpu().numpy(),
                                  x["seq_lens"], x["q_pos"], bound=U.higham_bound(w, x))
    U.log(f"  tie band, 128K planted, 16 seeds: {tot[0]} rows, {tot[1]} in the band, "
          f"{tot[2]} of them differ, 0 differ outside it")


def test_full_decode_b8_n32k():
    w = inputs.workload("decode_b8_n32k")
    x = inputs.make_inputs(w)
    _check_step(w, x, range(w.n_layers), w.name)


def test_full_decode_b32_ragged_paged():
    w = inputs.workload("decode_b32_ragged_paged")
    x = inputs.make_inputs(w)
    _check_step(w, x, range(w.n_layers), w.name)


def test_chunked_prefill_many_rows_chain():
    """More than 128 query rows through the whole step: the matrix-core indexer,
    the per-row top-k (including rows whose causal prefix holds no more than k
    keys, which select their whole prefix) and the key-range split attention
    (at least 4096 (row, KV head) units), every row and layer compared."""
    w = inputs.small_workload(batch=2, lens=(20000, 20000), n_q=512, causal=True,
                              q_pos0=(1800, 19488), top_k=2048, n_layers=2, wid=81)
    x = inputs.make_inputs(w)
    assert w.batch * w.n_q > 128 and w.batch * w.n_q * w.kv_heads >= 4096
    n = np.minimum(x["q_pos"] + 1, np.asarray(w.lens)[:, None])
    assert (n <= w.top_k).sum() > 100 and (n > w.top_k).sum() > 100
    gidx, gns, _ = _check_step(w, x, range(w.n_layers), "prefill 1024 rows")
    short = n <= w.top_k
    np.testing.assert_array_equal(gns[short], n[short])


@pytest.mark.parametrize("page_size,top_k,length", [(64, 256, 20000), (0, 40, 20000),
                                                    (0, 256, 20000), (0, 4096, 9000),
                                                    (0, 512, 140000)])
def test_chunked_prefill_many_rows_shapes(page_size, top_k, length):
    """More than 128 causal rows: the two-pass top-k (long rows next to short
    ones, whose dense candidates send them to the exact fallback) with paged
    and contiguous caches and small k, a k above 2048 (the top-k over full
    score rows), and a cache above 131072 tokens (more than 4096 samples per
    row: the 512-thread sampled-threshold workgroup); every row and layer
    compared."""
    w = inputs.small_workload(batch=2, lens=(length, length - 2000), n_q=96, causal=True,
                              q_pos0=(length - 96, 1500), top_k=top_k, n_layers=1,
                              page_size=page_size, wid=86)
    x = inputs.make_inputs(w)
    _check_step(w, x, range(1), f"prefill rows page {page_size} k {top_k}")


def test_chunked_prefill_candidate_fallback_rows():
    """The two-pass chunked-prefill top-k on rows whose candidates cannot decide
    the set, which their workgroups finish from recomputed scores: rows with a
    zero index query (every score 0: more candidates than the list holds; ties
    go to the lowest positions) and rows whose index keys at every 32nd
    position are aligned with their query (the sampled threshold is high, so
    fewer than k keys reach it), next to ordinary rows."""
    w = inputs.small_workload(batch=2, lens=(20000, 20000), n_q=160, causal=True,
                              q_pos0=(19840, 19840), top_k=256, n_layers=1, wid=85)
    x = inputs.make_inputs(w)
    q = x["q_idx"]
    q[0, :40] = 0                               # all-equal rows
    shared = q[1, 0].copy()                     # rows 40..79 of sequence 1 share one query
    q[1, 40:80] = shared
    qf = inputs.f32_from_bf16_bits(shared).astype(np.float64).reshape(-1)
    qhat = (qf / np.sqrt((qf * qf).sum())).reshape(4, 64)
    k1 = inputs.f32_from_bf16_bits(x["k_idx"][1, 0:20000:32]).astype(np.float64)
    x["k_idx"][1, 0:20000:32] = inputs.bf16_bits_from_f32((k1 + 4.0 * qhat / 8.0).astype(np.float32))
    gidx, gns, _ = _check_step(w, x, range(1), "prefill fallback rows")
    np.testing.assert_array_equal(gidx[0, :40], np.broadcast_to(np.arange(256), (40, 256)))


def test_many_single_query_rows():
    """160 decode rows (more than 128, some longer than 16384 keys): the
    per-row top-k fed by the decode indexer's coarse histograms, with empty
    rows, rows with fewer keys than k, exactly k and k + 1 keys."""
    g = np.random.default_rng(82)
    lens = [int(v) for v in g.integers(500, 20000, size=160)]
    lens[:4] = [0, 1024, 1025, 700]
    w = inputs.small_workload(batch=160, lens=lens, top_k=1024, n_layers=2, wid=82)
    x = inputs.make_inputs(w)
    gidx, gns, _ = _check_step(w, x, range(w.n_layers), "160 single-query rows")
    assert gns[0, 0] == 0 and gns[1, 0] == 1024 and gns[2, 0] == 1024 and gns[3, 0] == 700


def _slice_rows(w, x, rows):
    """The workload restricted to query rows ``rows`` of its one sequence (same
    caches and layers; each row keeps its own causal position)."""
    rows = np.asarray(rows)
    ws = dataclasses.replace(w, n_q=len(rows), q_pos0=None)
    xs = dict(x, q_idx=np.ascontiguousarray(x["q_idx"][:, rows]),
              q_layers=np.ascontiguousarray(x["q_layers"][:, :, rows]),
              q_pos=np.ascontiguousarray(x["q_pos"][:, rows]))
    return ws, xs


def test_full_prefill_t8k_n128k_sampled_rows():
    """The whole chunked-prefill step at full size (8192 causal rows over a
    131072-token cache, 16 layers) through clsa_decode_step; sampled rows (block
    edges and seeded rows) are compared with the oracle run on those rows alone:
    index sets bit-exact outside the tie band, every layer's output within the
    attention tolerances."""
    import torch
    from paper_2606_06467_amd import binding as B
    w = inputs.workload("prefill_t8k_n128k")
    x = inputs.make_inputs(w)
    g = np.random.default_rng(4004)
    rows = sorted(set([0, 15, 16, 127, 128, 4095, 4096, 8191] +
                      [int(v) for v in g.choice(w.n_q, size=16, replace=False)]))
    d = U.to_dev(x)
    sh = U.shape_of(w)
    L = w.n_layers
    out = torch.full((L, w.batch, w.n_q, w.q_heads, w.head_dim), float("nan"),
                     dtype=torch.bfloat16, device="cuda")
    lse = torch.full((L, w.batch, w.n_q, w.q_heads), float("nan"), device="cuda")
    idx = torch.full((w.batch, w.n_q, w.top_k), -7, dtype=torch.int32, device="cuda")
    ns = torch.full((w.batch, w.n_q), -7, dtype=torch.int32, device="cuda")
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L)
    U.log(f"  prefill_t8k_n128k: full step on the GPU, rows compared {rows}")
    B.clsa_decode_step(sh, d["q_idx"], d["k_idx"], d["k_cache"], d["v_cache"], d["page_table"],
                       d["seq_lens"], d["q_pos"], d["q_layers"], out, lse, idx, ns, ws)
    torch.cuda.synchronize()
    del ws
    r = torch.as_tensor(rows, device="cuda")
    g_out = B.bits_from_bf16(out[:, :, r].contiguous())
    g_lse = lse[:, :, r].cpu().numpy().astype(np.float64)
    gidx, gns = idx[:, r].cpu().numpy(), ns[:, r].cpu().numpy()
    del out, lse, idx, ns, d
    torch.cuda.empty_cache()
    assert np.all(gns == w.top_k)
    ws_, xs = _slice_rows(w, x, rows)
    osh = orc.shape_of(ws_)
    scores = orc.index_scores(osh, xs["q_idx"], xs["k_idx"], xs["seq_lens"], xs["q_pos"])
    oidx, ons = orc.topk(osh, scores.astype(np.float32), xs["seq_lens"], xs["q_pos"])
    nr, in_band, differ = U.check_index_sets(ws_, osh, scores, gidx, gns, xs["seq_lens"],
                                             xs["q_pos"], ref=(oidx, ons),
                                             bound=U.higham_bound(ws_, xs))
    U.log(f"  prefill sampled rows: {nr} rows, {in_band} in the tie band, {differ} of them "
          f"differ, 0 differ outside it")
    same = np.array([[np.array_equal(gidx[0, t], oidx[0, t]) for t in range(len(rows))]])
    assert same.sum() >= len(rows) - in_band
    for l in range(L):
        ro, rl = orc.sparse_attn(osh, xs["q_layers"][l], xs["k_cache"], xs["v_cache"], oidx, ons)
        U.compare_attn(g_out[l], g_lse[l], ro, rl, mask_rows=same, what=f"prefill layer {l}")


def test_device_error_bits_for_out_of_range_lengths():
    """seq_lens outside [0, max_len] are clamped (the step equals the one with
    clamped lengths) and raise CLSA_DEVERR_SEQ_LEN; n_sel outside [0, top_k] is
    clamped by the attention and raises CLSA_DEVERR_N_SEL; reading clears them."""
    import torch
    from paper_2606_06467_amd import binding as B
    w = inputs.small_workload(batch=3, lens=(3000, 3000, 0), top_k=512, n_layers=1, wid=83)
    x = inputs.make_inputs(w)
    B.clsa_get_device_error()                       # clear what earlier calls may have raised
    assert B.clsa_get_device_error() == 0
    ref = _gpu_step(w, x, 1)
    assert B.clsa_get_device_error() == 0
    bad = dict(x, seq_lens=np.array([w.max_len + 7, 3000, -5], np.int32))
    got = _gpu_step(w, bad, 1)
    assert B.clsa_get_device_error() == B.CLSA_DEVERR_SEQ_LEN
    assert B.clsa_get_device_error() == 0
    for u, v in zip(ref, got):
        np.testing.assert_array_equal(u, v)
    # n_sel past top_k on a stand-alone attention call
    d = U.to_dev(x)
    sh = U.shape_of(w)
    idx = torch.from_numpy(ref[2]).cuda()
    ns = torch.from_numpy(ref[3]).cuda()
    ws = B.workspace(sh, B.CLSA_OP_ATTN)
    q = d["q_layers"][0].contiguous()
    o1 = torch.empty_like(q)
    o2 = torch.empty_like(q)
    B.clsa_sparse_attn(sh, q, d["k_cache"], d["v_cache"], None, idx, ns, o1, None, ws)
    ns_bad = ns.clone()
    ns_bad[0, 0] = w.top_k + 9
    ns_full = ns.clone()
    ns_full[0, 0] = w.top_k
    B.clsa_sparse_attn(sh, q, d["k_cache"], d["v_cache"], None, idx, ns_bad, o2, None, ws)
    assert B.clsa_get_device_error() == B.CLSA_DEVERR_N_SEL
    B.clsa_sparse_attn(sh, q, d["k_cache"], d["v_cache"], None, idx, ns_full, o1, None, ws)
    assert B.clsa_get_device_error() == 0
    np.testing.assert_array_equal(B.bits_from_bf16(o1), B.bits_from_bf16(o2))


def test_concurrent_host_threads():
    """Four host threads, each with its own stream, workspace and outputs, run
    the step at the same time; every result equals the serial one bit for bit."""
    import threading
    import torch
    from paper_2606_06467_amd import binding as B
    ws_ = [inputs.small_workload(batch=2, lens=(6000 + 700 * i, 2500), top_k=1024, n_layers=2,
                                 page_size=64 if i % 2 else 0, wid=84 + i) for i in range(4)]
    xs = [inputs.make_inputs(w) for w in ws_]
    serial = [_gpu_step(w, x, 2) for w, x in zip(ws_, xs)]
    devs = [U.to_dev(x) for x in xs]
    results = [None] * 4
    errors = []

    def run(i):
        try:
            w, d = ws_[i], devs[i]
            sh = U.shape_of(w)
            st = torch.cuda.Stream()
            out = torch.empty((2, w.batch, 1, w.q_heads, w.head_dim), dtype=torch.bfloat16,
                              device="cuda")
            lse = torch.empty((2, w.batch, 1, w.q_heads), device="cuda")
            idx = torch.empty((w.batch, 1, w.top_k), dtype=torch.int32, device="cuda")
            ns = torch.empty((w.batch, 1), dtype=torch.int32, device="cuda")
            ws = B.workspace(sh, B.CLSA_OP_DECODE, 2)
            torch.cuda.synchronize()
            for _ in range(5):
                B.clsa_decode_step(sh, d["q_idx"], d["k_idx"], d["k_cache"], d["v_cache"],
                                   d["page_table"], d["seq_lens"], d["q_pos"], d["q_layers"],
                                   out, lse, idx, ns, ws, st)
            st.synchronize()
            results[i] = (B.bits_from_bf16(out), lse.cpu().numpy().astype(np.float64),
                          idx.cpu().numpy(), ns.cpu().numpy())
        except Exception as e:  # reported below
            errors.append(repr(e))

    th = [threading.Thread(target=run, args=(i,)) for i in range(4)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors, errors
    for a, b in zip(serial, results):
        for u, v in zip(a, b):
            np.testing.assert_array_equal(u, v)


def _grouped(w, q_idx_sets, k_idx_sets, x, group, stride_q, stride_k):
    import torch
    from paper_2606_06467_amd import binding as B
    d = U.to_dev(x)
    qi, ki = B.bf16_from_bits(q_idx_sets), B.bf16_from_bits(k_idx_sets)
    L = x["q_layers"].shape[0]
    n_sets = max(1, -(-L // group))
    out = torch.full((L, w.batch, w.n_q, w.q_heads, w.head_dim), float("nan"),
                     dtype=torch.bfloat16, device="cuda")
    lse = torch.full((L, w.batch, w.n_q, w.q_heads), float("nan"), device="cuda")
    idx = torch.full((n_sets, w.batch, w.n_q, w.top_k), -7, dtype=torch.int32, device="cuda")
    ns = torch.full((n_sets, w.batch, w.n_q), -7, dtype=torch.int32, device="cuda")
    sh = U.shape_of(w)
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L)
    B.clsa_decode_step_grouped(sh, qi, stride_q, ki, stride_k, d["k_cache"], d["v_cache"],
                               d["page_table"], d["seq_lens"], d["q_pos"], group, d["q_layers"],
                               out, lse, idx, ns, ws)
    torch.cuda.synchronize()
    return (B.bits_from_bf16(out), lse.cpu().numpy().astype(np.float64), idx.cpu().numpy(),
            ns.cpu().numpy())


def test_grouped_fresh_routing_per_layer():
    """group = 1 with a different indexer per layer: layer l attends over the set
    its own index keys select (per-layer routing)."""
    w = inputs.small_workload(batch=2, lens=(5000, 3100), top_k=512, n_layers=3, wid=96)
    x = inputs.make_inputs(w)
    sets = [inputs.make_inputs(w, seed_base=1000 * w.wid + 10000 * (s + 1), index_only=True)
            for s in range(3)]
    q_sets = np.stack([s_["q_idx"] for s_ in sets])
    k_sets = np.stack([s_["k_idx"] for s_ in sets])
    out, lse, gidx, gns = _grouped(w, q_sets, k_sets, x, 1, q_sets[0].size, k_sets[0].size)
    sh = orc.shape_of(w)
    for l in range(3):
        scores = orc.index_scores(sh, q_sets[l], k_sets[l], x["seq_lens"], x["q_pos"],
                                  x["page_table"])
        oidx, ons = orc.topk(sh, scores.astype(np.float32), x["seq_lens"], x["q_pos"])
        U.check_index_sets(w, sh, scores, gidx[l], gns[l], x["seq_lens"], x["q_pos"],
                           ref=(oidx, ons), bound=U.higham_bound(w, dict(x, q_idx=q_sets[l],
                                                                          k_idx=k_sets[l])))
        same = np.array([[np.array_equal(gidx[l][b, t], oidx[b, t]) for t in range(w.n_q)]
                         for b in range(w.batch)])
        ro, rl = orc.sparse_attn(sh, x["q_layers"][l], x["k_cache"], x["v_cache"], oidx, ons,
                                 x["page_table"])
        U.compare_attn(out[l], lse[l], ro, rl, mask_rows=same, what=f"per-layer routing l={l}")


def test_grouped_reused_keys_match_the_shared_step():
    """group = 2 over 3 layers with the same index keys for both sets: every set
    and every layer output equals the shared-routing step's, bit for bit."""
    w = inputs.small_workload(batch=3, lens=(4000, 2500, 700), top_k=1024, n_layers=3,
                              page_size=64, wid=97)
    x = inputs.make_inputs(w)
    out0, lse0, idx0, ns0 = _gpu_step(w, x, 3)
    out, lse, gidx, gns = _grouped(w, x["q_idx"], x["k_idx"], x, 2, 0, 0)
    for s in range(2):
        np.testing.assert_array_equal(gidx[s], idx0)
        np.testing.assert_array_equal(gns[s], ns0)
    np.testing.assert_array_equal(out, out0)
    np.testing.assert_array_equal(lse, lse0)
