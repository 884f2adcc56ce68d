"""clsa_decode_step_noalloc: the step on the library's fixed per-device scratch,
for callers that cannot allocate.  Checked through the C-ABI against
clsa_decode_step (the same kernels on a caller workspace): two calls in a row,
the second on a smaller input, so that the second runs on whatever the first
left in the shared scratch; and a step too large for the scratch is rejected
before anything is enqueued."""
import ctypes

import numpy as np
import pytest

from paper_2606_06467_amd import inputs


def _shape(w):
    from paper_2606_06467_amd import binding as B
    return B.make_shape(batch=w.batch, n_q=w.n_q, max_len=w.max_len, top_k=w.top_k,
                        page_size=w.page_size, max_pages=w.max_pages, causal=w.causal)


def _run(w, x, noalloc):
    import torch
    from paper_2606_06467_amd import binding as B
    dev = {k: (None if v is None else (B.bf16_from_bits(v) if v.dtype == np.uint16
                                       else torch.from_numpy(np.ascontiguousarray(v)).cuda()))
           for k, v in x.items()}
    sh = _shape(w)
    L = x["q_layers"].shape[0]
    out = torch.full((L, w.batch, w.n_q, w.q_heads, w.head_dim), float("nan"),
                     dtype=torch.bfloat16, device="cuda")
    lse = torch.full((L, w.batch, w.n_q, w.q_heads), float("nan"), device="cuda")
    idx = torch.full((w.batch, w.n_q, w.top_k), -7, dtype=torch.int32, device="cuda")
    ns = torch.full((w.batch, w.n_q), -7, dtype=torch.int32, device="cuda")
    args = (sh, dev["q_idx"], dev["k_idx"], dev["k_cache"], dev["v_cache"], dev["page_table"],
            dev["seq_lens"], dev["q_pos"], dev["q_layers"], out, lse, idx, ns)
    if noalloc:
        B.clsa_decode_step_noalloc(*args)
    else:
        B.clsa_decode_step(*args, B.workspace(sh, B.CLSA_OP_DECODE, L))
    torch.cuda.synchronize()
    return (B.bits_from_bf16(out), lse.cpu().numpy(), idx.cpu().numpy(), ns.cpu().numpy())


@pytest.mark.gpu
def test_noalloc_step_matches_the_workspace_step_twice():
    big = inputs.small_workload(batch=4, lens=(70000, 12000, 40000, 5000), top_k=2048,
                                n_layers=3, wid=61)
    small = inputs.small_workload(batch=2, lens=(6000, 900), top_k=512, n_layers=2,
                                  page_size=64, wid=62)
    for w in (big, small):
        x = inputs.make_inputs(w)
        got = _run(w, x, True)
        ref = _run(w, x, False)
        for name, a, b in zip(("out", "lse", "idx", "n_sel"), got, ref):
            assert np.array_equal(a, b, equal_nan=False), (w.lens, name)
        print(f"noalloc step = workspace step, lens {w.lens}, {x['q_layers'].shape[0]} layers",
              flush=True)


def test_noalloc_rejects_steps_beyond_the_scratch():
    """A step that needs more than the fixed scratch (chunked prefill of 8192
    rows over 131072 keys needs ~5.2 GB) is rejected on the host; invalid shapes
    keep their usual status."""
    from paper_2606_06467_amd import binding as B
    lib = B.lib()
    A = ctypes.c_void_p(1 << 20)
    w = inputs.workload("prefill_t8k_n128k")
    sh = _shape(w)
    assert B.clsa_workspace_bytes(sh, B.CLSA_OP_DECODE, 16) > B.CLSA_NOALLOC_SCRATCH_BYTES
    st = lib.clsa_decode_step_noalloc(ctypes.byref(sh), A, A, A, A, None, A, A, 16, A, A, None,
                                      A, A, None)
    assert st == B.CLSA_ERR_SCRATCH_LIMIT
    assert B.clsa_status_string(st) == "CLSA_ERR_SCRATCH_LIMIT"
    bad = _shape(inputs.small_workload(batch=2, lens=(100, 50), top_k=64))
    bad.top_k = 0
    assert lib.clsa_decode_step_noalloc(ctypes.byref(bad), A, A, A, A, None, A, None, 1, A, A,
                                        None, A, A, None) == B.CLSA_ERR_INVALID_ARG
    for name in ("decode_b1_n4k", "decode_b8_n32k", "decode_b4_n128k_planted",
                 "decode_b32_ragged_paged"):
        ww = inputs.workload(name)
        assert B.clsa_workspace_bytes(_shape(ww), B.CLSA_OP_DECODE, ww.n_layers) <= \
            B.CLSA_NOALLOC_SCRATCH_BYTES, name
