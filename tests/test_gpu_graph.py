"""The decode step captured in a HIP graph: every replay must give exactly the
eager step's index set and outputs, also when eager work runs between replays
(the library launches only kernels; it records no memset that a graph could
replay wrongly)."""
import numpy as np
import pytest

from paper_2606_06467_amd import inputs
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager_step():
    import torch
    from paper_2606_06467_amd import binding as B
    w = inputs.workload("decode_b1_n4k")
    x = inputs.make_inputs(w)
    d = U.to_dev(x)
    sh = U.shape_of(w)
    L = w.n_layers
    out = torch.empty((L, w.batch, 1, w.q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((L, w.batch, 1, w.q_heads), device="cuda")
    idx = torch.empty((w.batch, 1, w.top_k), dtype=torch.int32, device="cuda")
    ns = torch.empty((w.batch, 1), dtype=torch.int32, device="cuda")
    ws = B.workspace(sh, B.CLSA_OP_DECODE, L)

    def step():
        B.clsa_decode_step(sh, d["q_idx"], d["k_idx"], d["k_cache"], d["v_cache"], None,
                           d["seq_lens"], None, d["q_layers"], out, lse, idx, ns, ws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (out, lse, idx, ns)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for t in (out, lse, idx, ns):  # poison, then replay
            t.fill_(0 if t.dtype == torch.int32 else float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, r in zip((out, lse, idx, ns), ref):
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               r.view(torch.uint8) if r.dtype == torch.bfloat16 else r), rep
        step()  # eager work between replays
        torch.cuda.synchronize()
    U.log("  4 graph replays identical to the eager step")
