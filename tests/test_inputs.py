"""The seeded generator: determinism, bfloat16 rounding, structure of the workloads."""
import numpy as np
import pytest
import torch

from paper_2606_06467_amd import inputs


def test_deterministic_and_seed_sensitive():
    a = inputs.normal_bf16(5, (3, 1 << 20 | 7), 0.125)
    b = inputs.normal_bf16(5, (3, 1 << 20 | 7), 0.125)
    c = inputs.normal_bf16(6, (3, 1 << 20 | 7), 0.125)
    np.testing.assert_array_equal(a, b)
    assert (a != c).mean() > 0.9


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * 37,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.4e38, -1e-40,
                                  np.inf, -np.inf], np.float32)])
    ours = inputs.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(inputs.f32_from_bf16_bits(ours),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_value_distributions():
    a = inputs.f32_from_bf16_bits(inputs.normal_bf16(9, (1 << 21,), 1.0 / 8.0))
    assert abs(a.mean()) < 1e-3 and abs(a.std() - 0.125) < 1e-3


def test_named_workload_sizes():
    w = inputs.workload("decode_b4_n128k_planted")
    assert (w.batch, w.max_len, w.top_k, w.n_layers, w.planted) == (4, 131072, 2048, 16, 64)
    w = inputs.workload("decode_b32_ragged_paged")
    assert w.batch == 32 and all(16384 <= n <= 65536 for n in w.lens)
    assert w.page_size == 64 and w.max_len % 64 == 0 and max(w.lens) <= w.max_len
    assert min(w.lens) > w.top_k
    w = inputs.workload("prefill_t8k_n128k")
    assert w.n_q == 8192 and w.q_pos0 == [122880] and w.causal


def test_page_table_is_a_bijection():
    w = inputs.small_workload(lens=(64 * 5 + 1, 64, 130), batch=3, page_size=64)
    pt = inputs.page_table_for(w, 77)
    used = pt[pt >= 0]
    assert sorted(used.tolist()) == list(range(len(used)))
    assert [(pt[b] >= 0).sum() for b in range(3)] == [6, 1, 3]


def test_planting_raises_scores_by_three_sigma():
    w = inputs.small_workload(lens=(4096,), batch=1, top_k=64, wid=41)
    w.planted = 64
    x = inputs.make_inputs(w)
    pos = inputs.planted_positions(w)[0]
    q = inputs.f32_from_bf16_bits(x["q_idx"][0, 0]).astype(np.float64).reshape(-1)
    k = inputs.f32_from_bf16_bits(x["k_idx"][0]).astype(np.float64).reshape(4096, -1)
    s = k @ q
    sigma = np.linalg.norm(q) / 8
    rest = np.delete(s, pos)
    assert abs(rest.std() / sigma - 1) < 0.05
    assert abs((s[pos].mean() - rest.mean()) / sigma - 3.0) < 0.4
