"""Pins for the oracle's projections of new tokens (Eq. 2: Q_idx = H W_idx^Q,
K_idx = H W_idx^K, with the shared K = H W^K and V = H W^V) and the cache row
each new token occupies.

Each check compares the oracle with something other than itself: numpy's fp64
matrix product, exact integer arithmetic, unit-vector probes, and the cache
layout written out by hand."""
import numpy as np

from paper_2606_06467_amd import inputs


def _rand(seed, shape, scale):
    return inputs.normal_bf16(seed, shape, scale)


def test_matches_numpy_float64(orc):
    B, T, D, N = 2, 3, 96, 40
    h = _rand(301, (B * T, D), 1.0)
    w = _rand(302, (N, D), 0.05)
    sh = orc.shape(B, T, 64, 8)
    out, dest = orc.project(sh, h, w, np.array([5, 6, 7, 60, 61, 62], np.int32))
    hf = inputs.f32_from_bf16_bits(h).astype(np.float64)
    wf = inputs.f32_from_bf16_bits(w).astype(np.float64)
    np.testing.assert_allclose(out, hf @ wf.T, rtol=1e-13, atol=1e-14)


def test_exact_on_small_integers(orc):
    g = np.random.default_rng(7)
    D, N = 64, 9
    hi = g.integers(-9, 10, size=(2, D))
    wi = g.integers(-9, 10, size=(N, D))
    sh = orc.shape(2, 1, 16, 4)
    out, _ = orc.project(sh, inputs.bf16_bits_from_f32(hi.astype(np.float32)),
                         inputs.bf16_bits_from_f32(wi.astype(np.float32)),
                         np.array([0, 1], np.int32))
    for r in range(2):
        for c in range(N):
            assert out[r, c] == float(sum(int(a) * int(b) for a, b in zip(hi[r], wi[c])))


def test_unit_vector_probe(orc):
    """h = e_i picks column i of every output feature's weight vector: a transposed
    or mis-strided weight operand fails this."""
    D, N = 48, 12
    w = _rand(303, (N, D), 1.0)
    wf = inputs.f32_from_bf16_bits(w).astype(np.float64)
    one = inputs.bf16_bits_from_f32(np.array([1.0], np.float32))[0]
    sh = orc.shape(1, 1, 8, 4)
    for i in (0, 1, 17, D - 1):
        h = np.zeros((1, D), np.uint16)
        h[0, i] = one
        out, _ = orc.project(sh, h, w, np.array([3], np.int32))
        np.testing.assert_array_equal(out[0], wf[:, i])


def test_destination_rows(orc):
    """Contiguous caches: row b*max_len + pos; paged: the page table's page; outside
    [0, max_len): -1."""
    D = 16
    h = _rand(304, (6, D), 1.0)
    w = _rand(305, (4, D), 1.0)
    pos = np.array([0, 63, 64, 200, -1, 256], np.int32)
    sh = orc.shape(3, 2, 256, 4)
    _, dest = orc.project(sh, h, w, pos)
    np.testing.assert_array_equal(dest, [0, 63, 256 + 64, 256 + 200, -1, -1])
    pt = np.array([[5, 2, 7, 0], [1, 6, 3, 4], [8, 9, 10, 11]], np.int32)
    shp = orc.shape(3, 2, 256, 4, page_size=64, max_pages=4)
    _, dest = orc.project(shp, h, w, pos, pt)
    # rows 0,1: sequence 0, logical page 0 -> 5; row 2: sequence 1, page 1 -> 6;
    # row 3: sequence 1, position 200 = page 3 (-> 4), offset 8
    np.testing.assert_array_equal(dest, [5 * 64 + 0, 5 * 64 + 63, 6 * 64 + 0, 4 * 64 + 8, -1, -1])
