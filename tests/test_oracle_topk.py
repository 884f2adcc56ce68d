"""Pins for the oracle's top-k (Eq. 3: S_t = TopK(I_t, k)).

The oracle sorts; these checks use exhaustive subset search, numpy's stable
argsort and the order-statistic characterisation instead."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from paper_2606_06467_amd import inputs


def _run(orc, s, k, lens=None, q_pos=None, causal=False):
    s = np.asarray(s, np.float32)
    if s.ndim == 1:
        s = s[None, None, :]
    B, T, N = s.shape
    lens = np.full(B, N, np.int32) if lens is None else np.asarray(lens, np.int32)
    sh = orc.shape(B, T, N, k, causal=causal)
    return orc.topk(sh, s, lens, q_pos)


def _brute(s, k):
    """Best k-subset by exact sum; among equals, the lexicographically smallest sorted tuple."""
    n = len(s)
    if k >= n:
        return tuple(range(n))
    best, best_sum = None, None
    for c in itertools.combinations(range(n), k):   # generated in lexicographic order
        tot = sum(Fraction(float(s[i])) for i in c)
        if best_sum is None or tot > best_sum:
            best, best_sum = c, tot
    return best


@pytest.mark.parametrize("n", [1, 2, 5, 9, 11])
def test_exhaustive_subsets_tiny(orc, n):
    g = np.random.default_rng(100 + n)
    for trial in range(6):
        if trial % 2:
            s = (g.integers(-2, 3, size=n) / 4.0).astype(np.float32)   # many exact ties
        else:
            s = g.standard_normal(n).astype(np.float32)
        for k in range(1, n + 2):
            idx, nsel = _run(orc, s, k)
            m = min(k, n)
            assert nsel[0, 0] == m
            assert tuple(idx[0, 0, :m]) == _brute(s, k)
            assert (idx[0, 0, m:] == -1).all()


def test_matches_numpy_stable_argsort(orc):
    s = inputs.random_scores(7, 6, 3000, ties=0.3)
    s[2] = inputs.random_scores(8, 1, 3000, levels=16)[0]
    for k in (1, 17, 256, 2999, 3000, 4096):
        idx, nsel = _run(orc, s[:, None, :], k)
        for r in range(6):
            order = np.argsort(-s[r], kind="stable")        # descending score, ascending index on ties
            ref = np.sort(order[:min(k, 3000)])
            m = len(ref)
            assert nsel[r, 0] == m
            np.testing.assert_array_equal(idx[r, 0, :m], ref)
            assert (idx[r, 0, m:] == -1).all()


def test_order_statistic_characterisation(orc):
    s = inputs.random_scores(9, 4, 5000, levels=64)
    k = 300
    idx, nsel = _run(orc, s[:, None, :], k)
    for r in range(4):
        sel = idx[r, 0, :nsel[r, 0]]
        assert np.all(np.diff(sel) > 0)
        mask = np.zeros(5000, bool)
        mask[sel] = True
        tau = s[r, mask].min()
        assert s[r, ~mask].max() <= tau
        # ties at tau: every selected tie has a smaller index than every excluded tie
        sel_t = np.flatnonzero(mask & (s[r] == tau))
        exc_t = np.flatnonzero(~mask & (s[r] == tau))
        if len(exc_t):
            assert sel_t.max() < exc_t.min()


def test_signed_zero_is_a_tie(orc):
    idx, _ = _run(orc, [-0.0, 0.0, -1.0], 1)
    assert idx[0, 0, 0] == 0
    idx, _ = _run(orc, [0.0, -0.0, -1.0], 1)
    assert idx[0, 0, 0] == 0


def test_infinities_order(orc):
    idx, _ = _run(orc, [1.0, np.inf, -np.inf, 3.0], 2)
    assert list(idx[0, 0]) == [1, 3]
    idx, _ = _run(orc, [-np.inf, -np.inf, -np.inf], 2)
    assert list(idx[0, 0]) == [0, 1]


def test_k_at_least_len_selects_all_and_pads(orc):
    s = np.arange(10, dtype=np.float32)[None, None, :].repeat(3, 0)
    idx, nsel = _run(orc, s, 16, lens=[10, 4, 0])
    assert list(nsel[:, 0]) == [10, 4, 0]
    assert list(idx[0, 0]) == list(range(10)) + [-1] * 6
    assert list(idx[1, 0]) == [0, 1, 2, 3] + [-1] * 12
    assert (idx[2, 0] == -1).all()


def test_causal_rows_only_see_their_prefix(orc):
    N = 64
    s = np.tile(np.arange(N, 0, -1, dtype=np.float32), (1, 3, 1))   # larger score at lower j
    s[0, :, 50] = 1e6                                                # big score beyond the prefix
    q_pos = np.array([[5, 20, 63]], np.int32)
    idx, nsel = _run(orc, s, 8, q_pos=q_pos, causal=True)
    assert list(nsel[0]) == [6, 8, 8]
    assert list(idx[0, 0, :6]) == [0, 1, 2, 3, 4, 5]
    assert list(idx[0, 1]) == list(range(8))
    assert 50 in idx[0, 2]
