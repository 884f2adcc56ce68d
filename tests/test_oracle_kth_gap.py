"""Pins for ``oracle.kth_gap``, the tie-band classifier.

The parity rule for index sets (bit-exact outside the tie band) rests on this
function: a row is in the band when the relative gap between its k-th and
(k+1)-th largest exact scores, (s_(k) - s_(k+1)) / |s_(k)|, is below 1e-5.
Nothing here re-types that expression on the oracle's own partition: the pins
are hand-worked rows whose gap follows by arithmetic, a brute force over a
full Python sort (``sorted``) of the valid prefix, invariances of the
definition (row permutation, positive scaling, junk past the valid prefix), and
mutants of the function that each pin set must reject."""
import inspect
import math
import textwrap

import numpy as np
import pytest

import oracle

# (row, n_valid, k, expected gap), every expected value worked out by hand:
# sorted descending, s_(k) is the k-th entry (1-based), s_(k+1) the next one.
HAND = [
    ([5.0, 4.0, 3.0, 2.0], 4, 2, (4.0 - 3.0) / 4.0),          # 0.25
    ([2.0, 3.0, 5.0, 4.0], 4, 1, (5.0 - 4.0) / 5.0),          # 0.2, order in the row ignored
    ([2.0, 3.0, 5.0, 4.0], 4, 3, (3.0 - 2.0) / 3.0),
    ([1.0, 1.0, 1.0], 3, 1, 0.0),                              # exact tie at k / k+1
    ([1.0, 1.0, 1.0], 3, 2, 0.0),
    ([3.0, 1.0, 1.0], 3, 1, (3.0 - 1.0) / 3.0),                # tie below k+1 is irrelevant
    ([-1.0, -2.0, -3.0], 3, 1, (-1.0 - -2.0) / 1.0),           # negative k-th score: |s_(k)|
    ([-1.0, -2.0, -3.0], 3, 2, (-2.0 - -3.0) / 2.0),
    ([0.5, -0.5, 2.0], 3, 2, (0.5 - -0.5) / 0.5),              # mixed signs
    ([1e-40, 0.0, -1.0], 3, 1, (1e-40 - 0.0) / 1e-30),         # |s_(k)| below the 1e-30 floor
    ([0.0, 0.0, -1.0], 3, 2, (0.0 - -1.0) / 1e-30),            # s_(k) = 0 uses the floor
    ([7.0, 6.0], 2, 2, math.inf),                              # n == k: nothing excluded
    ([7.0, 6.0, 100.0, 200.0], 2, 2, math.inf),                # n_valid == k, junk past it
    ([7.0, 6.0], 2, 5, math.inf),                              # n < k
    ([9.0, 8.0, 100.0], 2, 1, (9.0 - 8.0) / 9.0),              # junk past n_valid ignored
    ([0.0, 0.0, 0.0, 0.0], 0, 1, math.inf),                    # empty row
]


def _brute(row, n, k):
    """Gap from a full descending sort of the valid prefix (Python's sorted)."""
    if n <= k:
        return math.inf
    s = sorted((float(v) for v in row[:n]), reverse=True)
    return (s[k - 1] - s[k]) / max(abs(s[k - 1]), 1e-30)


def _one(fn, row, n, k):
    a = np.asarray(row, dtype=np.float64)[None, :]
    return float(fn(a, np.array([n]), k)[0])


def pin_hand_worked(fn):
    for row, n, k, want in HAND:
        got = _one(fn, row, n, k)
        if math.isinf(want):
            assert math.isinf(got) and got > 0, (row, n, k, got)
        else:
            assert got == pytest.approx(want, rel=1e-12, abs=0.0), (row, n, k, got, want)


def pin_brute_force(fn):
    g = np.random.default_rng(7)
    for trial in range(60):
        n_max = int(g.integers(1, 40))
        rows = int(g.integers(1, 5))
        if trial % 3 == 0:
            s = g.integers(-3, 4, size=(rows, n_max)).astype(np.float64) / 2.0  # many ties
        else:
            s = g.standard_normal((rows, n_max)) * (10.0 ** g.integers(-3, 4))
        nv = g.integers(0, n_max + 1, size=rows)
        k = int(g.integers(1, n_max + 2))
        got = fn(s, nv, k)
        assert got.shape == nv.shape
        for r in range(rows):
            want = _brute(s[r], int(nv[r]), k)
            if math.isinf(want):
                assert math.isinf(got[r]) and got[r] > 0, (trial, r)
            else:
                assert got[r] == pytest.approx(want, rel=1e-12, abs=1e-300), (trial, r)


def pin_invariances(fn):
    g = np.random.default_rng(11)
    for _ in range(20):
        n = int(g.integers(3, 200))
        k = int(g.integers(1, n))
        row = g.standard_normal(n)
        base = _one(fn, row, n, k)
        assert _one(fn, g.permutation(row), n, k) == pytest.approx(base, rel=1e-12)
        assert _one(fn, row * 3.5, n, k) == pytest.approx(base, rel=1e-12)
        padded = np.concatenate([row, g.standard_normal(17) * 1e6])
        assert _one(fn, padded, n, k) == pytest.approx(base, rel=1e-12)
        # the gap is non-negative, and zero exactly when s_(k) == s_(k+1)
        assert base >= 0.0
        tied = row.copy()
        order = np.argsort(-row, kind="stable")
        tied[order[k]] = tied[order[k - 1]]
        assert _one(fn, tied, n, k) == 0.0


def pin_batch_shape(fn):
    """Rows keep their [B, T] shape and each uses its own n_valid."""
    s = np.array([[[3.0, 2.0, 1.0], [1.0, 1.0, 0.0]],
                  [[4.0, 2.0, 0.0], [5.0, 1.0, 9.0]]])
    nv = np.array([[3, 3], [2, 2]])
    got = fn(s, nv, 1)
    want = np.array([[(3 - 2) / 3, 0.0], [(4 - 2) / 4, (5 - 1) / 5]])
    assert got.shape == (2, 2)
    np.testing.assert_allclose(got, want, rtol=1e-12)


PINS = [pin_hand_worked, pin_brute_force, pin_invariances, pin_batch_shape]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_kth_gap(pin):
    pin(oracle.kth_gap)


# Plausible mistakes in the function, each planted in a copy of its source.
MUTANTS = {
    "partition_at_k_and_k_plus_1": ("(k - 1, k)", "(k, k + 1)"),
    "index_k_and_k_plus_1": ("sk, sk1 = part[k - 1], part[k]", "sk, sk1 = part[k], part[k + 1]"),
    "zero_instead_of_inf": ("gap = np.full(rows.shape[0], np.inf)",
                            "gap = np.full(rows.shape[0], 0.0)"),
    "no_abs_on_kth": ("max(abs(sk), 1e-30)", "max(sk, 1e-30)"),
    "divide_by_k_plus_1": ("max(abs(sk), 1e-30)", "max(abs(sk1), 1e-30)"),
    "ignores_n_valid": ("rows[r, :n]", "rows[r, :]"),
    "n_equal_k_not_excluded": ("if n <= k:", "if n < k:"),
    "ascending_partition": ("part = -np.partition(-rows[r, :n], (k - 1, k))",
                            "part = np.partition(rows[r, :n], (k - 1, k))"),
    "gap_sign_flipped": ("(sk - sk1)", "(sk1 - sk)"),
}


def _mutant(name):
    find, repl = MUTANTS[name]
    src = textwrap.dedent(inspect.getsource(oracle.kth_gap))
    assert src.count(find) >= 1, f"mutation {name} does not apply"
    ns = {"np": np}
    exec(compile(src.replace(find, repl), f"<kth_gap mutant {name}>", "exec"), ns)
    return ns["kth_gap"]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_kth_gap_mutant(name):
    fn = _mutant(name)
    caught = []
    for pin in PINS:
        try:
            pin(fn)
        except (AssertionError, IndexError, ValueError) as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught the kth_gap mutant {name}"
