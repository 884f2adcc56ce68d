"""Pins for the oracle's distillation target (Eq. 5) and loss with gradient (Eq. 6).

Each check compares the oracle with something other than itself: scipy's softmax,
log-softmax and relative entropy, invariants (rows of a mixture of distributions
sum to one; KL of a distribution with itself is zero), and central finite
differences of the loss for the gradient."""
import numpy as np
from scipy import special

from paper_2606_06467_amd import inputs


def _w(batch=2, lens=(40, 25), n_q=6, q_heads=4, kv_heads=2, n_layers=2, causal=True,
       q_pos0=(34, 19), wid=111):
    return inputs.small_workload(batch=batch, lens=lens, n_q=n_q, causal=causal, q_pos0=q_pos0,
                                 q_heads=q_heads, kv_heads=kv_heads, n_layers=n_layers, wid=wid)


def _f(bits):
    return inputs.f32_from_bf16_bits(bits).astype(np.float64)


def _valid(w, x, b, t):
    n = w.lens[b]
    if w.causal:
        n = min(n, int(x["q_pos"][b, t]) + 1)
    return max(n, 0)


def test_target_is_a_mean_of_scipy_softmaxes(orc):
    w = _w()
    x = inputs.make_inputs(w)
    sh = orc.shape_of(w)
    a = orc.kd_target(sh, x["q_layers"], x["k_cache"], x["seq_lens"], x["q_pos"])
    q = _f(x["q_layers"])             # [L, B, T, Hq, D]
    k = _f(x["k_cache"])              # [B, N, Hkv, D]
    G = w.q_heads // w.kv_heads
    for b in range(w.batch):
        for t in range(w.n_q):
            n = _valid(w, x, b, t)
            ref = np.zeros(n)
            for l in range(w.n_layers):
                for h in range(w.q_heads):
                    z = w.softmax_scale * (k[b, :n, h // G] @ q[l, b, t, h])
                    ref += special.softmax(z)
            ref /= w.n_layers * w.q_heads
            np.testing.assert_allclose(a[b, t, :n], ref, rtol=1e-12, atol=1e-15)
            assert np.isnan(a[b, t, n:]).all()          # masked positions are not written


def test_target_rows_sum_to_one(orc):
    w = _w(lens=(70, 70), q_pos0=(60, 3))
    x = inputs.make_inputs(w)
    a = orc.kd_target(orc.shape_of(w), x["q_layers"], x["k_cache"], x["seq_lens"], x["q_pos"])
    sums = np.nansum(a, axis=-1)
    np.testing.assert_allclose(sums, 1.0, rtol=1e-13)


def _softmax_scores(w, x, q_idx=None, k_idx=None):
    q = _f(x["q_idx"] if q_idx is None else q_idx).reshape(w.batch, w.n_q, 256)
    k = _f(x["k_idx"] if k_idx is None else k_idx).reshape(w.batch, w.max_len, 256)
    return q, k


def test_kl_of_the_indexer_distribution_with_itself_is_zero(orc):
    w = _w()
    x = inputs.make_inputs(w)
    q, k = _softmax_scores(w, x)
    abar = np.full((w.batch, w.n_q, w.max_len), np.nan)
    for b in range(w.batch):
        for t in range(w.n_q):
            n = _valid(w, x, b, t)
            abar[b, t, :n] = special.softmax(k[b, :n] @ q[b, t])
    loss, dq, dk = orc.kd_loss(orc.shape_of(w), abar, x["q_idx"], x["k_idx"], x["seq_lens"],
                               x["q_pos"])
    assert abs(loss) < 1e-13
    assert np.abs(dq).max() < 1e-13 and np.nanmax(np.abs(dk)) < 1e-13


def _loss_ref(w, x, abar, q, k):
    """Eq. 6 through scipy: mean over rows of sum rel_entr(P, Q), Q = softmax(I)."""
    tot, rows = 0.0, 0
    for b in range(w.batch):
        for t in range(w.n_q):
            n = _valid(w, x, b, t)
            if n == 0:
                continue
            logq = special.log_softmax(k[b, :n] @ q[b, t])
            p = abar[b, t, :n]
            tot += float(np.sum(special.rel_entr(p, np.exp(logq))))
            rows += 1
    return tot / rows


def _random_target(w, x, seed):
    g = np.random.default_rng(seed)
    abar = np.full((w.batch, w.n_q, w.max_len), np.nan)
    for b in range(w.batch):
        for t in range(w.n_q):
            n = _valid(w, x, b, t)
            p = g.dirichlet(np.full(n, 0.5))
            p[g.random(n) < 0.2] = 0.0                  # exact zeros: 0 log 0 terms
            abar[b, t, :n] = p / p.sum()
    return abar


def test_loss_matches_scipy_relative_entropy(orc):
    w = _w()
    x = inputs.make_inputs(w)
    abar = _random_target(w, x, 5)
    loss, _, _ = orc.kd_loss(orc.shape_of(w), abar, x["q_idx"], x["k_idx"], x["seq_lens"],
                             x["q_pos"])
    q, k = _softmax_scores(w, x)
    assert abs(loss - _loss_ref(w, x, abar, q, k)) < 1e-12 * max(1.0, abs(loss))


def test_gradient_matches_central_differences(orc):
    w = _w(lens=(30, 18), n_q=3, q_pos0=(27, 15))
    x = inputs.make_inputs(w)
    abar = _random_target(w, x, 6)
    _, dq, dk = orc.kd_loss(orc.shape_of(w), abar, x["q_idx"], x["k_idx"], x["seq_lens"],
                            x["q_pos"])
    q, k = _softmax_scores(w, x)
    eps = 1e-6
    g = np.random.default_rng(7)
    for _ in range(12):
        b, t, e = int(g.integers(w.batch)), int(g.integers(w.n_q)), int(g.integers(256))
        qp, qm = q.copy(), q.copy()
        qp[b, t, e] += eps
        qm[b, t, e] -= eps
        fd = (_loss_ref(w, x, abar, qp, k) - _loss_ref(w, x, abar, qm, k)) / (2 * eps)
        assert abs(fd - dq.reshape(w.batch, w.n_q, 256)[b, t, e]) < 1e-7, (b, t, e)
    dkr = dk.reshape(w.batch, w.max_len, 256)
    for _ in range(12):
        b, j, e = int(g.integers(w.batch)), int(g.integers(w.lens[1])), int(g.integers(256))
        kp, km = k.copy(), k.copy()
        kp[b, j, e] += eps
        km[b, j, e] -= eps
        fd = (_loss_ref(w, x, abar, q, kp) - _loss_ref(w, x, abar, q, km)) / (2 * eps)
        assert abs(fd - dkr[b, j, e]) < 1e-7, (b, j, e)


def test_rows_without_keys_do_not_count(orc):
    """A sequence of length 0 adds no row to the mean; its dq rows are zero."""
    w = _w(lens=(30, 0), q_pos0=(24, 0))
    x = inputs.make_inputs(w)
    abar = _random_target(w, x, 8)
    loss, dq, _ = orc.kd_loss(orc.shape_of(w), abar, x["q_idx"], x["k_idx"], x["seq_lens"],
                              x["q_pos"])
    q, k = _softmax_scores(w, x)
    assert abs(loss - _loss_ref(w, x, abar, q, k)) < 1e-12
    assert not dq.reshape(w.batch, w.n_q, 256)[1].any()
