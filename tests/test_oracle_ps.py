"""Pins of the oracle's parameter-server apply and loss-statistics filter
(Section 4 parameter server, Section 4.2 stability; AdaGrad of Duchi, Hazan and
Singer 2011).  Each pin comes from somewhere other than the oracle's own loop:
hand-computed closed forms, AdaGrad written as cumulative sums, brute-force
staleness bookkeeping, numpy's mean/variance, and the weighted-sum form of the
exponentially weighted statistics."""
import math

import numpy as np
import pytest


# ---------------------------------------------------------------------------
# AdaGrad apply
# ---------------------------------------------------------------------------
def test_adagrad_closed_form_two_steps(oracle_mod):
    # g = 4 twice, lr = 0.5, eps = 1: h = 16 then 32;
    # theta: 0 - 0.5*4/(1+4) = -0.4, then - 0.5*4/(1+sqrt(32)) = -2/(1+4*sqrt(2))
    r = oracle_mod.ps_apply(np.zeros(1), np.zeros(1), np.array([[4.0], [4.0]]), [0, 0], 0,
                            10, 0.5, 1.0)
    assert r["accum"][0] == 32.0
    assert math.isclose(r["theta"][0], -0.4 - 2.0 / (1.0 + 4.0 * math.sqrt(2.0)), rel_tol=1e-15)
    assert list(r["applied"]) == [1, 1] and r["ps_version"] == 2


def test_adagrad_matches_cumulative_sum_form(oracle_mod):
    """theta_T = theta_0 - lr sum_t g_t / (eps + sqrt(h_0 + sum_{s<=t} g_s^2))."""
    rng = np.random.default_rng(11)
    G, n = 7, 50
    g = rng.standard_normal((G, n))
    th0, h0 = rng.standard_normal(n), rng.random(n)
    lr, eps = 0.25, 0.125
    h = h0 + np.cumsum(g * g, axis=0)
    want = th0 - lr * np.sum(g / (eps + np.sqrt(h)), axis=0)
    r = oracle_mod.ps_apply(th0, h0, g, np.zeros(G, np.int64), 0, 100, lr, eps)
    np.testing.assert_allclose(r["theta"], want, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(r["accum"], h[-1], rtol=1e-14)


def test_staleness_brute_force(oracle_mod):
    rng = np.random.default_rng(12)
    for trial in range(200):
        G = int(rng.integers(1, 9))
        V0 = int(rng.integers(0, 20))
        ver = rng.integers(max(0, V0 - 8), V0 + 1, G)
        keep = (rng.random(G) < 0.8).astype(np.uint8)
        max_delay = int(rng.integers(0, 6))
        # bookkeeping written out: the server version when each gradient's turn comes
        V, want = V0, []
        for i in range(G):
            ok = bool(keep[i]) and V - ver[i] <= max_delay
            want.append(int(ok))
            V += ok
        g = rng.standard_normal((G, 3))
        r = oracle_mod.ps_apply(np.zeros(3), np.zeros(3), g, ver, V0, max_delay, 0.1, 1e-3, keep)
        assert list(r["applied"]) == want, trial
        assert r["ps_version"] == V
        # the result equals applying only the accepted gradients, all fresh
        sel = g[np.array(want, bool)]
        ref = oracle_mod.ps_apply(np.zeros(3), np.zeros(3), sel.reshape(-1, 3),
                                  np.zeros(len(sel), np.int64), 0, 10**9, 0.1, 1e-3)
        np.testing.assert_array_equal(r["theta"], ref["theta"])


def test_earlier_updates_make_later_gradients_stale(oracle_mod):
    # versions 4,4,4 at server version 5, max delay 2: delays 1, 2, 3 at their turns
    r = oracle_mod.ps_apply(np.zeros(2), np.zeros(2), np.ones((3, 2)), [4, 4, 4], 5, 2, 0.1, 1.0)
    assert list(r["applied"]) == [1, 1, 0] and r["ps_version"] == 7


def test_discarded_and_zero_gradients_leave_theta(oracle_mod):
    th = np.array([1.0, -2.0, 3.0])
    r = oracle_mod.ps_apply(th, np.ones(3), np.array([[5.0, 5.0, 5.0], [0.0, 0.0, 0.0]]),
                            [0, 0], 0, 5, 0.5, 0.1, keep=np.array([0, 1], np.uint8))
    np.testing.assert_array_equal(r["theta"], th)
    np.testing.assert_array_equal(r["accum"], np.ones(3))
    assert list(r["applied"]) == [0, 1] and r["ps_version"] == 1


def test_ps_apply_rejects_nonpositive_eps(oracle_mod):
    with pytest.raises(ValueError):
        oracle_mod.ps_apply(np.zeros(1), np.zeros(1), np.ones((1, 1)), [0], 0, 1, 0.1, 0.0)


# ---------------------------------------------------------------------------
# Loss-statistics filter
# ---------------------------------------------------------------------------
def _run_filter(oracle_mod, xs, alpha, k, warmup):
    st = np.zeros((1, 3))
    keeps, hist = [], []
    for x in xs:
        keep, st = oracle_mod.loss_filter(st, [x], alpha, k, warmup)
        keeps.append(int(keep[0]))
        hist.append(st[0].copy())
    return keeps, hist


def test_filter_cumulative_matches_numpy(oracle_mod):
    rng = np.random.default_rng(13)
    xs = np.abs(rng.standard_normal(300)).astype(np.float32)
    xs[[50, 120, 250]] = [9.0, 12.0, 20.0]  # outliers
    k, warmup = 3.0, 10
    keeps, hist = _run_filter(oracle_mod, xs, 0.0, k, warmup)
    x64 = xs.astype(np.float64)
    for i in range(len(xs)):
        seen = x64[: i + 1]
        assert hist[i][0] == i + 1
        assert math.isclose(hist[i][1], seen.mean(), rel_tol=1e-12)
        assert math.isclose(hist[i][2], seen.var(), rel_tol=1e-10, abs_tol=1e-15)
        if i >= warmup:
            prev = x64[:i]
            want = not (x64[i] > prev.mean() + k * prev.std())
            assert keeps[i] == int(want), i
        else:
            assert keeps[i] == 1
    assert keeps[50] == 0 and keeps[120] == 0 and keeps[250] == 0


def test_filter_exponential_hand_computed(oracle_mod):
    # alpha 0.5: x = 1 -> (1, 0); x = 3 -> d = 2, mean 2, var 0.5*(0 + 0.5*4) = 1;
    # x = 10 with k = 3, warmup 2: 10 > 2 + 3*1, discarded; then d = 8, mean 6,
    # var = 0.5*(1 + 0.5*64) = 16.5
    keeps, hist = _run_filter(oracle_mod, [1.0, 3.0, 10.0], 0.5, 3.0, 2)
    assert keeps == [1, 1, 0]
    assert list(hist[1]) == [2.0, 2.0, 1.0]
    assert list(hist[2]) == [3.0, 6.0, 16.5]


def test_filter_exponential_matches_weighted_sums(oracle_mod):
    """The recursion equals the mean and variance under weights
    w_1 = (1-a)^(n-1), w_i = a (1-a)^(n-i) (i >= 2), which sum to one."""
    rng = np.random.default_rng(14)
    xs = (rng.random(40) * 4).astype(np.float32).astype(np.float64)
    a = 0.125
    _, hist = _run_filter(oracle_mod, xs, a, 2.0, 5)
    for n in (1, 2, 7, 40):
        w = np.array([(1 - a) ** (n - 1)] + [a * (1 - a) ** (n - i) for i in range(2, n + 1)])
        mu = float(np.sum(w * xs[:n]))
        var = float(np.sum(w * (xs[:n] - mu) ** 2))
        assert math.isclose(hist[n - 1][1], mu, rel_tol=1e-12)
        assert math.isclose(hist[n - 1][2], var, rel_tol=1e-9, abs_tol=1e-15)


def test_filter_absolute_value_and_independent_learners(oracle_mod):
    st = np.zeros((2, 3))
    keep, st = oracle_mod.loss_filter(st, [-2.0, 5.0], 0.0, 1.0, 0)
    assert list(keep) == [1, 1]  # n = 0: nothing to compare against
    assert st[0, 1] == 2.0 and st[1, 1] == 5.0
    keep, st2 = oracle_mod.loss_filter(st, [2.0, 100.0], 0.0, 1.0, 0)
    # learner 0 sees |x| = mean: kept; learner 1: var 0 and x > mean: discarded
    assert list(keep) == [1, 0]
    assert st2[0, 0] == 2.0 and st2[1, 0] == 2.0


def test_filter_threshold_is_k_standard_deviations(oracle_mod):
    # after 1, 3 (alpha 0.5): mean 2, var 1, so the bar at k = 3 is 2 + 3*1 = 5
    assert _run_filter(oracle_mod, [1.0, 3.0, 4.5], 0.5, 3.0, 2)[0] == [1, 1, 1]
    assert _run_filter(oracle_mod, [1.0, 3.0, 5.5], 0.5, 3.0, 2)[0] == [1, 1, 0]
    # warmup 3: the third loss is compared only once three have been seen
    assert _run_filter(oracle_mod, [1.0, 3.0, 50.0], 0.5, 3.0, 3)[0] == [1, 1, 1]
