"""Closed-form pins for the oracle's TD target, Huber loss and dLoss/dQ.

A bias-only network (every weight and hidden bias zero, b5 = v) has
Q(s, .) = v for every state, so the DQN loss of eq. (1) and the terminal rule of
Algorithm 1 reduce to scalars that can be written down by hand:
  y = r + gamma * (1 - t) * max v-,  delta = y - v[a],
  loss = mean Huber(delta),  db5[a] = -sum_{b: a_b = a} clamp(delta_b) / B,
and every other gradient is exactly zero (ReLU'(0) = 0 kills the hidden path).
"""
import math

import numpy as np
import pytest

TINY = dict(in_c=2, in_h=12, in_w=12, c1=3, k1=4, s1=2, c2=4, k2=3, s2=1,
            c3=2, k3=2, s3=1, hidden=6, n_actions=3)


def _bias_only(oracle_mod, net, v, v_tgt):
    off = oracle_mod.param_offsets(net)
    theta = np.zeros(off[-1])
    theta[off[9]:off[10]] = v
    tgt = np.zeros(off[-1])
    tgt[off[9]:off[10]] = v_tgt
    return off, theta, tgt


@pytest.mark.parametrize("full", [False, True])
def test_bias_only_network_closed_form(oracle_mod, full):
    net = oracle_mod.Net() if full else oracle_mod.Net(**TINY)
    A = net.n_actions
    rng = np.random.default_rng(3)
    v = rng.normal(size=A).round(3)
    v_tgt = rng.normal(size=A).round(3)
    off, theta, tgt = _bias_only(oracle_mod, net, v, v_tgt)
    B = 6
    shape = (B, net.in_c, net.in_h, net.in_w)
    s = rng.integers(0, 256, shape, dtype=np.uint8)
    s2 = rng.integers(0, 256, shape, dtype=np.uint8)
    a = np.array([0, 1, 2, 0, 1, 2], np.int32) % A
    r = np.array([1.0, 0.0, -1.0, 0.5, 2.0, 0.0], np.float32)
    term = np.array([0, 1, 0, 0, 1, 0], np.uint8)
    gamma, clip = np.float32(0.99), 1.0
    out = oracle_mod.learner_step(net, theta, tgt, s, s2, a, r, term, gamma, clip)
    np.testing.assert_array_equal(out["q"], np.tile(v, (B, 1)))
    np.testing.assert_array_equal(out["q2"], np.tile(v_tgt, (B, 1)))
    g = float(gamma)
    m = max(v_tgt)
    loss, db5 = 0.0, np.zeros(A)
    for b in range(B):
        y = float(r[b]) if term[b] else float(r[b]) + g * m
        d = y - v[a[b]]
        ell = 0.5 * d * d if abs(d) <= clip else clip * abs(d) - 0.5 * clip * clip
        loss += ell
        db5[a[b]] -= max(-clip, min(clip, d)) / B
        # the per-sample pieces the oracle reports
        assert out["max_q2"][b] == m
        assert out["y"][b] == pytest.approx(y, rel=1e-15, abs=1e-15)
        assert out["delta"][b] == pytest.approx(d, rel=1e-14, abs=1e-15)
        assert out["ell"][b] == pytest.approx(ell, rel=1e-14, abs=1e-15)
    assert out["loss"] == pytest.approx(loss / B, rel=1e-14)
    np.testing.assert_allclose(out["grads"][off[9]:off[10]], db5, rtol=1e-14, atol=1e-16)
    assert not out["grads"][:off[9]].any()


@pytest.mark.parametrize("r,clip,loss,coef", [
    (0.5, 1.0, 0.125, -0.5),      # inside the quadratic zone
    (-0.5, 1.0, 0.125, 0.5),
    (2.0, 1.0, 1.5, -1.0),        # linear zone: c|d| - c^2/2, slope clipped
    (-2.0, 1.0, 1.5, 1.0),
    (2.0, math.inf, 2.0, -2.0),   # no clip: eq. (1) with a factor 1/2
    (3.0, 2.0, 4.0, -2.0),
])
def test_huber_values(oracle_mod, r, clip, loss, coef):
    net = oracle_mod.Net(**TINY)
    off, theta, tgt = _bias_only(oracle_mod, net, np.zeros(3), np.full(3, 7.0))
    s = np.zeros((1, 2, 12, 12), np.uint8)
    out = oracle_mod.learner_step(net, theta, tgt, s, s, np.array([1], np.int32),
                                  np.array([r], np.float32), np.array([1], np.uint8),
                                  0.99, clip)
    # terminal: y = r (the target net's 7.0 must not leak in), delta = r - 0
    assert out["loss"] == loss
    assert out["y"][0] == r and out["delta"][0] == r and out["ell"][0] == loss
    assert out["max_q2"][0] == 7.0
    assert out["grads"][off[9] + 1] == coef
    assert out["grads"][off[9]] == 0 and out["grads"][off[9] + 2] == 0


def test_gamma_zero_and_nonterminal(oracle_mod):
    net = oracle_mod.Net(**TINY)
    off, theta, tgt = _bias_only(oracle_mod, net, np.array([0.25, 0.0, 0.0]),
                                 np.array([0.5, 0.75, -1.0]))
    s = np.zeros((2, 2, 12, 12), np.uint8)
    a = np.array([0, 0], np.int32)
    r = np.array([0.5, 0.5], np.float32)
    t = np.array([0, 0], np.uint8)
    out0 = oracle_mod.learner_step(net, theta, tgt, s, s, a, r, t, 0.0, math.inf)
    assert out0["loss"] == 0.5 * 0.25 ** 2          # y = r, delta = 0.25
    out1 = oracle_mod.learner_step(net, theta, tgt, s, s, a, r, t, 0.5, math.inf)
    d = 0.5 + 0.5 * 0.75 - 0.25                      # max over v- is 0.75
    assert out1["loss"] == pytest.approx(0.5 * d * d, rel=1e-15)
    assert out1["grads"][off[9]] == pytest.approx(-d, rel=1e-15)


def test_rejects_bad_arguments(oracle_mod):
    net = oracle_mod.Net(**TINY)
    off, theta, tgt = _bias_only(oracle_mod, net, np.zeros(3), np.zeros(3))
    s = np.zeros((1, 2, 12, 12), np.uint8)
    one = np.ones(1, np.float32)
    with pytest.raises(ValueError):
        oracle_mod.learner_step(net, theta, tgt, s, s, np.array([3], np.int32), one,
                                np.zeros(1, np.uint8), 0.99)
    with pytest.raises(ValueError):
        oracle_mod.learner_step(net, theta, tgt, s, s, np.array([0], np.int32), one,
                                np.zeros(1, np.uint8), 0.99, clip=0.0)
