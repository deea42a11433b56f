"""Pins for the oracle's epsilon-greedy behaviour policy (Algorithm 1).

The draws come from the SplitMix64 output function.  It is pinned by the first
outputs of the published SplitMix64 generator for seed 1234567 (the sequence
printed with the reference implementation by Steele, Lea and Flood / Vigna:
6457827717110365317, 3203168211198807973, 9817491932198370423), which a
generator stepping its state by the golden gamma produces at states
seed + 1*G, seed + 2*G, seed + 3*G.
"""
import math

import numpy as np
import pytest

M64 = (1 << 64) - 1
G = 0x9E3779B97F4A7C15
TINY = dict(in_c=1, in_h=10, in_w=10, c1=2, k1=3, s1=1, c2=2, k2=3, s2=1,
            c3=2, k3=2, s3=2, hidden=8, n_actions=7)


def mix(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def test_splitmix64_published_outputs():
    seed = 1234567
    outs = [mix((seed + k * G) & M64) for k in (1, 2, 3)]
    assert outs == [6457827717110365317, 3203168211198807973, 9817491932198370423]


def _net_theta(oracle_mod, rng, A=7):
    net = oracle_mod.Net(**dict(TINY, n_actions=A))
    theta = rng.normal(0, 0.5, oracle_mod.param_count(net))
    return net, theta


def test_eps_zero_is_lowest_index_argmax(oracle_mod):
    rng = np.random.default_rng(41)
    net, theta = _net_theta(oracle_mod, rng)
    states = rng.integers(0, 256, (64, 1, 10, 10), dtype=np.uint8)
    acts, q = oracle_mod.act(net, theta, states, 0.0, 99)
    np.testing.assert_array_equal(acts, np.argmax(q, axis=1))  # numpy: first max
    assert q.shape == (64, 7)


def test_ties_break_to_lowest_index(oracle_mod):
    rng = np.random.default_rng(43)
    net, theta = _net_theta(oracle_mod, rng)
    off = oracle_mod.param_offsets(net)
    theta[:off[9]] = 0.0                     # Q = b5 for every state
    theta[off[9]:off[10]] = [0.1, 0.7, -1, 0.7, 0.2, 0.7, 0.0]
    states = np.zeros((3, 1, 10, 10), np.uint8)
    acts, _ = oracle_mod.act(net, theta, states, 0.0, 0)
    assert list(acts) == [1, 1, 1]


@pytest.mark.parametrize("A", [7, 18])
def test_eps_one_draws_from_the_action_counter(oracle_mod, A):
    rng = np.random.default_rng(47)
    net, theta = _net_theta(oracle_mod, rng, A)
    n, seed = 500, 0xDEADBEEF12345
    states = rng.integers(0, 256, (n, 1, 10, 10), dtype=np.uint8)
    acts, _ = oracle_mod.act(net, theta, states, 1.0, seed)
    want = [(((mix((seed + (2 * e + 2) * G) & M64) >> 32) * A) >> 32) for e in range(n)]
    assert list(acts) == want
    counts = np.bincount(acts, minlength=A)
    chi2 = ((counts - n / A) ** 2 / (n / A)).sum()
    assert chi2 < A + 6 * math.sqrt(2 * A)   # ~6 sigma for a chi-square(A-1)


def test_explore_rate_and_determinism(oracle_mod):
    rng = np.random.default_rng(53)
    net, theta = _net_theta(oracle_mod, rng)
    n, eps, seed = 4096, 0.05, 1507001
    states = rng.integers(0, 256, (n, 1, 10, 10), dtype=np.uint8)
    acts, q = oracle_mod.act(net, theta, states, eps, seed)
    acts2, _ = oracle_mod.act(net, theta, states, eps, seed)
    np.testing.assert_array_equal(acts, acts2)
    thr = math.floor(float(np.float32(eps)) * 2.0 ** 53)
    explore = np.array([(mix((seed + (2 * e + 1) * G) & M64) >> 11) < thr for e in range(n)])
    k = int(explore.sum())
    assert abs(k - n * eps) < 5 * math.sqrt(n * eps * (1 - eps))
    greedy = np.argmax(q, axis=1)
    np.testing.assert_array_equal(acts[~explore], greedy[~explore])
    acts3, _ = oracle_mod.act(net, theta, states, eps, seed + 1)
    assert (acts3 != acts).any()
