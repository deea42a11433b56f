"""Pins of the oracle's actor side: replay insert (Algorithm 1 "store the
transition in D", Section 4 replay memory) against a bounded-deque model of the
same memory, and the epsilon schedule of Section 5.1 (1 -> 0.1 over the first
million updates) against its closed form."""
import collections

import numpy as np


def _ring(cap, fshape=(3, 5)):
    return (np.zeros((cap,) + fshape, np.uint8), np.zeros(cap, np.uint8),
            np.zeros(cap, np.int32), np.zeros(cap, np.float32))


def test_insert_matches_bounded_deque(oracle_mod):
    rng = np.random.default_rng(21)
    cap = 11
    frames, ep, act, rew = _ring(cap)
    model = collections.deque(maxlen=cap)  # logical order, oldest first
    head, size = 0, 0
    for call in range(40):
        m = int(rng.integers(0, 6))
        fi = rng.integers(0, 256, (m, 3, 5)).astype(np.uint8)
        ei = (rng.random(m) < 0.3).astype(np.uint8)
        ai = rng.integers(0, 18, m).astype(np.int32)
        ri = rng.standard_normal(m).astype(np.float32)
        head, size = oracle_mod.replay_insert(frames, ep, act, rew, head, size, fi, ei, ai, ri)
        for j in range(m):
            model.append((fi[j].copy(), int(ei[j]), int(ai[j]), float(ri[j])))
        assert size == len(model)
        for k, (f, e, a, r) in enumerate(model):
            slot = (head + k) % cap
            np.testing.assert_array_equal(frames[slot], f)
            assert (ep[slot], act[slot], rew[slot]) == (e, a, np.float32(r)), (call, k)


def test_insert_then_gather_stacks_a_trajectory(oracle_mod):
    """Frames stored by insert come back as four-frame stacks with zero-fill
    at the episode starts the actor flagged (checked by brute force)."""
    rng = np.random.default_rng(22)
    cap, T = 9, 23  # the ring wraps twice
    frames, ep, act, rew = _ring(cap, (2, 2))
    traj_f = rng.integers(1, 256, (T, 2, 2)).astype(np.uint8)
    traj_e = np.zeros(T, np.uint8)
    traj_e[[0, 5, 6, 14, 20]] = 1
    traj_a = np.arange(T, dtype=np.int32) % 18
    traj_r = np.linspace(-1, 1, T).astype(np.float32)
    head, size = 0, 0
    for t in range(T):  # one record per environment step
        head, size = oracle_mod.replay_insert(frames, ep, act, rew, head, size, traj_f[t:t + 1],
                                              traj_e[t:t + 1], traj_a[t:t + 1], traj_r[t:t + 1])
    assert size == cap and head == T % cap
    first = T - cap  # trajectory index of logical 0
    idx = np.arange(0, cap - 1, dtype=np.int64)
    out = oracle_mod.gather(frames, ep, act, rew, head, idx)
    for k in idx:
        for w, key in ((0, "s"), (1, "s2")):
            kn = k + w
            # latest episode start at or before kn, logical 0 counting as one
            e = max([0] + [j for j in range(1, kn + 1) if traj_e[first + j]])
            for c in range(4):
                l = kn - 3 + c
                want = traj_f[first + l] if l >= e else np.zeros((2, 2), np.uint8)
                np.testing.assert_array_equal(out[key][k, c], want, err_msg=f"k={k} {key} c={c}")
        assert out["a"][k] == traj_a[first + k] and out["r"][k] == traj_r[first + k]
        assert out["term"][k] == traj_e[first + k + 1]


def test_insert_rejects_more_than_capacity(oracle_mod):
    frames, ep, act, rew = _ring(4)
    import pytest
    with pytest.raises(ValueError):
        oracle_mod.replay_insert(frames, ep, act, rew, 0, 0, np.zeros((5, 3, 5), np.uint8),
                                 np.zeros(5), np.zeros(5), np.zeros(5))


def test_epsilon_schedule_closed_form(oracle_mod):
    assert oracle_mod.epsilon(0) == 1.0
    assert oracle_mod.epsilon(-5) == 1.0
    assert abs(oracle_mod.epsilon(500_000) - 0.55) < 1e-15
    assert abs(oracle_mod.epsilon(250_000) - 0.775) < 1e-15
    assert oracle_mod.epsilon(1_000_000) == 0.1 and oracle_mod.epsilon(5_000_000) == 0.1
    e = [oracle_mod.epsilon(u) for u in range(0, 1_000_001, 50_000)]
    assert all(a > b for a, b in zip(e, e[1:]))
    # linear: equal steps per update
    d = np.diff(e)
    np.testing.assert_allclose(d, -0.9 / 20, rtol=1e-12)


def test_insert_accepts_strided_inputs(oracle_mod):
    """Column views of [m, rings] record arrays (copied by the wrapper) store
    the same records as contiguous inputs."""
    rng = np.random.default_rng(23)
    m, rings, cap = 6, 3, 10
    fi = rng.integers(0, 256, (m, rings, 3, 5)).astype(np.uint8)
    ei = (rng.random((m, rings)) < 0.5).astype(np.uint8)
    ai = rng.integers(0, 18, (m, rings)).astype(np.int32)
    ri = rng.standard_normal((m, rings)).astype(np.float32)
    a = _ring(cap)
    b = _ring(cap)
    oracle_mod.replay_insert(*a, 0, 0, fi[:, 1], ei[:, 1], ai[:, 1], ri[:, 1])
    oracle_mod.replay_insert(*b, 0, 0, fi[:, 1].copy(), ei[:, 1].copy(), ai[:, 1].copy(),
                             ri[:, 1].copy())
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(a[2][:m], ai[:, 1])
    np.testing.assert_array_equal(a[3][:m], ri[:, 1])


# ---------------------------------------------------------------------------
# Parameter pull / target sync (Algorithm 1; Section 5.1 N = 60K)
# ---------------------------------------------------------------------------
def test_bf16_rounding_hand_values(oracle_mod):
    assert oracle_mod.f32_to_bf16(1.0) == 0x3F80
    assert oracle_mod.f32_to_bf16(1 + 2 ** -8) == 0x3F80          # tie, even stays
    assert oracle_mod.f32_to_bf16(1 + 3 * 2 ** -8) == 0x3F82      # tie, rounds up to even
    assert oracle_mod.f32_to_bf16(1 + 2 ** -8 + 2 ** -20) == 0x3F81  # above the tie
    assert oracle_mod.f32_to_bf16(1.9921875 + 2 ** -8) == 0x4000   # tie carrying into the exponent
    assert oracle_mod.f32_to_bf16(-2.5) == 0xC020
    assert oracle_mod.f32_to_bf16(0.0) == 0 and oracle_mod.f32_to_bf16(-0.0) == 0x8000


def test_bf16_rounding_matches_torch():
    """torch's float32 -> bfloat16 conversion (round to nearest even) is a
    library special case of the oracle's rounding."""
    import torch

    import oracle
    rng = np.random.default_rng(24)
    x = np.concatenate([rng.standard_normal(20000), rng.standard_normal(20000) * 1e-39,
                        rng.standard_normal(20000) * 1e30]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    d, _, _ = oracle.params_sync(x, [0], 1, 0, 1, True)
    np.testing.assert_array_equal(d[0], want)


def test_sync_period_crossing(oracle_mod):
    """Copied iff some multiple of the period lies in (held version, current]."""
    rng = np.random.default_rng(25)
    src = rng.standard_normal(5).astype(np.float32)
    for trial in range(300):
        period = int(rng.integers(1, 12))
        held = rng.integers(0, 60, 4)
        now = int(held.max() + rng.integers(0, 30))
        d, v, synced = oracle_mod.params_sync(src, held, now, period, 4, False)
        for c in range(4):
            want = any(m % period == 0 for m in range(int(held[c]) + 1, now + 1))
            assert synced[c] == want, (trial, period, held[c], now)
            if want:
                np.testing.assert_array_equal(d[c], src)
                assert v[c] == now
            else:
                assert not d[c].any() and v[c] == held[c]


def test_pull_without_period_always_copies(oracle_mod):
    src = np.arange(7, dtype=np.float32) - 3.5
    d, v, synced = oracle_mod.params_sync(src, [5, 9], 9, 0, 2, False)
    assert list(synced) == [1, 1] and list(v) == [9, 9]
    np.testing.assert_array_equal(d, np.stack([src, src]))
