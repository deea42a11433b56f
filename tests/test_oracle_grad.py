"""Pins for the oracle's forward pass and gradient.

- Forward and gradient against torch CPU fp64 conv2d/linear + autograd (a
  library special case of the same definitions: catches transposed operands,
  wrong strides, flatten order, sign and scale of the gradient).
- Central finite differences on tiny topologies (every parameter) and on
  sampled coordinates of the full Atari network.
- Batch semantics: the minibatch gradient is the mean of single-sample
  gradients, permutation invariant, and a duplicated row counts twice.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

TINY = dict(in_c=2, in_h=12, in_w=12, c1=3, k1=4, s1=2, c2=4, k2=3, s2=1,
            c3=2, k3=2, s3=1, hidden=6, n_actions=3)
TINY2 = dict(in_c=1, in_h=10, in_w=9, c1=2, k1=3, s1=3, c2=3, k2=2, s2=1,
             c3=3, k3=2, s3=1, hidden=4, n_actions=5)


def _tensors(oracle_mod, net, theta):
    off = oracle_mod.param_offsets(net)
    t = torch.from_numpy(np.asarray(theta, np.float64))
    W1 = t[off[0]:off[1]].view(net.c1, net.in_c, net.k1, net.k1)
    W2 = t[off[2]:off[3]].view(net.c2, net.c1, net.k2, net.k2)
    W3 = t[off[4]:off[5]].view(net.c3, net.c2, net.k3, net.k3)
    W4 = t[off[6]:off[7]].view(net.hidden, -1)
    W5 = t[off[8]:off[9]].view(net.n_actions, net.hidden)
    return [W1, t[off[1]:off[2]], W2, t[off[3]:off[4]], W3, t[off[5]:off[6]],
            W4, t[off[7]:off[8]], W5, t[off[9]:off[10]]]


def _torch_q(net, ts, states):
    W1, b1, W2, b2, W3, b3, W4, b4, W5, b5 = ts
    x = torch.from_numpy(states.astype(np.float64)) / 255.0
    h = F.relu(F.conv2d(x, W1, b1, stride=net.s1))
    h = F.relu(F.conv2d(h, W2, b2, stride=net.s2))
    h = F.relu(F.conv2d(h, W3, b3, stride=net.s3))
    h = F.relu(F.linear(h.flatten(1), W4, b4))
    return F.linear(h, W5, b5)


def _random_theta(oracle_mod, net, rng, scale=1.0, bias=0.1):
    off = oracle_mod.param_offsets(net)
    theta = np.zeros(off[-1])
    fan = [net.in_c * net.k1 ** 2, None, net.c1 * net.k2 ** 2, None,
           net.c2 * net.k3 ** 2, None, (off[7] - off[6]) // net.hidden, None,
           net.hidden, None]
    for t in range(10):
        n = off[t + 1] - off[t]
        std = scale * math.sqrt(2.0 / fan[t]) if fan[t] else bias
        theta[off[t]:off[t + 1]] = rng.normal(0, std, n)
    return theta


def _batch(net, rng, B):
    shape = (B, net.in_c, net.in_h, net.in_w)
    s = rng.integers(0, 256, shape, dtype=np.uint8)
    s2 = rng.integers(0, 256, shape, dtype=np.uint8)
    a = rng.integers(0, net.n_actions, B).astype(np.int32)
    r = rng.choice(np.array([-1.0, 0.0, 1.0], np.float32), B)
    t = (rng.random(B) < 0.3).astype(np.uint8)
    return s, s2, a, r, t


@pytest.mark.parametrize("topo", ["tiny", "tiny2", "full"])
def test_forward_matches_torch_fp64(oracle_mod, topo):
    net = {"tiny": oracle_mod.Net(**TINY), "tiny2": oracle_mod.Net(**TINY2),
           "full": oracle_mod.Net()}[topo]
    rng = np.random.default_rng(11)
    theta = _random_theta(oracle_mod, net, rng)
    states = rng.integers(0, 256, (3, net.in_c, net.in_h, net.in_w), dtype=np.uint8)
    q = oracle_mod.q_forward(net, theta, states)
    qt = _torch_q(net, _tensors(oracle_mod, net, theta), states).numpy()
    np.testing.assert_allclose(q, qt, rtol=1e-12, atol=1e-12 * np.abs(qt).max())


@pytest.mark.parametrize("clip", [1.0, math.inf])
@pytest.mark.parametrize("topo", ["tiny", "full"])
def test_gradient_matches_torch_autograd(oracle_mod, topo, clip):
    net = oracle_mod.Net(**TINY) if topo == "tiny" else oracle_mod.Net(n_actions=6)
    rng = np.random.default_rng(5)
    theta = _random_theta(oracle_mod, net, rng)
    tgt = theta + rng.normal(0, 0.01, theta.shape)
    B = 4
    s, s2, a, r, t = _batch(net, rng, B)
    gamma = 0.99
    out = oracle_mod.learner_step(net, theta, tgt, s, s2, a, r, t, gamma, clip)

    ts = [x.clone().requires_grad_(True) for x in _tensors(oracle_mod, net, theta)]
    with torch.no_grad():
        q2 = _torch_q(net, _tensors(oracle_mod, net, tgt), s2)
        y = torch.from_numpy(r.astype(np.float64)) + float(np.float32(gamma)) * \
            (1 - torch.from_numpy(t.astype(np.float64))) * q2.max(1).values
    q = _torch_q(net, ts, s)
    qa = q[torch.arange(B), torch.from_numpy(a).long()]
    if math.isinf(clip):
        loss = (0.5 * (y - qa) ** 2).mean()
    else:
        loss = F.huber_loss(qa, y, delta=clip, reduction="mean")
    loss.backward()
    assert out["loss"] == pytest.approx(loss.item(), rel=1e-12)
    off = oracle_mod.param_offsets(net)
    for k, x in enumerate(ts):
        g = out["grads"][off[k]:off[k + 1]]
        gt = x.grad.flatten().numpy()
        scale = max(np.abs(gt).max(), 1e-300)
        np.testing.assert_allclose(g, gt, rtol=1e-10, atol=1e-11 * scale, err_msg=f"tensor {k}")
    # sanity: the sample really exercises both ReLU branches and nonzero grads
    assert np.abs(out["grads"]).max() > 0


def _loss(oracle_mod, net, theta, tgt, batch, gamma, clip):
    s, s2, a, r, t = batch
    return oracle_mod.learner_step(net, theta, tgt, s, s2, a, r, t, gamma, clip)["loss"]


@pytest.mark.parametrize("topo", ["tiny", "tiny2"])
@pytest.mark.parametrize("clip", [1.0, math.inf])
def test_finite_differences_tiny_all_parameters(oracle_mod, topo, clip):
    net = oracle_mod.Net(**(TINY if topo == "tiny" else TINY2))
    rng = np.random.default_rng(17)
    theta = _random_theta(oracle_mod, net, rng, scale=1.5, bias=0.3)
    tgt = theta + rng.normal(0, 0.05, theta.shape)
    batch = _batch(net, rng, 3)
    # push rewards so that some samples sit in Huber's linear zone
    batch = (batch[0], batch[1], batch[2], batch[3] * 3, batch[4])
    gamma = 0.9
    g = oracle_mod.learner_step(net, theta, tgt, *batch, gamma, clip)["grads"]
    fd = np.zeros_like(g)
    for i in range(theta.shape[0]):
        h = 1e-6 * max(1.0, abs(theta[i]))
        tp = theta.copy(); tp[i] += h
        tm = theta.copy(); tm[i] -= h
        fd[i] = (_loss(oracle_mod, net, tp, tgt, batch, gamma, clip) -
                 _loss(oracle_mod, net, tm, tgt, batch, gamma, clip)) / (2 * h)
    scale = np.abs(g).max()
    assert scale > 0
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-7 * scale)


@pytest.mark.slow
def test_finite_differences_full_network_sampled(oracle_mod):
    net = oracle_mod.Net()
    rng = np.random.default_rng(23)
    theta = _random_theta(oracle_mod, net, rng)
    tgt = theta + rng.normal(0, 0.01, theta.shape)
    batch = _batch(net, rng, 2)
    gamma, clip = 0.99, 1.0
    g = oracle_mod.learner_step(net, theta, tgt, *batch, gamma, clip)["grads"]
    off = oracle_mod.param_offsets(net)
    for k in range(10):
        lo, hi = off[k], off[k + 1]
        # prefer coordinates with a non-negligible gradient
        cand = np.arange(lo, hi)
        big = cand[np.abs(g[lo:hi]) > 1e-3 * np.abs(g[lo:hi]).max()] if g[lo:hi].any() else cand
        pick = rng.choice(big, size=min(4, big.size), replace=False)
        for i in pick:
            h = 1e-5 * max(1.0, abs(theta[i]))
            tp = theta.copy(); tp[i] += h
            tm = theta.copy(); tm[i] -= h
            fd = (_loss(oracle_mod, net, tp, tgt, batch, gamma, clip) -
                  _loss(oracle_mod, net, tm, tgt, batch, gamma, clip)) / (2 * h)
            assert fd == pytest.approx(g[i], rel=1e-5, abs=1e-9), (k, i)


def test_batch_mean_permutation_and_duplicates(oracle_mod):
    net = oracle_mod.Net(**TINY)
    rng = np.random.default_rng(29)
    theta = _random_theta(oracle_mod, net, rng)
    tgt = theta + rng.normal(0, 0.02, theta.shape)
    s, s2, a, r, t = _batch(net, rng, 5)
    gamma = 0.99
    full = oracle_mod.learner_step(net, theta, tgt, s, s2, a, r, t, gamma)
    singles = [oracle_mod.learner_step(net, theta, tgt, s[i:i + 1], s2[i:i + 1], a[i:i + 1],
                                       r[i:i + 1], t[i:i + 1], gamma) for i in range(5)]
    np.testing.assert_allclose(full["grads"], np.mean([x["grads"] for x in singles], 0),
                               rtol=1e-12, atol=1e-15)
    assert full["loss"] == pytest.approx(np.mean([x["loss"] for x in singles]), rel=1e-13)
    perm = np.array([3, 0, 4, 2, 1])
    pf = oracle_mod.learner_step(net, theta, tgt, s[perm], s2[perm], a[perm], r[perm],
                                 t[perm], gamma)
    np.testing.assert_allclose(pf["grads"], full["grads"], rtol=1e-12, atol=1e-15)
    dup = np.array([0, 0, 1])
    d = oracle_mod.learner_step(net, theta, tgt, s[dup], s2[dup], a[dup], r[dup], t[dup], gamma)
    want = (2 * singles[0]["grads"] + singles[1]["grads"]) / 3
    np.testing.assert_allclose(d["grads"], want, rtol=1e-12, atol=1e-15)


def test_no_gradient_flows_into_target(oracle_mod):
    """theta- only enters through y; changing it moves y but the gradient is
    still taken w.r.t. theta alone (eq. (2))."""
    net = oracle_mod.Net(**TINY)
    rng = np.random.default_rng(31)
    theta = _random_theta(oracle_mod, net, rng)
    s, s2, a, r, t = _batch(net, rng, 3)
    t[:] = 1  # terminal everywhere: theta- cannot matter at all
    o1 = oracle_mod.learner_step(net, theta, theta, s, s2, a, r, t, 0.99)
    o2 = oracle_mod.learner_step(net, theta, theta * 3.0 + 1.0, s, s2, a, r, t, 0.99)
    np.testing.assert_array_equal(o1["grads"], o2["grads"])
    assert o1["loss"] == o2["loss"]


def test_kink_margin_closed_form(oracle_mod):
    """A hidden unit built to sit exactly on the ReLU kink has margin 0; moving
    one of its weights by a relative 1e-3 moves the margin to the closed-form
    |h0 - (1 + 1e-3) h0| / (h0 + (1 + 1e-3) h0)."""
    net = oracle_mod.Net(**TINY)
    off = oracle_mod.param_offsets(net)
    rng = np.random.default_rng(37)
    theta = _random_theta(oracle_mod, net, rng, bias=0.0)
    # conv3 channels 0 and 1 identical -> h3[c=0] == h3[c=1] elementwise
    W3 = theta[off[4]:off[5]].reshape(net.c3, net.c2, net.k3, net.k3)
    W3[1] = W3[0]
    theta[off[5]:off[6]] = 0.0
    W4 = theta[off[6]:off[7]].reshape(net.hidden, -1)
    W4[:] = np.abs(W4) + 0.1          # every other hidden unit clearly positive
    theta[off[7]:off[8]] = 0.0
    P3 = (off[7] - off[6]) // net.hidden // net.c3   # conv3 output pixels
    W4[0] = 0.0
    W4[0, 0], W4[0, P3] = 1.0, -1.0                  # z4[0] = h3[0,0] - h3[1,0] = 0
    s = rng.integers(0, 256, (1, net.in_c, net.in_h, net.in_w), dtype=np.uint8)
    args = (s, s, np.array([0], np.int32), np.zeros(1, np.float32), np.zeros(1, np.uint8), 0.9)
    out = oracle_mod.learner_step(net, theta, theta, *args)
    assert out["margin"][0] == 0.0
    W4[0, P3] = -(1.0 + 1e-3)
    out = oracle_mod.learner_step(net, theta, theta, *args)
    h0 = out["margin"][0]
    assert 0 < h0 <= 1e-3 / (2 + 1e-3) * (1 + 1e-12)
