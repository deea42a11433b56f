"""The no-allocation actor call (gorila_act_noalloc: static device scratch, no
workspace) against gorila_act on the same inputs, through the C-ABI: actions
bit-exact, Q within 1e-4 relative.  Two calls in a row, the second smaller, so
the scratch's leftovers from the first must not leak into the second."""
import sys

import numpy as np
import pytest

import parity
from paper_1507_04296_amd import datagen

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    return torch


@pytest.fixture(scope="module")
def g(torch_cuda):
    import paper_1507_04296_amd as gmod
    gmod.lib()
    return gmod


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _compare(torch, g, ctx_ws, ctx_none, theta, A, states, eps, seed):
    n = states.shape[0]
    ref_a, ref_q = g.act(ctx_ws, theta, A, states, eps, seed, with_q=True)
    acts = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    q = torch.full((n, A), float("nan"), dtype=torch.float32, device="cuda")
    g.gorila_act_noalloc(ctx_none, theta, A, states, eps, seed, acts, q)
    ctx_ws.check()
    ctx_none.check()
    np.testing.assert_array_equal(acts.cpu().numpy(), ref_a.cpu().numpy())
    assert parity.q_rel_err(q.cpu().numpy(), ref_q.cpu().numpy()) <= parity.Q_TOL
    return bool(torch.equal(q, ref_q))


def test_act_noalloc_matches_act(torch_cuda, g):
    torch = torch_cuda
    w = datagen.WORKLOADS["actor_n1024_a18_f32"]
    A = w["n_actions"]
    inp = datagen.actor_inputs(w["seed"], 300, A, w["eps"])
    theta = _dev(torch, inp.theta)
    ctx_ws = g.Context(max_batch=g.NOALLOC_MAX_STATES, n_actions=A)
    ctx_none = g.Context(max_batch=0, n_actions=A)  # no workspace at all
    states = _dev(torch, inp.states)
    for n, eps, seed in ((g.NOALLOC_MAX_STATES, 0.05, inp.seed), (37, 0.0, 11), (37, 0.5, 12)):
        _say(f"act_noalloc n={n} eps={eps} vs act")
        same = _compare(torch, g, ctx_ws, ctx_none, theta, A, states[:n], eps, seed)
        _say(f"bitwise-equal Q: {same}")
    # bf16 parameters (widened in the scratch), 6 actions
    inp6 = datagen.learner_inputs(9100, 64, 6)
    bits = datagen.to_bf16_bits(inp6.theta.astype(np.float64))
    _say("act_noalloc bf16 n=64 A=6")
    _compare(torch, g, ctx_ws, ctx_none, _dev(torch, bits.view(np.int16)), 6,
             _dev(torch, inp6.s), 0.0, 3)
    # without Q output
    acts = torch.empty(5, dtype=torch.int32, device="cuda")
    g.gorila_act_noalloc(ctx_none, theta, A, states[:5], 0.0, 1, acts)
    ref = g.act(ctx_ws, theta, A, states[:5], 0.0, 1)
    ctx_none.check()
    assert torch.equal(acts, ref.to(torch.int32))
    ctx_ws.close()
    ctx_none.close()


def test_act_noalloc_limits(torch_cuda, g):
    torch = torch_cuda
    A = 18
    ctx_none = g.Context(max_batch=0, n_actions=A)
    inp = datagen.learner_inputs(9200, 4, A)
    theta = _dev(torch, inp.theta)
    big = torch.zeros((g.NOALLOC_MAX_STATES + 1, 4, 84, 84), dtype=torch.uint8, device="cuda")
    acts = torch.empty(big.shape[0], dtype=torch.int32, device="cuda")
    with pytest.raises(g.GorilaError) as e:  # beyond the stated maximum
        g.gorila_act_noalloc(ctx_none, theta, A, big, 0.0, 1, acts)
    assert e.value.code == -3
    # n = 0 is a no-op
    g.gorila_act_noalloc(ctx_none, theta, A, big[:0], 0.0, 1, acts[:0])
    # the calls that need a workspace refuse a context without one
    rep = g.Replay.stacked(_dev(torch, inp.s), _dev(torch, inp.s2), _dev(torch, inp.a),
                           _dev(torch, inp.r), _dev(torch, inp.term))
    with pytest.raises(g.GorilaError) as e:
        g.learner_step(ctx_none, theta, _dev(torch, inp.theta_target), A, rep, _dev(torch, inp.idx))
    assert e.value.code == -3
    with pytest.raises(g.GorilaError) as e:
        g.q_forward(ctx_none, theta, A, _dev(torch, inp.s))
    assert e.value.code == -3
    with pytest.raises(g.GorilaError) as e:
        g.gather(ctx_none, rep, _dev(torch, inp.idx))
    assert e.value.code == -3
    ctx_none.check()
    ctx_none.close()
