"""GPU parity of the parameter-server side (Section 4 parameter server,
Section 4.2 stability) against the fp64 oracle on the same seeded inputs.

Bars: the apply decisions and the server version are integers (bit-exact);
the loss-filter statistics and decisions are fp64 operations rounded once on
both sides in the same order (bit-exact); theta+ and the AdaGrad accumulator
are fp32 on the GPU and fp64 in the oracle, so they are compared against an
error bound derived from the arithmetic: each AdaGrad step rounds the
accumulator once (relative 2^-24) and the update lr g / (eps + sqrt h) in at
most five operations, then rounds theta once, so after T applied gradients
    |theta - theta*| <= 2^-22 (T |theta| + 8 sum_t |u_t|),
    |h - h*| <= 2^-22 T h*,
with u_t the oracle's update at step t (the factor 4 over 2^-24 covers
propagation into later steps).
"""
import sys

import numpy as np
import pytest

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


@pytest.fixture(scope="module")
def ctx(g):
    c = g.Context(max_batch=1, n_actions=18)
    yield c
    c.close()


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _apply_case(torch, g, ctx, oracle_mod, inp, max_delay, lr, eps, use_keep=True):
    G, n = inp.grads.shape
    theta, accum = _dev(torch, inp.theta), _dev(torch, inp.accum)
    grads = _dev(torch, inp.grads)
    ver = _dev(torch, inp.version)
    psv = _dev(torch, np.array([inp.ps_version], np.int64))
    applied = torch.empty(G, dtype=torch.uint8, device="cuda")
    keep = _dev(torch, inp.keep) if use_keep else None
    g.gorila_ps_apply(ctx, theta, accum, grads, ver, psv, max_delay, lr, eps, applied, keep)
    ctx.check()
    ref = oracle_mod.ps_apply(inp.theta, inp.accum, inp.grads, inp.version, inp.ps_version,
                              max_delay, lr, eps, inp.keep if use_keep else None)
    np.testing.assert_array_equal(applied.cpu().numpy(), ref["applied"])
    assert int(psv.cpu()[0]) == ref["ps_version"]
    # error bound from the arithmetic (see the module docstring)
    sel = inp.grads[ref["applied"].astype(bool)].astype(np.float64)
    T = sel.shape[0]
    lr32, eps32 = float(np.float32(lr)), float(np.float32(eps))
    h = inp.accum.astype(np.float64) + np.cumsum(sel * sel, axis=0) if T else None
    usum = (np.sum(lr32 * np.abs(sel) / (eps32 + np.sqrt(h)), axis=0) if T
            else np.zeros(n))
    bound_t = 2.0 ** -22 * (max(T, 1) * np.abs(ref["theta"]) + 8 * usum) + 1e-30
    bound_h = 2.0 ** -22 * max(T, 1) * ref["accum"] + 1e-30
    got_t = theta.cpu().numpy().astype(np.float64)
    got_h = accum.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got_t - ref["theta"]) <= bound_t), \
        float(np.max(np.abs(got_t - ref["theta"]) / bound_t))
    assert np.all(np.abs(got_h - ref["accum"]) <= bound_h), \
        float(np.max(np.abs(got_h - ref["accum"]) / bound_h))
    return ref, T


def test_ps_apply_16_gradients_full_network(torch_cuda, g, ctx, oracle_mod):
    """16 learner gradients of the 18-action network (P = 1,693,362)."""
    w = datagen.WORKLOADS["ps_apply_g16_a18_f32"]
    P = datagen.param_count(w["n_actions"])
    _say(f"ps_apply G={w['groups']} n={P} seed={w['seed']}")
    inp = datagen.ps_inputs(w["seed"], w["groups"], P)
    ref, T = _apply_case(torch_cuda, g, ctx, oracle_mod, inp, max_delay=10, lr=0.01, eps=1e-3)
    assert 0 < T < w["groups"]  # some gradients stale or not kept, some applied
    _say(f"applied {T} of {w['groups']}")


@pytest.mark.parametrize("G,n,max_delay", [(1, 1, 10), (3, 7, 10), (5, 1000003, 2), (0, 33, 1),
                                           (9, 4096, 0)])
def test_ps_apply_ragged(torch_cuda, g, ctx, oracle_mod, G, n, max_delay):
    _say(f"ps_apply ragged G={G} n={n} max_delay={max_delay}")
    inp = datagen.ps_inputs(9000 + n + G, G, n)
    _apply_case(torch_cuda, g, ctx, oracle_mod, inp, max_delay, 0.05, 1e-4)


def test_ps_apply_without_keep_mask(torch_cuda, g, ctx, oracle_mod):
    _say("ps_apply keep=NULL")
    inp = datagen.ps_inputs(9100, 6, 5000, max_lag=1)
    ref, T = _apply_case(torch_cuda, g, ctx, oracle_mod, inp, 100, 0.1, 1e-2, use_keep=False)
    assert T == 6


def test_ps_apply_argument_errors(torch_cuda, g, ctx):
    torch = torch_cuda
    th = torch.zeros(8, device="cuda")
    acc = torch.zeros(8, device="cuda")
    gr = torch.zeros((2, 8), device="cuda")
    ver = torch.zeros(2, dtype=torch.int64, device="cuda")
    psv = torch.zeros(1, dtype=torch.int64, device="cuda")
    app = torch.empty(2, dtype=torch.uint8, device="cuda")
    for lr, eps in ((0.1, 0.0), (-1.0, 1e-3), (0.1, -1e-3)):
        with pytest.raises(g.GorilaError) as e:
            g.gorila_ps_apply(ctx, th, acc, gr, ver, psv, 1, lr, eps, app)
        assert e.value.code == -1


@pytest.mark.parametrize("alpha", [0.0, 0.05])
def test_loss_filter_sequences(torch_cuda, g, ctx, oracle_mod, alpha):
    """200 steps of 16 learners; statistics and decisions bit-exact at every step."""
    torch = torch_cuda
    _say(f"loss_filter 200 x 16 alpha={alpha}")
    seq = datagen.loss_sequences(9200, 200, 16)
    k, warmup = 3.0, 10
    stats_d = torch.zeros((16, 3), dtype=torch.float64, device="cuda")
    stats_o = np.zeros((16, 3))
    keep_d = torch.empty(16, dtype=torch.uint8, device="cuda")
    discarded = 0
    for t in range(seq.shape[0]):
        g.gorila_loss_filter(ctx, stats_d, _dev(torch, seq[t]), alpha, k, warmup, keep_d)
        keep_o, stats_o = oracle_mod.loss_filter(stats_o, seq[t], alpha, k, warmup)
        np.testing.assert_array_equal(keep_d.cpu().numpy(), keep_o, err_msg=f"step {t}")
        np.testing.assert_array_equal(stats_d.cpu().numpy(), stats_o, err_msg=f"step {t}")
        discarded += int((keep_o == 0).sum())
    ctx.check()
    assert discarded > 0
    _say(f"discarded {discarded} of {seq.size}")


def test_loss_filter_argument_errors(torch_cuda, g, ctx):
    torch = torch_cuda
    st = torch.zeros((2, 3), dtype=torch.float64, device="cuda")
    loss = torch.zeros(2, device="cuda")
    keep = torch.empty(2, dtype=torch.uint8, device="cuda")
    for alpha, k in ((1.5, 3.0), (-0.1, 3.0), (0.1, -1.0)):
        with pytest.raises(g.GorilaError) as e:
            g.gorila_loss_filter(ctx, st, loss, alpha, k, 5, keep)
        assert e.value.code == -1


# ---------------------------------------------------------------------------
# Parameter pull / periodic target sync (Algorithm 1; Section 5.1)
# ---------------------------------------------------------------------------
def test_pull_16_bf16_replicas_full_network(torch_cuda, g, ctx, oracle_mod):
    """theta+ of the 18-action network rounded into 16 bf16 replicas: bit-exact."""
    torch = torch_cuda
    P = datagen.param_count(18)
    _say(f"params_sync pull 16 bf16 replicas n={P}")
    rng = np.random.default_rng(9300)
    src = (0.05 * rng.standard_normal(P)).astype(np.float32)
    held = np.arange(16, dtype=np.int64)
    dst = torch.zeros((16, P), dtype=torch.int16, device="cuda")
    ver = _dev(torch, held)
    psv = _dev(torch, np.array([40], np.int64))
    synced = torch.empty(16, dtype=torch.uint8, device="cuda")
    g.gorila_params_sync(ctx, _dev(torch, src), dst, ver, psv, 0, synced)
    ctx.check()
    want, wver, wsync = oracle_mod.params_sync(src, held, 40, 0, 16, True)
    np.testing.assert_array_equal(dst.cpu().numpy().view(np.uint16), want)
    np.testing.assert_array_equal(ver.cpu().numpy(), wver)
    np.testing.assert_array_equal(synced.cpu().numpy(), wsync)


@pytest.mark.parametrize("bf16", [False, True])
def test_periodic_target_sync(torch_cuda, g, ctx, oracle_mod, bf16):
    torch = torch_cuda
    _say(f"params_sync period 60 bf16={bf16}")
    rng = np.random.default_rng(9400 + bf16)
    n, copies, period, now = 10007, 6, 60, 245
    src = rng.standard_normal(n).astype(np.float32)
    held = np.array([0, 180, 239, 240, 241, 245], np.int64)  # due: 0, 180, 239
    prev_np = (rng.integers(0, 2 ** 15, (copies, n)).astype(np.uint16) if bf16 else
               rng.standard_normal((copies, n)).astype(np.float32))
    dst = _dev(torch, prev_np.view(np.int16) if bf16 else prev_np)
    ver = _dev(torch, held)
    psv = _dev(torch, np.array([now], np.int64))
    synced = torch.empty(copies, dtype=torch.uint8, device="cuda")
    g.gorila_params_sync(ctx, _dev(torch, src), dst, ver, psv, period, synced)
    ctx.check()
    want, wver, wsync = oracle_mod.params_sync(src, held, now, period, copies, bf16, dst=prev_np)
    got = dst.cpu().numpy()
    np.testing.assert_array_equal(got.view(np.uint16) if bf16 else got, want)
    np.testing.assert_array_equal(ver.cpu().numpy(), wver)
    np.testing.assert_array_equal(synced.cpu().numpy(), wsync)
    assert list(wsync) == [1, 1, 1, 0, 0, 0]
