"""GPU parity of the grouped learner step (Section 4: many learners, each on its
own possibly stale copy of theta, one shared target theta-) and of bf16
parameter sets, against the fp64 oracle run once per group.

bf16 parameters are bit patterns; the oracle takes their exact fp64 values.
When every parameter set of a step is bf16 the HIP path multiplies bf16 MFMA
operands with fp32 accumulation (forward activations as two bf16 terms,
backward operands rounded to bf16): every gradient tensor within 2e-2
relative L2 and the loss within 1e-4 relative.  Mixed fp32 / bf16 steps and
the forward-only calls compute in fp32 from the exactly widened values and
meet the fp32 bars (Q and loss 1e-4 relative, gradients 1e-3 relative L2).
The stale-replica workload is checked on exactly the rows bench.py times.
"""
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


def _group_rows(G, pool, batch):
    """idx [G*batch]: group g takes the first `batch` of its `pool` rows."""
    return np.concatenate([gi * pool + np.arange(batch) for gi in range(G)]).astype(np.int64)


def _oracle_groups(oracle_mod, net, thetas64, target64, inp, idx, batch, clip=1.0):
    out = []
    for gi, th in enumerate(thetas64):
        ix = idx[gi * batch:(gi + 1) * batch]
        out.append(oracle_mod.learner_step(net, th, target64, inp.s[ix], inp.s2[ix], inp.a[ix],
                                           inp.r[ix], inp.term[ix], inp.gamma, clip))
    return out


def _replay(torch, g, inp):
    return g.Replay.stacked(_dev(torch, inp.s), _dev(torch, inp.s2), _dev(torch, inp.a),
                            _dev(torch, inp.r), _dev(torch, inp.term))


def test_grouped_16x64_bf16_a18(torch_cuda, g, oracle_mod):
    """The stale-replica workload: 16 bf16 replicas x 64 transitions, 18 actions."""
    torch = torch_cuda
    w = datagen.WORKLOADS["grouped_g16_b64_a18_bf16"]
    G, b, A = w["groups"], w["batch"], w["n_actions"]
    _say(f"grouped G={G} b={b} A={A} bf16 seed={w['seed']}")
    inp = datagen.grouped_inputs(w["seed"], G, b, A)
    net = oracle_mod.Net(n_actions=A)
    th64 = [datagen.bf16_bits_to_f64(t) for t in inp.theta_bf16]
    tg64 = datagen.bf16_bits_to_f64(inp.target_bf16)
    idx = _group_rows(G, b, b)
    np.testing.assert_array_equal(idx, np.arange(G * b))  # the rows bench.py times
    ctx = g.Context(max_batch=b, n_actions=A, groups=G, dtype=g.GORILA_BF16)
    thetas = _dev(torch, inp.theta_bf16.view(np.int16))
    target = _dev(torch, inp.target_bf16.view(np.int16))
    grads, loss = g.learner_step_grouped(ctx, thetas, target, A, _replay(torch, g, inp),
                                         _dev(torch, idx), inp.gamma, 1.0)
    ctx.check()
    q, qn, td = g.learner_td(ctx, G * b, A)
    got_g, got_l = grads.cpu().numpy(), loss.cpu().numpy()
    q, qn, td = q.cpu().numpy(), qn.cpu().numpy(), td.cpu().numpy()
    ref = _oracle_groups(oracle_mod, net, th64, tg64, inp, idx, b)
    worst, worst_td = {}, {}
    for gi in range(G):
        errs = parity.assert_grads_close(got_g[gi], ref[gi]["grads"], A, parity.GRAD_TOL_BF16)
        assert abs(got_l[gi] - ref[gi]["loss"]) <= parity.LOSS_TOL * abs(ref[gi]["loss"]), gi
        rows = slice(gi * b, (gi + 1) * b)
        tde = parity.assert_td_close(q[rows], qn[rows], td[rows], ref[gi], 1.0)
        for k, v in errs.items():
            worst[k] = max(worst.get(k, 0.0), v)
        for k, v in tde.items():
            worst_td[k] = max(worst_td.get(k, 0.0), v)
    _say(f"worst grad rel-L2 over groups {worst}; td errors / Q scale {worst_td}")
    # replicas differ, so their gradients must too
    assert not np.array_equal(got_g[0], got_g[1])
    ctx.close()


def test_grouped_ragged_mixed_dtypes(torch_cuda, g, oracle_mod):
    """3 groups of 37 rows, 7 actions; replicas fp32, bf16, fp32; bf16 target."""
    torch = torch_cuda
    G, b, A, pool = 3, 37, 7, 60
    _say(f"grouped ragged G={G} b={b} A={A} mixed dtypes")
    inp = datagen.grouped_inputs(8100, G, pool, A)
    net = oracle_mod.Net(n_actions=A)
    th64 = [datagen.bf16_bits_to_f64(t) for t in inp.theta_bf16]
    # replica 0 and 2 in fp32: perturb so they are not bf16-representable
    rng = np.random.default_rng(8101)
    th64[0] = (th64[0] + 1e-4 * rng.standard_normal(th64[0].shape[0])).astype(np.float32)
    th64[2] = (th64[2] - 1e-4 * rng.standard_normal(th64[2].shape[0])).astype(np.float32)
    th64 = [np.asarray(t, np.float64) for t in th64]
    tg64 = datagen.bf16_bits_to_f64(inp.target_bf16)
    idx = _group_rows(G, pool, b)
    ctx = g.Context(max_batch=b, n_actions=A, groups=G, dtype=g.GORILA_BF16)
    thetas = [_dev(torch, th64[0].astype(np.float32)),
              _dev(torch, inp.theta_bf16[1].view(np.int16)),
              _dev(torch, th64[2].astype(np.float32))]
    target = _dev(torch, inp.target_bf16.view(np.int16))
    grads, loss = g.learner_step_grouped(ctx, thetas, target, A, _replay(torch, g, inp),
                                         _dev(torch, idx), inp.gamma, 0.5)
    ctx.check()
    ref = _oracle_groups(oracle_mod, net, th64, tg64, inp, idx, b, clip=0.5)
    for gi in range(G):
        parity.assert_grads_close(grads[gi].cpu().numpy(), ref[gi]["grads"], A)
        l = float(loss[gi].cpu())
        assert abs(l - ref[gi]["loss"]) <= parity.LOSS_TOL * abs(ref[gi]["loss"]), gi
    ctx.close()


@pytest.mark.parametrize("G,b,A,clip", [(3, 37, 7, 0.5), (1, 100, 4, 1.0), (2, 24, 5, 1.0),
                                          (5, 53, 6, 1.0)])
def test_grouped_all_bf16_ragged(torch_cuda, g, oracle_mod, G, b, A, clip):
    """All-bf16 steps (bf16 MFMA operands) at ragged batch sizes: partial
    row tiles, one group on its own; 48 learner rows cut the fc1 and conv3
    data-gradient reductions into four parts (fp32 partial planes), 265 rows
    into none (gradients handed on as bf16)."""
    torch = torch_cuda
    pool = b + b // 2 + 8
    _say(f"grouped all-bf16 G={G} b={b} A={A}")
    inp = datagen.grouped_inputs(8300 + G, G, pool, A)
    net = oracle_mod.Net(n_actions=A)
    th64 = [datagen.bf16_bits_to_f64(t) for t in inp.theta_bf16]
    tg64 = datagen.bf16_bits_to_f64(inp.target_bf16)
    idx = _group_rows(G, pool, b)
    ctx = g.Context(max_batch=b, n_actions=A, groups=G, dtype=g.GORILA_BF16)
    thetas = _dev(torch, inp.theta_bf16.view(np.int16))
    target = _dev(torch, inp.target_bf16.view(np.int16))
    grads, loss = g.learner_step_grouped(ctx, thetas, target, A, _replay(torch, g, inp),
                                         _dev(torch, idx), inp.gamma, clip)
    ctx.check()
    ref = _oracle_groups(oracle_mod, net, th64, tg64, inp, idx, b, clip=clip)
    for gi in range(G):
        errs = parity.assert_grads_close(grads[gi].cpu().numpy(), ref[gi]["grads"], A,
                                         parity.GRAD_TOL_BF16)
        l = float(loss[gi].cpu())
        assert abs(l - ref[gi]["loss"]) <= parity.LOSS_TOL * abs(ref[gi]["loss"]), gi
    _say(f"grad rel-L2 of the last group {errs}")
    ctx.close()


def test_grouped_one_group_matches_single_step(torch_cuda, g):
    """G = 1 runs the single learner step's launches: results are bitwise equal."""
    torch = torch_cuda
    _say("grouped G=1 == learner_step")
    inp = datagen.learner_inputs(8200, 48, 18)
    ctx = g.Context(max_batch=48, n_actions=18)
    theta, tgt = _dev(torch, inp.theta), _dev(torch, inp.theta_target)
    rep = g.Replay.stacked(_dev(torch, inp.s), _dev(torch, inp.s2), _dev(torch, inp.a),
                           _dev(torch, inp.r), _dev(torch, inp.term))
    idx = _dev(torch, inp.idx)
    g1, l1 = g.learner_step(ctx, theta, tgt, 18, rep, idx)
    g2, l2 = g.learner_step_grouped(ctx, [theta], tgt, 18, rep, idx)
    ctx.check()
    assert torch.equal(g1, g2[0]) and torch.equal(l1, l2)
    ctx.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_grouped_step_is_deterministic(torch_cuda, g, dtype):
    """Every reduction is a fixed-order sum: two calls of the grouped step
    (bf16 and fp32 parameter sets, 4 groups of 40 rows) give bitwise equal
    gradients and losses."""
    torch = torch_cuda
    G, b, A = 4, 40, 9
    _say(f"grouped determinism G={G} b={b} A={A} {dtype}")
    inp = datagen.grouped_inputs(8400, G, b, A)
    if dtype == "bf16":
        thetas = _dev(torch, inp.theta_bf16.view(np.int16))
        target = _dev(torch, inp.target_bf16.view(np.int16))
        ctx = g.Context(max_batch=b, n_actions=A, groups=G, dtype=g.GORILA_BF16)
    else:
        thetas = [_dev(torch, datagen.bf16_bits_to_f64(t).astype(np.float32)) for t in inp.theta_bf16]
        target = _dev(torch, datagen.bf16_bits_to_f64(inp.target_bf16).astype(np.float32))
        ctx = g.Context(max_batch=b, n_actions=A, groups=G)
    idx = _dev(torch, np.arange(G * b, dtype=np.int64))
    rep = _replay(torch, g, inp)
    g1, l1 = g.learner_step_grouped(ctx, thetas, target, A, rep, idx, inp.gamma, 1.0)
    g1, l1 = g1.clone(), l1.clone()
    g2, l2 = g.learner_step_grouped(ctx, thetas, target, A, rep, idx, inp.gamma, 1.0)
    ctx.check()
    assert torch.equal(g1, g2) and torch.equal(l1, l2)
    ctx.close()


def test_grouped_argument_errors(torch_cuda, g):
    torch = torch_cuda
    inp = datagen.learner_inputs(8300, 4, 18)
    ctx = g.Context(max_batch=4, n_actions=18, groups=2)
    theta, tgt = _dev(torch, inp.theta), _dev(torch, inp.theta_target)
    rep = g.Replay.stacked(_dev(torch, inp.s), _dev(torch, inp.s2), _dev(torch, inp.a),
                           _dev(torch, inp.r), _dev(torch, inp.term))
    idx = _dev(torch, np.tile(inp.idx, 2))
    grads = torch.empty((17, g.param_count(18)), device="cuda")
    loss = torch.empty(17, device="cuda")
    with pytest.raises(g.GorilaError) as e:  # 17 groups: over the limit
        g.gorila_learner_step_grouped(ctx, [theta] * 17, tgt, 18, rep, idx, 4, 0.99, 1.0,
                                      grads, loss)
    assert e.value.code == -1
    with pytest.raises(g.GorilaError) as e:  # 3 groups need more workspace
        g.gorila_learner_step_grouped(ctx, [theta] * 3, tgt, 18, rep, _dev(torch, np.tile(inp.idx, 3)),
                                      4, 0.99, 1.0, grads, loss)
    assert e.value.code == -3
    # bf16 parameters are not accepted by the single learner step
    bf = _dev(torch, datagen.to_bf16_bits(inp.theta.astype(np.float64)).view(np.int16))
    with pytest.raises(g.GorilaError) as e:
        g.learner_step(ctx, bf, tgt, 18, rep, _dev(torch, inp.idx))
    assert e.value.code == -5
    ctx.close()


@pytest.mark.parametrize("n", [5, 300])
def test_q_forward_bf16_params(torch_cuda, g, oracle_mod, n):
    torch = torch_cuda
    _say(f"q_forward bf16 n={n}")
    inp = datagen.learner_inputs(8400 + n, n, 18)
    bits = datagen.to_bf16_bits(inp.theta.astype(np.float64))
    ctx = g.Context(max_batch=n, n_actions=18, dtype=g.GORILA_BF16)
    q = g.q_forward(ctx, _dev(torch, bits.view(np.int16)), 18, _dev(torch, inp.s))
    acts = g.act(ctx, _dev(torch, bits.view(np.int16)), 18, _dev(torch, inp.s), 0.0, 5)
    ctx.check()
    net = oracle_mod.Net(n_actions=18)
    th64 = datagen.bf16_bits_to_f64(bits)
    ref_a, ref_q = oracle_mod.act(net, th64, inp.s, 0.0, 5)
    assert parity.q_rel_err(q.cpu().numpy(), ref_q) <= parity.Q_TOL
    parity.assert_actions_match(acts.cpu().numpy(), ref_q, ref_a, np.zeros(n, bool))
    ctx.close()
