"""The learner step captured into a HIP graph (through torch.cuda.graph) and
replayed: every replay, with eager calls and synchronisations between them,
must equal the eager result bit for bit (the step's reductions have a fixed
order), and a replay must pick up new contents of its input buffers.  At
batch 512 the step splits the last tiles of two launches into reduction
pieces whose per-tile counters every launch must leave at zero (no memset is
recorded): replays after the first would otherwise hand the epilogue to the
wrong piece."""
import sys

import numpy as np
import pytest

from paper_1507_04296_amd import datagen

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("B", [32, 512])
def test_learner_step_graph_replays_match_eager(B):
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    import paper_1507_04296_amd as g
    g.lib()
    _say(f"learner B={B} A=18 captured in a HIP graph")
    inp = datagen.learner_inputs(datagen.SEED_BASE + 0, B, 18, rows=3 * B)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    theta, tgt = t(inp.theta), t(inp.theta_target)
    rep = g.Replay.stacked(t(inp.s), t(inp.s2), t(inp.a), t(inp.r), t(inp.term))
    idx_a = t(np.arange(B, dtype=np.int64))
    idx_b = t(np.arange(B + 8, 2 * B + 8, dtype=np.int64))
    idx = idx_a.clone()
    ctx = g.Context(B, 18, device=dev)
    grads = torch.empty(g.param_count(18), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)

    def step():
        g.gorila_learner_step(ctx, theta, tgt, 18, rep, idx, 0.99, 1.0, grads, loss)

    ref_a, lref_a = g.learner_step(ctx, theta, tgt, 18, rep, idx_a)
    ref_b, lref_b = g.learner_step(ctx, theta, tgt, 18, rep, idx_b)
    ctx.check()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rnd in range(3):
        grads.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(grads, ref_a) and torch.equal(loss, lref_a), rnd
        # eager work on the same context between replays
        e, le = g.learner_step(ctx, theta, tgt, 18, rep, idx_b)
        ctx.check()
        assert torch.equal(e, ref_b) and torch.equal(le, lref_b), rnd
    # the graph reads idx in place: new indices, same graph
    idx.copy_(idx_b)
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(grads, ref_b) and torch.equal(loss, lref_b)
    ctx.check()
    ctx.close()
