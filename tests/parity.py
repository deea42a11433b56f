"""Comparison helpers shared by the GPU parity tests (no method arithmetic).

Tolerances: Q values within 1e-4 relative (max |q - q*| / max |q*|), the loss
within 1e-4 relative, every gradient tensor within 1e-3 relative L2 for the fp32
path and 2e-2 for bf16 operands with fp32 accumulation; integer outputs (gathered bytes, frame maps, actions) bit-exact.

ReLU derivatives are a discrete choice taken from a float: a pre-activation
within rounding of zero may be switched on in fp32 and off in fp64, and a single
such flip moves a whole sample's backward pass by ~1/sqrt(512 B).  Gradient
parity therefore runs on rows whose online pre-activations all clear the
oracle's kink margin KINK_TAU (|z| / (|b| + sum |w||x|)); the batch size, and so
the launch configuration, stays the one under test.
"""
import numpy as np

from paper_1507_04296_amd import datagen

Q_TOL = 1e-4
LOSS_TOL = 1e-4
GRAD_TOL = 1e-3
GRAD_TOL_BF16 = 2e-2  # bf16 operands with fp32 accumulation
TENSORS = ("W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4", "W5", "b5")
KINK_TAU = 1e-6


def kink_certified(margins, want, tau=KINK_TAU):
    """Positions of the first `want` rows whose kink margin is at least tau."""
    ok = np.nonzero(np.asarray(margins) >= tau)[0]
    assert ok.size >= want, f"only {ok.size} of {len(margins)} rows clear the kink margin"
    return ok[:want]


def q_rel_err(q, q_ref):
    q, q_ref = np.asarray(q, np.float64), np.asarray(q_ref, np.float64)
    return float(np.abs(q - q_ref).max() / max(np.abs(q_ref).max(), 1e-30))


def grad_errors(g, g_ref, n_actions):
    """Relative L2 error per parameter tensor (absolute when the reference is 0)."""
    sl = datagen.tensor_slices(n_actions)
    out = {}
    for name in TENSORS:
        a = np.asarray(g[sl[name]], np.float64)
        b = np.asarray(g_ref[sl[name]], np.float64)
        nb = np.linalg.norm(b)
        out[name] = float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))
    return out


def assert_grads_close(g, g_ref, n_actions, tol=GRAD_TOL):
    errs = grad_errors(g, g_ref, n_actions)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"gradient tensors over {tol}: {bad} (all: {errs})"
    return errs


def assert_actions_match(actions, q_oracle, acts_oracle, explored):
    """Bit-exact where the greedy choice is well posed; elsewhere the GPU's
    greedy action must be one of the oracle's near-maxima."""
    q = np.asarray(q_oracle, np.float64)
    scale = np.abs(q).max()
    srt = np.sort(q, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    certified = explored | (gap > 4 * Q_TOL * scale)
    np.testing.assert_array_equal(np.asarray(actions)[certified], acts_oracle[certified])
    for e in np.nonzero(~certified)[0]:
        assert q[e, actions[e]] >= q[e].max() - 4 * Q_TOL * scale, e
    return int((~certified).sum())
