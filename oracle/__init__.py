"""fp64 CPU oracle for the Gorila DQN learner step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the HIP library and its binding) never imports, links or calls it, and the
oracle shares no code with it.

The arithmetic lives in ``gorila_oracle.c`` (plain C, fp64, OpenMP over
samples), ``ps_oracle.c`` (the parameter-server apply and the loss-statistics
filter, Section 4 and 4.2) and ``actor_oracle.c`` (replay insert and the
epsilon schedule, Algorithm 1 and Section 5.1); this module only marshals
numpy arrays through ctypes.  Each function
cites the passage of Nair et al. 2015 it follows; the readings used where the
paper is silent are listed at the top of the C source.

Pins: every function here is pinned by tests in ``tests/test_oracle_*.py``
(finite differences, closed forms, a hand-enumerated replay-ring fixture, a
published SplitMix64 output, torch fp64 convolutions as a library special
case, batch invariants).  The whole learner step at full size has no value
printed in the paper to compare against: beyond those pins it is parity
unpinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, f) for f in ("gorila_oracle.c", "ps_oracle.c", "actor_oracle.c")]
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no BLAS; no contraction of
    a*b+c into fused multiply-adds, so every fp64 operation rounds once)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
             "-Wall", "-Wextra", "-o", tmp] + _SRCS + ["-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Net(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "in_c", "in_h", "in_w", "c1", "k1", "s1", "c2", "k2", "s2",
        "c3", "k3", "s3", "hidden", "n_actions")]


@dataclass(frozen=True)
class Net:
    """Q-network topology (Section 5.1: 84x84x4 input, conv 32@8x8/4,
    conv 64@4x4/2, conv 64@3x3/1, FC 512, linear FC with one unit per action).
    Tiny topologies exist only for finite-difference tests."""
    in_c: int = 4
    in_h: int = 84
    in_w: int = 84
    c1: int = 32
    k1: int = 8
    s1: int = 4
    c2: int = 64
    k2: int = 4
    s2: int = 2
    c3: int = 64
    k3: int = 3
    s3: int = 1
    hidden: int = 512
    n_actions: int = 18

    def c(self) -> _Net:
        return _Net(*[getattr(self, name) for name, _ in _Net._fields_])

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        P = ctypes.POINTER
        net_p = P(_Net)
        dp, u8p, i32p, i64p, f32p = (ctypes.c_void_p,) * 5
        L.oracle_param_count.argtypes = [net_p]
        L.oracle_param_count.restype = ctypes.c_int64
        L.oracle_param_offsets.argtypes = [net_p, i64p]
        L.oracle_num_threads.restype = ctypes.c_int
        L.oracle_set_num_threads.argtypes = [ctypes.c_int32]
        L.oracle_q_forward.argtypes = [net_p, dp, u8p, ctypes.c_int32, dp]
        L.oracle_act.argtypes = [net_p, dp, u8p, ctypes.c_int32, ctypes.c_double,
                                 ctypes.c_uint64, i32p, dp]
        L.oracle_learner_step.argtypes = [
            net_p, dp, dp, u8p, u8p, i32p, dp, u8p, ctypes.c_int32,
            ctypes.c_double, ctypes.c_double, dp, dp, dp, dp, dp, dp]
        L.oracle_gather.argtypes = [
            u8p, u8p, i32p, f32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
            ctypes.c_int64, i64p, ctypes.c_int32, u8p, u8p, i64p, i32p, f32p, u8p]
        L.oracle_loss_filter.argtypes = [dp, dp, ctypes.c_int32, ctypes.c_double,
                                         ctypes.c_double, ctypes.c_int64, u8p]
        L.oracle_ps_apply.argtypes = [dp, dp, ctypes.c_int64, dp, ctypes.c_int32, u8p, i64p,
                                      i64p, ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                      u8p]
        L.oracle_replay_insert.argtypes = [u8p, u8p, i32p, f32p, ctypes.c_int64, ctypes.c_int64,
                                           i64p, i64p, u8p, u8p, i32p, f32p, ctypes.c_int32]
        L.oracle_epsilon.argtypes = [ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_int64]
        L.oracle_epsilon.restype = ctypes.c_double
        L.oracle_params_sync.argtypes = [f32p, dp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int64, i64p, ctypes.c_int64, u8p]
        L.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        L.oracle_f32_to_bf16.restype = ctypes.c_uint16
        for f in ("oracle_param_offsets", "oracle_q_forward", "oracle_act",
                  "oracle_learner_step", "oracle_gather", "oracle_loss_filter",
                  "oracle_ps_apply", "oracle_replay_insert", "oracle_params_sync"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"{what}: oracle rejected the arguments (rc={rc})")


def param_count(net: Net) -> int:
    """Length of the flat parameter vector (layout in gorila_oracle.h)."""
    return int(lib().oracle_param_count(ctypes.byref(net.c())))


def param_offsets(net: Net) -> list[int]:
    """Offsets of W1,b1,W2,b2,W3,b3,W4,b4,W5,b5 and the total."""
    off = np.zeros(11, np.int64)
    _check(lib().oracle_param_offsets(ctypes.byref(net.c()), _ptr(off)), "param_offsets")
    return [int(x) for x in off]


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    _check(lib().oracle_set_num_threads(int(n)), "set_num_threads")


def q_forward(net: Net, theta, states) -> np.ndarray:
    """Q(s, .; theta) for a batch of uint8 states (Section 5.1 network)."""
    theta = _c(theta, np.float64)
    states = _c(states, np.uint8)
    n = states.shape[0]
    q = np.zeros((n, net.n_actions), np.float64)
    _check(lib().oracle_q_forward(ctypes.byref(net.c()), _ptr(theta), _ptr(states),
                                  n, _ptr(q)), "q_forward")
    return q


def act(net: Net, theta, states, eps: float, seed: int):
    """epsilon-greedy behaviour (Algorithm 1); returns (actions i32, Q f64).
    eps is taken as a float32 value promoted exactly to fp64."""
    theta = _c(theta, np.float64)
    states = _c(states, np.uint8)
    n = states.shape[0]
    acts = np.zeros(n, np.int32)
    q = np.zeros((n, net.n_actions), np.float64)
    _check(lib().oracle_act(ctypes.byref(net.c()), _ptr(theta), _ptr(states), n,
                            float(np.float32(eps)), ctypes.c_uint64(seed & (2**64 - 1)),
                            _ptr(acts), _ptr(q)), "act")
    return acts, q


def learner_step(net: Net, theta, theta_target, s, s2, a, r, term, gamma: float,
                 clip: float = 1.0):
    """DQN loss (eq. (1)) and its gradient (eq. (2)) on one minibatch.

    Returns dict(grads [P] f64, loss f64, q [B,A], q2 [B,A], margin [B],
    max_q2 [B], y [B], delta [B], ell [B]).  margin is each sample's smallest
    ReLU kink margin over the online network (min |z| / (|b| + sum |w||x|));
    max_q2, y, delta and ell are the per-sample pieces of Algorithm 1's target
    and eq. (1)'s error (max_a' Q(s',a';theta-), y, y - Q(s,a;theta), Huber).  gamma, r and clip are float32 values
    promoted exactly to fp64 (clip may be +inf)."""
    theta = _c(theta, np.float64)
    theta_target = _c(theta_target, np.float64)
    s = _c(s, np.uint8)
    s2 = _c(s2, np.uint8)
    a = _c(a, np.int32)
    r = _c(np.asarray(r, np.float32), np.float64)
    term = _c(term, np.uint8)
    B = s.shape[0]
    P = param_count(net)
    grads = np.zeros(P, np.float64)
    loss = np.zeros(1, np.float64)
    q = np.zeros((B, net.n_actions), np.float64)
    q2 = np.zeros((B, net.n_actions), np.float64)
    margin = np.zeros(B, np.float64)
    td = np.zeros((B, 4), np.float64)
    _check(lib().oracle_learner_step(
        ctypes.byref(net.c()), _ptr(theta), _ptr(theta_target), _ptr(s), _ptr(s2),
        _ptr(a), _ptr(r), _ptr(term), B, float(np.float32(gamma)),
        float(np.float32(clip)), _ptr(grads), _ptr(loss), _ptr(q), _ptr(q2),
        _ptr(margin), _ptr(td)), "learner_step")
    return dict(grads=grads, loss=float(loss[0]), q=q, q2=q2, margin=margin, max_q2=td[:, 0],
                y=td[:, 1], delta=td[:, 2], ell=td[:, 3])


def gather(frames, ep_start, action, reward, head: int, idx, hist: int = 4):
    """Frame stacking out of the replay ring (Section 4 replay memory,
    Section 5.1 four-frame input).  frames is [capacity, ...] uint8.

    Returns dict(s, s2 [n, hist, ...] u8, frame_map [n, 2, hist] i64,
    a i32, r f32, term u8)."""
    frames = np.asarray(frames)
    assert frames.dtype == np.uint8 and frames.flags["C_CONTIGUOUS"]
    cap = frames.shape[0]
    fshape = frames.shape[1:]
    fbytes = int(np.prod(fshape)) if fshape else 1
    ep_start = _c(ep_start, np.uint8)
    action = _c(action, np.int32)
    reward = _c(reward, np.float32)
    idx = _c(idx, np.int64)
    n = idx.shape[0]
    s = np.zeros((n, hist) + fshape, np.uint8)
    s2 = np.zeros((n, hist) + fshape, np.uint8)
    fmap = np.zeros((n, 2, hist), np.int64)
    a = np.zeros(n, np.int32)
    r = np.zeros(n, np.float32)
    t = np.zeros(n, np.uint8)
    _check(lib().oracle_gather(_ptr(frames), _ptr(ep_start), _ptr(action), _ptr(reward),
                               cap, head, hist, fbytes, _ptr(idx), n, _ptr(s), _ptr(s2),
                               _ptr(fmap), _ptr(a), _ptr(r), _ptr(t)), "gather")
    return dict(s=s, s2=s2, frame_map=fmap, a=a, r=r, term=t)


def loss_filter(stats, loss, alpha: float, k: float, warmup: int):
    """Section 4.2 loss-statistics filter for G learners.

    stats [G, 3] = (n, mean, var) of each learner's absolute loss (fp64; a new
    array is returned, the input is not modified); loss [G] (float32 values
    promoted exactly).  Returns (keep [G] uint8, new stats)."""
    st = _c(stats, np.float64).copy()
    x = _c(np.asarray(loss, np.float32), np.float64)
    G = x.shape[0]
    assert st.shape == (G, 3)
    keep = np.zeros(G, np.uint8)
    _check(lib().oracle_loss_filter(_ptr(st), _ptr(x), G, float(alpha), float(k), int(warmup),
                                    _ptr(keep)), "loss_filter")
    return keep, st


def ps_apply(theta, accum, grads, version, ps_version: int, max_delay: int, lr: float,
             eps: float, keep=None):
    """Section 4 / 4.2 parameter-server apply: AdaGrad updates of theta+ by the
    gradients grads [G, n] taken in index order, skipping those not kept and
    those older than max_delay server updates at their turn.  lr and eps are
    float32 values promoted exactly.  Returns dict(theta, accum (fp64 [n]),
    applied [G] uint8, ps_version)."""
    th = _c(theta, np.float64).copy()
    acc = _c(accum, np.float64).copy()
    gr = _c(grads, np.float64)
    G, n = gr.shape
    ver = _c(version, np.int64)
    kp = None if keep is None else _c(keep, np.uint8)
    psv = np.array([ps_version], np.int64)
    applied = np.zeros(G, np.uint8)
    _check(lib().oracle_ps_apply(_ptr(th), _ptr(acc), n, _ptr(gr), G, _ptr(kp), _ptr(ver),
                                 _ptr(psv), int(max_delay), float(np.float32(lr)),
                                 float(np.float32(eps)), _ptr(applied)), "ps_apply")
    return dict(theta=th, accum=acc, applied=applied, ps_version=int(psv[0]))


def replay_insert(frames, ep_start, action, reward, head: int, size: int, frames_in, ep_in,
                  act_in, rew_in):
    """Algorithm 1 / Section 4: append m records to a replay ring in place
    (frames [capacity, ...] u8, ep_start u8, action i32, reward f32, all
    modified); returns the new (head, size)."""
    for a, dt in ((frames, np.uint8), (ep_start, np.uint8), (action, np.int32),
                  (reward, np.float32)):
        assert a.dtype == dt and a.flags["C_CONTIGUOUS"]
    cap = frames.shape[0]
    fb = int(np.prod(frames.shape[1:]))
    # every array handed to C is held by a name until the call returns
    fi = _c(frames_in, np.uint8)
    ei = _c(ep_in, np.uint8)
    ai = _c(act_in, np.int32)
    ri = _c(rew_in, np.float32)
    m = fi.shape[0]
    h = np.array([head], np.int64)
    sz = np.array([size], np.int64)
    _check(lib().oracle_replay_insert(_ptr(frames), _ptr(ep_start), _ptr(action), _ptr(reward),
                                      cap, fb, _ptr(h), _ptr(sz), _ptr(fi), _ptr(ei), _ptr(ai),
                                      _ptr(ri), m), "replay_insert")
    return int(h[0]), int(sz[0])


def epsilon(update: int, eps_start: float = 1.0, eps_end: float = 0.1,
            anneal_updates: int = 1_000_000) -> float:
    """Section 5.1 behaviour-policy epsilon after `update` global updates."""
    return float(lib().oracle_epsilon(int(update), float(eps_start), float(eps_end),
                                      int(anneal_updates)))


def params_sync(src, dst_versions, ps_version: int, period: int, copies: int, to_bf16: bool,
                dst=None):
    """Algorithm 1 parameter pull / periodic target sync.  src fp32 [n];
    dst [copies, n] (fp32, or uint16 bf16 bits; zeros if None) and
    dst_versions [copies] are copied, updated and returned as
    (dst, versions, synced)."""
    s = _c(src, np.float32)
    n = s.shape[0]
    dt = np.uint16 if to_bf16 else np.float32
    d = np.zeros((copies, n), dt) if dst is None else _c(dst, dt).copy()
    v = _c(dst_versions, np.int64).copy()
    synced = np.zeros(copies, np.uint8)
    _check(lib().oracle_params_sync(_ptr(s), _ptr(d), n, copies, int(bool(to_bf16)),
                                    int(ps_version), _ptr(v), int(period), _ptr(synced)),
           "params_sync")
    return d, v, synced


def f32_to_bf16(x: float) -> int:
    return int(lib().oracle_f32_to_bf16(float(x)))
