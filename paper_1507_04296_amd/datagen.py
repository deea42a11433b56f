"""Seeded synthetic inputs for the Gorila DQN learner step.

This module draws inputs only: parameters, transitions, replay rings and actor
states.  It holds none of the method's arithmetic, and it is the one piece of
code that both the HIP path (through the tests and the benchmark) and the fp64
oracle consume.  Everything comes from numpy's PCG64 (``default_rng``), so an
input is fixed by its seed.

The paper trains on Atari 2600 frames (Section 5.1: 84x84 luminance, four-frame
stacks, up to 18 actions, rewards clipped as in DQN); those frames are not
available here, so these generators stand in for them with the same shapes,
value ranges and structure.

Parameter layout (flat, this order): W1 [32,4,8,8], b1 [32], W2 [64,32,4,4],
b2 [64], W3 [64,64,3,3], b3 [64], W4 [512,3136], b4 [512], W5 [A,512], b5 [A].
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

FRAME_H = FRAME_W = 84
HIST = 4
FRAME_BYTES = FRAME_H * FRAME_W
STATE_BYTES = HIST * FRAME_BYTES

SEED_BASE = 1507000


def tensor_shapes(n_actions: int):
    """(name, shape, fan_in) of the ten parameter tensors in layout order."""
    return [
        ("W1", (32, 4, 8, 8), 4 * 8 * 8), ("b1", (32,), None),
        ("W2", (64, 32, 4, 4), 32 * 4 * 4), ("b2", (64,), None),
        ("W3", (64, 64, 3, 3), 64 * 3 * 3), ("b3", (64,), None),
        ("W4", (512, 3136), 3136), ("b4", (512,), None),
        ("W5", (n_actions, 512), 512), ("b5", (n_actions,), None),
    ]


def param_count(n_actions: int) -> int:
    return sum(int(np.prod(s)) for _, s, _ in tensor_shapes(n_actions))


def tensor_slices(n_actions: int):
    """name -> slice of the flat vector."""
    out, off = {}, 0
    for name, shape, _ in tensor_shapes(n_actions):
        n = int(np.prod(shape))
        out[name] = slice(off, off + n)
        off += n
    return out


def he_normal_params(rng: np.random.Generator, n_actions: int) -> np.ndarray:
    """He-normal weights (std sqrt(2 / fan_in)), zero biases, drawn tensor by
    tensor in layout order in fp64; returned in fp64 (cast by the caller)."""
    parts = []
    for _, shape, fan_in in tensor_shapes(n_actions):
        n = int(np.prod(shape))
        if fan_in is None:
            parts.append(np.zeros(n, np.float64))
        else:
            parts.append(rng.standard_normal(n) * np.sqrt(2.0 / fan_in))
    return np.concatenate(parts)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to bfloat16 (round to nearest even, one rounding
    straight from fp64) and return the 16-bit patterns.  Values are assumed
    finite and inside bf16's normal range (true for these weights) or zero."""
    x = np.asarray(x, np.float64)
    bits = x.view(np.uint64).copy()
    drop = np.uint64(45)  # fp64 has 52 stored mantissa bits, bf16 keeps 7
    lsb = (bits >> drop) & np.uint64(1)
    bits = bits + (np.uint64(1) << np.uint64(44)) - np.uint64(1) + lsb
    bits &= ~((np.uint64(1) << drop) - np.uint64(1))
    f32 = bits.view(np.float64).astype(np.float32)  # exact: 8 significant bits
    return (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32).astype(np.float64)


def random_frames(rng: np.random.Generator, n_bytes: int) -> np.ndarray:
    """n_bytes uniform bytes 0..255 (raw PCG64 output reinterpreted)."""
    words = rng.bit_generator.random_raw((n_bytes + 7) // 8)
    return words.view(np.uint8)[:n_bytes].copy() if n_bytes % 8 else words.view(np.uint8)


def rewards(rng: np.random.Generator, n: int) -> np.ndarray:
    """Rewards in {-1, 0, +1} with probabilities {0.05, 0.9, 0.05}."""
    u = rng.random(n)
    return np.where(u < 0.05, -1.0, np.where(u < 0.95, 0.0, 1.0)).astype(np.float32)


@dataclass
class LearnerInputs:
    """One minibatch of stacked transitions plus both parameter sets."""
    n_actions: int
    theta: np.ndarray          # f32 [P] (bf16-valued when grouped)
    theta_target: np.ndarray   # f32 [P]
    s: np.ndarray              # u8 [rows, 4, 84, 84]
    s2: np.ndarray             # u8 [rows, 4, 84, 84]
    a: np.ndarray              # i32 [rows]
    r: np.ndarray              # f32 [rows]
    term: np.ndarray           # u8 [rows]
    idx: np.ndarray            # i64 [B] row indices
    gamma: float = 0.99
    extra: dict = field(default_factory=dict)


def learner_inputs(seed: int, batch: int, n_actions: int, gamma: float = 0.99,
                   term_p: float = 0.01, target_sigma: float = 0.01,
                   rows: int | None = None, idx: np.ndarray | None = None) -> LearnerInputs:
    """Learner-step workload: He-normal theta, theta- = theta + N(0, sigma^2),
    uniform random uint8 states s and s', actions uniform over A, rewards in
    {-1,0,1} w.p. {.05,.9,.05}, terminal w.p. term_p.  Drawn in that order."""
    rng = np.random.default_rng(seed)
    rows = batch if rows is None else rows
    theta64 = he_normal_params(rng, n_actions)
    tgt64 = theta64 + target_sigma * rng.standard_normal(theta64.shape[0])
    s = random_frames(rng, rows * STATE_BYTES).reshape(rows, HIST, FRAME_H, FRAME_W)
    s2 = random_frames(rng, rows * STATE_BYTES).reshape(rows, HIST, FRAME_H, FRAME_W)
    a = rng.integers(0, n_actions, rows).astype(np.int32)
    r = rewards(rng, rows)
    term = (rng.random(rows) < term_p).astype(np.uint8)
    if idx is None:
        idx = np.arange(batch, dtype=np.int64)
    return LearnerInputs(n_actions, theta64.astype(np.float32), tgt64.astype(np.float32),
                         s, s2, a, r, term, np.asarray(idx, np.int64), gamma)


def sprite_states(rng: np.random.Generator, n: int, n_sprites: int = 3) -> np.ndarray:
    """Actor states with smooth synthetic content: a dark background (uniform
    0..24) with n_sprites 8x8 bright sprites (brightness uniform 160..255)
    moving with integer velocities in [-4, 4]^2 px/frame; frame j (oldest = 0)
    draws each sprite at clip(p0 + v*j, 0, 76), overlaps combined with max."""
    out = rng.integers(0, 25, (n, HIST, FRAME_H, FRAME_W), dtype=np.uint8)
    bright = rng.integers(160, 256, (n, n_sprites))
    p0 = rng.integers(0, 77, (n, n_sprites, 2))
    vel = rng.integers(-4, 5, (n, n_sprites, 2))
    for e in range(n):
        for k in range(n_sprites):
            for j in range(HIST):
                y, x = np.clip(p0[e, k] + vel[e, k] * j, 0, 76)
                blk = out[e, j, y:y + 8, x:x + 8]
                np.maximum(blk, np.uint8(bright[e, k]), out=blk)
    return out


@dataclass
class ActorInputs:
    n_actions: int
    theta: np.ndarray
    states: np.ndarray
    eps: float
    seed: int


def actor_inputs(seed: int, n: int, n_actions: int, eps: float = 0.05) -> ActorInputs:
    rng = np.random.default_rng(seed)
    theta = he_normal_params(rng, n_actions).astype(np.float32)
    states = sprite_states(rng, n)
    return ActorInputs(n_actions, theta, states, eps, seed)


@dataclass
class RingInputs:
    """A replay ring of single frames (Section 4 replay memory, 1M frames)."""
    frames: np.ndarray    # u8 [capacity, 84, 84] (or [capacity, fh, fw])
    ep_start: np.ndarray  # u8 [capacity], physical slots
    action: np.ndarray    # i32 [capacity]
    reward: np.ndarray    # f32 [capacity]
    head: int             # physical slot of the oldest frame (logical 0)


def ring_inputs(rng: np.random.Generator, capacity: int, n_actions: int,
                mean_episode: float = 2000.0, frame_shape=(FRAME_H, FRAME_W)) -> RingInputs:
    """Uniform random frames; episode lengths Geometric(1/mean) laid out from
    logical 0 until the end of the ring; head uniform over the slots."""
    fbytes = int(np.prod(frame_shape))
    frames = random_frames(rng, capacity * fbytes).reshape((capacity,) + tuple(frame_shape))
    starts_logical = [0]
    pos = 0
    while True:
        pos += int(rng.geometric(1.0 / mean_episode))
        if pos >= capacity:
            break
        starts_logical.append(pos)
    head = int(rng.integers(0, capacity))
    ep_start = np.zeros(capacity, np.uint8)
    ep_start[(head + np.asarray(starts_logical, np.int64)) % capacity] = 1
    action = rng.integers(0, n_actions, capacity).astype(np.int32)
    reward = rewards(rng, capacity)
    return RingInputs(frames, ep_start, action, reward, head)


def boundary_dense_idx(ring: RingInputs, n_starts: int = 50) -> np.ndarray:
    """Logical positions around episode starts (m-1 .. m+4 for the first
    n_starts starts after logical 0) plus logical 0 and capacity-2: the places
    where zero-fill and terminal flags change."""
    cap = ring.frames.shape[0]
    logical_flags = np.roll(ring.ep_start, -ring.head)
    starts = np.nonzero(logical_flags)[0]
    starts = starts[starts > 0][:n_starts]
    idx = [0, cap - 2]
    for m in starts:
        idx.extend(int(k) for k in range(m - 1, m + 5) if 0 <= k <= cap - 2)
    return np.asarray(idx, np.int64)


@dataclass
class GroupedInputs:
    """Stale-replica workload: G learners, each with its own bf16 parameters."""
    n_actions: int
    groups: int
    batch: int
    theta_bf16: np.ndarray      # u16 [G, P] bf16 bit patterns
    target_bf16: np.ndarray     # u16 [P]
    s: np.ndarray
    s2: np.ndarray
    a: np.ndarray
    r: np.ndarray
    term: np.ndarray
    gamma: float = 0.99


def grouped_inputs(seed: int, groups: int, batch: int, n_actions: int,
                   drift_sigma: float = 0.005, target_sigma: float = 0.01,
                   gamma: float = 0.99) -> GroupedInputs:
    """Base He-normal weights; replica g = bf16(base + N(0, drift^2)); one
    shared target bf16(base + N(0, target_sigma^2)); transitions as in the
    single-learner workload, rows g*batch .. g*batch+batch-1 for group g."""
    rng = np.random.default_rng(seed)
    base = he_normal_params(rng, n_actions)
    P = base.shape[0]
    theta = np.stack([to_bf16_bits(base + drift_sigma * rng.standard_normal(P))
                      for _ in range(groups)])
    target = to_bf16_bits(base + target_sigma * rng.standard_normal(P))
    rows = groups * batch
    s = random_frames(rng, rows * STATE_BYTES).reshape(rows, HIST, FRAME_H, FRAME_W)
    s2 = random_frames(rng, rows * STATE_BYTES).reshape(rows, HIST, FRAME_H, FRAME_W)
    a = rng.integers(0, n_actions, rows).astype(np.int32)
    r = rewards(rng, rows)
    term = (rng.random(rows) < 0.01).astype(np.uint8)
    return GroupedInputs(n_actions, groups, batch, theta, target, s, s2, a, r, term, gamma)


class SpriteEnv:
    """A synthetic stand-in for the Atari environments (none are available):
    n independent games on a dark 84x84 screen with one 8x8 sprite the agent
    moves and one fixed target.  Action a in [0, A) moves the sprite by
    (dy, dx) = ((a % 9) // 3 - 1, (a % 9) % 3 - 1) * 4 px (the 9 joystick
    directions; higher actions repeat them); reaching the target gives +1 and
    ends the episode, every other step gives 0, and an episode also ends after
    `max_steps` steps.  A new episode draws fresh positions from the env's
    seeded generator.  Pure host numpy: shared by both sides of a test as an
    input generator."""

    def __init__(self, seed: int, n: int, max_steps: int = 25):
        self.rng = np.random.default_rng(seed)
        self.n, self.max_steps = n, max_steps
        self.bg = self.rng.integers(0, 25, (n, FRAME_H, FRAME_W), dtype=np.uint8)
        self.pos = np.zeros((n, 2), np.int64)
        self.goal = np.zeros((n, 2), np.int64)
        self.t = np.zeros(n, np.int64)
        for e in range(n):
            self._reset(e)

    def _reset(self, e: int):
        self.pos[e] = self.rng.integers(0, 77, 2)
        self.goal[e] = self.rng.integers(0, 77, 2)
        self.t[e] = 0

    def frames(self) -> np.ndarray:
        """Current screens, u8 [n, 84, 84]."""
        out = self.bg.copy()
        for e in range(self.n):
            gy, gx = self.goal[e]
            out[e, gy:gy + 8, gx:gx + 8] = np.maximum(out[e, gy:gy + 8, gx:gx + 8], 120)
            y, x = self.pos[e]
            out[e, y:y + 8, x:x + 8] = 255
        return out

    def step(self, actions: np.ndarray):
        """Apply one action per game: returns (reward f32 [n], done u8 [n]); a
        finished game has already been reset to its next episode's start."""
        a = np.asarray(actions, np.int64) % 9
        d = np.stack([a // 3 - 1, a % 3 - 1], axis=1) * 4
        self.pos = np.clip(self.pos + d, 0, 76)
        self.t += 1
        hit = np.all(np.abs(self.pos - self.goal) < 8, axis=1)
        reward = hit.astype(np.float32)
        done = (hit | (self.t >= self.max_steps)).astype(np.uint8)
        for e in np.nonzero(done)[0]:
            self._reset(int(e))
        return reward, done


@dataclass
class PsInputs:
    """Parameter-server apply inputs: theta+ and AdaGrad accumulator [n],
    G learner gradients [G, n] with the server versions they were computed at."""
    theta: np.ndarray      # f32 [n]
    accum: np.ndarray      # f32 [n], >= 0
    grads: np.ndarray      # f32 [G, n]
    version: np.ndarray    # i64 [G]
    ps_version: int
    keep: np.ndarray       # u8 [G]


def ps_inputs(seed: int, groups: int, n: int, max_lag: int = 6, keep_p: float = 0.9,
              ps_version: int = 1000) -> PsInputs:
    """theta ~ N(0, 0.05^2), accum ~ U[0, 0.01), gradients ~ N(0, 1e-3^2),
    version = ps_version - U{0..max_lag-1}, keep ~ Bernoulli(keep_p); drawn in
    that order."""
    rng = np.random.default_rng(seed)
    theta = (0.05 * rng.standard_normal(n)).astype(np.float32)
    accum = (0.01 * rng.random(n)).astype(np.float32)
    grads = (1e-3 * rng.standard_normal((groups, n))).astype(np.float32)
    version = (ps_version - rng.integers(0, max_lag, groups)).astype(np.int64)
    keep = (rng.random(groups) < keep_p).astype(np.uint8)
    return PsInputs(theta, accum, grads, version, ps_version, keep)


def loss_sequences(seed: int, steps: int, groups: int, outlier_p: float = 0.02) -> np.ndarray:
    """f32 [steps, groups] learner losses: lognormal around 0.05 with a slow
    drift, and outliers 5-50x the typical value with probability outlier_p;
    some values negative, to exercise the absolute value."""
    rng = np.random.default_rng(seed)
    t = np.arange(steps)[:, None]
    base = 0.05 * np.exp(0.3 * rng.standard_normal((steps, groups))) * (1.0 + 0.002 * t)
    out = rng.random((steps, groups)) < outlier_p
    base = np.where(out, base * rng.uniform(5, 50, (steps, groups)), base)
    sign = np.where(rng.random((steps, groups)) < 0.1, -1.0, 1.0)
    return (sign * base).astype(np.float32)


# Named workloads (sizes of the paper's setting: 4x84x84 uint8 stacks, 18 or 6
# actions, replay of one million frames, gamma 0.99).
WORKLOADS = {
    "learner_b32_a18_f32": dict(kind="learner", batch=32, n_actions=18, seed=SEED_BASE + 0),
    "actor_n1024_a18_f32": dict(kind="act", n=1024, n_actions=18, eps=0.05, seed=SEED_BASE + 1),
    "learner_b512_a6_f32": dict(kind="learner", batch=512, n_actions=6, seed=SEED_BASE + 2),
    "ring1m_gather_learner_b256_a18_f32": dict(kind="ring", batch=256, n_actions=18,
                                                capacity=1_000_000, seed=SEED_BASE + 3),
    "grouped_g16_b64_a18_bf16": dict(kind="grouped", groups=16, batch=64, n_actions=18,
                                     seed=SEED_BASE + 4),
    # the server side of the stale-replica workload: 16 gradients of the
    # 18-action network applied to theta+
    "ps_apply_g16_a18_f32": dict(kind="ps_apply", groups=16, n_actions=18, seed=SEED_BASE + 5),
}
