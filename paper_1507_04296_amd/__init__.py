"""Gorila DQN learner step on MI355X (gfx950): HIP kernels behind a C-ABI.

This module is the thin Python binding of ``libgorila.so`` (declared in
``include/gorila.h``): it only marshals torch tensors (device pointers) and the
current HIP stream into the C calls.  Every step of the computation runs in the
library's kernels; there is no Python or CPU fallback.  If the library is not
built, every call raises.

Method: Nair et al. 2015, "Massively Parallel Methods for Deep Reinforcement
Learning" -- the learner's DQN gradient step (Algorithm 1, eq. (1) and (2)) and
the actors' epsilon-greedy inference (Algorithm 1), on the Q-network of
Section 5.1.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgorila.so")

GORILA_F32, GORILA_BF16 = 0, 1
REPLAY_STACKED, REPLAY_RING = 0, 1
ERRORS = {0: "OK", -1: "EINVAL", -2: "ERANGE", -3: "EWORKSPACE", -4: "EHIP", -5: "EUNSUPPORTED"}

# Every function declared in include/gorila.h.
EXPORTS = (
    "gorila_param_count", "gorila_workspace_bytes", "gorila_ctx_create", "gorila_ctx_destroy",
    "gorila_ctx_set_stream", "gorila_ctx_check", "gorila_strerror", "gorila_gather",
    "gorila_q_forward", "gorila_act", "gorila_learner_step", "gorila_learner_step_grouped",
    "gorila_ctx_timing_begin", "gorila_ctx_timing_end", "gorila_stage_name",
    "gorila_loss_filter", "gorila_ps_apply", "gorila_replay_insert", "gorila_epsilon",
    "gorila_params_sync", "gorila_learner_td", "gorila_act_noalloc",
)
NOALLOC_MAX_STATES = 256  # GORILA_NOALLOC_MAX_STATES


class GorilaError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {ERRORS.get(code, code)} ({strerror(code)})")


class _Params(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("n_actions", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class _Replay(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("s", ctypes.c_void_p), ("s2", ctypes.c_void_p), ("term", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("frames", ctypes.c_void_p),
                ("ep_start", ctypes.c_void_p), ("capacity", ctypes.c_int64),
                ("head", ctypes.c_int64), ("size", ctypes.c_int64), ("action", ctypes.c_void_p),
                ("reward", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libgorila.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback implementation)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64, f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                              ctypes.c_float)
    P, R = ctypes.POINTER(_Params), ctypes.POINTER(_Replay)
    sig = {
        "gorila_param_count": (i64, [i32]),
        "gorila_workspace_bytes": (ctypes.c_size_t, [i32, i32, i32, i32]),
        "gorila_ctx_create": (ctypes.c_int, [ctypes.POINTER(vp), vp, vp, ctypes.c_size_t]),
        "gorila_ctx_destroy": (ctypes.c_int, [vp]),
        "gorila_ctx_set_stream": (ctypes.c_int, [vp, vp]),
        "gorila_ctx_check": (ctypes.c_int, [vp]),
        "gorila_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "gorila_gather": (ctypes.c_int, [R, vp, i32, vp, vp, vp, vp, vp, vp, vp]),
        "gorila_q_forward": (ctypes.c_int, [P, vp, i32, vp, vp]),
        "gorila_act": (ctypes.c_int, [P, vp, i32, f32, u64, vp, vp, vp]),
        "gorila_learner_step": (ctypes.c_int, [P, P, R, vp, i32, f32, f32, vp, vp, vp]),
        "gorila_learner_step_grouped": (ctypes.c_int, [P, i32, P, R, vp, i32, f32, f32, vp, vp, vp]),
        "gorila_ctx_timing_begin": (ctypes.c_int, [vp, ctypes.c_uint32, i32]),
        "gorila_ctx_timing_end": (ctypes.c_int, [vp, vp, vp, i32]),
        "gorila_stage_name": (ctypes.c_char_p, [i32]),
        "gorila_loss_filter": (ctypes.c_int, [vp, vp, i32, ctypes.c_double, ctypes.c_double, i64,
                                              vp, vp]),
        "gorila_replay_insert": (ctypes.c_int, [vp, vp, vp, vp, i64, i32, ctypes.POINTER(i64),
                                                ctypes.POINTER(i64), vp, vp, vp, vp, i32, vp]),
        "gorila_epsilon": (ctypes.c_double, [i64, ctypes.c_double, ctypes.c_double, i64]),
        "gorila_params_sync": (ctypes.c_int, [vp, vp, i64, i32, i32, vp, vp, i64, vp, vp]),
        "gorila_ps_apply": (ctypes.c_int, [vp, vp, i64, vp, i32, vp, vp, vp, i64, f32, f32, vp,
                                           vp]),
        "gorila_learner_td": (ctypes.c_int, [vp, vp, vp, vp]),
        "gorila_act_noalloc": (ctypes.c_int, [P, vp, i32, f32, u64, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype, fn.argtypes = res, args
    _lib = L
    return L


def strerror(code: int) -> str:
    return lib().gorila_strerror(code).decode()


def stage_names() -> list:
    out, i = [], 0
    while True:
        name = lib().gorila_stage_name(i)
        if name is None:
            return out
        out.append(name.decode())
        i += 1


def param_count(n_actions: int) -> int:
    return int(lib().gorila_param_count(n_actions))


def workspace_bytes(max_batch: int, n_actions: int, dtype: int = GORILA_F32, groups: int = 1) -> int:
    return int(lib().gorila_workspace_bytes(max_batch, n_actions, dtype, groups))


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _check(rc: int, what: str):
    if rc != 0:
        raise GorilaError(rc, what)


class Context:
    """A gorila_ctx bound to a torch-allocated device workspace.

    The workspace is sized for calls with batch <= max_batch (learner step) or
    n <= 2 * max_batch states (forward / act); max_batch = 0 makes a context
    without one (for gorila_act_noalloc and the calls that need none)."""

    def __init__(self, max_batch: int, n_actions: int, groups: int = 1, device=None,
                 dtype: int = GORILA_F32):
        import torch
        self.device = torch.device(device if device is not None else "cuda")
        if max_batch == 0:  # a context without a workspace (gorila_act_noalloc)
            self.ws_bytes, self.workspace = 0, None
        else:
            self.ws_bytes = workspace_bytes(max_batch, n_actions, dtype, groups)
            if self.ws_bytes == 0:
                raise ValueError("invalid workspace request")
        with torch.cuda.device(self.device):
            if self.ws_bytes:
                self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
            h = ctypes.c_void_p()
            _check(lib().gorila_ctx_create(ctypes.byref(h), self._stream(), _ptr(self.workspace),
                                           self.ws_bytes), "gorila_ctx_create")
        self.handle = h

    def _stream(self):
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream)

    def bind_stream(self):
        _check(lib().gorila_ctx_set_stream(self.handle, self._stream()), "gorila_ctx_set_stream")
        return self.handle

    def check(self) -> None:
        """Synchronise and raise GorilaError(ERANGE) if the device saw a bad index/action."""
        _check(lib().gorila_ctx_check(self.handle), "gorila_ctx_check")

    def timing_begin(self, stages, max_records: int = 4096):
        """Record HIP events around the named stages of the following calls."""
        mask = 0
        for name in stages:
            mask |= 1 << stage_names().index(name)
        _check(lib().gorila_ctx_timing_begin(self.handle, mask, max_records), "timing_begin")

    def timing_end(self) -> dict:
        """{stage: (total_ms, launches)} for the stages timed since timing_begin."""
        import numpy as np
        names = stage_names()
        ms = np.zeros(len(names), np.float64)
        cnt = np.zeros(len(names), np.int32)
        _check(lib().gorila_ctx_timing_end(self.handle, ms.ctypes.data, cnt.ctypes.data, len(names)),
               "timing_end")
        return {n: (float(ms[i]), int(cnt[i])) for i, n in enumerate(names) if cnt[i]}

    def close(self):
        if getattr(self, "handle", None) is not None:
            lib().gorila_ctx_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dtype_of(theta) -> int:
    """GORILA_F32 for a float32 tensor, GORILA_BF16 for bfloat16 or 16-bit integer bit patterns."""
    import torch
    if theta.dtype == torch.float32:
        return GORILA_F32
    if theta.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return GORILA_BF16
    raise TypeError(f"parameters must be float32 or bf16 (bits), got {theta.dtype}")


def params(theta, n_actions: int, dtype: int | None = None) -> _Params:
    """gorila_params over a flat device tensor (fp32, or bf16 bits as int16/uint16/bfloat16)."""
    return _Params(theta.data_ptr(), n_actions, dtype_of(theta) if dtype is None else dtype)


@dataclass
class Replay:
    """Device tensors of a replay memory (see gorila_replay in include/gorila.h)."""
    kind: int
    action: object
    reward: object
    s: object = None
    s2: object = None
    term: object = None
    frames: object = None
    ep_start: object = None
    head: int = 0
    rings: int = 1
    size: int | None = None  # RING: frames stored per ring (None: full)

    @staticmethod
    def stacked(s, s2, action, reward, term) -> "Replay":
        return Replay(REPLAY_STACKED, action, reward, s=s, s2=s2, term=term)

    @staticmethod
    def ring(frames, ep_start, action, reward, head: int, size: int | None = None) -> "Replay":
        """One ring: frames [capacity, 84, 84] holding `size` frames (default: full)."""
        return Replay(REPLAY_RING, action, reward, frames=frames, ep_start=ep_start, head=head,
                      size=size)

    @staticmethod
    def rings_of(frames, ep_start, action, reward, head: int, size: int | None = None) -> "Replay":
        """R rings filled in lockstep: frames [R, capacity, 84, 84], the others [R, capacity];
        minibatch index r * capacity + k is logical position k of ring r."""
        return Replay(REPLAY_RING, action, reward, frames=frames, ep_start=ep_start, head=head,
                      rings=frames.shape[0], size=size)

    def c(self) -> _Replay:
        if self.kind == REPLAY_RING:
            rows = self.rings if self.rings > 1 else 0
            cap = self.frames.shape[1] if self.rings > 1 else self.frames.shape[0]
            size = cap if self.size is None else int(self.size)
        else:
            rows = self.s.shape[0] if self.s is not None else 0
            cap = size = 0
        return _Replay(self.kind, 0, _ptr(self.s), _ptr(self.s2), _ptr(self.term), rows,
                       _ptr(self.frames), _ptr(self.ep_start), cap, int(self.head), size,
                       _ptr(self.action), _ptr(self.reward))


def gorila_gather(ctx: Context, replay: Replay, idx, s_out, s2_out, frame_map_out, a_out, r_out,
                  term_out) -> None:
    rv = replay.c()
    _check(lib().gorila_gather(ctypes.byref(rv), _ptr(idx), idx.shape[0], _ptr(s_out), _ptr(s2_out),
                               _ptr(frame_map_out), _ptr(a_out), _ptr(r_out), _ptr(term_out),
                               ctx.bind_stream()), "gorila_gather")


def gorila_q_forward(ctx: Context, theta, n_actions: int, states, q_out) -> None:
    p = params(theta, n_actions)
    _check(lib().gorila_q_forward(ctypes.byref(p), _ptr(states), states.shape[0], _ptr(q_out),
                                  ctx.bind_stream()), "gorila_q_forward")


def gorila_act(ctx: Context, theta, n_actions: int, states, eps: float, seed: int, actions_out,
               q_out=None) -> None:
    p = params(theta, n_actions)
    _check(lib().gorila_act(ctypes.byref(p), _ptr(states), states.shape[0], eps,
                            ctypes.c_uint64(seed & (2 ** 64 - 1)), _ptr(actions_out), _ptr(q_out),
                            ctx.bind_stream()), "gorila_act")


def gorila_act_noalloc(ctx: Context, theta, n_actions: int, states, eps: float, seed: int,
                       actions_out, q_out=None) -> None:
    """gorila_act on the library's static scratch (no workspace, n <= NOALLOC_MAX_STATES)."""
    p = params(theta, n_actions)
    _check(lib().gorila_act_noalloc(ctypes.byref(p), _ptr(states), states.shape[0], eps,
                                    ctypes.c_uint64(seed & (2 ** 64 - 1)), _ptr(actions_out),
                                    _ptr(q_out), ctx.bind_stream()), "gorila_act_noalloc")


def gorila_learner_step(ctx: Context, theta, theta_target, n_actions: int, replay: Replay, idx,
                        gamma: float, clip_delta: float, grads_out, loss_out) -> None:
    p, pt, rv = params(theta, n_actions), params(theta_target, n_actions), replay.c()
    _check(lib().gorila_learner_step(ctypes.byref(p), ctypes.byref(pt), ctypes.byref(rv), _ptr(idx),
                                     idx.shape[0], gamma, clip_delta, _ptr(grads_out),
                                     _ptr(loss_out), ctx.bind_stream()), "gorila_learner_step")


def gorila_learner_step_grouped(ctx: Context, thetas, theta_target, n_actions: int,
                                replay: Replay, idx, batch: int, gamma: float, clip_delta: float,
                                grads_out, loss_out) -> None:
    """thetas: a [G, P] tensor or a sequence of G flat tensors; idx [G * batch]."""
    rows = [thetas[g] for g in range(len(thetas))]
    arr = (_Params * len(rows))(*[params(t, n_actions) for t in rows])
    pt, rv = params(theta_target, n_actions), replay.c()
    _check(lib().gorila_learner_step_grouped(arr, len(rows), ctypes.byref(pt), ctypes.byref(rv),
                                             _ptr(idx), batch, gamma, clip_delta, _ptr(grads_out),
                                             _ptr(loss_out), ctx.bind_stream()),
           "gorila_learner_step_grouped")


def gorila_learner_td(ctx: Context, q_out=None, q_next_out=None, td_out=None) -> None:
    """Per-row Q(s), Q(s'), and (max Q(s'), y, delta, Huber) of the last learner call."""
    _check(lib().gorila_learner_td(ctx.bind_stream(), _ptr(q_out), _ptr(q_next_out), _ptr(td_out)),
           "gorila_learner_td")


def learner_td(ctx: Context, rows: int, n_actions: int, device=None):
    """Allocating wrapper of gorila_learner_td: (q [rows, A], q_next [rows, A], td [rows, 4])."""
    import torch
    dev = ctx.device if device is None else device
    q = torch.empty((rows, n_actions), dtype=torch.float32, device=dev)
    qn = torch.empty_like(q)
    td = torch.empty((rows, 4), dtype=torch.float32, device=dev)
    gorila_learner_td(ctx, q, qn, td)
    return q, qn, td


def gorila_loss_filter(ctx: Context, stats, loss, alpha: float, k: float, warmup: int,
                       keep_out) -> None:
    """stats: float64 [G, 3] device tensor (updated in place); loss [G] fp32."""
    _check(lib().gorila_loss_filter(_ptr(stats), _ptr(loss), loss.shape[0], alpha, k, warmup,
                                    _ptr(keep_out), ctx.bind_stream()), "gorila_loss_filter")


def gorila_ps_apply(ctx: Context, theta_plus, accum, grads, grad_version, ps_version,
                    max_delay: int, lr: float, eps: float, applied_out, keep=None) -> None:
    """theta_plus / accum fp32 [n] (updated in place); grads [G, n]; grad_version
    int64 [G]; ps_version int64 [1] (advanced in place); applied_out uint8 [G]."""
    G = grads.shape[0] if grads.dim() == 2 else 0
    _check(lib().gorila_ps_apply(_ptr(theta_plus), _ptr(accum), theta_plus.numel(), _ptr(grads),
                                 G, _ptr(keep), _ptr(grad_version), _ptr(ps_version), max_delay,
                                 lr, eps, _ptr(applied_out), ctx.bind_stream()),
           "gorila_ps_apply")


class RingSet:
    """Replay rings of one or more actors on the device (Section 4 bundled mode:
    one ring per actor, filled in lockstep), with the host-side head / size."""

    def __init__(self, rings: int, capacity: int, device=None):
        import torch
        dev = torch.device(device if device is not None else "cuda")
        self.rings, self.capacity = rings, capacity
        self.frames = torch.zeros((rings, capacity, 84, 84), dtype=torch.uint8, device=dev)
        self.ep_start = torch.zeros((rings, capacity), dtype=torch.uint8, device=dev)
        self.action = torch.zeros((rings, capacity), dtype=torch.int32, device=dev)
        self.reward = torch.zeros((rings, capacity), dtype=torch.float32, device=dev)
        self.head, self.size = 0, 0

    def replay(self) -> Replay:
        if self.rings == 1:
            return Replay.ring(self.frames[0], self.ep_start[0], self.action[0], self.reward[0],
                               self.head, self.size)
        return Replay.rings_of(self.frames, self.ep_start, self.action, self.reward, self.head,
                               self.size)


def gorila_replay_insert(ctx: Context, rs: RingSet, frames_in, ep_in, act_in, rew_in) -> None:
    """Append m records to every ring: frames_in [m, rings, 84, 84] u8, the others [m, rings]."""
    m = frames_in.shape[0]
    h, sz = ctypes.c_int64(rs.head), ctypes.c_int64(rs.size)
    _check(lib().gorila_replay_insert(_ptr(rs.frames), _ptr(rs.ep_start), _ptr(rs.action),
                                      _ptr(rs.reward), rs.capacity, rs.rings, ctypes.byref(h),
                                      ctypes.byref(sz), _ptr(frames_in), _ptr(ep_in), _ptr(act_in),
                                      _ptr(rew_in), m, ctx.bind_stream()), "gorila_replay_insert")
    rs.head, rs.size = h.value, sz.value


def gorila_params_sync(ctx: Context, src, dst, dst_version, ps_version, period: int,
                       synced_out=None) -> None:
    """Pull (period 0) or periodic target sync of theta+ (src fp32 [n]) into
    dst [copies, n] (fp32, or bf16 bits as int16 / uint16 / bfloat16)."""
    copies = dst.shape[0]
    _check(lib().gorila_params_sync(_ptr(src), _ptr(dst), src.numel(), copies, dtype_of(dst),
                                    _ptr(ps_version), _ptr(dst_version), period,
                                    _ptr(synced_out), ctx.bind_stream()), "gorila_params_sync")


def epsilon(update: int, eps_start: float = 1.0, eps_end: float = 0.1,
            anneal_updates: int = 1_000_000) -> float:
    """Section 5.1 schedule (gorila_epsilon)."""
    return float(lib().gorila_epsilon(update, eps_start, eps_end, anneal_updates))


# Convenience wrappers that allocate the outputs (torch) and return them.
def q_forward(ctx: Context, theta, n_actions: int, states):
    import torch
    q = torch.empty((states.shape[0], n_actions), dtype=torch.float32, device=states.device)
    gorila_q_forward(ctx, theta, n_actions, states, q)
    return q


def act(ctx: Context, theta, n_actions: int, states, eps: float, seed: int, with_q: bool = False):
    import torch
    n = states.shape[0]
    actions = torch.empty(n, dtype=torch.int32, device=states.device)
    q = torch.empty((n, n_actions), dtype=torch.float32, device=states.device) if with_q else None
    gorila_act(ctx, theta, n_actions, states, eps, seed, actions, q)
    return (actions, q) if with_q else actions


def learner_step(ctx: Context, theta, theta_target, n_actions: int, replay: Replay, idx,
                 gamma: float = 0.99, clip_delta: float = 1.0):
    import torch
    grads = torch.empty(param_count(n_actions), dtype=torch.float32, device=theta.device)
    loss = torch.empty(1, dtype=torch.float32, device=theta.device)
    gorila_learner_step(ctx, theta, theta_target, n_actions, replay, idx, gamma, clip_delta,
                        grads, loss)
    return grads, loss


def learner_step_grouped(ctx: Context, thetas, theta_target, n_actions: int, replay: Replay, idx,
                         gamma: float = 0.99, clip_delta: float = 1.0):
    """G learner steps sharing theta_target; returns grads [G, P] fp32 and loss [G]."""
    import torch
    G = len(thetas)
    batch = idx.shape[0] // G
    grads = torch.empty((G, param_count(n_actions)), dtype=torch.float32, device=idx.device)
    loss = torch.empty(G, dtype=torch.float32, device=idx.device)
    gorila_learner_step_grouped(ctx, thetas, theta_target, n_actions, replay, idx, batch, gamma,
                                clip_delta, grads, loss)
    return grads, loss


def gather(ctx: Context, replay: Replay, idx):
    import torch
    n, dev = idx.shape[0], idx.device
    s = torch.empty((n, 4, 84, 84), dtype=torch.uint8, device=dev)
    s2 = torch.empty_like(s)
    fmap = torch.empty((n, 2, 4), dtype=torch.int64, device=dev)
    a = torch.empty(n, dtype=torch.int32, device=dev)
    r = torch.empty(n, dtype=torch.float32, device=dev)
    t = torch.empty(n, dtype=torch.uint8, device=dev)
    gorila_gather(ctx, replay, idx, s, s2, fmap, a, r, t)
    return dict(s=s, s2=s2, frame_map=fmap, a=a, r=r, term=t)


INF = math.inf
