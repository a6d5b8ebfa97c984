"""CPU oracle for the DQN TD-gradient and parameter-server hot path.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg, never by the HIP library or its binding.
It shares no code with the HIP path.  The arithmetic lives in oracle.c
(double precision, direct loops); this module marshals numpy arrays and
drives multi-step runs (sequential SGD, target-network refresh, and the
staleness-bounded replica schedule) from the per-step functions.

Parity pins: every function here is checked by the CPU tests against facts
the paper and the mathematics fix (finite differences, closed forms,
hand-built transitions, brute force, invariants); none is left unpinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
RULE_SGD, RULE_RMSPROP, RULE_ADAGRAD = 0, 1, 2
_RULES = {"sgd": RULE_SGD, "rmsprop": RULE_RMSPROP, "adagrad": RULE_ADAGRAD}


class _Net(ctypes.Structure):
    _fields_ = [("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32), ("in_w", ctypes.c_int32),
                ("n_conv", ctypes.c_int32), ("conv_out", ctypes.c_int32 * 3),
                ("conv_k", ctypes.c_int32 * 3), ("conv_stride", ctypes.c_int32 * 3),
                ("fc_hidden", ctypes.c_int32), ("n_actions", ctypes.c_int32),
                ("bf16_inputs", ctypes.c_int32)]


def lib_path():
    return os.path.join(HERE, "liboracle.so")


def build():
    src = os.path.join(HERE, "oracle.c")
    out = lib_path()
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-Wall",
                           "-Wextra", "-Werror", src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


_LIB = None
_P = ctypes.c_void_p


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(lib_path()):
            build()
        lib = ctypes.CDLL(lib_path())
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_num_threads.restype = ctypes.c_int
        lib.oracle_param_count.argtypes = [ctypes.POINTER(_Net)]
        lib.oracle_param_count.restype = ctypes.c_int64
        lib.oracle_param_offset.argtypes = [ctypes.POINTER(_Net), ctypes.c_int32, ctypes.c_int32]
        lib.oracle_param_offset.restype = ctypes.c_int64
        lib.oracle_replay_gather.argtypes = [_P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                             _P, _P, _P, _P, ctypes.c_int64, ctypes.c_int64,
                                             _P, _P, _P, _P, _P]
        lib.oracle_forward_q.argtypes = [ctypes.POINTER(_Net), _P, _P, ctypes.c_int64, _P]
        lib.oracle_relu_margins.argtypes = [ctypes.POINTER(_Net), _P, _P, ctypes.c_int64, _P]
        lib.oracle_select_actions.argtypes = [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
                                              _P, _P]
        lib.oracle_td_gradient.argtypes = [ctypes.POINTER(_Net), _P, _P, _P, _P, _P, _P, _P,
                                           ctypes.c_int64, ctypes.c_double, _P, _P, _P, _P, _P]
        lib.oracle_apply_update.argtypes = [ctypes.c_int32, _P, _P, _P, _P, ctypes.c_int64,
                                            ctypes.c_double, ctypes.c_double, ctypes.c_double]
        lib.oracle_bf16_round.argtypes = [_P, ctypes.c_int64, _P]
        lib.oracle_snake_reset.argtypes = [_P, ctypes.c_int64, _P, _P]
        lib.oracle_snake_step.argtypes = [_P, ctypes.c_int64, _P, _P, _P, _P, _P]
        lib.oracle_replay_append.argtypes = [_P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                             ctypes.c_int64, _P, _P, _P, _P, _P, _P, _P]
        lib.oracle_anneal_epsilon.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_double,
                                              ctypes.c_double]
        lib.oracle_anneal_epsilon.restype = ctypes.c_double
        lib.oracle_preprocess.argtypes = [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_int32, _P]
        for f in ("oracle_snake_reset", "oracle_snake_step", "oracle_replay_append", "oracle_preprocess"):
            getattr(lib, f).restype = ctypes.c_int
        for f in ("oracle_replay_gather", "oracle_forward_q", "oracle_relu_margins", "oracle_bf16_round",
                  "oracle_select_actions",
                  "oracle_td_gradient", "oracle_apply_update"):
            getattr(lib, f).restype = ctypes.c_int
        _LIB = lib
    return _LIB


def _net(net, bf16=False):
    """bf16: the bf16-input variant (every layer-contraction operand rounded
    to bfloat16, round to nearest even, before the double-precision products)."""
    n = _Net()
    n.in_c, n.in_h, n.in_w = net.in_c, net.in_h, net.in_w
    n.n_conv = len(net.conv)
    for i, (o, k, s) in enumerate(net.conv):
        n.conv_out[i], n.conv_k[i], n.conv_stride[i] = o, k, s
    n.fc_hidden, n.n_actions = net.fc_hidden, net.n_actions
    n.bf16_inputs = 1 if bf16 else 0
    return n


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what} failed with status {rc}")


def num_threads() -> int:
    return int(_lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (the results do not
    depend on the count)."""
    _check(_lib().oracle_set_num_threads(int(n)), "oracle_set_num_threads")


def param_count(net) -> int:
    return int(_lib().oracle_param_count(ctypes.byref(_net(net))))


def param_offset(net, layer: int, is_bias: bool) -> int:
    return int(_lib().oracle_param_offset(ctypes.byref(_net(net)), layer, int(is_bias)))


def replay_gather(frames, record_stride, rec_bytes, size, action, reward, terminal, idx,
                  with_next=True, max_index=None):
    """Returns (s, s_next, a int32, r float32, term uint8)."""
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    B = idx.shape[0]
    s = np.empty((B, rec_bytes), np.uint8)
    sn = np.empty((B, rec_bytes), np.uint8) if with_next else None
    a = np.empty(B, np.int32)
    r = np.empty(B, np.float32)
    t = np.empty(B, np.uint8)
    if max_index is None:
        max_index = size - 2 if with_next else size - 1
    rc = _lib().oracle_replay_gather(frames.ctypes.data, record_stride, rec_bytes, size,
                                     action.ctypes.data, reward.ctypes.data, terminal.ctypes.data,
                                     idx.ctypes.data, B, max_index, s.ctypes.data, _ptr(sn),
                                     a.ctypes.data, r.ctypes.data, t.ctypes.data)
    _check(rc, "oracle_replay_gather")
    return s, sn, a, r, t


def gather_from_host_replay(rep, idx, with_next=True):
    """Gather from a dqn_inputs.HostReplay (record i = frames i..i+3)."""
    rec_bytes = rep.c * rep.frames.shape[1] * rep.frames.shape[2]
    return replay_gather(rep.frames, rep.record_stride, rec_bytes, rep.size, rep.action,
                         rep.reward, rep.terminal, idx, with_next)


def bf16_round(x) -> np.ndarray:
    """x rounded to float32 and then to bfloat16 (nearest, ties to even), as float64."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    _check(_lib().oracle_bf16_round(x.ctypes.data, x.size, out.ctypes.data), "oracle_bf16_round")
    return out


def forward_q(net, theta, states, bf16=False) -> np.ndarray:
    th = np.ascontiguousarray(theta, dtype=np.float64)
    st = np.ascontiguousarray(states, dtype=np.uint8)
    B = st.shape[0]
    q = np.empty((B, net.n_actions), np.float64)
    _check(_lib().oracle_forward_q(ctypes.byref(_net(net, bf16)), th.ctypes.data, st.ctypes.data, B,
                                   q.ctypes.data), "oracle_forward_q")
    return q


def relu_margins(net, theta, states) -> np.ndarray:
    """Per-sample smallest normalized ReLU margin |z| / (|b| + sum |w x|) of
    Q(state; theta) over every conv and hidden fc unit (float64)."""
    th = np.ascontiguousarray(theta, dtype=np.float64)
    st = np.ascontiguousarray(states, dtype=np.uint8)
    B = st.shape[0]
    m = np.empty(B, np.float64)
    _check(_lib().oracle_relu_margins(ctypes.byref(_net(net)), th.ctypes.data, st.ctypes.data, B,
                                      m.ctypes.data), "oracle_relu_margins")
    return m


def select_actions(q, epsilon, draws=None) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.float64)
    B, A = q.shape
    act = np.empty(B, np.int32)
    d = None if draws is None else np.ascontiguousarray(draws, dtype=np.uint64)
    _check(_lib().oracle_select_actions(q.ctypes.data, B, A, float(epsilon), _ptr(d),
                                        act.ctypes.data), "oracle_select_actions")
    return act


def td_gradient(net, theta, theta_tgt, s, s_next, a, r, term, gamma, bf16=False):
    """Returns dict(grad fp64 [p], loss, q [B][A], qn [B][A], y [B]).
    bf16: the bf16-input variant (see _net)."""
    th = np.ascontiguousarray(theta, dtype=np.float64)
    tt = th if theta_tgt is None else np.ascontiguousarray(theta_tgt, dtype=np.float64)
    s = np.ascontiguousarray(s, dtype=np.uint8)
    sn = np.ascontiguousarray(s_next, dtype=np.uint8)
    a = np.ascontiguousarray(a, dtype=np.int32)
    r = np.ascontiguousarray(r, dtype=np.float32)
    t = np.ascontiguousarray(term, dtype=np.uint8)
    B = s.shape[0]
    P = param_count(net)
    grad = np.empty(P, np.float64)
    loss = np.zeros(1, np.float64)
    q = np.empty((B, net.n_actions), np.float64)
    qn = np.empty((B, net.n_actions), np.float64)
    y = np.empty(B, np.float64)
    rc = _lib().oracle_td_gradient(ctypes.byref(_net(net, bf16)), th.ctypes.data, tt.ctypes.data,
                                   s.ctypes.data, sn.ctypes.data, a.ctypes.data, r.ctypes.data,
                                   t.ctypes.data, B, float(gamma), grad.ctypes.data,
                                   loss.ctypes.data, q.ctypes.data, qn.ctypes.data, y.ctypes.data)
    _check(rc, "oracle_td_gradient")
    return dict(grad=grad, loss=float(loss[0]), q=q, qn=qn, y=y)


def apply_update(rule, theta, state, grad, lr, decay=0.9, eps=0.0):
    """Returns (theta' float32, state' float32 or None); inputs are not modified."""
    rule = _RULES.get(rule, rule)
    th = np.ascontiguousarray(theta, dtype=np.float32)
    out = np.empty_like(th)
    st = None if state is None else np.array(state, dtype=np.float32, copy=True)
    g = np.ascontiguousarray(grad, dtype=np.float64)
    _check(_lib().oracle_apply_update(rule, th.ctypes.data, out.ctypes.data, _ptr(st),
                                      g.ctypes.data, th.shape[0], float(lr), float(decay),
                                      float(eps)), "oracle_apply_update")
    return out, st


# ----------------------------------------------------------------------------
# Multi-step drivers

def sequential_training(net, theta0, rep, idx_stream, gamma, lr, rule="sgd", decay=0.9, eps=0.0,
                        target_period=None, steps=None, state0=None, callback=None, bf16=False):
    """Sequential worker + server: for n = 0..steps-1, gather the minibatch
    idx_stream[n] from the host replay, compute the TD gradient with the
    target network, and apply the update (Alg. 1 then Alg. 2 with one
    worker).  Target network: theta^- = theta_n when target_period is None;
    otherwise it is refreshed to theta_n at n = 0, C, 2C, ... (Alg. 1's
    refresh test n >= l*C with generation l starting at 0).
    Returns (theta float32, state, losses)."""
    theta = np.array(theta0, dtype=np.float32, copy=True)
    state = None if rule == "sgd" else (np.zeros_like(theta) if state0 is None else state0.copy())
    tgt = theta.copy()
    gen = 0
    steps = idx_stream.shape[0] if steps is None else steps
    losses = []
    for n in range(steps):
        if target_period is None:
            tgt = theta
        elif n >= gen * target_period:
            tgt = theta.copy()
            gen = n // target_period + 1
        s, sn, a, r, t = gather_from_host_replay(rep, idx_stream[n])
        out = td_gradient(net, theta, tgt, s, sn, a, r, t, gamma, bf16)
        losses.append(out["loss"])
        theta, state = apply_update(rule, theta, state, out["grad"], lr, decay, eps)
        if callback is not None:
            callback(n, theta, state, out)
    return theta, state, np.array(losses)


def stale_replica_training(net, theta0, rep, idx_stream, gamma, lr, staleness, rule="adagrad",
                           decay=0.9, eps=1e-8, updates=None, callback=None, state0=None):
    """Asynchronous workers with bounded staleness, replayed deterministically
    (Sec. IV.A, Alg. 2): update u is a gradient computed on the parameter
    version v(u) = max(0, u - staleness), which also serves as that worker's
    target network; the server applies updates in order u = 0, 1, ...,
    producing version u + 1.  Which replica computed update u does not
    change the arithmetic.  state0 is the optimizer state before update 0
    (zero when None).  Returns (theta, state, losses)."""
    updates = idx_stream.shape[0] if updates is None else updates
    versions = [np.array(theta0, dtype=np.float32, copy=True)]
    state = None if rule == "sgd" else (np.zeros_like(versions[0]) if state0 is None
                                        else np.array(state0, dtype=np.float32, copy=True))
    losses = []
    for u in range(updates):
        v = max(0, u - staleness)
        th_v = versions[v]
        s, sn, a, r, t = gather_from_host_replay(rep, idx_stream[u])
        out = td_gradient(net, th_v, th_v, s, sn, a, r, t, gamma)
        losses.append(out["loss"])
        new, state = apply_update(rule, versions[-1], state, out["grad"], lr, decay, eps)
        versions.append(new)
        if len(versions) > staleness + 2:
            versions[len(versions) - staleness - 3] = None  # no longer reachable
        if callback is not None:
            callback(u, new, state, out)
    return versions[-1], state, np.array(losses)


# ----------------------------------------------------------------------------
# The actor side of Alg. 1: Snake games and the replay memory they fill

SNAKE_GRID = 12
SNAKE_STATE_INTS = SNAKE_GRID * SNAKE_GRID + 3   # body cells, length, heading, apple


class SnakeGames:
    """E Snake games (oracle.c states the rules and the readings) with their
    stacked-frame states uint8 [E][4][84][84]."""

    def __init__(self, E: int, draws):
        self.E = E
        self.games = np.zeros((E, SNAKE_STATE_INTS), np.int32)
        self.states = np.zeros((E, 4, 84, 84), np.uint8)
        d = np.ascontiguousarray(draws, dtype=np.uint64).reshape(E, 2)
        _check(_lib().oracle_snake_reset(self.games.ctypes.data, E, d.ctypes.data, self.states.ctypes.data),
               "oracle_snake_reset")

    def step(self, actions, draws):
        """Returns (reward float32 [E], terminal uint8 [E]); states advance."""
        a = np.ascontiguousarray(actions, dtype=np.int32)
        d = np.ascontiguousarray(draws, dtype=np.uint64).reshape(self.E, 2)
        r = np.empty(self.E, np.float32)
        t = np.empty(self.E, np.uint8)
        _check(_lib().oracle_snake_step(self.games.ctypes.data, self.E, a.ctypes.data, d.ctypes.data,
                                        self.states.ctypes.data, r.ctypes.data, t.ctypes.data),
               "oracle_snake_step")
        return r, t

    def lengths(self):
        return self.games[:, SNAKE_GRID * SNAKE_GRID].copy()


class SegmentedReplay:
    """Replay memory pooled over E games, each keeping its last N states in
    N + 1 records (slot N repeats slot 0): see oracle_replay_append."""

    def __init__(self, E: int, N: int, rec_bytes: int = 4 * 84 * 84):
        self.E, self.N, self.rec = E, N, rec_bytes
        self.frames = np.zeros((E * (N + 1), rec_bytes), np.uint8)
        self.action = np.zeros(E * (N + 1), np.uint8)
        self.reward = np.zeros(E * (N + 1), np.int8)
        self.terminal = np.zeros(E * (N + 1), np.uint8)

    def append(self, t, states, actions=None, reward=None, terminal=None):
        st = np.ascontiguousarray(states, dtype=np.uint8)
        a = None if actions is None else np.ascontiguousarray(actions, dtype=np.int32)
        r = None if reward is None else np.ascontiguousarray(reward, dtype=np.float32)
        tt = None if terminal is None else np.ascontiguousarray(terminal, dtype=np.uint8)
        _check(_lib().oracle_replay_append(self.frames.ctypes.data, self.rec, self.E, self.N, int(t),
                                           st.ctypes.data, _ptr(a), _ptr(r), _ptr(tt),
                                           self.action.ctypes.data, self.reward.ctypes.data,
                                           self.terminal.ctypes.data), "oracle_replay_append")


def anneal_epsilon(n, n_max, eps_min, eps_max) -> float:
    """Alg. 1: q = max((N_max - n)/N_max, 0); epsilon = (1 - q) eps_min + q eps_max."""
    return float(_lib().oracle_anneal_epsilon(int(n), int(n_max), float(eps_min), float(eps_max)))


def preprocess(rgb, top, left, factor) -> np.ndarray:
    """phi of uint8 RGB frames [n][h][w][3] -> uint8 [n][84][84] (oracle.c states the reading)."""
    x = np.ascontiguousarray(rgb, dtype=np.uint8)
    n, h, w, _ = x.shape
    out = np.empty((n, 84, 84), np.uint8)
    _check(_lib().oracle_preprocess(x.ctypes.data, n, h, w, top, left, factor, out.ctypes.data),
           "oracle_preprocess")
    return out


def stack_frames(states, frames, terminal, t) -> np.ndarray:
    """Alg. 1's next state over the last four preprocessed frames: a state
    drops its oldest frame and appends the new one, oldest first; a game that
    starts (t = -1) or restarts (its terminal flag) holds four copies of its
    first frame.  states uint8 [n][4][84][84], frames uint8 [n][84][84]."""
    out = np.empty_like(states)
    for e in range(states.shape[0]):
        if t < 0 or terminal[e]:
            out[e] = frames[e][None]
        else:
            out[e, :3] = states[e, 1:]
            out[e, 3] = frames[e]
    return out
