"""ctypes binding of libdqn.so.  Argument marshalling only."""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))

DQN_OK, DQN_EINVAL, DQN_EWORKSPACE, DQN_EHIP, DQN_EUNSUPPORTED = 0, -1, -2, -3, -4
PS_SGD, PS_RMSPROP, PS_ADAGRAD = 0, 1, 2
DQN_OP_FORWARD, DQN_OP_TD_GRADIENT = 0, 1
_RULES = {"sgd": PS_SGD, "rmsprop": PS_RMSPROP, "adagrad": PS_ADAGRAD}


class DqnError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {dqn_status_string(status)} ({status})")


class _CNet(ctypes.Structure):
    _fields_ = [("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32), ("in_w", ctypes.c_int32),
                ("n_conv", ctypes.c_int32), ("conv_out", ctypes.c_int32 * 3),
                ("conv_k", ctypes.c_int32 * 3), ("conv_stride", ctypes.c_int32 * 3),
                ("fc_hidden", ctypes.c_int32), ("n_actions", ctypes.c_int32),
                ("precision", ctypes.c_int32)]


class _CReplay(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_void_p), ("action", ctypes.c_void_p),
                ("reward", ctypes.c_void_p), ("terminal", ctypes.c_void_p),
                ("record_stride", ctypes.c_int64), ("size", ctypes.c_int64),
                ("c", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32)]


class _CReplayOut(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_void_p), ("action", ctypes.c_void_p), ("reward", ctypes.c_void_p),
                ("terminal", ctypes.c_void_p), ("record_stride", ctypes.c_int64), ("capacity", ctypes.c_int64)]


@dataclass(frozen=True)
class Net:
    """Q-network shape: conv layers as (out_channels, kernel, stride)."""
    in_c: int
    in_h: int
    in_w: int
    conv: tuple
    fc_hidden: int
    n_actions: int
    precision: int = 0


DQN_FP32, DQN_BF16 = 0, 1   # Net.precision (include/dqn.h)
NET_SMALL = Net(4, 84, 84, ((16, 8, 4), (32, 4, 2)), 256, 6)
NET_LARGE = Net(4, 84, 84, ((32, 8, 4), (64, 4, 2), (64, 3, 1)), 512, 18)
# The large network with bf16-input contractions (fp32 accumulation).
NET_LARGE_BF16 = Net(4, 84, 84, ((32, 8, 4), (64, 4, 2), (64, 3, 1)), 512, 18, DQN_BF16)


@dataclass
class Replay:
    """Device replay memory: records [size][c][h][w] uint8 (or any tensor
    whose record i starts at i*record_stride bytes) and side arrays."""
    frames: object      # torch uint8 tensor on the device
    action: object      # uint8 [size]
    reward: object      # int8 [size]
    terminal: object    # uint8 [size]
    size: int
    c: int = 4
    h: int = 84
    w: int = 84
    record_stride: int | None = None


def lib_path():
    return os.path.join(HERE, "libdqn.so")


_LIB = None
_P = ctypes.c_void_p


def lib():
    """The loaded libdqn.so.  Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        # torch ships its own HIP runtime under the same SONAME; importing it
        # first makes libdqn.so bind to that one, so there is a single HIP
        # runtime (and one set of streams) in the process.
        import torch  # noqa: F401
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError(f"libdqn.so not found at {path}; build it with "
                               "`python -m paper_1508_04186_amd.build`")
        L = ctypes.CDLL(path)
        L.dqn_param_count.argtypes = [ctypes.POINTER(_CNet)]
        L.dqn_param_count.restype = ctypes.c_int64
        L.dqn_param_offset.argtypes = [ctypes.POINTER(_CNet), ctypes.c_int32, ctypes.c_int32]
        L.dqn_param_offset.restype = ctypes.c_int64
        L.dqn_workspace_bytes.argtypes = [ctypes.POINTER(_CNet), ctypes.c_int32, ctypes.c_int32]
        L.dqn_workspace_bytes.restype = ctypes.c_int64
        L.replay_gather.argtypes = [ctypes.POINTER(_CReplay), _P, ctypes.c_int32, _P, _P, _P, _P,
                                    _P, _P]
        L.dqn_forward.argtypes = [ctypes.POINTER(_CNet), _P, _P, ctypes.c_int32, ctypes.c_float,
                                  _P, _P, _P, _P, ctypes.c_size_t, _P]
        L.dqn_td_gradient.argtypes = [ctypes.POINTER(_CNet), _P, _P, _P, _P, _P, _P, _P,
                                      ctypes.c_int32, ctypes.c_float, _P, _P, _P, _P, _P,
                                      ctypes.c_size_t, _P]
        L.dqn_forward_replay.argtypes = [ctypes.POINTER(_CNet), _P, ctypes.POINTER(_CReplay), _P,
                                         ctypes.c_int32, ctypes.c_float, _P, _P, _P, _P, ctypes.c_size_t,
                                         _P]
        L.dqn_forward_replay.restype = ctypes.c_int
        L.dqn_td_gradient_replay.argtypes = [ctypes.POINTER(_CNet), _P, _P, ctypes.POINTER(_CReplay),
                                             _P, ctypes.c_int32, ctypes.c_float, _P, _P, _P, _P,
                                             _P, ctypes.c_size_t, _P]
        L.dqn_td_gradient_replay.restype = ctypes.c_int
        L.dqn_td_gradient_noalloc.argtypes = [ctypes.POINTER(_CNet), _P, _P, _P, _P, _P, _P, _P,
                                              ctypes.c_int32, ctypes.c_float, _P, _P, _P, _P, _P]
        L.dqn_td_gradient_noalloc.restype = ctypes.c_int
        L.ps_apply_update.argtypes = [ctypes.c_int32, _P, _P, _P, _P, ctypes.c_int64,
                                      ctypes.c_float, ctypes.c_float, ctypes.c_float, _P]
        for f in ("replay_gather", "dqn_forward", "dqn_td_gradient", "ps_apply_update"):
            getattr(L, f).restype = ctypes.c_int
        L.dqn_status_string.argtypes = [ctypes.c_int]
        L.dqn_status_string.restype = ctypes.c_char_p
        L.dqn_train_ring_stride.argtypes = [ctypes.POINTER(_CNet)]
        L.dqn_train_ring_stride.restype = ctypes.c_int64
        L.dqn_train_workspace_bytes.argtypes = [ctypes.POINTER(_CNet), ctypes.c_int32, ctypes.c_int32]
        L.dqn_train_workspace_bytes.restype = ctypes.c_int64
        L.dqn_train_steps.argtypes = [ctypes.POINTER(_CNet), _P, _P, _P, ctypes.c_int32,
                                      ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                      ctypes.POINTER(_CReplay), _P, ctypes.c_int32, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int64, _P, _P, ctypes.c_size_t, _P]
        L.dqn_train_steps.restype = ctypes.c_int
        L.dqn_train_replicas.argtypes = [ctypes.POINTER(_CNet), _P, _P, ctypes.c_int32,
                                         ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                         ctypes.c_float, ctypes.POINTER(_CReplay), _P,
                                         ctypes.c_int32, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, _P, _P, ctypes.c_size_t, _P]
        L.dqn_train_replicas.restype = ctypes.c_int
        L.dqn_profile_attach.argtypes = [ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32]
        L.dqn_profile_attach.restype = ctypes.c_int
        L.dqn_profile_set_fusion.argtypes = [ctypes.c_int32]
        L.dqn_profile_set_fusion.restype = ctypes.c_int
        L.dqn_profile_used.argtypes = [ctypes.c_int32]
        L.dqn_profile_used.restype = ctypes.c_int32
        L.snake_state_bytes.argtypes = [ctypes.c_int32]
        L.snake_state_bytes.restype = ctypes.c_int64
        L.snake_reset.argtypes = [_P, ctypes.c_int32, _P, _P, ctypes.POINTER(_CReplayOut), _P]
        L.snake_reset.restype = ctypes.c_int
        L.snake_step.argtypes = [_P, ctypes.c_int32, _P, _P, _P, _P, _P, ctypes.POINTER(_CReplayOut),
                                 ctypes.c_int64, _P]
        L.snake_step.restype = ctypes.c_int
        L.dqn_anneal_epsilon.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_double, ctypes.c_double]
        L.dqn_anneal_epsilon.restype = ctypes.c_double
        L.dqn_act.argtypes = [ctypes.POINTER(_CNet), _P, _P, ctypes.c_int32, _P, ctypes.c_float, _P, _P, _P,
                              _P, _P, ctypes.POINTER(_CReplayOut), ctypes.c_int64, _P, ctypes.c_size_t, _P]
        L.dqn_act.restype = ctypes.c_int
        L.replay_gather_validate.argtypes = [ctypes.POINTER(_CReplay), _P, ctypes.c_int32, ctypes.c_int32, _P, _P]
        L.replay_gather_validate.restype = ctypes.c_int
        L.replay_fill_synthetic.argtypes = [ctypes.POINTER(_CReplay), ctypes.c_int32, ctypes.c_uint64, _P]
        L.replay_fill_synthetic.restype = ctypes.c_int
        L.dqn_preprocess.argtypes = [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64, _P]
        L.dqn_preprocess.restype = ctypes.c_int
        L.dqn_observe.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P, ctypes.POINTER(_CReplayOut),
                                  ctypes.c_int64, _P]
        L.dqn_observe.restype = ctypes.c_int
        L.dqn_profile_mfma_peak.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P]
        L.dqn_profile_mfma_peak.restype = ctypes.c_int64
        L.dqn_profile_stream_copy.argtypes = [_P, _P, ctypes.c_int64, ctypes.c_int32, _P]
        L.dqn_profile_stream_copy.restype = ctypes.c_int
        _LIB = L
    return _LIB


def dqn_status_string(status: int) -> str:
    return lib().dqn_status_string(int(status)).decode()


def _cnet(net) -> _CNet:
    n = _CNet()
    n.in_c, n.in_h, n.in_w = net.in_c, net.in_h, net.in_w
    n.n_conv = len(net.conv)
    for i, (o, k, s) in enumerate(net.conv):
        n.conv_out[i], n.conv_k[i], n.conv_stride[i] = o, k, s
    n.fc_hidden, n.n_actions = net.fc_hidden, net.n_actions
    n.precision = getattr(net, "precision", 0)
    return n


def _ptr(t, dtype=None, what="tensor"):
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{what} must live in device memory")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(rc, what):
    if rc != DQN_OK:
        raise DqnError(rc, what)


def dqn_param_count(net) -> int:
    v = lib().dqn_param_count(ctypes.byref(_cnet(net)))
    _check(0 if v >= 0 else v, "dqn_param_count")
    return int(v)


def dqn_param_offset(net, layer: int, is_bias: bool) -> int:
    v = lib().dqn_param_offset(ctypes.byref(_cnet(net)), layer, int(is_bias))
    _check(0 if v >= 0 else v, "dqn_param_offset")
    return int(v)


def dqn_workspace_bytes(net, batch: int, op: int) -> int:
    v = lib().dqn_workspace_bytes(ctypes.byref(_cnet(net)), batch, op)
    _check(0 if v >= 0 else v, "dqn_workspace_bytes")
    return int(v)


def workspace(net, batch: int, op: int, device="cuda"):
    """A device workspace tensor large enough for (net, batch, op)."""
    import torch
    return torch.empty(dqn_workspace_bytes(net, batch, op), dtype=torch.uint8, device=device)


def _creplay(replay: Replay) -> _CReplay:
    import torch
    rp = _CReplay()
    rp.frames = _ptr(replay.frames, torch.uint8, "replay.frames")
    rp.action = _ptr(replay.action, torch.uint8, "replay.action")
    rp.reward = _ptr(replay.reward, torch.int8, "replay.reward")
    rp.terminal = _ptr(replay.terminal, torch.uint8, "replay.terminal")
    rec = replay.c * replay.h * replay.w
    rp.record_stride = replay.record_stride if replay.record_stride is not None else rec
    rp.size = replay.size
    rp.c, rp.h, rp.w = replay.c, replay.h, replay.w
    return rp


def replay_gather(replay: Replay, idx, s_out, s_next_out=None, a_out=None, r_out=None,
                  term_out=None, stream=None):
    import torch
    rp = _CReplay()
    rp.frames = _ptr(replay.frames, torch.uint8, "replay.frames")
    rp.action = _ptr(replay.action, torch.uint8, "replay.action")
    rp.reward = _ptr(replay.reward, torch.int8, "replay.reward")
    rp.terminal = _ptr(replay.terminal, torch.uint8, "replay.terminal")
    rec = replay.c * replay.h * replay.w
    rp.record_stride = replay.record_stride if replay.record_stride is not None else rec
    rp.size = replay.size
    rp.c, rp.h, rp.w = replay.c, replay.h, replay.w
    B = idx.shape[0]
    for name, t, n in (("s_out", s_out, B * rec), ("s_next_out", s_next_out, B * rec),
                       ("a_out", a_out, B), ("r_out", r_out, B), ("term_out", term_out, B)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().replay_gather(ctypes.byref(rp), _ptr(idx, torch.int64, "idx"), B,
                             _ptr(s_out, torch.uint8, "s_out"),
                             _ptr(s_next_out, torch.uint8, "s_next_out"),
                             _ptr(a_out, torch.int32, "a_out"), _ptr(r_out, torch.float32, "r_out"),
                             _ptr(term_out, torch.uint8, "term_out"), _stream(stream))
    _check(rc, "replay_gather")


def dqn_forward(net, theta, states, epsilon=0.0, draws=None, q_out=None, action_out=None,
                ws=None, stream=None):
    import torch
    B = states.shape[0]
    if ws is None:
        ws = workspace(net, B, DQN_OP_FORWARD, states.device)
    if q_out is not None and q_out.numel() < B * net.n_actions:
        raise ValueError("q_out too small")
    if action_out is not None and action_out.numel() < B:
        raise ValueError("action_out too small")
    if draws is not None and draws.numel() < B:
        raise ValueError("draws too small")
    rc = lib().dqn_forward(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                           _ptr(states, torch.uint8, "states"), B, float(epsilon),
                           _ptr(draws, torch.uint64, "draws"), _ptr(q_out, torch.float32, "q_out"),
                           _ptr(action_out, torch.int32, "action_out"),
                           _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    _check(rc, "dqn_forward")


def dqn_forward_replay(net, theta, replay: Replay, idx, epsilon=0.0, draws=None, q_out=None,
                       action_out=None, ws=None, stream=None):
    """dqn_forward on the states idx (device int64 [B]) read in place from the
    replay (include/dqn.h dqn_forward_replay)."""
    import torch
    B = idx.shape[0]
    if ws is None:
        ws = workspace(net, B, DQN_OP_FORWARD, theta.device)
    if q_out is not None and q_out.numel() < B * net.n_actions:
        raise ValueError("q_out too small")
    if action_out is not None and action_out.numel() < B:
        raise ValueError("action_out too small")
    if draws is not None and draws.numel() < B:
        raise ValueError("draws too small")
    rc = lib().dqn_forward_replay(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                                  ctypes.byref(_creplay(replay)), _ptr(idx, torch.int64, "idx"), B,
                                  float(epsilon), _ptr(draws, torch.uint64, "draws"),
                                  _ptr(q_out, torch.float32, "q_out"),
                                  _ptr(action_out, torch.int32, "action_out"),
                                  _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    _check(rc, "dqn_forward_replay")


def dqn_td_gradient(net, theta, theta_target, s, s_next, action, reward, terminal, gamma,
                    grad_out, loss_out, q_out=None, y_out=None, ws=None, stream=None):
    import torch
    B = s.shape[0]
    if ws is None:
        ws = workspace(net, B, DQN_OP_TD_GRADIENT, s.device)
    P = dqn_param_count(net)
    for name, t, n in (("theta", theta, P), ("theta_target", theta_target, P),
                       ("grad_out", grad_out, P), ("s_next", s_next, s.numel()),
                       ("action", action, B), ("reward", reward, B), ("terminal", terminal, B),
                       ("loss_out", loss_out, 1), ("q_out", q_out, B * net.n_actions),
                       ("y_out", y_out, B)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().dqn_td_gradient(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                               _ptr(theta_target, torch.float32, "theta_target"),
                               _ptr(s, torch.uint8, "s"), _ptr(s_next, torch.uint8, "s_next"),
                               _ptr(action, torch.int32, "action"),
                               _ptr(reward, torch.float32, "reward"),
                               _ptr(terminal, torch.uint8, "terminal"), B, float(gamma),
                               _ptr(grad_out, torch.float32, "grad_out"),
                               _ptr(loss_out, torch.float32, "loss_out"),
                               _ptr(q_out, torch.float32, "q_out"), _ptr(y_out, torch.float32, "y_out"),
                               _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    _check(rc, "dqn_td_gradient")


def dqn_td_gradient_noalloc(net, theta, theta_target, s, s_next, action, reward, terminal, gamma,
                            grad_out, loss_out, q_out=None, y_out=None, stream=None):
    """dqn_td_gradient on the library's static per-GPU scratch instead of a
    caller workspace (include/dqn.h dqn_td_gradient_noalloc)."""
    import torch
    B = s.shape[0]
    P = dqn_param_count(net)
    for name, t, n in (("theta", theta, P), ("theta_target", theta_target, P),
                       ("grad_out", grad_out, P), ("s_next", s_next, s.numel()),
                       ("action", action, B), ("reward", reward, B), ("terminal", terminal, B),
                       ("loss_out", loss_out, 1), ("q_out", q_out, B * net.n_actions),
                       ("y_out", y_out, B)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().dqn_td_gradient_noalloc(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                                       _ptr(theta_target, torch.float32, "theta_target"),
                                       _ptr(s, torch.uint8, "s"), _ptr(s_next, torch.uint8, "s_next"),
                                       _ptr(action, torch.int32, "action"),
                                       _ptr(reward, torch.float32, "reward"),
                                       _ptr(terminal, torch.uint8, "terminal"), B, float(gamma),
                                       _ptr(grad_out, torch.float32, "grad_out"),
                                       _ptr(loss_out, torch.float32, "loss_out"),
                                       _ptr(q_out, torch.float32, "q_out"), _ptr(y_out, torch.float32, "y_out"),
                                       _stream(stream))
    _check(rc, "dqn_td_gradient_noalloc")


def dqn_td_gradient_replay(net, theta, theta_target, replay: Replay, idx, gamma, grad_out, loss_out,
                           q_out=None, y_out=None, ws=None, stream=None):
    """TD gradient of the minibatch idx (device int64 [B]) read in place from
    the replay (include/dqn.h dqn_td_gradient_replay)."""
    import torch
    B = idx.shape[0]
    if ws is None:
        ws = workspace(net, B, DQN_OP_TD_GRADIENT, theta.device)
    P = dqn_param_count(net)
    for name, t, n in (("theta", theta, P), ("theta_target", theta_target, P),
                       ("grad_out", grad_out, P), ("loss_out", loss_out, 1),
                       ("q_out", q_out, B * net.n_actions), ("y_out", y_out, B)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().dqn_td_gradient_replay(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                                      _ptr(theta_target, torch.float32, "theta_target"),
                                      ctypes.byref(_creplay(replay)), _ptr(idx, torch.int64, "idx"),
                                      B, float(gamma), _ptr(grad_out, torch.float32, "grad_out"),
                                      _ptr(loss_out, torch.float32, "loss_out"),
                                      _ptr(q_out, torch.float32, "q_out"),
                                      _ptr(y_out, torch.float32, "y_out"),
                                      _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    _check(rc, "dqn_td_gradient_replay")


def ps_apply_update(rule, theta_in, theta_out, state, grad, lr, decay=0.9, eps=0.0, stream=None,
                    n=None):
    import torch
    rule = _RULES.get(rule, rule)
    n = theta_in.numel() if n is None else n
    for name, t in (("theta_out", theta_out), ("state", state), ("grad", grad)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().ps_apply_update(int(rule), _ptr(theta_in, torch.float32, "theta_in"),
                               _ptr(theta_out, torch.float32, "theta_out"),
                               _ptr(state, torch.float32, "state"), _ptr(grad, torch.float32, "grad"),
                               n, float(lr), float(decay), float(eps), _stream(stream))
    _check(rc, "ps_apply_update")


# ----------------------------------------------------------------------------
# Worker and parameter-server loops (include/dqn_train.h)

class HipStreams:
    """n distinct HIP streams at the default priority (torch's stream pool may
    hand out the same stream twice).  They synchronize with the legacy
    default stream like torch's own; release them with close()."""

    def __init__(self, n: int):
        import torch
        path = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
        self._hip = ctypes.CDLL(path if os.path.exists(path) else "libamdhip64.so")
        self._hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipStreamCreate.restype = ctypes.c_int
        self._hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        self._hip.hipStreamDestroy.restype = ctypes.c_int
        torch.cuda.init()
        self.handles = []
        for _ in range(n):
            h = ctypes.c_void_p()
            if self._hip.hipStreamCreate(ctypes.byref(h)) != 0:
                self.close()
                raise RuntimeError("hipStreamCreate failed")
            self.handles.append(h.value)

    def close(self):
        for h in self.handles:
            self._hip.hipStreamDestroy(h)
        self.handles = []

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def dqn_train_ring_stride(net) -> int:
    v = lib().dqn_train_ring_stride(ctypes.byref(_cnet(net)))
    _check(0 if v >= 0 else v, "dqn_train_ring_stride")
    return int(v)


def dqn_train_workspace_bytes(net, batch: int, replicas: int = 1) -> int:
    v = lib().dqn_train_workspace_bytes(ctypes.byref(_cnet(net)), batch, replicas)
    _check(0 if v >= 0 else v, "dqn_train_workspace_bytes")
    return int(v)


def dqn_train_steps(net, theta, theta_target, opt_state, rule, lr, decay, eps, gamma, replay, idx,
                    step0=0, target_period=0, losses_out=None, ws=None, stream=None):
    """idx: device int64 [n_steps][batch]."""
    import torch
    rule = _RULES.get(rule, rule)
    n_steps, batch = idx.shape
    P = dqn_param_count(net)
    if ws is None:
        ws = torch.empty(dqn_train_workspace_bytes(net, batch, 1), dtype=torch.uint8,
                         device=theta.device)
    for name, t, n in (("theta", theta, P), ("theta_target", theta_target, P),
                       ("opt_state", opt_state, P), ("losses_out", losses_out, n_steps)):
        if t is not None and t.numel() < n:
            raise ValueError(f"{name} too small")
    rc = lib().dqn_train_steps(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                               _ptr(theta_target, torch.float32, "theta_target"),
                               _ptr(opt_state, torch.float32, "opt_state"), int(rule), float(lr),
                               float(decay), float(eps), float(gamma), ctypes.byref(_creplay(replay)),
                               _ptr(idx, torch.int64, "idx"), batch, n_steps, int(step0),
                               int(target_period), _ptr(losses_out, torch.float32, "losses_out"),
                               _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    _check(rc, "dqn_train_steps")


def dqn_train_replicas(net, theta_ring, opt_state, rule, lr, decay, eps, gamma, replay, idx,
                       replicas, staleness, streams, losses_out=None, ws=None):
    """theta_ring: device float [staleness+1][dqn_train_ring_stride(net)]
    (slot 0 = initial parameters);
    streams: replicas + 1 distinct streams (HipStreams handles or
    torch.cuda.Stream objects): the replica streams, then the server stream.
    idx: device int64 [n_updates][batch]."""
    import torch
    rule = _RULES.get(rule, rule)
    n_updates, batch = idx.shape
    if theta_ring.numel() < (staleness + 1) * dqn_train_ring_stride(net):
        raise ValueError("theta_ring too small")
    if len(streams) != replicas + 1:
        raise ValueError("need replicas + 1 streams")
    if ws is None:
        ws = torch.empty(dqn_train_workspace_bytes(net, batch, replicas), dtype=torch.uint8,
                         device=theta_ring.device)
    if losses_out is not None and losses_out.numel() < n_updates:
        raise ValueError("losses_out too small")
    arr = (ctypes.c_void_p * (replicas + 1))(*[_stream(s) for s in streams])
    rc = lib().dqn_train_replicas(ctypes.byref(_cnet(net)), _ptr(theta_ring, torch.float32, "theta_ring"),
                                  _ptr(opt_state, torch.float32, "opt_state"), int(rule), float(lr),
                                  float(decay), float(eps), float(gamma),
                                  ctypes.byref(_creplay(replay)), _ptr(idx, torch.int64, "idx"),
                                  batch, n_updates, replicas, staleness,
                                  _ptr(losses_out, torch.float32, "losses_out"),
                                  _ptr(ws, torch.uint8, "ws"), ws.numel(),
                                  ctypes.cast(arr, ctypes.c_void_p))
    _check(rc, "dqn_train_replicas")


# ----------------------------------------------------------------------------
# Measurement hook (include/dqn_profile.h)

KERNEL_NAMES = ["gather", "conv1_fwd", "conv2_fwd", "conv3_fwd", "fc1_fwd", "head", "fc1_wgrad",
                "fc1_dgrad", "conv1_wgrad", "conv2_wgrad", "conv3_wgrad", "conv2_dgrad",
                "conv3_dgrad", "finalize", "apply", "fc1_bwd", "conv2_bwd", "conv3_bwd",
                "finalize_apply", "conv12_fwd", "conv12_bwd", "snake_step", "observe", "weight_repack"]
_ATTACHED = {}


def profile_attach(kernel: int, events, stride: int = 1) -> None:
    """Bracket every stride-th launch of `kernel`, up to len(events)//2 of
    them, with the given hipEvent_t handles (ints), pairwise.  events=None
    detaches."""
    if events is None or len(events) < 2:
        rc = lib().dqn_profile_attach(kernel, None, 0, 1)
        _ATTACHED.pop(kernel, None)
    else:
        arr = (ctypes.c_void_p * len(events))(*events)
        _ATTACHED[kernel] = arr
        rc = lib().dqn_profile_attach(kernel, ctypes.cast(arr, ctypes.c_void_p), len(events) // 2,
                                      int(stride))
    _check(rc, "dqn_profile_attach")


def profile_set_fusion(enabled: bool) -> None:
    """Enable (default) or disable the fused two-layer conv launches of the
    small network (include/dqn_profile.h dqn_profile_set_fusion)."""
    _check(lib().dqn_profile_set_fusion(1 if enabled else 0), "dqn_profile_set_fusion")


def profile_used(kernel: int) -> int:
    return int(lib().dqn_profile_used(kernel))


DQN_PEAK_FP32, DQN_PEAK_BF16 = 0, 1


def profile_mfma_peak(dtype: int, workgroups: int, iters: int, out, stream=None) -> int:
    """Enqueue the pure matrix-core loop (include/dqn_profile.h); returns its FLOP count.
    out: device float32 tensor with at least `workgroups` elements."""
    import torch
    if out.numel() < workgroups:
        raise ValueError("out needs one float per workgroup")
    v = lib().dqn_profile_mfma_peak(int(dtype), int(workgroups), int(iters),
                                    _ptr(out, torch.float32, "out"), _stream(stream))
    _check(0 if v > 0 else int(v), "dqn_profile_mfma_peak")
    return int(v)


def profile_stream_copy(src, dst, workgroups: int, stream=None) -> None:
    """Enqueue the streaming copy dst <- src (equal-sized device tensors, bytes a multiple of 16)."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb:
        raise ValueError("src and dst must have the same byte size")
    _check(lib().dqn_profile_stream_copy(_ptr(src, None, "src"), _ptr(dst, None, "dst"), nb,
                                         int(workgroups), _stream(stream)), "dqn_profile_stream_copy")


# ----------------------------------------------------------------------------
# The actor side of Alg. 1 (include/dqn_actor.h)

SNAKE_STATE_BYTES = 512


class ActorReplay:
    """Replay memory pooled over n_games games, each keeping its last
    `capacity` states in capacity + 1 device records (include/dqn_actor.h);
    `view` is the same memory as a Replay for replay_gather and
    dqn_td_gradient_replay."""

    def __init__(self, n_games: int, capacity: int, device="cuda"):
        import torch
        self.n_games, self.capacity = n_games, capacity
        n = n_games * (capacity + 1)
        self.frames = torch.zeros((n, 4, 84, 84), dtype=torch.uint8, device=device)
        self.action = torch.zeros(n, dtype=torch.uint8, device=device)
        self.reward = torch.zeros(n, dtype=torch.int8, device=device)
        self.terminal = torch.zeros(n, dtype=torch.uint8, device=device)
        self.view = Replay(self.frames, self.action, self.reward, self.terminal, n)

    def _c(self):
        r = _CReplayOut()
        r.frames, r.action = self.frames.data_ptr(), self.action.data_ptr()
        r.reward, r.terminal = self.reward.data_ptr(), self.terminal.data_ptr()
        r.record_stride, r.capacity = 4 * 84 * 84, self.capacity
        return r


def snake_games(n_games: int, device="cuda"):
    """Device state of n_games games (uninitialized until snake_reset)."""
    import torch
    v = lib().snake_state_bytes(n_games)
    _check(0 if v > 0 else int(v), "snake_state_bytes")
    return torch.empty(int(v), dtype=torch.uint8, device=device)


def snake_reset(games, draws, states, replay: ActorReplay | None = None, stream=None) -> None:
    import torch
    E = states.shape[0]
    rp = replay._c() if replay is not None else None
    _check(lib().snake_reset(_ptr(games, torch.uint8, "games"), E, _ptr(draws, torch.uint64, "draws"),
                             _ptr(states, torch.uint8, "states"), ctypes.byref(rp) if rp else None,
                             _stream(stream)), "snake_reset")


def snake_step(games, actions, draws, states, reward_out, terminal_out, replay: ActorReplay | None = None,
               t: int = 0, stream=None) -> None:
    import torch
    E = states.shape[0]
    rp = replay._c() if replay is not None else None
    _check(lib().snake_step(_ptr(games, torch.uint8, "games"), E, _ptr(actions, torch.int32, "actions"),
                            _ptr(draws, torch.uint64, "draws"), _ptr(states, torch.uint8, "states"),
                            _ptr(reward_out, torch.float32, "reward_out"),
                            _ptr(terminal_out, torch.uint8, "terminal_out"), ctypes.byref(rp) if rp else None,
                            int(t), _stream(stream)), "snake_step")


def dqn_anneal_epsilon(n: int, n_max: int, eps_min: float, eps_max: float) -> float:
    return float(lib().dqn_anneal_epsilon(int(n), int(n_max), float(eps_min), float(eps_max)))


def dqn_act(net, theta, games, states, epsilon, eps_draws, env_draws, actions_out, reward_out, terminal_out,
            replay: ActorReplay | None = None, t: int = 0, ws=None, stream=None) -> None:
    """One acting step of Alg. 1 (include/dqn_actor.h dqn_act)."""
    import torch
    E = states.shape[0]
    if ws is None:
        ws = workspace(net, E, DQN_OP_FORWARD, states.device)
    rp = replay._c() if replay is not None else None
    _check(lib().dqn_act(ctypes.byref(_cnet(net)), _ptr(theta, torch.float32, "theta"),
                         _ptr(games, torch.uint8, "games"), E, _ptr(states, torch.uint8, "states"),
                         ctypes.c_float(epsilon), _ptr(eps_draws, torch.uint64, "eps_draws"),
                         _ptr(env_draws, torch.uint64, "env_draws"), _ptr(actions_out, torch.int32, "actions_out"),
                         _ptr(reward_out, torch.float32, "reward_out"),
                         _ptr(terminal_out, torch.uint8, "terminal_out"), ctypes.byref(rp) if rp else None,
                         int(t), _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream)), "dqn_act")


def dqn_preprocess(rgb, top: int, left: int, factor: int, out=None, stream=None):
    """phi of raw screens rgb uint8 [n][h][w][3] (include/dqn_actor.h).  out:
    uint8 [n][84][84], or any uint8 tensor whose dim-0 slices hold one 84 x 84
    frame each at a 16-byte multiple stride (e.g. states[:, 3] of a
    [n][4][84][84] state array).  Returns out."""
    import torch
    n, h, w, c = rgb.shape
    if c != 3:
        raise ValueError("rgb must be [n][h][w][3]")
    if out is None:
        out = torch.empty((n, 84, 84), dtype=torch.uint8, device=rgb.device)
    if out.dtype != torch.uint8 or not out.is_cuda:
        raise TypeError("out must be a uint8 device tensor")
    if out.shape[0] != n or (n > 0 and (out[0].numel() != 84 * 84 or not out[0].is_contiguous())):
        raise ValueError("out must hold n contiguous 84 x 84 frames")
    stride = out.stride(0) if n > 1 else 84 * 84
    _check(lib().dqn_preprocess(_ptr(rgb, torch.uint8, "rgb"), n, h, w, top, left, factor, out.data_ptr(),
                                stride, _stream(stream)), "dqn_preprocess")
    return out


def dqn_observe(rgb, top: int, left: int, factor: int, states, actions=None, rewards=None, terminal=None,
                replay: ActorReplay | None = None, t: int = -1, stream=None) -> None:
    """Observe step of Alg. 1 for games with raw screens (include/dqn_actor.h):
    phi of each game's screen into its state stack and, with a replay, the
    experience into it.  t = -1 starts the games."""
    import torch
    E, h, w, _ = rgb.shape
    if tuple(states.shape) != (E, 4, 84, 84):
        raise ValueError("states must be [n_games][4][84][84]")
    rp = replay._c() if replay is not None else None
    _check(lib().dqn_observe(_ptr(rgb, torch.uint8, "rgb"), E, h, w, top, left, factor,
                             _ptr(actions, torch.int32, "actions"), _ptr(rewards, torch.int8, "rewards"),
                             _ptr(terminal, torch.uint8, "terminal"), _ptr(states, torch.uint8, "states"),
                             ctypes.byref(rp) if rp else None, int(t), _stream(stream)), "dqn_observe")


def replay_fill_synthetic(replay: "Replay", n_actions: int, seed: int, stream=None) -> None:
    """Fill a replay memory with the seeded synthetic stream (include/dqn.h)."""
    _check(lib().replay_fill_synthetic(ctypes.byref(_creplay(replay)), int(n_actions), int(seed) & (2**64 - 1),
                                       _stream(stream)), "replay_fill_synthetic")


def replay_gather_validate(replay: "Replay", idx, bad_count, with_next: bool = True, stream=None) -> None:
    """Count the indices of idx outside the valid range into bad_count
    (device int32 [1]; include/dqn.h)."""
    import torch
    _check(lib().replay_gather_validate(ctypes.byref(_creplay(replay)), _ptr(idx, torch.int64, "idx"),
                                        int(idx.numel()), 1 if with_next else 0,
                                        _ptr(bad_count, torch.int32, "bad_count"), _stream(stream)),
           "replay_gather_validate")
