"""Seeded synthetic inputs for the DQN hot path.

This package is shared by the CPU oracle, the tests and the benchmark.  It
generates inputs only (network shapes, initial weights, replay contents, index
streams, exploration draws); it computes no part of the Q-learning method.

Workload stand-ins (the paper's Snake game and its frames are not available):
  * frames: 84x84 uint8 screens, dark noisy background plus 1..4 moving bright
    rectangles (frames.c), stacked four at a time as in Sec. III.A;
  * replay side arrays: action uniform on {0..A-1}, reward uniform on
    {-1, 0, +1}, terminal Bernoulli(0.01);
  * weights: Xavier-uniform, biases zero (the paper's N(0, xi) init leaves xi
    unvalued, Alg. 2);
  * minibatch indices: uniform with replacement over valid transitions
    (Sec. III.C, Alg. 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
FRAME_H = FRAME_W = 84
FRAME_BYTES = FRAME_H * FRAME_W


@dataclass(frozen=True)
class NetShape:
    """Shape of a DQN Q-network: conv layers (out, kernel, stride), then
    FC hidden + ReLU, then a linear FC with one output per action."""
    name: str
    in_c: int
    in_h: int
    in_w: int
    conv: tuple  # ((out, k, stride), ...)
    fc_hidden: int
    n_actions: int

    def conv_dims(self):
        """[(cin, ih, iw, cout, k, s, oh, ow), ...] for valid-padding convs."""
        out = []
        c, h, w = self.in_c, self.in_h, self.in_w
        for (o, k, s) in self.conv:
            oh = (h - k) // s + 1
            ow = (w - k) // s + 1
            out.append((c, h, w, o, k, s, oh, ow))
            c, h, w = o, oh, ow
        return out

    def flat(self):
        c, h, w = self.in_c, self.in_h, self.in_w
        for (o, k, s) in self.conv:
            h = (h - k) // s + 1
            w = (w - k) // s + 1
            c = o
        return c * h * w

    def tensors(self):
        """[(name, shape, fan_in, fan_out), ...] in flat-parameter order:
        conv1.W, conv1.b, ..., fc1.W, fc1.b, fc2.W, fc2.b."""
        out = []
        for i, (cin, _, _, cout, k, _, _, _) in enumerate(self.conv_dims()):
            out.append((f"conv{i+1}.W", (cout, cin, k, k), cin * k * k, cout * k * k))
            out.append((f"conv{i+1}.b", (cout,), None, None))
        f = self.flat()
        out.append(("fc1.W", (self.fc_hidden, f), f, self.fc_hidden))
        out.append(("fc1.b", (self.fc_hidden,), None, None))
        out.append(("fc2.W", (self.n_actions, self.fc_hidden), self.fc_hidden, self.n_actions))
        out.append(("fc2.b", (self.n_actions,), None, None))
        return out

    def param_count(self):
        return int(sum(int(np.prod(s)) for _, s, _, _ in self.tensors()))

    def slices(self):
        """{name: (offset, shape)} for the flat parameter vector."""
        off = 0
        res = {}
        for name, shape, _, _ in self.tensors():
            n = int(np.prod(shape))
            res[name] = (off, shape)
            off += n
        return res


NET_S = NetShape("net_s", 4, 84, 84, ((16, 8, 4), (32, 4, 2)), 256, 6)
NET_L = NetShape("net_l", 4, 84, 84, ((32, 8, 4), (64, 4, 2), (64, 3, 1)), 512, 18)
NETS = {"net_s": NET_S, "net_l": NET_L}


def tiny_net(in_c=2, in_h=12, in_w=12, conv=((3, 4, 2),), fc_hidden=5, n_actions=3):
    return NetShape("tiny", in_c, in_h, in_w, tuple(conv), fc_hidden, n_actions)


def xavier_theta(net: NetShape, seed: int, bias_scale: float = 0.0) -> np.ndarray:
    """Flat float32 parameters: W ~ U(+-sqrt(6/(fan_in+fan_out))), biases zero
    (or U(+-bias_scale) when bias_scale > 0, used by small test cases)."""
    rng = np.random.default_rng(seed)
    parts = []
    for _, shape, fi, fo in net.tensors():
        n = int(np.prod(shape))
        if fi is None:
            if bias_scale > 0:
                parts.append(rng.uniform(-bias_scale, bias_scale, n))
            else:
                parts.append(np.zeros(n))
        else:
            lim = np.sqrt(6.0 / (fi + fo))
            parts.append(rng.uniform(-lim, lim, n))
    return np.concatenate(parts).astype(np.float32)


def random_states(batch: int, seed: int, c=4, h=84, w=84) -> np.ndarray:
    """uint8 [batch][c][h][w], i.i.d. uniform on 0..255."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=(batch, c, h, w), dtype=np.uint8)


def random_transitions(batch: int, n_actions: int, seed: int, p_terminal=0.01):
    """(a int32 [B], r float32 [B] in {-1,0,1}, term uint8 [B])."""
    rng = np.random.default_rng(seed)
    a = rng.integers(0, n_actions, size=batch).astype(np.int32)
    r = rng.integers(-1, 2, size=batch).astype(np.float32)
    t = (rng.random(batch) < p_terminal).astype(np.uint8)
    return a, r, t


def side_arrays(size: int, n_actions: int, seed: int, p_terminal=0.01):
    """Replay side arrays: action uint8 [N], reward int8 [N], terminal uint8 [N]."""
    rng = np.random.default_rng(seed ^ 0x5EED)
    a = rng.integers(0, n_actions, size=size).astype(np.uint8)
    r = rng.integers(-1, 2, size=size).astype(np.int8)
    t = (rng.random(size) < p_terminal).astype(np.uint8)
    return a, r, t


def side_arrays_hashed(size: int, n_actions: int, seed: int):
    """The hashed side arrays of the seeded stream (action uint8, reward int8,
    terminal uint8 [size]): the ones replay_fill_synthetic writes."""
    a = np.empty(size, np.uint8)
    r = np.empty(size, np.int8)
    t = np.empty(size, np.uint8)
    _lib().synth_side(seed, n_actions, 0, size, a.ctypes.data, r.ctypes.data, t.ctypes.data)
    return a, r, t


def index_stream(steps: int, batch: int, size: int, seed: int) -> np.ndarray:
    """int64 [steps][batch], uniform with replacement on [0, size-2]: valid
    transitions i need record i+1 for the next state."""
    rng = np.random.default_rng(seed ^ 0x1D5)
    return rng.integers(0, size - 1, size=(steps, batch), dtype=np.int64)


def game_draws(n_games: int, seed: int, step: int) -> np.ndarray:
    """uint64 [n_games][2] placement words for the games at one step (a new
    game's head and heading from word 0, an apple's cell from word 1); step
    -1 is the first reset."""
    rng = np.random.default_rng([seed, 0x5A4E, step + 1])
    return rng.integers(0, 2**64, size=(n_games, 2), dtype=np.uint64)


def actor_minibatch(batch: int, seed: int, step: int, n_games: int, capacity: int, moves: int) -> np.ndarray:
    """int64 [batch] record indices drawn uniformly with replacement over the
    valid experiences of a replay pooled over n_games games that each keep
    their last `capacity` states (include/dqn_actor.h), after `moves` moves
    of every game: experiences t = max(0, moves-capacity+1) .. moves-1 of game
    e sit at record e*(capacity+1) + t mod capacity."""
    count = min(moves, capacity - 1)
    if count <= 0:
        raise ValueError("no complete experience yet")
    rng = np.random.default_rng([seed, 0xAC70, step])
    k = rng.integers(0, n_games * count, size=batch)
    e, off = k // count, k % count
    t = moves - count + off
    return (e * (capacity + 1) + t % capacity).astype(np.int64)


def rgb_screens(n: int, seed: int, h: int = 176, w: int = 176) -> np.ndarray:
    """uint8 [n][h][w][3] raw color screens: a dark noisy background with 1-4
    solid colored rectangles each (stand-ins for a game's raw frames)."""
    rng = np.random.default_rng([seed, 0x26B])
    out = rng.integers(0, 24, size=(n, h, w, 3), dtype=np.uint8)
    for i in range(n):
        for _ in range(int(rng.integers(1, 5))):
            rh, rw = int(rng.integers(4, h // 3)), int(rng.integers(4, w // 3))
            y0, x0 = int(rng.integers(0, h - rh)), int(rng.integers(0, w - rw))
            out[i, y0:y0 + rh, x0:x0 + rw] = rng.integers(64, 256, size=3, dtype=np.uint8)
    return out


def egreedy_draws(batch: int, seed: int) -> np.ndarray:
    """uint64 [batch] exploration draws: high 32 bits decide exploration,
    low 32 bits pick the random action."""
    rng = np.random.default_rng(seed ^ 0xE95)
    return rng.integers(0, 2**64, size=batch, dtype=np.uint64)


def random_gradient(n: int, seed: int, scale=1e-2) -> np.ndarray:
    rng = np.random.default_rng(seed ^ 0x6AD)
    g = rng.standard_normal(n) * scale
    g[rng.random(n) < 0.01] = 0.0
    return g.astype(np.float32)


# ----------------------------------------------------------------------------
# frames (C, OpenMP)

_LIB = None


def frames_lib_path():
    return os.path.join(HERE, "libframes.so")


def build_frames_lib():
    src = os.path.join(HERE, "frames.c")
    out = frames_lib_path()
    tmp = out + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", src, "-o", tmp])
    os.replace(tmp, out)
    return out


def _lib():
    global _LIB
    if _LIB is None:
        path = frames_lib_path()
        if not os.path.exists(path):
            build_frames_lib()
        lib = ctypes.CDLL(path)
        lib.synth_frames.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.synth_frames.restype = None
        lib.synth_side.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64, ctypes.c_int64,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.synth_side.restype = None
        lib.synth_hash.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64]
        lib.synth_hash.restype = ctypes.c_uint64
        _LIB = lib
    return _LIB


def synth_hash(seed: int, stream: int, i: int) -> int:
    return int(_lib().synth_hash(seed, stream, i))


def frames(seed: int, t0: int, count: int, out: np.ndarray | None = None) -> np.ndarray:
    """uint8 [count][84][84]: frames t0 .. t0+count-1 of the seeded stream."""
    if out is None:
        out = np.empty((count, FRAME_H, FRAME_W), dtype=np.uint8)
    assert out.dtype == np.uint8 and out.flags.c_contiguous and out.size == count * FRAME_BYTES
    _lib().synth_frames(seed, t0, count, out.ctypes.data)
    return out


def stacked_records(frame_stream: np.ndarray, first: int, count: int, c: int = 4) -> np.ndarray:
    """Records first..first+count-1 as a copy [count][c][84][84]; record i
    stacks frames i..i+c-1, oldest first."""
    out = np.empty((count, c, FRAME_H, FRAME_W), dtype=np.uint8)
    for k in range(c):
        out[:, k] = frame_stream[first + k: first + k + count]
    return out


@dataclass
class HostReplay:
    """Replay memory on the host.  ``frames`` holds the frame stream; record i
    is the 4-frame stack starting at frame i, so records overlap in memory
    (record stride = one frame) while holding the same bytes a stacked
    replay would."""
    frames: np.ndarray      # uint8 [size + 3][84][84]
    action: np.ndarray      # uint8 [size]
    reward: np.ndarray      # int8 [size]
    terminal: np.ndarray    # uint8 [size]
    size: int
    c: int = 4

    @property
    def record_stride(self):
        return self.frames.shape[1] * self.frames.shape[2]

    def record(self, i):
        return self.frames[i:i + self.c]


def host_replay(size: int, n_actions: int, seed: int, c: int = 4) -> HostReplay:
    fr = frames(seed, 0, size + c - 1)
    a, r, t = side_arrays_hashed(size, n_actions, seed)
    return HostReplay(fr, a, r, t, size, c)


def device_replay(size: int, n_actions: int, seed: int, device="cuda", c: int = 4,
                  chunk_records: int = 65536, host: HostReplay | None = None):
    """Replay memory in device memory as uint8 [size][c][84][84] stacked
    records (28,224 bytes each), plus side arrays.  Frames are generated on
    the host in chunks and expanded to stacked records on the device.
    Returns (records, action, reward, terminal) torch tensors."""
    import torch
    rec = torch.empty((size, c, FRAME_H, FRAME_W), dtype=torch.uint8, device=device)
    pinned = torch.empty((chunk_records + c - 1, FRAME_H, FRAME_W), dtype=torch.uint8).pin_memory()
    dev_frames = torch.empty((chunk_records + c - 1, FRAME_H, FRAME_W), dtype=torch.uint8, device=device)
    for first in range(0, size, chunk_records):
        n = min(chunk_records, size - first)
        if host is not None:
            pinned[: n + c - 1].numpy()[:] = host.frames[first: first + n + c - 1]
        else:
            frames(seed, first, n + c - 1, pinned[: n + c - 1].numpy())
        dev_frames[: n + c - 1].copy_(pinned[: n + c - 1], non_blocking=False)
        for k in range(c):
            rec[first: first + n, k].copy_(dev_frames[k: k + n])
    if host is not None:
        a, r, t = host.action, host.reward, host.terminal
    else:
        a, r, t = side_arrays_hashed(size, n_actions, seed)
    torch.cuda.synchronize()
    return (rec, torch.from_numpy(a).to(device), torch.from_numpy(r).to(device),
            torch.from_numpy(t).to(device))


def transitions_at(seed: int, idx, n_actions: int, size: int, c: int = 4):
    """The transitions idx of the seeded replay of `size` records (the same
    bytes device_replay(size, n_actions, seed) holds), regenerated from the
    frame stream without materializing the whole replay.
    Returns (s, s_next uint8 [B][c][84][84], a int32, r float32, term uint8)."""
    idx = np.asarray(idx, dtype=np.int64)
    B = idx.shape[0]
    s = np.empty((B, c, FRAME_H, FRAME_W), np.uint8)
    sn = np.empty_like(s)
    buf = np.empty((c + 1, FRAME_H, FRAME_W), np.uint8)
    for j, i in enumerate(idx):
        frames(seed, int(i), c + 1, buf)
        s[j] = buf[:c]
        sn[j] = buf[1:]
    a, r, t = side_arrays_hashed(size, n_actions, seed)
    return s, sn, a[idx].astype(np.int32), r[idx].astype(np.float32), t[idx].astype(np.uint8)
