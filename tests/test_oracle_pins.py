"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test would fail on a plausible mistake in the oracle: a dropped term
(bias, 1/2, 1/b, gamma), a wrong sign, a transposed weight, a wrong stride
or flatten order, a mask taken on the wrong tensor, the target computed
from the wrong network, or an optimizer reading the old state.
"""
import os

import numpy as np
import pytest

import dqn_inputs as di
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#")[0].strip()
        if not line:
            continue
        k, *v = line.split()
        vals.setdefault(k, []).append(v)
    return vals


# ---------------------------------------------------------------------------
# An independent forward pass: im2col with numpy's sliding windows and a
# matrix product, in float64.

def np_forward(net, theta, states):
    th = np.asarray(theta, np.float64)
    sl = net.slices()
    x = states.astype(np.float64) / 255.0                      # [B][C][H][W]
    for i, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(net.conv_dims()):
        o, shp = sl[f"conv{i+1}.W"]
        Wt = th[o:o + np.prod(shp)].reshape(shp)
        ob, bs = sl[f"conv{i+1}.b"]
        b = th[ob:ob + bs[0]]
        win = np.lib.stride_tricks.sliding_window_view(x, (k, k), axis=(2, 3))  # B C H' W' k k
        win = win[:, :, ::s, ::s][:, :, :oh, :ow]                               # B C oh ow k k
        cols = win.transpose(0, 2, 3, 1, 4, 5).reshape(x.shape[0], oh * ow, cin * k * k)
        z = cols @ Wt.reshape(cout, -1).T + b                                  # B P O
        x = np.maximum(z, 0).transpose(0, 2, 1).reshape(x.shape[0], cout, oh, ow)
    flat = x.reshape(x.shape[0], -1)
    o, shp = sl["fc1.W"]; W1 = th[o:o + np.prod(shp)].reshape(shp)
    o, shp = sl["fc1.b"]; b1 = th[o:o + shp[0]]
    o, shp = sl["fc2.W"]; W2 = th[o:o + np.prod(shp)].reshape(shp)
    o, shp = sl["fc2.b"]; b2 = th[o:o + shp[0]]
    h = np.maximum(flat @ W1.T + b1, 0)
    return h @ W2.T + b2


TINY_NETS = [
    di.tiny_net(2, 12, 12, ((3, 4, 2),), 5, 3),
    di.tiny_net(3, 14, 14, ((4, 4, 2), (3, 3, 1)), 6, 4),
    di.tiny_net(2, 20, 20, ((3, 8, 4), (4, 2, 1), (2, 2, 1)), 4, 5),
]


@pytest.mark.parametrize("net", TINY_NETS + [di.NET_S], ids=lambda n: str(n.conv))
def test_forward_matches_im2col_matmul(net):
    th = di.xavier_theta(net, 11, bias_scale=0.1)
    st = di.random_states(3, 12, net.in_c, net.in_h, net.in_w)
    q = oracle.forward_q(net, th, st)
    ref = np_forward(net, th, st)
    assert np.allclose(q, ref, rtol=1e-12, atol=1e-13)


def test_forward_net_l_matches_im2col():
    net = di.NET_L
    th = di.xavier_theta(net, 5, bias_scale=0.05)
    st = di.random_states(2, 6)
    assert np.allclose(oracle.forward_q(net, th, st), np_forward(net, th, st), rtol=1e-12, atol=1e-13)


def test_delta_filter_reproduces_strided_input():
    # conv 1@2x2 stride 2 with W = delta at (0,0): output = input[::2, ::2]/255;
    # identity FC layers pass it through to Q.
    net = di.tiny_net(1, 8, 8, ((1, 2, 2),), 16, 16)
    th = np.zeros(net.param_count(), np.float32)
    sl = net.slices()
    th[sl["conv1.W"][0]] = 1.0
    o, _ = sl["fc1.W"]; th[o:o + 256] = np.eye(16, dtype=np.float32).ravel()
    o, _ = sl["fc2.W"]; th[o:o + 256] = np.eye(16, dtype=np.float32).ravel()
    st = di.random_states(2, 3, 1, 8, 8)
    q = oracle.forward_q(net, th, st)
    assert np.array_equal(q, st[:, 0, ::2, ::2].reshape(2, 16).astype(np.float64) / 255.0)


def test_flatten_is_channel_major():
    # one fc1 unit reads exactly flat index c*OH*OW + y*OW + x of the last conv
    net = di.tiny_net(2, 6, 6, ((2, 2, 2),), 1, 1)      # conv out 2x3x3, flat 18
    th = np.zeros(net.param_count(), np.float32)
    sl = net.slices()
    w, _ = sl["conv1.W"]
    th[w + (1 * 2 + 0) * 4 + 0] = 1.0                   # out ch 1 <- in ch 0 tap (0,0)
    f, _ = sl["fc1.W"]
    th[f + 1 * 9 + 2 * 3 + 1] = 1.0                     # (c=1, y=2, x=1)
    th[sl["fc2.W"][0]] = 1.0
    st = di.random_states(1, 4, 2, 6, 6)
    q = oracle.forward_q(net, th, st)
    assert q[0, 0] == st[0, 0, 4, 2] / 255.0


# ---------------------------------------------------------------------------
# Backward: central finite differences of the oracle's own loss.

@pytest.mark.parametrize("net", TINY_NETS, ids=lambda n: str(n.conv))
def test_gradient_matches_finite_differences(net):
    rng = np.random.default_rng(3)
    th = di.xavier_theta(net, 21, bias_scale=0.2).astype(np.float64)
    tgt = th + rng.normal(0, 0.05, th.shape)           # a distinct held network
    B = 3
    s = di.random_states(B, 22, net.in_c, net.in_h, net.in_w)
    sn = di.random_states(B, 23, net.in_c, net.in_h, net.in_w)
    a = np.array([0, net.n_actions - 1, 1], np.int32)
    r = np.array([1.0, -1.0, 0.0], np.float32)
    t = np.array([0, 1, 0], np.uint8)
    gamma = 0.9
    g = oracle.td_gradient(net, th, tgt, s, sn, a, r, t, gamma)["grad"]
    h = 1e-6
    fd = np.empty_like(th)
    for i in range(th.size):
        tp = th.copy(); tp[i] += h
        tm = th.copy(); tm[i] -= h
        lp = oracle.td_gradient(net, tp, tgt, s, sn, a, r, t, gamma)["loss"]
        lm = oracle.td_gradient(net, tm, tgt, s, sn, a, r, t, gamma)["loss"]
        fd[i] = (lp - lm) / (2 * h)
    err = np.linalg.norm(g - fd) / np.linalg.norm(fd)
    assert err < 1e-6, err
    assert np.abs(g - fd).max() < 1e-7


def test_gradient_ignores_target_path_when_target_is_theta():
    # y is a constant even when theta-hat == theta: the gradient is the one of
    # a fixed-target regression, so it equals the gradient with a frozen copy.
    net = TINY_NETS[0]
    th = di.xavier_theta(net, 2, bias_scale=0.1).astype(np.float64)
    s = di.random_states(4, 1, 2, 12, 12); sn = di.random_states(4, 2, 2, 12, 12)
    a, r, t = di.random_transitions(4, 3, 3)
    g_same = oracle.td_gradient(net, th, None, s, sn, a, r, t, 0.99)["grad"]
    g_copy = oracle.td_gradient(net, th, th.copy(), s, sn, a, r, t, 0.99)["grad"]
    assert np.array_equal(g_same, g_copy)
    # and it is NOT the total derivative through y (finite differences that
    # move theta-hat together with theta give a different number)
    i = net.slices()["fc2.b"][0]
    h = 1e-6
    tp = th.copy(); tp[i] += h
    tm = th.copy(); tm[i] -= h
    lp = oracle.td_gradient(net, tp, tp, s, sn, a, r, t, 0.99)["loss"]
    lm = oracle.td_gradient(net, tm, tm, s, sn, a, r, t, 0.99)["loss"]
    assert abs((lp - lm) / (2 * h) - g_same[i]) > 1e-4


# ---------------------------------------------------------------------------
# TD targets and loss: hand-worked example (golden file).

def _bias_only_net():
    return di.tiny_net(1, 4, 4, ((1, 2, 2),), 2, 3)


def test_td_targets_hand_worked():
    gd = _read_golden("td_targets_hand.txt")
    net = _bias_only_net()
    sl = net.slices()
    th = np.zeros(net.param_count()); tg = np.zeros(net.param_count())
    o, _ = sl["fc2.b"]
    th[o:o + 3] = [float(v) for v in gd["bq"][0]]
    tg[o:o + 3] = [float(v) for v in gd["bt"][0]]
    a = np.array(gd["action"][0], np.int32)
    r = np.array(gd["reward"][0], np.float32)
    t = np.array(gd["terminal"][0], np.uint8)
    s = di.random_states(4, 1, 1, 4, 4); sn = di.random_states(4, 2, 1, 4, 4)
    out = oracle.td_gradient(net, th, tg, s, sn, a, r, t, float(gd["gamma"][0][0]))
    assert np.array_equal(out["y"], np.array(gd["y"][0], float))
    assert out["loss"] == float(gd["loss"][0][0])
    assert np.array_equal(out["grad"][o:o + 3], np.array(gd["grad_bq"][0], float))
    # every weight is zero, so nothing else receives gradient except fc2.W,
    # whose input h1 = ReLU(b1) = 0 here
    rest = np.delete(out["grad"], np.arange(o, o + 3))
    assert np.all(rest == 0)


def test_gamma_zero_and_all_terminal_give_reward_targets():
    net = TINY_NETS[1]
    th = di.xavier_theta(net, 7, bias_scale=0.3)
    s = di.random_states(5, 1, 3, 14, 14); sn = di.random_states(5, 2, 3, 14, 14)
    a, r, _ = di.random_transitions(5, 4, 3)
    y0 = oracle.td_gradient(net, th, None, s, sn, a, r, np.zeros(5, np.uint8), 0.0)["y"]
    y1 = oracle.td_gradient(net, th, None, s, sn, a, r, np.ones(5, np.uint8), 0.99)["y"]
    assert np.array_equal(y0, r.astype(float)) and np.array_equal(y1, r.astype(float))
    # non-terminal target uses the max over the target network's outputs
    out = oracle.td_gradient(net, th, None, s, sn, a, r, np.zeros(5, np.uint8), 0.99)
    qn = oracle.forward_q(net, th, sn)
    assert np.allclose(out["y"], r + 0.99 * qn.max(axis=1), rtol=0, atol=1e-14)
    assert np.allclose(out["qn"], qn, rtol=0, atol=1e-15)


def test_zero_gradient_when_q_equals_target():
    # all transitions terminal and Q(s, a_j) = r_j: every residual is 0
    net = TINY_NETS[0]
    sl = net.slices()
    th = di.xavier_theta(net, 3).astype(np.float64)
    o, shp = sl["fc2.W"]; th[o:o + np.prod(shp)] = 0.0
    o, _ = sl["fc2.b"]; th[o:o + 3] = 0.5
    s = di.random_states(6, 1, 2, 12, 12); sn = di.random_states(6, 2, 2, 12, 12)
    a = np.array([0, 1, 2, 2, 1, 0], np.int32)
    r = np.full(6, 0.5, np.float32)
    out = oracle.td_gradient(net, th, None, s, sn, a, r, np.ones(6, np.uint8), 0.99)
    assert out["loss"] == 0.0 and np.all(out["grad"] == 0.0)
    th2, _ = oracle.apply_update("sgd", th.astype(np.float32), None, out["grad"], 0.1)
    assert np.array_equal(th2, th.astype(np.float32))


def test_relu_derivative_at_zero_is_zero():
    # fc1 pre-activations are exactly 0 (W1 = 0, b1 = 0): no gradient reaches
    # fc1 or the convs even though W2 != 0.
    net = TINY_NETS[0]
    sl = net.slices()
    th = di.xavier_theta(net, 4).astype(np.float64)
    o, shp = sl["fc1.W"]; th[o:o + np.prod(shp)] = 0.0
    s = di.random_states(3, 1, 2, 12, 12); sn = di.random_states(3, 2, 2, 12, 12)
    a, r, t = di.random_transitions(3, 3, 5)
    g = oracle.td_gradient(net, th, None, s, sn, a, r, t, 0.9)["grad"]
    o_fc2 = sl["fc2.W"][0]
    assert np.all(g[:o_fc2] == 0.0)
    assert np.any(g[sl["fc2.b"][0]:] != 0.0)


def test_batch_gradient_is_mean_of_sample_gradients_and_order_free():
    net = TINY_NETS[1]
    th = di.xavier_theta(net, 9, bias_scale=0.1)
    B = 6
    s = di.random_states(B, 1, 3, 14, 14); sn = di.random_states(B, 2, 3, 14, 14)
    a, r, t = di.random_transitions(B, 4, 3, p_terminal=0.3)
    full = oracle.td_gradient(net, th, None, s, sn, a, r, t, 0.99)
    singles = [oracle.td_gradient(net, th, None, s[j:j+1], sn[j:j+1], a[j:j+1], r[j:j+1],
                                  t[j:j+1], 0.99) for j in range(B)]
    mean_g = sum(o["grad"] for o in singles) / B
    assert np.allclose(full["grad"], mean_g, rtol=1e-12, atol=1e-16)
    assert np.isclose(full["loss"], sum(o["loss"] for o in singles) / B, rtol=1e-13)
    p = np.random.default_rng(0).permutation(B)
    perm = oracle.td_gradient(net, th, None, s[p], sn[p], a[p], r[p], t[p], 0.99)
    assert np.allclose(full["grad"], perm["grad"], rtol=1e-12, atol=1e-16)


# ---------------------------------------------------------------------------
# Optimizers: closed forms for a constant gradient.

def test_sgd_closed_form():
    th0 = np.array([1.0, -2.0, 0.5, 0.0], np.float32)
    g = np.array([0.5, -0.25, 0.0, 2.0])
    th, st = th0, None
    for _ in range(4):
        th, st = oracle.apply_update("sgd", th, st, g, 0.125)
    # all values exact in binary
    assert np.array_equal(th, (th0 - 4 * 0.125 * g).astype(np.float32))


def test_rmsprop_closed_form_and_zero_gradient():
    # Alg. 2: r_k = (1 - 0.9^k) g^2, step_k = lr * sign(g) / sqrt(1 - 0.9^k)
    g = np.array([0.3, -2.0, 1e-3, 0.0])
    th = np.array([0.0, 0.0, 0.0, 0.7], np.float32)
    st = np.zeros(4, np.float32)
    lr = 1e-2
    ref = np.zeros(4)
    for k in range(1, 6):
        prev = th.copy()
        th, st = oracle.apply_update("rmsprop", th, st, g, lr, 0.9)
        ref_r = (1 - 0.9 ** k) * g ** 2
        assert np.allclose(st, ref_r, rtol=3e-7, atol=0)
        step = np.where(g != 0, lr * np.sign(g) / np.sqrt(1 - 0.9 ** k), 0.0)
        ref = ref - step
        assert np.allclose(th[:3], ref[:3], rtol=1e-6, atol=1e-9)
        assert th[3] == np.float32(0.7) == prev[3]     # r stays 0: parameter unchanged


def test_adagrad_closed_form():
    g = np.array([0.3, -2.0, 1e-5, 0.0])
    th = np.zeros(4, np.float32)
    st = np.zeros(4, np.float32)
    lr, eps = 0.01, 1e-8
    ref = np.zeros(4)
    for k in range(1, 6):
        th, st = oracle.apply_update("adagrad", th, st, g, lr, 0.0, eps)
        assert np.allclose(st, k * g ** 2, rtol=3e-7, atol=0)
        ref = ref - lr * g / (np.sqrt(k) * np.abs(g) + eps)
        assert np.allclose(th, ref, rtol=1e-6, atol=1e-12)


# ---------------------------------------------------------------------------
# Greedy / epsilon-greedy action choice.

def test_argmax_ties_take_lowest_index():
    q = np.array([[1.0, 3.0, 3.0, 2.0], [0.0, 0.0, 0.0, 0.0], [-1.0, -2.0, -1.0, -5.0],
                  [0.0, 0.0, 0.0, 1e-300]])
    assert list(oracle.select_actions(q, 0.0)) == [1, 0, 0, 3]


def test_egreedy_threshold_golden():
    gd = _read_golden("egreedy_threshold.txt")
    eps = np.frombuffer(int(gd["epsilon_f32_hex"][0][0], 16).to_bytes(4, "little"), np.float32)[0]
    assert eps == np.float32(0.05)
    for row in gd["draw"]:
        w = int(row[0], 16); A = int(row[2]); explore = int(row[4]); act = int(row[6])
        q = np.zeros((1, A)); q[0, 1] = 1.0      # greedy action is 1
        got = oracle.select_actions(q, float(eps), np.array([w], np.uint64))[0]
        assert got == (act if explore else 1)


def test_egreedy_extremes():
    rng = np.random.default_rng(1)
    q = rng.normal(size=(500, 6))
    draws = di.egreedy_draws(500, 2)
    assert np.array_equal(oracle.select_actions(q, 0.0, draws), q.argmax(axis=1))
    all_rand = oracle.select_actions(q, 1.0, draws)
    assert np.array_equal(all_rand, ((draws & np.uint64(0xffffffff)) * np.uint64(6)) >> np.uint64(32))
    # exploration rate close to epsilon
    frac = np.mean((draws >> np.uint64(32)) < np.uint64(214748368))
    assert 0.02 < frac < 0.09


# ---------------------------------------------------------------------------
# Replay gather: brute force against the frame stream.

def test_gather_brute_force_and_bounds():
    size = 300
    rep = di.host_replay(size, 6, seed=5)
    idx = np.array([0, 1, 99, 100, 101, size - 2, 7, 7], np.int64)
    s, sn, a, r, t = oracle.gather_from_host_replay(rep, idx)
    for j, i in enumerate(idx):
        assert np.array_equal(s[j].reshape(4, 84, 84), di.frames(5, i, 4))
        assert np.array_equal(sn[j].reshape(4, 84, 84), di.frames(5, i + 1, 4))
        assert a[j] == rep.action[i] and r[j] == rep.reward[i] and t[j] == rep.terminal[i]
    with pytest.raises(RuntimeError):
        oracle.gather_from_host_replay(rep, np.array([size - 1]))
    with pytest.raises(RuntimeError):
        oracle.gather_from_host_replay(rep, np.array([-1]))


# ---------------------------------------------------------------------------
# Multi-step schedules reduce to each other in their special cases.

def _small_replay_setup(net, size=64, steps=4, B=3):
    rep_frames = di.frames(8, 0, size + 3)
    a, r, t = di.side_arrays(size, net.n_actions, 8, p_terminal=0.2)
    # shrink frames to the tiny net's input by cropping the top-left corner
    crop = np.ascontiguousarray(rep_frames[:, :net.in_h, :net.in_w])
    rep = di.HostReplay(crop, a, r, t, size, c=net.in_c)
    idx = di.index_stream(steps, B, size, 9)
    return rep, idx


def _crop_gather(rep, idx):
    rec_bytes = rep.c * rep.frames.shape[1] * rep.frames.shape[2]
    return oracle.replay_gather(rep.frames, rep.frames.shape[1] * rep.frames.shape[2], rec_bytes,
                                rep.size, rep.action, rep.reward, rep.terminal, idx)


def test_zero_staleness_replicas_equal_sequential_adagrad():
    net = di.tiny_net(4, 12, 12, ((3, 4, 2),), 5, 3)
    rep, idx = _small_replay_setup(net)
    th0 = di.xavier_theta(net, 1, bias_scale=0.1)
    a1, s1, l1 = oracle.sequential_training(net, th0, rep, idx, 0.99, 0.01, rule="adagrad", eps=1e-8)
    a2, s2, l2 = oracle.stale_replica_training(net, th0, rep, idx, 0.99, 0.01, staleness=0,
                                               rule="adagrad", eps=1e-8)
    assert np.array_equal(a1, a2) and np.array_equal(s1, s2) and np.array_equal(l1, l2)


def test_stale_schedule_uses_old_versions():
    net = di.tiny_net(4, 12, 12, ((3, 4, 2),), 5, 3)
    rep, idx = _small_replay_setup(net, steps=5)
    th0 = di.xavier_theta(net, 1, bias_scale=0.1)
    S = 2
    got, _, losses = oracle.stale_replica_training(net, th0, rep, idx, 0.99, 0.01, staleness=S,
                                                   rule="adagrad", eps=1e-8)
    # manual replay of the schedule
    vers = [th0.copy()]
    G = np.zeros_like(th0)
    ml = []
    for u in range(5):
        v = vers[max(0, u - S)]
        s, sn, a, r, t = _crop_gather(rep, idx[u])
        out = oracle.td_gradient(net, v, v, s, sn, a, r, t, 0.99)
        ml.append(out["loss"])
        new, G = oracle.apply_update("adagrad", vers[-1], G, out["grad"], 0.01, 0.0, 1e-8)
        vers.append(new)
    assert np.array_equal(got, vers[-1]) and np.array_equal(losses, np.array(ml))
    # losses of updates 1 and 2 were computed on version 0 (same as update 0's)
    assert not np.array_equal(got, oracle.sequential_training(
        net, th0, rep, idx, 0.99, 0.01, rule="adagrad", eps=1e-8)[0])


def test_target_refresh_schedule():
    net = di.tiny_net(4, 12, 12, ((3, 4, 2),), 5, 3)
    rep, idx = _small_replay_setup(net, steps=5)
    th0 = di.xavier_theta(net, 2, bias_scale=0.1)
    # period 1 is the same as always using the current parameters
    a1, _, l1 = oracle.sequential_training(net, th0, rep, idx, 0.99, 0.05, target_period=1)
    a2, _, l2 = oracle.sequential_training(net, th0, rep, idx, 0.99, 0.05, target_period=None)
    assert np.array_equal(a1, a2) and np.array_equal(l1, l2)
    # period 2: steps 0,1 use theta_0 as target, steps 2,3 use theta_2, step 4 theta_4
    got, _, _ = oracle.sequential_training(net, th0, rep, idx, 0.99, 0.05, target_period=2)
    th = th0.copy(); tgt = None
    for n in range(5):
        if n % 2 == 0:
            tgt = th.copy()
        s, sn, a, r, t = _crop_gather(rep, idx[n])
        g = oracle.td_gradient(net, th, tgt, s, sn, a, r, t, 0.99)["grad"]
        th, _ = oracle.apply_update("sgd", th, None, g, 0.05)
    assert np.array_equal(got, th)


# ---------------------------------------------------------------------------
# Parameter layout and input generator.

@pytest.mark.parametrize("net", [di.NET_S, di.NET_L] + TINY_NETS, ids=lambda n: n.name + str(n.conv))
def test_param_layout_agrees_with_generator(net):
    sl = net.slices()
    assert oracle.param_count(net) == net.param_count()
    for l in range(len(net.conv)):
        assert oracle.param_offset(net, l, False) == sl[f"conv{l+1}.W"][0]
        assert oracle.param_offset(net, l, True) == sl[f"conv{l+1}.b"][0]
    L = len(net.conv)
    assert oracle.param_offset(net, L, False) == sl["fc1.W"][0]
    assert oracle.param_offset(net, L + 1, True) == sl["fc2.b"][0]


def test_paper_net_sizes():
    assert di.NET_S.param_count() == 677686 and di.NET_S.flat() == 2592
    assert di.NET_L.param_count() == 1693362 and di.NET_L.flat() == 3136


def test_frames_are_pure_function_of_index():
    whole = di.frames(3, 0, 250)
    assert np.array_equal(whole[120:140], di.frames(3, 120, 20))
    assert not np.array_equal(whole[:10], di.frames(4, 0, 10))
    assert whole.max() >= 192 and np.median(whole) <= 8
    # rectangles move within a segment and are redrawn at segment boundaries
    assert not np.array_equal(whole[10], whole[11])


# ---------------------------------------------------------------------------
# Normalized ReLU margins (used to tell unique gradients from ones that the
# working precision does not decide).

def np_margins(net, theta, states):
    th = np.asarray(theta, np.float64)
    sl = net.slices()
    B = states.shape[0]
    x = states.astype(np.float64) / 255.0
    m = np.full(B, np.inf)
    for i, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(net.conv_dims()):
        o, shp = sl[f"conv{i+1}.W"]
        Wt = th[o:o + np.prod(shp)].reshape(cout, -1)
        ob, bs = sl[f"conv{i+1}.b"]
        b = th[ob:ob + bs[0]]
        win = np.lib.stride_tricks.sliding_window_view(x, (k, k), axis=(2, 3))[:, :, ::s, ::s][:, :, :oh, :ow]
        cols = win.transpose(0, 2, 3, 1, 4, 5).reshape(B, oh * ow, -1)
        z = cols @ Wt.T + b
        den = np.abs(cols) @ np.abs(Wt).T + np.abs(b)
        m = np.minimum(m, (np.abs(z) / den).reshape(B, -1).min(axis=1))
        x = np.maximum(z, 0).transpose(0, 2, 1).reshape(B, cout, oh, ow)
    flat = x.reshape(B, -1)
    o, shp = sl["fc1.W"]; W1 = th[o:o + np.prod(shp)].reshape(shp)
    o, shp = sl["fc1.b"]; b1 = th[o:o + shp[0]]
    z = flat @ W1.T + b1
    den = np.abs(flat) @ np.abs(W1).T + np.abs(b1)
    return np.minimum(m, (np.abs(z) / den).min(axis=1))


@pytest.mark.parametrize("net", TINY_NETS, ids=lambda n: str(n.conv))
def test_relu_margins_match_independent_formulation(net):
    th = di.xavier_theta(net, 31, bias_scale=0.1)
    st = di.random_states(5, 32, net.in_c, net.in_h, net.in_w)
    assert np.allclose(oracle.relu_margins(net, th, st), np_margins(net, th, st), rtol=1e-10, atol=0)


def test_relu_margin_hand_worked():
    # conv 1@1x1/1 with weight 1 and bias -x0 puts pixel 0 exactly on the
    # kink (margin 0); the other pixels have margin |x - x0| / (|x| + x0).
    net = di.tiny_net(1, 2, 2, ((1, 1, 1),), 1, 1)
    st = np.array([[[[51, 102], [153, 255]]]], np.uint8)
    x0 = 51 / 255.0
    th = np.zeros(net.param_count())
    sl = net.slices()
    th[sl["conv1.W"][0]] = 1.0
    th[sl["conv1.b"][0]] = -x0
    th[sl["fc1.b"][0]] = 1.0           # fc1 unit: z = 1, margin 1
    assert oracle.relu_margins(net, th, st)[0] == 0.0
    th[sl["conv1.b"][0]] = -0.5 * x0   # now the smallest is pixel 0: (x0/2) / (1.5 x0) = 1/3
    assert np.isclose(oracle.relu_margins(net, th, st)[0], 1.0 / 3.0, rtol=1e-15)


def test_transitions_at_regenerates_replay_records():
    hr = di.host_replay(500, 18, 9)
    idx = np.array([0, 7, 250, 497])
    s, sn, a, r, t = di.transitions_at(9, idx, 18, 500)
    rs, rsn, ra, rr, rt = oracle.gather_from_host_replay(hr, idx)
    assert np.array_equal(s.reshape(4, -1), rs) and np.array_equal(sn.reshape(4, -1), rsn)
    assert np.array_equal(a, ra) and np.array_equal(r, rr) and np.array_equal(t, rt)
