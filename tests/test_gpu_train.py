"""GPU parity of the worker / parameter-server loops (include/dqn_train.h)
against the oracle's drivers over whole trajectories: sequential training
with and without target-network refresh (Alg. 1's n >= l*C test) under each
update rule, and the bounded-staleness replica schedule (Sec. IV.A, Alg. 2)
with AdaGrad.  Compared per step: the loss; at the end: the total parameter
change per tensor and the optimizer state."""
import numpy as np
import pytest

import dqn_inputs as di
import oracle
import paper_1508_04186_amd as dq
from gpu_util import FP32_TOL, assert_grad_close, dev_tensor, host, rel_l2, say

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module")
def small_replay(dev):
    size = 3000
    say(f"[setup] host replay size={size} seed=41 -> device")
    hr = di.host_replay(size, 6, seed=41)
    rec, a, r, t = di.device_replay(size, 6, seed=41, host=hr)
    return hr, dq.Replay(rec, a, r, t, size)


def _check_trajectory(shape, th0, th_gpu, th_ref, losses_gpu, losses_ref, st_gpu=None, st_ref=None):
    assert np.allclose(losses_gpu, losses_ref, rtol=FP32_TOL, atol=0), (losses_gpu, losses_ref)
    d_gpu = th_gpu.astype(np.float64) - th0
    d_ref = th_ref.astype(np.float64) - th0
    assert_grad_close(shape, d_gpu, d_ref, what="parameter change")
    if st_gpu is not None:
        assert_grad_close(shape, st_gpu, st_ref, what="optimizer state")


@pytest.mark.parametrize("rule,lr,period", [("sgd", 1e-2, 0), ("sgd", 1e-2, 4), ("rmsprop", 1e-3, 3),
                                            ("adagrad", 1e-3, 0)])
def test_train_steps_trajectory(dev, small_replay, rule, lr, period):
    import torch
    hr, rp = small_replay
    net, shape = dq.NET_SMALL, di.NET_S
    N, B = 10, 32
    idx = di.index_stream(N, B, hr.size, 42)
    th0 = di.xavier_theta(shape, 43)
    theta = dev_tensor(th0)
    tgt = torch.empty_like(theta) if period else None
    state = None if rule == "sgd" else torch.zeros_like(theta)
    losses = torch.empty(N, dtype=torch.float32, device=dev)
    decay, eps = (0.9, 0.0) if rule != "adagrad" else (0.0, 1e-8)
    say(f"[train] rule={rule} lr={lr} period={period}: GPU {N} steps")
    dq.dqn_train_steps(net, theta, tgt, state, rule, lr, decay, eps, 0.99, rp, dev_tensor(idx),
                       target_period=period, losses_out=losses)
    torch.cuda.synchronize()
    say(f"[train] rule={rule}: oracle")
    th_ref, st_ref, l_ref = oracle.sequential_training(
        shape, th0, hr, idx, float(F32(0.99)), float(F32(lr)), rule=rule, decay=float(F32(decay)),
        eps=float(F32(eps)), target_period=period or None)
    _check_trajectory(shape, th0, host(theta), th_ref, host(losses), l_ref,
                      None if state is None else host(state), st_ref)


def test_train_steps_resumes_across_calls(dev, small_replay):
    """Two calls (steps 0-5 then 6-11, step0 = 6) equal one call of 12 steps,
    bit for bit, including the target refresh at step 8."""
    import torch
    hr, rp = small_replay
    net, shape = dq.NET_SMALL, di.NET_S
    idx = dev_tensor(di.index_stream(12, 32, hr.size, 44))
    th0 = dev_tensor(di.xavier_theta(shape, 45))
    a, ta = th0.clone(), torch.empty_like(th0)
    b, tb = th0.clone(), torch.empty_like(th0)
    say("[train] resume: one call of 12 vs 6 + 6")
    dq.dqn_train_steps(net, a, ta, None, "sgd", 1e-2, 0.9, 0.0, 0.99, rp, idx, target_period=4)
    dq.dqn_train_steps(net, b, tb, None, "sgd", 1e-2, 0.9, 0.0, 0.99, rp, idx[:6], target_period=4)
    dq.dqn_train_steps(net, b, tb, None, "sgd", 1e-2, 0.9, 0.0, 0.99, rp, idx[6:], step0=6,
                       target_period=4)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(ta, tb)


@pytest.mark.parametrize("B", [32, 300])
@pytest.mark.parametrize("rule,lr,decay,eps", [("sgd", 1e-2, 0.9, 0.0), ("rmsprop", 1e-3, 0.9, 0.0),
                                               ("adagrad", 1e-3, 0.0, 1e-8)])
def test_train_steps_fused_update_is_bitwise_two_calls(dev, small_replay, rule, lr, decay, eps, B):
    """The update fused into each step's last kernel equals, bit for bit,
    dqn_td_gradient_replay followed by ps_apply_update (target refresh
    every 3 steps, so both theta and theta^- paths run); batch 300 runs the
    reductions for batches above 128."""
    import torch
    _, rp = small_replay
    net = dq.NET_SMALL
    N, C = 7, 3
    idx = dev_tensor(di.index_stream(N, B, rp.size, 50))
    th0 = dev_tensor(di.xavier_theta(di.NET_S, 51))
    a, ta = th0.clone(), torch.empty_like(th0)
    b, tb = th0.clone(), torch.empty_like(th0)
    sa = None if rule == "sgd" else torch.full_like(th0, 0.01)
    sb = None if sa is None else sa.clone()
    la = torch.empty(N, dtype=torch.float32, device=dev)
    lb = torch.empty(N, dtype=torch.float32, device=dev)
    say(f"[train] fused vs two calls, rule={rule} batch={B}")
    dq.dqn_train_steps(net, a, ta, sa, rule, lr, decay, eps, 0.99, rp, idx, target_period=C,
                       losses_out=la)
    g = torch.empty_like(th0)
    for n in range(N):
        if n % C == 0:
            tb.copy_(b)
        dq.dqn_td_gradient_replay(net, b, tb, rp, idx[n], 0.99, g, lb[n:n + 1])
        dq.ps_apply_update(rule, b, b, sb, g, lr, decay, eps)
    torch.cuda.synchronize()
    assert torch.equal(la, lb)
    assert torch.equal(a, b) and torch.equal(ta, tb)
    if sa is not None:
        assert torch.equal(sa, sb)


def _replica_run(dev, rp, shape, net, th0, idx, R, S, lr=0.01, eps=1e-8):
    import torch
    P = dq.dqn_param_count(net)
    RS = dq.dqn_train_ring_stride(net)
    ring = torch.empty((S + 1) * RS, dtype=torch.float32, device=dev)
    ring[:P].copy_(dev_tensor(th0))
    G = torch.zeros(P, dtype=torch.float32, device=dev)
    U = idx.shape[0]
    losses = torch.empty(U, dtype=torch.float32, device=dev)
    with dq.HipStreams(R + 1) as hs:
        torch.cuda.synchronize()
        dq.dqn_train_replicas(net, ring, G, "adagrad", lr, 0.0, eps, 0.99, rp, idx, R, S, hs.handles,
                              losses_out=losses)
        torch.cuda.synchronize()
    slot = U % (S + 1)
    return host(ring[slot * RS:slot * RS + P]), host(G), host(losses)


def test_replicas_match_stale_schedule_oracle(dev, small_replay):
    hr, rp = small_replay
    net, shape = dq.NET_SMALL, di.NET_S
    U, B, R, S = 24, 32, 16, 4
    idx = di.index_stream(U, B, hr.size, 46)
    th0 = di.xavier_theta(shape, 47)
    say(f"[replicas] R={R} S={S} U={U}: GPU")
    th, G, losses = _replica_run(dev, rp, shape, net, th0, dev_tensor(idx), R, S)
    say("[replicas] oracle")
    th_ref, G_ref, l_ref = oracle.stale_replica_training(
        shape, th0, hr, idx, float(F32(0.99)), float(F32(0.01)), S, rule="adagrad",
        eps=float(F32(1e-8)))
    _check_trajectory(shape, th0, th, th_ref, losses, l_ref, G, G_ref)


def test_replicas_zero_staleness_is_sequential_and_deterministic(dev, small_replay):
    import torch
    hr, rp = small_replay
    net, shape = dq.NET_SMALL, di.NET_S
    U, B = 8, 32
    idx = dev_tensor(di.index_stream(U, B, hr.size, 48))
    th0 = di.xavier_theta(shape, 49)
    say("[replicas] R=1 S=0 vs train_steps adagrad")
    th_r, G_r, l_r = _replica_run(dev, rp, shape, net, th0, idx, 1, 0)
    theta = dev_tensor(th0)
    G = torch.zeros_like(theta)
    losses = torch.empty(U, dtype=torch.float32, device=dev)
    dq.dqn_train_steps(net, theta, None, G, "adagrad", 0.01, 0.0, 1e-8, 0.99, rp, idx,
                       losses_out=losses)
    torch.cuda.synchronize()
    assert np.array_equal(th_r, host(theta)) and np.array_equal(G_r, host(G))
    assert np.array_equal(l_r, host(losses))
    say("[replicas] R=16 S=4 twice: bitwise identical")
    a = _replica_run(dev, rp, shape, net, th0, idx, 16, 4)
    b = _replica_run(dev, rp, shape, net, th0, idx, 16, 4)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))


def test_train_argument_errors(dev, small_replay):
    import torch
    _, rp = small_replay
    net = dq.NET_SMALL
    P = dq.dqn_param_count(net)
    th = torch.zeros(P, dtype=torch.float32, device=dev)
    idx = torch.zeros((2, 4), dtype=torch.int64, device=dev)
    with pytest.raises(dq.DqnError):   # RMSProp without its state
        dq.dqn_train_steps(net, th, None, None, "rmsprop", 1e-3, 0.9, 0.0, 0.99, rp, idx)
    with pytest.raises(dq.DqnError):   # refresh without a target buffer
        dq.dqn_train_steps(net, th, None, None, "sgd", 1e-3, 0.9, 0.0, 0.99, rp, idx, target_period=2)
    ring = torch.zeros(3 * dq.dqn_train_ring_stride(net), dtype=torch.float32, device=dev)
    G = torch.zeros(P, dtype=torch.float32, device=dev)
    with dq.HipStreams(3) as hs:
        streams = hs.handles
        with pytest.raises(dq.DqnError):   # replicas must exceed staleness
            dq.dqn_train_replicas(net, ring, G, "adagrad", 1e-2, 0.0, 1e-8, 0.99, rp, idx, 2, 2, streams)
        with pytest.raises(dq.DqnError):   # streams must be distinct
            dq.dqn_train_replicas(net, ring, G, "adagrad", 1e-2, 0.0, 1e-8, 0.99, rp, idx, 2, 1,
                                  [streams[0], streams[0], streams[1]])
