"""GPU parity at the full workload sizes: the large Q-network at batch 256,
517 and 2,048 (TD gradient), the small one at batch 700 (its large-batch
launch shapes), and an 8,192-state epsilon-greedy forward pass whose Q values and
actions are compared with the oracle on a 1,024-state sample.

TD batches are drawn from transitions whose forward pass keeps every ReLU
pre-activation at least MARGIN_MIN (normalized) away from the kink, where
the gradient is unique; the transitions left out are checked separately
(their Q values, targets and loss are unique and must match)."""
import numpy as np
import pytest

import dqn_inputs as di
import oracle
import paper_1508_04186_amd as dq
from gpu_util import (FP32_TOL, assert_close, assert_grad_close, check_actions, dev_tensor, host, rel_l2, say,
                      split_by_margin)

pytestmark = pytest.mark.gpu
F32 = np.float32


def _run_td(dev, net, th, tt, s, sn, a, r, t, gamma):
    import torch
    B = s.shape[0]
    P = dq.dqn_param_count(net)
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    q = torch.empty((B, net.n_actions), dtype=torch.float32, device=dev)
    y = torch.empty(B, dtype=torch.float32, device=dev)
    th_d = dev_tensor(th)
    tt_d = th_d if tt is None else dev_tensor(tt)
    dq.dqn_td_gradient(net, th_d, tt_d, dev_tensor(s), dev_tensor(sn), dev_tensor(a), dev_tensor(r),
                       dev_tensor(t), gamma, g, loss, q, y)
    torch.cuda.synchronize()
    return host(g), float(host(loss)[0]), host(q), host(y)


# large 517: ragged weight-gradient slots (the float32 six-product kernels:
# conv2 slots of 5 samples, the last of 2; conv3 slots of 3, the last of 1)
@pytest.mark.parametrize("name,B,target", [("small", 700, "same"), ("small", 1024, "held"),
                                           ("large", 131, "held"), ("large", 256, "held"),
                                           ("large", 517, "held"), ("large", 2048, "same")])
def test_td_gradient_full_size(dev, name, B, target):
    net, shape = (dq.NET_SMALL, di.NET_S) if name == "small" else (dq.NET_LARGE, di.NET_L)
    size = 4 * B + 10
    say(f"[td-large] net={name} batch={B} target={target}: host replay {size}")
    hr = di.host_replay(size, shape.n_actions, seed=B)
    n_cand = B + B // 2
    idx = di.index_stream(1, n_cand, size, B + 1)[0]
    s, sn, a, r, t = oracle.gather_from_host_replay(hr, idx)
    s = s.reshape(n_cand, 4, 84, 84)
    sn = sn.reshape(n_cand, 4, 84, 84)
    a = a.astype(np.int32)
    th = di.xavier_theta(shape, 3 * B, bias_scale=0.02)
    tt = None if target == "same" else di.xavier_theta(shape, 3 * B + 1, bias_scale=0.02)
    say(f"[td-large] net={name} batch={B}: oracle margins of {n_cand} candidates")
    keep = np.nonzero(split_by_margin(shape, th, s))[0]
    assert keep.size >= B, f"only {keep.size} of {n_cand} candidates have a unique gradient"
    sel = keep[:B]
    s, sn, a, r, t = s[sel], sn[sel], a[sel], r[sel], t[sel]
    say(f"[td-large] net={name} batch={B}: GPU")
    g, loss, q, y = _run_td(dev, net, th, tt, s, sn, a, r, t, 0.99)
    say(f"[td-large] net={name} batch={B}: oracle")
    ref = oracle.td_gradient(shape, th, tt, s, sn, a, r, t, float(F32(0.99)))
    assert_close(q, ref["q"], FP32_TOL, "q")
    assert_close(y, ref["y"], FP32_TOL, "y")
    assert abs(loss - ref["loss"]) <= FP32_TOL * abs(ref["loss"])
    assert_grad_close(shape, g, ref["grad"])


def test_forward_8192_states_egreedy(dev):
    import torch
    net, shape = dq.NET_LARGE, di.NET_L
    B = 8192
    size = 20000
    say(f"[fwd-large] batch={B}: replay {size} -> device gather")
    hr = di.host_replay(size, shape.n_actions, seed=77)
    rec, ra, rr, rt = di.device_replay(size, shape.n_actions, seed=77, host=hr)
    rp = dq.Replay(rec, ra, rr, rt, size)
    idx = np.random.default_rng(78).integers(0, size, B).astype(np.int64)
    st = torch.empty((B, 4, 84, 84), dtype=torch.uint8, device=dev)
    dq.replay_gather(rp, dev_tensor(idx), st)
    th = di.xavier_theta(shape, 79, bias_scale=0.02)
    draws = di.egreedy_draws(B, 80)
    q = torch.empty((B, net.n_actions), dtype=torch.float32, device=dev)
    act = torch.empty(B, dtype=torch.int32, device=dev)
    say(f"[fwd-large] batch={B}: GPU forward eps=0.05")
    dq.dqn_forward(net, dev_tensor(th), st, float(F32(0.05)), dev_tensor(draws), q, act)
    torch.cuda.synchronize()
    sample = np.sort(np.random.default_rng(81).choice(B, 1024, replace=False))
    states, _, _, _, _ = oracle.gather_from_host_replay(hr, idx[sample], with_next=False)
    say("[fwd-large] oracle on 1,024 sampled states")
    q_ref = oracle.forward_q(shape, th, states.reshape(-1, 4, 84, 84))
    qg = host(q)[sample]
    assert_close(qg, q_ref, FP32_TOL, "qg")
    act_ref = oracle.select_actions(q_ref, float(F32(0.05)), draws[sample])
    explore = (draws[sample] >> np.uint64(32)) < np.uint64(214748368)
    check_actions(host(act)[sample], qg, q_ref, act_ref, explore)
    # every state, not just the sample: greedy actions are the argmax of q_out
    all_explore = (draws >> np.uint64(32)) < np.uint64(214748368)
    own = np.argmax(host(q), axis=1)
    assert np.array_equal(host(act)[~all_explore], own[~all_explore])


def test_td_precision_ambiguous_transitions(dev):
    """Transitions with a ReLU pre-activation within float32 rounding of zero:
    Q, the targets and the loss are still unique and must match; the
    gradient may legitimately differ where a ReLU derivative flips, and is
    only required to be finite and the same on a second run."""
    net, shape = dq.NET_LARGE, di.NET_L
    size = 8202
    hr = di.host_replay(size, shape.n_actions, seed=2048)
    idx = di.index_stream(1, 3072, size, 2049)[0]
    s, sn, a, r, t = oracle.gather_from_host_replay(hr, idx)
    s = s.reshape(-1, 4, 84, 84)
    sn = sn.reshape(-1, 4, 84, 84)
    th = di.xavier_theta(shape, 6144, bias_scale=0.02)
    say("[td-ambiguous] oracle margins")
    amb = np.nonzero(~split_by_margin(shape, th, s))[0]
    assert amb.size > 0
    sel = amb[:256]
    s, sn, a, r, t = s[sel], sn[sel], a[sel].astype(np.int32), r[sel], t[sel]
    say(f"[td-ambiguous] {sel.size} transitions: GPU twice")
    g1, l1, q, y = _run_td(dev, net, th, None, s, sn, a, r, t, 0.99)
    g2, l2, _, _ = _run_td(dev, net, th, None, s, sn, a, r, t, 0.99)
    assert np.array_equal(g1, g2) and l1 == l2 and np.all(np.isfinite(g1))
    ref = oracle.td_gradient(shape, th, None, s, sn, a, r, t, float(F32(0.99)))
    assert_close(q, ref["q"], FP32_TOL, "q")
    assert_close(y, ref["y"], FP32_TOL, "y")
    assert abs(l1 - ref["loss"]) <= FP32_TOL * abs(ref["loss"])
