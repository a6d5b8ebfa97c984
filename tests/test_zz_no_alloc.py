"""The TD-gradient entry point that allocates nothing
(dqn_td_gradient_noalloc, on the library's static per-GPU scratch) against
the workspace entry point dqn_td_gradient: bitwise the same outputs on two
calls in a row, the second with a smaller batch, both within the fp32 bar of
the oracle (Alg. 1; Eq. (1)); a batch whose workspace exceeds the scratch is
rejected before anything is enqueued."""
import numpy as np
import pytest

import dqn_inputs as di
import oracle
import paper_1508_04186_amd as dq
from gpu_util import FP32_TOL, assert_close, assert_grad_close, dev_tensor, host, say, split_by_margin

pytestmark = pytest.mark.gpu
F32 = np.float32


def _inputs(shape, B, seed):
    """Seeded inputs; the states are drawn from 2B uniform candidates whose
    oracle ReLU margins are at least MARGIN_MIN (a unique gradient)."""
    th = di.xavier_theta(shape, seed, bias_scale=0.05)
    tt = di.xavier_theta(shape, seed + 1, bias_scale=0.05)
    cand = di.random_states(2 * B, seed + 2)
    keep = np.nonzero(split_by_margin(shape, th, cand))[0]
    assert keep.size >= B
    s = cand[keep[:B]]
    sn = di.random_states(B, seed + 3)
    a, r, t = di.random_transitions(B, shape.n_actions, seed + 4, p_terminal=0.2)
    return th, tt, s, sn, a.astype(np.int32), r.astype(F32), t.astype(np.uint8)


def _outputs(dev, net, B):
    import torch
    P = dq.dqn_param_count(net)
    return (torch.full((P,), np.nan, dtype=torch.float32, device=dev),
            torch.full((1,), np.nan, dtype=torch.float32, device=dev),
            torch.full((B, net.n_actions), np.nan, dtype=torch.float32, device=dev),
            torch.full((B,), np.nan, dtype=torch.float32, device=dev))


@pytest.mark.parametrize("name,batches", [("small", (32, 9)), ("large", (94, 17))])
def test_noalloc_equals_workspace_entry_point(dev, name, batches):
    import torch
    net, shape = (dq.NET_SMALL, di.NET_S) if name == "small" else (dq.NET_LARGE, di.NET_L)
    for call, B in enumerate(batches):
        say(f"[noalloc] net={name} call={call} batch={B}")
        th, tt, s, sn, a, r, t = _inputs(shape, B, 700 + 10 * call + B)
        d = [dev_tensor(x) for x in (th, tt, s, sn, a, r, t)]
        g0, l0, q0, y0 = _outputs(dev, net, B)
        g1, l1, q1, y1 = _outputs(dev, net, B)
        dq.dqn_td_gradient_noalloc(net, *d[:7], 0.99, g0, l0, q0, y0)
        dq.dqn_td_gradient(net, *d[:7], 0.99, g1, l1, q1, y1)
        torch.cuda.synchronize()
        for x, y_, what in ((g0, g1, "grad"), (l0, l1, "loss"), (q0, q1, "q"), (y0, y1, "y")):
            assert torch.equal(x, y_), f"{what} differs from dqn_td_gradient (batch {B})"
        ref = oracle.td_gradient(shape, th, tt, s, sn, a, r, t, float(F32(0.99)))
        assert_close(host(q0), ref["q"], FP32_TOL, "q")
        assert_close(host(y0), ref["y"], FP32_TOL, "y")
        assert abs(float(host(l0)[0]) - ref["loss"]) <= FP32_TOL * abs(ref["loss"])
        assert_grad_close(shape, host(g0), ref["grad"])


def test_noalloc_rejects_a_batch_beyond_the_scratch(dev):
    import torch
    net, shape = dq.NET_LARGE, di.NET_L
    B = 128     # its workspace exceeds the 64 MiB scratch
    assert dq.dqn_workspace_bytes(net, B, dq.DQN_OP_TD_GRADIENT) > 64 << 20
    th, tt, s, sn, a, r, t = _inputs(shape, B, 800)
    d = [dev_tensor(x) for x in (th, tt, s, sn, a, r, t)]
    g, loss, q, y = _outputs(dev, net, B)
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_td_gradient_noalloc(net, *d, 0.99, g, loss, q, y)
    assert e.value.status == dq.DQN_EWORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(g).all() and torch.isnan(loss).all()   # nothing was enqueued
