"""GPU parity of the bf16-input variant of the large Q-network (every conv
and fc1 contraction operand rounded to bfloat16, fp32 accumulation).

Two references, both per tensor (each W and b separately):
  - the oracle's bf16-input variant, which computes the same definition with
    exact (double) sums: within 3e-2, normwise and element by element;
  - the unrounded float64 oracle: Q within 3e-2; the gradients within the
    error of the exact bf16-input computation itself plus 3e-2, i.e.
    |g_gpu - g64| / |g64| <= |g_bf16 - g64| / |g64| + 3e-2.  On these
    workloads an exact bf16-input computation already differs from the
    float64 gradients by several percent (the TD residual Q - y is small next
    to Q, so the bf16-sized error of Q is amplified in dQ), so 3e-2 alone
    is not met against the float64 oracle by any bf16-input computation."""
import numpy as np
import pytest

import dqn_inputs as di
import oracle
import paper_1508_04186_amd as dq
from gpu_util import assert_close, assert_grad_close, check_actions, dev_tensor, grad_errors, host, rel_l2, say

pytestmark = pytest.mark.gpu
F32 = np.float32
BF16_TOL = 3e-2
NET, SHAPE = dq.NET_LARGE_BF16, di.NET_L


def _inputs(B, seed, held):
    size = 2 * B + 20
    hr = di.host_replay(size, SHAPE.n_actions, seed=seed)
    idx = di.index_stream(1, B, size, seed + 1)[0]
    s, sn, a, r, t = oracle.gather_from_host_replay(hr, idx)
    th = di.xavier_theta(SHAPE, seed + 2, bias_scale=0.02)
    tt = di.xavier_theta(SHAPE, seed + 3, bias_scale=0.02) if held else None
    return th, tt, s.reshape(B, 4, 84, 84), sn.reshape(B, 4, 84, 84), a.astype(np.int32), r, t


def _run_td(dev, th, tt, s, sn, a, r, t, gamma=0.99):
    import torch
    B = s.shape[0]
    g = torch.empty(dq.dqn_param_count(NET), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    q = torch.empty((B, NET.n_actions), dtype=torch.float32, device=dev)
    y = torch.empty(B, dtype=torch.float32, device=dev)
    th_d = dev_tensor(th)
    tt_d = th_d if tt is None else dev_tensor(tt)
    dq.dqn_td_gradient(NET, th_d, tt_d, dev_tensor(s), dev_tensor(sn), dev_tensor(a), dev_tensor(r),
                       dev_tensor(t), gamma, g, loss, q, y)
    torch.cuda.synchronize()
    return host(g), float(host(loss)[0]), host(q), host(y)


@pytest.mark.parametrize("B,held", [(3, False), (17, True), (64, False), (131, True), (256, True), (2048, False)])
def test_bf16_td_gradient_matches_oracle(dev, B, held):
    say(f"[bf16-td] batch={B} held={held}: inputs")
    th, tt, s, sn, a, r, t = _inputs(B, 500 + B, held)
    say(f"[bf16-td] batch={B}: GPU")
    g, loss, q, y = _run_td(dev, th, tt, s, sn, a, r, t)
    say(f"[bf16-td] batch={B}: oracle (bf16-input variant)")
    ref = oracle.td_gradient(SHAPE, th, tt, s, sn, a, r, t, float(F32(0.99)), bf16=True)
    assert_close(q, ref["q"], BF16_TOL, "q")
    assert_close(y, ref["y"], BF16_TOL, "y")
    assert abs(loss - ref["loss"]) <= BF16_TOL * abs(ref["loss"])
    errs = assert_grad_close(SHAPE, g, ref["grad"], tol=BF16_TOL, what="bf16 grad")
    say(f"[bf16-td] batch={B}: worst per-tensor error vs the bf16-input oracle {max(errs.values()):.2e}")
    say(f"[bf16-td] batch={B}: oracle (float64)")
    ref64 = oracle.td_gradient(SHAPE, th, tt, s, sn, a, r, t, float(F32(0.99)))
    assert_close(q, ref64["q"], BF16_TOL, "q against the float64 oracle")
    e64 = grad_errors(SHAPE, g, ref64["grad"])
    b64 = grad_errors(SHAPE, ref["grad"], ref64["grad"])
    for k in e64:
        say(f"[bf16-td] batch={B} {k}: GPU vs float64 {e64[k]:.3e}; exact bf16-input vs float64 {b64[k]:.3e}")
    bad = {k: (e64[k], b64[k]) for k in e64 if not e64[k] <= b64[k] + BF16_TOL}
    assert not bad, f"bf16 gradients against the float64 oracle: {bad}"


def test_bf16_td_gradient_is_deterministic_and_differs_from_fp32(dev):
    th, tt, s, sn, a, r, t = _inputs(40, 900, False)
    g1, l1, q1, _ = _run_td(dev, th, tt, s, sn, a, r, t)
    g2, l2, q2, _ = _run_td(dev, th, tt, s, sn, a, r, t)
    assert np.array_equal(g1, g2) and l1 == l2 and np.array_equal(q1, q2)
    # the fp32 network on the same inputs gives a different (more exact) Q
    import torch
    qf = torch.empty((40, 18), dtype=torch.float32, device=dev)
    dq.dqn_forward(dq.NET_LARGE, dev_tensor(th), dev_tensor(s), 0.0, None, qf, None)
    torch.cuda.synchronize()
    assert not np.array_equal(host(qf), q1)
    q64 = oracle.forward_q(SHAPE, th, s)
    assert rel_l2(host(qf), q64) < rel_l2(q1, q64)


@pytest.mark.parametrize("B", [5, 300])
def test_bf16_forward_matches_oracle(dev, B):
    import torch
    th = di.xavier_theta(SHAPE, 40 + B, bias_scale=0.05)
    st = di.random_states(B, 41 + B)
    q = torch.empty((B, NET.n_actions), dtype=torch.float32, device=dev)
    act = torch.empty(B, dtype=torch.int32, device=dev)
    dq.dqn_forward(NET, dev_tensor(th), dev_tensor(st), 0.0, None, q, act)
    torch.cuda.synchronize()
    q_ref = oracle.forward_q(SHAPE, th, st, bf16=True)
    assert_close(host(q), q_ref, BF16_TOL, "host(q)")
    act_ref = oracle.select_actions(q_ref, 0.0)
    check_actions(host(act), host(q), q_ref, act_ref, np.zeros(B, bool), tol=BF16_TOL)


def test_bf16_forward_8192_states_egreedy(dev):
    import torch
    B = 8192
    th = di.xavier_theta(SHAPE, 88, bias_scale=0.02)
    st = di.random_states(B, 89)
    draws = di.egreedy_draws(B, 90)
    q = torch.empty((B, NET.n_actions), dtype=torch.float32, device=dev)
    act = torch.empty(B, dtype=torch.int32, device=dev)
    say(f"[bf16-fwd] batch={B}: GPU forward eps=0.05")
    dq.dqn_forward(NET, dev_tensor(th), dev_tensor(st), float(F32(0.05)), dev_tensor(draws), q, act)
    torch.cuda.synchronize()
    sample = np.sort(np.random.default_rng(91).choice(B, 512, replace=False))
    say("[bf16-fwd] oracle (bf16-input variant) on 512 sampled states")
    q_ref = oracle.forward_q(SHAPE, th, st[sample], bf16=True)
    qg = host(q)[sample]
    assert_close(qg, q_ref, BF16_TOL, "qg")
    act_ref = oracle.select_actions(q_ref, float(F32(0.05)), draws[sample])
    explore = (draws[sample] >> np.uint64(32)) < np.uint64(214748368)
    check_actions(host(act)[sample], qg, q_ref, act_ref, explore, tol=BF16_TOL)
    all_explore = (draws >> np.uint64(32)) < np.uint64(214748368)
    own = np.argmax(host(q), axis=1)
    assert np.array_equal(host(act)[~all_explore], own[~all_explore])
