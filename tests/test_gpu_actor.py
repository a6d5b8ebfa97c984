"""GPU parity of the actor side of Alg. 1 (include/dqn_actor.h) against the
oracle: the Snake games, their stacked frames and the replay memory they
fill, bit for bit over long runs that restart games and wrap the replay;
acting with the Q-network (dqn_act); and the TD gradient of minibatches
drawn from that replay."""
import numpy as np
import pytest

import dqn_inputs as di
import oracle
import paper_1508_04186_amd as dq
from gpu_util import FP32_TOL, assert_grad_close, check_actions, dev_tensor, host, rel_l2, say

pytestmark = pytest.mark.gpu


def _run_both(dev, E, N, T, seed, check_every=1):
    import torch
    rng = np.random.default_rng(seed)
    d0 = di.game_draws(E, seed, -1)
    og = oracle.SnakeGames(E, d0)
    orp = oracle.SegmentedReplay(E, N)
    orp.append(-1, og.states)
    games = dq.snake_games(E, dev)
    states = torch.empty((E, 4, 84, 84), dtype=torch.uint8, device=dev)
    rp = dq.ActorReplay(E, N, dev)
    dq.snake_reset(games, dev_tensor(d0), states, rp)
    rew = torch.empty(E, dtype=torch.float32, device=dev)
    term = torch.empty(E, dtype=torch.uint8, device=dev)
    n_term = n_eat = 0
    for t in range(T):
        a = rng.integers(0, 6, E).astype(np.int32)
        d = di.game_draws(E, seed, t)
        dq.snake_step(games, dev_tensor(a), dev_tensor(d), states, rew, term, rp, t)
        r, tt = og.step(a, d)
        orp.append(t, og.states, a, r, tt)
        n_term += int(tt.sum())
        n_eat += int((r > 0).sum())
        if t % check_every == 0 or t == T - 1:
            torch.cuda.synchronize()
            assert np.array_equal(host(rew), r), f"reward differs at step {t}"
            assert np.array_equal(host(term), tt), f"terminal differs at step {t}"
            assert np.array_equal(host(states), og.states), f"states differ at step {t}"
    torch.cuda.synchronize()
    return rp, orp, n_term, n_eat


@pytest.mark.parametrize("E,N,T", [(1, 2, 40), (37, 50, 400)])
def test_games_and_replay_bit_exact(dev, E, N, T):
    say(f"[actor] games={E} capacity={N} moves={T}")
    rp, orp, n_term, n_eat = _run_both(dev, E, N, T, seed=11 + E, check_every=1 if E == 1 else 7)
    assert np.array_equal(host(rp.frames).reshape(len(orp.frames), -1), orp.frames)
    assert np.array_equal(host(rp.action), orp.action)
    assert np.array_equal(host(rp.reward), orp.reward)
    assert np.array_equal(host(rp.terminal), orp.terminal)
    if E > 1:
        assert n_term > 0 and n_eat > 0   # the run covered restarts and apples


def test_act_with_the_network(dev):
    import torch
    net, shape = dq.NET_SMALL, di.NET_S
    E, T = 24, 6
    th = di.xavier_theta(shape, 5, bias_scale=0.05)
    th_d = dev_tensor(th)
    d0 = di.game_draws(E, 3, -1)
    og = oracle.SnakeGames(E, d0)
    games = dq.snake_games(E, dev)
    states = torch.empty((E, 4, 84, 84), dtype=torch.uint8, device=dev)
    dq.snake_reset(games, dev_tensor(d0), states)
    acts = torch.empty(E, dtype=torch.int32, device=dev)
    rew = torch.empty(E, dtype=torch.float32, device=dev)
    term = torch.empty(E, dtype=torch.uint8, device=dev)
    q = torch.empty((E, 6), dtype=torch.float32, device=dev)
    for t in range(T):
        eps = dq.dqn_anneal_epsilon(t, 4, 0.1, 1.0)
        assert eps == pytest.approx(oracle.anneal_epsilon(t, 4, 0.1, 1.0), abs=0)
        ed = di.egreedy_draws(E, 100 + t)
        gd = di.game_draws(E, 3, t)
        # Q of the current states, for the action check
        dq.dqn_forward(net, th_d, states, 0.0, None, q, None)
        dq.dqn_act(net, th_d, games, states, float(np.float32(eps)), dev_tensor(ed), dev_tensor(gd), acts, rew,
                   term)
        torch.cuda.synchronize()
        a = host(acts)
        q_ref = oracle.forward_q(shape, th, og.states)
        act_ref = oracle.select_actions(q_ref, float(np.float32(eps)), ed)
        te = np.floor(np.float64(np.float32(eps)) * 2**32)
        explore = (ed >> np.uint64(32)).astype(np.float64) < te
        check_actions(a, host(q), q_ref, act_ref, explore)
        r, tt = og.step(a, gd)                      # the oracle game moves with the GPU's actions
        assert np.array_equal(host(rew), r) and np.array_equal(host(term), tt)
        assert np.array_equal(host(states), og.states)


def test_td_gradient_on_the_actor_replay(dev):
    import torch
    net, shape = dq.NET_SMALL, di.NET_S
    E, N, T, B = 16, 30, 45, 32
    rp, orp, _, _ = _run_both(dev, E, N, T, seed=23, check_every=50)
    idx = di.actor_minibatch(B, 4, 0, E, N, T)
    th = di.xavier_theta(shape, 8, bias_scale=0.05)
    th_d = dev_tensor(th)
    P = dq.dqn_param_count(net)
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    dq.dqn_td_gradient_replay(net, th_d, th_d, rp.view, dev_tensor(idx), 0.99, g, loss)
    torch.cuda.synchronize()
    s, sn, a, r, t = oracle.replay_gather(orp.frames, orp.rec, orp.rec, len(orp.frames), orp.action,
                                          orp.reward, orp.terminal, idx)
    a = np.minimum(a, 5)
    ref = oracle.td_gradient(shape, th, None, s.reshape(B, 4, 84, 84), sn.reshape(B, 4, 84, 84), a, r, t,
                             float(np.float32(0.99)))
    assert abs(float(host(loss)[0]) - ref["loss"]) <= FP32_TOL * abs(ref["loss"])
    assert_grad_close(shape, host(g), ref["grad"])
