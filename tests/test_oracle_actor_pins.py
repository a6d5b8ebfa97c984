"""Pins of the oracle's actor side (Alg. 1's act / store steps): the Snake
rules of Sec. V.A on hand-built positions, the rendering, the random
placements against their definition, the replay memory that keeps the last
N states per game against a brute-force history, and the annealed
exploration rate against its closed form."""
import numpy as np
import pytest

import oracle

G = oracle.SNAKE_GRID
CELLS = G * G


def draws_for(head=None, heading=0, apple_k=None, free=None):
    """A (w0, w1) pair: w0 puts a new game's head on `head` with `heading`;
    w1 picks the apple_k-th of `free` free cells."""
    w0 = 0
    if head is not None:
        lo = -(-head * 2**32 // CELLS)          # smallest lo with floor(lo*144/2^32) = head
        w0 = (heading << 62) | lo
    w1 = 0
    if apple_k is not None:
        w1 = (-(-apple_k * 2**32 // free)) << 32
    return np.array([w0, w1], np.uint64)


def set_game(games, e, body, heading, apple):
    games.games[e, :] = 0
    games.games[e, :len(body)] = body
    games.games[e, CELLS] = len(body)
    games.games[e, CELLS + 1] = heading
    games.games[e, CELLS + 2] = apple


def head_of(games, e):
    return int(games.games[e, 0])


def test_new_game_from_draws():
    d = draws_for(head=50, heading=1, apple_k=51, free=CELLS - 2)
    g = oracle.SnakeGames(1, d)
    assert list(g.games[0, :2]) == [50, 49]            # second cell behind the head
    assert g.games[0, CELLS] == 2 and g.games[0, CELLS + 1] == 1
    # free cells before 53 in row-major order: 0..52 minus the body (49, 50) = 51
    assert g.games[0, CELLS + 2] == 53
    st = g.states[0]
    assert all(np.array_equal(st[f], st[0]) for f in range(4))   # four copies


def test_render_blocks():
    d = draws_for(head=50, heading=1, apple_k=51, free=CELLS - 2)
    g = oracle.SnakeGames(1, d)
    f = g.states[0, 3]
    assert (f == 255).sum() == 49 and (f == 128).sum() == 49 and (f == 192).sum() == 49
    assert (f == 0).sum() == 84 * 84 - 3 * 49
    # head cell (4, 2) -> pixels [28, 35) x [14, 21); apple (4, 5) -> x [35, 42)
    assert np.all(f[28:35, 14:21] == 255) and np.all(f[28:35, 7:14] == 128) and np.all(f[28:35, 35:42] == 192)


def test_moves_eat_and_grow():
    d = draws_for(head=50, heading=1, apple_k=51, free=CELLS - 2)
    g = oracle.SnakeGames(1, d)
    nxt = draws_for(apple_k=0, free=CELLS - 3)           # next apple: the first free cell, 0
    rewards = []
    for _ in range(3):
        r, t = g.step(np.array([1], np.int32), nxt)
        rewards.append((float(r[0]), int(t[0])))
    assert rewards == [(0.0, 0), (0.0, 0), (1.0, 0)]      # 51, 52, then the apple on 53
    assert list(g.games[0, :3]) == [53, 52, 51] and g.games[0, CELLS] == 3
    assert g.games[0, CELLS + 2] == 0


def test_state_stack_shifts_by_one_frame():
    d = draws_for(head=50, heading=1, apple_k=51, free=CELLS - 2)
    g = oracle.SnakeGames(1, d)
    before = g.states[0].copy()
    g.step(np.array([1], np.int32), draws_for(apple_k=0, free=CELLS - 3))
    assert np.array_equal(g.states[0, :3], before[1:])
    assert g.states[0, 3, 28:35, 21:28].min() == 255     # head now on cell 51


def test_reverse_and_noop_keep_heading_and_board_wraps():
    g = oracle.SnakeGames(1, draws_for(head=50, heading=1, apple_k=0, free=CELLS - 2))
    set_game(g, 0, [59, 58], 1, 0)                       # head at (4, 11) heading right
    g.step(np.array([3], np.int32), draws_for())          # left is the reverse: ignored
    assert head_of(g, 0) == 48                           # wrapped to (4, 0)
    g.step(np.array([5], np.int32), draws_for())          # action >= 4 keeps the heading
    assert head_of(g, 0) == 49
    g.step(np.array([0], np.int32), draws_for())          # up
    assert head_of(g, 0) == 37
    set_game(g, 0, [5, 17], 0, 100)                      # (0, 5) heading up wraps to (11, 5)
    g.step(np.array([0], np.int32), draws_for())
    assert head_of(g, 0) == 137


def test_self_hit_ends_the_game_and_restarts():
    g = oracle.SnakeGames(1, draws_for(head=0, heading=0, apple_k=0, free=CELLS - 2))
    set_game(g, 0, [50, 49, 48, 47, 46], 1, 100)
    restart = draws_for(head=70, heading=2, apple_k=3, free=CELLS - 2)
    out = []
    for a in (2, 3, 0):                                  # down, left, up into the body at 49
        r, t = g.step(np.array([a], np.int32), restart)
        out.append((float(r[0]), int(t[0])))
    assert out == [(0.0, 0), (0.0, 0), (-1.0, 1)]
    # restarted at once from the draws: head 70 heading down, tail behind it
    assert list(g.games[0, :2]) == [70, 58] and g.games[0, CELLS] == 2
    st = g.states[0]
    assert all(np.array_equal(st[f], st[0]) for f in range(4))


def test_moving_into_the_leaving_tail_is_not_a_hit():
    g = oracle.SnakeGames(1, draws_for(head=0, heading=0, apple_k=0, free=CELLS - 2))
    set_game(g, 0, [50, 62, 61, 49], 2, 100)             # a 2x2 loop; the tail sits on 49
    r, t = g.step(np.array([3], np.int32), draws_for())  # left from 50 onto 49
    assert float(r[0]) == 0.0 and int(t[0]) == 0 and head_of(g, 0) == 49


def test_apples_never_on_the_snake_and_placement_follows_the_draw():
    rng = np.random.default_rng(5)
    E = 16
    g = oracle.SnakeGames(E, rng.integers(0, 2**64, size=(E, 2), dtype=np.uint64))
    for _ in range(1500):
        before = g.games.copy()
        d = rng.integers(0, 2**64, size=(E, 2), dtype=np.uint64)
        r, t = g.step(rng.integers(0, 6, E).astype(np.int32), d)
        for e in range(E):
            L = g.games[e, CELLS]
            apple = g.games[e, CELLS + 2]
            body = set(g.games[e, :L])
            assert len(body) == L and apple not in body
            if r[e] == 1.0:
                # the apple is the k-th free cell of the grown snake
                free = [c for c in range(CELLS) if c not in body]
                k = ((int(d[e, 1]) >> 32) * len(free)) >> 32
                assert apple == free[k]
                assert L == before[e, CELLS] + 1


def test_replay_keeps_the_last_n_states_per_game():
    rng = np.random.default_rng(7)
    E, N, T = 3, 7, 25                                   # wraps the segments three times
    rec = 4 * 84 * 84
    g = oracle.SnakeGames(E, rng.integers(0, 2**64, size=(E, 2), dtype=np.uint64))
    rp = oracle.SegmentedReplay(E, N)
    rp.append(-1, g.states)
    hist_s = [g.states.copy()]
    hist = []
    for t in range(T):
        a = rng.integers(0, 6, E).astype(np.int32)
        r, term = g.step(a, rng.integers(0, 2**64, size=(E, 2), dtype=np.uint64))
        rp.append(t, g.states, a, r, term)
        hist_s.append(g.states.copy())
        hist.append((a, r, term))
    for e in range(E):
        base = e * (N + 1)
        # transitions T-N+1 .. T-1 are stored; transition t at slot t mod N
        for t in range(T - N + 1, T):
            i = base + t % N
            assert np.array_equal(rp.frames[i], hist_s[t][e].reshape(-1))
            assert np.array_equal(rp.frames[i + 1], hist_s[t + 1][e].reshape(-1))   # successor record
            a, r, term = hist[t]
            assert rp.action[i] == a[e] and rp.reward[i] == int(r[e]) and rp.terminal[i] == term[e]
        assert np.array_equal(rp.frames[base + N], rp.frames[base])                   # slot N repeats slot 0


@pytest.mark.parametrize("n,expect", [(0, 1.0), (500, 0.55), (1000, 0.1), (5000, 0.1)])
def test_annealed_epsilon(n, expect):
    assert oracle.anneal_epsilon(n, 1000, 0.1, 1.0) == pytest.approx(expect, abs=1e-15)


# ---------------------------------------------------------------------------
# Preprocessing phi (Sec. III.A): gray-scale, crop, f x f box down-sampling.

def test_preprocess_constant_colors_closed_form():
    for (r, g, b) in [(0, 0, 0), (255, 255, 255), (255, 0, 0), (0, 255, 0), (0, 0, 255), (12, 200, 77)]:
        rgb = np.zeros((1, 170, 172, 3), np.uint8)
        rgb[...] = (r, g, b)
        gray = (299 * r + 587 * g + 114 * b + 500) // 1000
        out = oracle.preprocess(rgb, 1, 2, 2)
        assert np.all(out == gray)
    # the BT.601 weights on the primaries
    assert [(299 * 255 + 500) // 1000, (587 * 255 + 500) // 1000, (114 * 255 + 500) // 1000] == [76, 150, 29]


def test_preprocess_one_bright_pixel_lands_in_its_block():
    rgb = np.zeros((1, 260, 260, 3), np.uint8)
    top, left, f = 5, 7, 3
    yy, xx = 40, 61                                   # output block (40, 61), offset (1, 2) inside it
    rgb[0, top + f * yy + 1, left + f * xx + 2] = (255, 255, 255)
    out = oracle.preprocess(rgb, top, left, f)
    expect = np.zeros((84, 84), np.uint8)
    expect[yy, xx] = (255 + 4) // 9                   # (sum + f*f/2) / (f*f)
    assert np.array_equal(out[0], expect)


def test_preprocess_is_the_mean_of_blocks_of_gray():
    rgb = np.random.default_rng(3).integers(0, 256, size=(2, 180, 175, 3), dtype=np.uint8)
    c = rgb.astype(np.int64)
    g = (299 * c[..., 0] + 587 * c[..., 1] + 114 * c[..., 2] + 500) // 1000
    win = g[:, 6:6 + 168, 3:3 + 168].reshape(2, 84, 2, 84, 2).sum(axis=(2, 4))
    assert np.array_equal(oracle.preprocess(rgb, 6, 3, 2), ((win + 2) // 4).astype(np.uint8))
