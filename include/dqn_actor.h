/*
 * dqn_actor.h -- the actor side of Alg. 1 in libdqn.so: games that the
 * Q-network plays, and the replay memory their experiences fill.
 *
 * Alg. 1 has each worker select an action epsilon-greedily with an annealed
 * epsilon, execute it, observe the reward and the next frame, and store the
 * experience (phi_t, a_t, r_t, phi_{t+1}) in its replay memory, which keeps
 * the last N experiences (Sec. III.C) pooled over game instances.  The game
 * is Snake as Sec. V.A describes it: an n x n board; the snake starts with
 * two cells and grows by one when it eats an apple, which scores +1; hitting
 * itself ends the game and scores -1.  Readings where the text is silent:
 *  - n = 12 and the board wraps around at its edges, so hitting itself is
 *    the only way a game ends;
 *  - actions 0..3 set the heading (up, right, down, left) unless it is the
 *    reverse of the current heading; other actions (the networks have 6 or
 *    18 outputs) keep it;
 *  - the tail leaves its cell in the same move, so moving into it is not a
 *    hit; when the snake eats, the tail stays;
 *  - placement draws come from the caller, two 64-bit words per game and
 *    step (w0, w1): a new game puts the head on cell
 *    floor(lo32(w0) * 144 / 2^32), heading w0 >> 62, the second cell behind
 *    it; an apple goes to the k-th free cell in row-major order,
 *    k = floor(hi32(w1) * free / 2^32) (none on a full board);
 *  - a finished game restarts at once; the experience that ended it stores
 *    the new game's first state as its next state (its target is r alone);
 *  - frames are 84 x 84 bytes rendered directly in gray (each cell a 7 x 7
 *    block: 0 empty, 128 body, 255 head, 192 apple), so the preprocessing
 *    phi is the identity; a state stacks the last four frames, oldest first,
 *    and a new game's state is four copies of its first frame.
 *
 * Replay layout (dqn_replay_out): game e keeps its last N states in records
 * e*(N+1) .. e*(N+1)+N; state t of the game is in slot t mod N and slot N
 * repeats slot 0, so every state's successor is the next record.  The side
 * fields of experience t (a_t, r_t, terminal_t) sit at the record of state
 * t.  After T steps (states 0..T stored), experiences t = max(0, T-N+1) ..
 * T-1 of every game are valid, at record e*(N+1) + t mod N; the same arrays
 * viewed as a dqn_replay of size n_games*(N+1) feed replay_gather and
 * dqn_td_gradient_replay with those indices.
 *
 * Games whose screens come from outside the library (an emulator stepped on
 * the host, its raw screens copied to the device) use dqn_preprocess and
 * dqn_observe instead of the Snake entry points.  Sec. III.A and Fig. 2 say
 * that phi gray-scales the RGB screen, down-samples it to a fixed size and
 * crops it to the network's 84 x 84 input, and stacks the last four frames;
 * the text gives no formulas.  Readings:
 *  - gray = (299 R + 587 G + 114 B + 500) / 1000 per pixel in integers (the
 *    ITU-R BT.601 luma weights, rounded half up);
 *  - down-sampling by an integer factor F (1..8) averages F x F blocks,
 *    (sum + F*F/2) / (F*F) in integers, over the 84F x 84F window of the
 *    screen whose top-left pixel is (top, left): the crop.  Gray-scaling a
 *    block mean and averaging gray pixels agree in exact arithmetic, so the
 *    order of the two steps only decides where the roundings fall; gray is
 *    rounded per pixel, then the block mean;
 *  - the stack and replay rules are those of the Snake games above: a
 *    terminal flag means the screen passed is the first one of a new game.
 *
 * Conventions as in dqn.h: device pointers, caller-owned memory, work
 * enqueued on `stream`, DQN_OK or a negative dqn_status, checks on the host
 * before anything is enqueued.
 */
#ifndef DQN_ACTOR_H
#define DQN_ACTOR_H

#include <stddef.h>
#include <stdint.h>

#include "dqn.h"

#ifdef __cplusplus
extern "C" {
#endif

#define DQN_SNAKE_GRID 12
#define DQN_SNAKE_STATE_BYTES 512   /* device bytes per game */

typedef struct {
    uint8_t* frames;        /* records [n_games*(capacity+1)] of 4x84x84 bytes at record_stride */
    uint8_t* action;        /* [n_games*(capacity+1)] */
    int8_t* reward;         /* [n_games*(capacity+1)] */
    uint8_t* terminal;      /* [n_games*(capacity+1)] */
    int64_t record_stride;  /* bytes between records: a multiple of 16, >= 4*84*84 */
    int64_t capacity;       /* N >= 2 states kept per game */
} dqn_replay_out;

/* Device bytes of the state of n_games games (16-byte aligned buffer), or a
 * negative dqn_status. */
int64_t snake_state_bytes(int32_t n_games);

/* Start every game: games (device, snake_state_bytes), draws uint64
 * [n_games][2], states uint8 [n_games][4][84][84] (16-byte aligned) receive
 * four copies of each game's first frame.  replay (nullable): the first
 * states are stored as state 0 of every game. */
int snake_reset(void* games, int32_t n_games, const uint64_t* draws, uint8_t* states,
                const dqn_replay_out* replay, void* stream);

/* One move of every game with actions int32 [n_games]; draws uint64
 * [n_games][2] (used when the game restarts or places an apple).  states
 * advance by one frame (or restart); reward_out float [n_games] (+1, -1 or
 * 0), terminal_out uint8 [n_games].  replay (nullable): stores experience t
 * (side fields of state t, state t+1 into its slot).  t >= 0 counts the
 * moves since snake_reset. */
int snake_step(void* games, int32_t n_games, const int32_t* actions, const uint64_t* draws, uint8_t* states,
               float* reward_out, uint8_t* terminal_out, const dqn_replay_out* replay, int64_t t, void* stream);

/* Exploration rate of Alg. 1 at iteration n: q = max((n_max - n)/n_max, 0),
 * epsilon = (1 - q) eps_min + q eps_max (host function). */
double dqn_anneal_epsilon(int64_t n, int64_t n_max, double eps_min, double eps_max);

/* One acting step of Alg. 1 for n_games games: the Q-network picks actions
 * on the current states with epsilon-greedy exploration (as dqn_forward,
 * eps_draws uint64 [n_games]), written to actions_out int32 [n_games], and
 * every game moves (as snake_step).  ws: dqn_workspace_bytes(net, n_games,
 * DQN_OP_FORWARD) bytes. */
int dqn_act(const dqn_net* net, const float* theta, void* games, int32_t n_games, uint8_t* states,
            float epsilon, const uint64_t* eps_draws, const uint64_t* env_draws, int32_t* actions_out,
            float* reward_out, uint8_t* terminal_out, const dqn_replay_out* replay, int64_t t, void* ws,
            size_t ws_bytes, void* stream);

/* phi of n raw screens: rgb uint8 [n][h][w][3] (16-byte aligned), window
 * top-left (top, left), factor 1..8 with top + 84*factor <= h and left +
 * 84*factor <= w.  Screen i's 84 x 84 result goes to out + i*out_stride (out
 * 16-byte aligned, out_stride a multiple of 16, >= 84*84; so out may be the
 * newest frame of a [n][4][84][84] state array with out_stride 4*84*84).
 * out must not overlap rgb.  n = 0 does nothing (rgb and out may then be
 * NULL). */
int dqn_preprocess(const uint8_t* rgb, int64_t n, int32_t h, int32_t w, int32_t top, int32_t left,
                   int32_t factor, uint8_t* out, int64_t out_stride, void* stream);

/* Observe step of Alg. 1 for n_games games with raw screens rgb (as in
 * dqn_preprocess, one screen per game).  t = -1 starts the games: each state
 * (uint8 [n_games][4][84][84], 16-byte aligned) becomes four copies of phi of
 * its screen and is stored as state 0 (replay nullable; actions, rewards,
 * terminal unused and nullable).  t >= 0 stores experience t: terminal uint8
 * [n_games] (required) restarts a game's state from its screen, otherwise the
 * state drops its oldest frame and appends phi of the screen; with a replay,
 * actions int32 [n_games] and rewards int8 [n_games] (required) go into the
 * side fields of state t, and state t+1 into its slot, as snake_step does. */
int dqn_observe(const uint8_t* rgb, int32_t n_games, int32_t h, int32_t w, int32_t top, int32_t left,
                int32_t factor, const int32_t* actions, const int8_t* rewards, const uint8_t* terminal,
                uint8_t* states, const dqn_replay_out* replay, int64_t t, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DQN_ACTOR_H */
