// The actor side of Alg. 1 ("execute action a_t, observe r_t and frame
// x_{t+1}, store the experience in D"): E Snake games (Sec. V.A), one
// wavefront each, and the replay memory they fill.
//
// Game rules and readings (include/dqn_actor.h): a 12 x 12 board that wraps
// at its edges; the snake starts with two cells and grows by one per apple
// (+1); hitting itself ends the game (-1) and a new one starts at once;
// actions 0..3 set the heading unless it is the reverse of the current one,
// other actions keep it; the tail leaves its cell in the same move unless the
// snake eats.  Placement is drawn from two caller-supplied words per game and
// step.  A frame is 84 x 84 bytes, 7 x 7 per cell: 0 empty, 128 body, 255
// head, 192 apple; a state stacks the last four frames, oldest first.
//
// Device game state: a ring of body cells (segment i at ring[(hp + i) % 144])
// and an occupancy grid, so a move touches two cells; the workgroup (four
// waves) copies them to LDS, every thread runs the same control logic on the
// same values, the lanes of each wave compute the free-cell count of an apple
// placement (a prefix sum over three cells per lane), and the threads share
// the rendering (16-byte vectors) and the state and replay writes, with the
// kept frames read before the game logic runs.
#include "common.h"
#include "dqn_actor.h"
#include "dqn_profile.h"

namespace dqn {
namespace {

constexpr int SG = DQN_SNAKE_GRID;           // board side
constexpr int SC = SG * SG;                  // cells
constexpr int SPX = 84 / SG;                 // pixels per cell side
constexpr int FB = 84 * 84;                  // frame bytes
constexpr int FV = FB / 16;                  // 16-byte vectors per frame
constexpr int AW = 256;                      // threads per game (four waves)
constexpr int WL = 64;                       // wavefront
constexpr int VPT = (FV + AW - 1) / AW;      // frame vectors per thread (2)
static_assert(SG * SPX == 84 && FB % 16 == 0, "frame geometry");

struct SnakeDev {
    int16_t ring[SC];
    uint8_t occ[SC];
    int32_t hp, len, heading, apple;
};
static_assert(sizeof(SnakeDev) <= DQN_SNAKE_STATE_BYTES, "game state size");

__device__ __forceinline__ int cell_move(int cell, int heading) {
    int y = cell / SG, x = cell - (cell / SG) * SG;
    y += heading == 0 ? -1 : heading == 2 ? 1 : 0;
    x += heading == 1 ? 1 : heading == 3 ? -1 : 0;
    y = (y + SG) % SG;
    x = (x + SG) % SG;
    return y * SG + x;
}

struct Lds {
    int16_t ring[SC];
    uint8_t occ[SC];
    int32_t hp, len, heading, apple;
};

// k-th free cell in row-major order (k from the high 32 bits of w1 scaled to
// the free count), or -1 on a full board.  Lane l counts cells 3l .. 3l+2;
// every wave computes the same result.
__device__ int place_apple(const Lds& g, uint64_t w1) {
    const int l = threadIdx.x & (WL - 1);
    int cnt = 0;
    if (l * 3 < SC)
        for (int i = 0; i < 3; ++i) cnt += g.occ[3 * l + i] == 0;
    int incl = cnt;
#pragma unroll
    for (int d = 1; d < WL; d <<= 1) {
        const int v = __shfl_up(incl, d, WL);
        if (l >= d) incl += v;
    }
    const int free_cells = __shfl(incl, WL - 1, WL);
    if (free_cells == 0) return -1;
    const uint32_t k = (uint32_t)(((w1 >> 32) * (uint64_t)free_cells) >> 32);
    const int excl = incl - cnt;
    int found = -1;
    if (cnt > 0 && (int)k >= excl && (int)k < incl) {
        int r = (int)k - excl;
        for (int i = 0; i < 3; ++i)
            if (g.occ[3 * l + i] == 0) {
                if (r == 0) { found = 3 * l + i; break; }
                --r;
            }
    }
    // exactly one lane found it
    const uint64_t m = __ballot(found >= 0);
    return __shfl(found, __ffsll((unsigned long long)m) - 1, WL);
}

__device__ void new_game(Lds& g, uint64_t w0, uint64_t w1) {
    const int l = threadIdx.x;  // 0 .. AW-1
    for (int c = l; c < SC; c += AW) g.occ[c] = 0;
    __syncthreads();
    const int head = (int)(((w0 & 0xffffffffull) * (uint64_t)SC) >> 32);
    const int heading = (int)(w0 >> 62);
    const int tail = cell_move(head, (heading + 2) & 3);
    if (l == 0) {
        g.hp = 0;
        g.len = 2;
        g.heading = heading;
        g.ring[0] = (int16_t)head;
        g.ring[1] = (int16_t)tail;
        g.occ[head] = 1;
        g.occ[tail] = 1;
    }
    __syncthreads();
    const int apple = place_apple(g, w1);
    __syncthreads();
    if (l == 0) g.apple = apple;
    __syncthreads();
}

// Pixels 16q .. 16q+15 of the frame of game g.
__device__ __forceinline__ uint4 render16(const Lds& g, int q) {
    uint8_t v[16];
    const int head = g.ring[g.hp];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int p = 16 * q + i;
        const int y = p / 84, x = p - (p / 84) * 84;
        const int cell = (y / SPX) * SG + x / SPX;
        v[i] = cell == head ? 255 : g.occ[cell] ? 128 : cell == g.apple ? 192 : 0;
    }
    uint4 o;
    o.x = v[0] | (v[1] << 8) | (v[2] << 16) | ((uint32_t)v[3] << 24);
    o.y = v[4] | (v[5] << 8) | (v[6] << 16) | ((uint32_t)v[7] << 24);
    o.z = v[8] | (v[9] << 8) | (v[10] << 16) | ((uint32_t)v[11] << 24);
    o.w = v[12] | (v[13] << 8) | (v[14] << 16) | ((uint32_t)v[15] << 24);
    return o;
}

__device__ void load_game(Lds& g, const SnakeDev* src) {
    const int l = threadIdx.x;
    for (int c = l; c < SC; c += AW) {
        g.ring[c] = src->ring[c];
        g.occ[c] = src->occ[c];
    }
    if (l == 0) {
        g.hp = src->hp;
        g.len = src->len;
        g.heading = src->heading;
        g.apple = src->apple;
    }
    __syncthreads();
}

__device__ void store_game(const Lds& g, SnakeDev* dst) {
    const int l = threadIdx.x;
    for (int c = l; c < SC; c += AW) {
        dst->ring[c] = g.ring[c];
        dst->occ[c] = g.occ[c];
    }
    if (l == 0) {
        dst->hp = g.hp;
        dst->len = g.len;
        dst->heading = g.heading;
        dst->apple = g.apple;
    }
}

// The three frames a move keeps (frames 1..3 of the state), read by each
// thread for its vectors before anything is written.
struct Kept {
    uint4 f[3][VPT];
};

__device__ void read_kept(const uint8_t* st, Kept& k) {
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int q = threadIdx.x + i * AW;
        if (q < FV)
#pragma unroll
            for (int f = 0; f < 3; ++f) k.f[f][i] = ((const uint4*)(st + (f + 1) * FB))[q];
    }
}

// State write of game e (the new frame in every slot, or the kept frames
// shifted by one) and the replay copy of the same state.
__device__ void write_state(const Lds& g, uint8_t* st, bool fresh, const Kept& kept, const ReplayOut& rp, int e) {
    uint8_t* rec = nullptr;
    uint8_t* mirror = nullptr;
    if (rp.frames) {
        const int64_t base = (int64_t)e * (rp.cap + 1);
        const int64_t slot = (rp.t + 1) % rp.cap;
        rec = rp.frames + (base + slot) * rp.stride;
        if (slot == 0) mirror = rp.frames + (base + rp.cap) * rp.stride;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int q = threadIdx.x + i * AW;
        if (q >= FV) continue;
        const uint4 nf = render16(g, q);
        uint4 f[4];
        if (fresh) {
            f[0] = f[1] = f[2] = f[3] = nf;
        } else {
            f[0] = kept.f[0][i];
            f[1] = kept.f[1][i];
            f[2] = kept.f[2][i];
            f[3] = nf;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) ((uint4*)(st + k * FB))[q] = f[k];
        if (rec)
#pragma unroll
            for (int k = 0; k < 4; ++k) ((uint4*)(rec + k * FB))[q] = f[k];
        if (mirror)
#pragma unroll
            for (int k = 0; k < 4; ++k) ((uint4*)(mirror + k * FB))[q] = f[k];
    }
}

__global__ __launch_bounds__(AW) void snake_reset_kernel(SnakeDev* games, const uint64_t* draws, uint8_t* states,
                                                         ReplayOut rp) {
    __shared__ Lds g;
    const int e = blockIdx.x;
    new_game(g, draws[2 * e], draws[2 * e + 1]);
    store_game(g, games + e);
    Kept none;
    write_state(g, states + (size_t)e * 4 * FB, true, none, rp, e);
}

__global__ __launch_bounds__(AW) void snake_step_kernel(SnakeDev* games, const int32_t* actions,
                                                        const uint64_t* draws, uint8_t* states, float* reward,
                                                        uint8_t* terminal, ReplayOut rp) {
    __shared__ Lds g;
    const int e = blockIdx.x;
    const int l = threadIdx.x;
    Kept kept;
    read_kept(states + (size_t)e * 4 * FB, kept);   // in flight during the game logic
    load_game(g, games + e);
    const uint64_t w0 = draws[2 * e], w1 = draws[2 * e + 1];
    const int a = actions[e];
    int heading = g.heading;
    if (a >= 0 && a < 4 && a != ((heading + 2) & 3)) heading = a;
    const int head = g.ring[g.hp];
    const int nh = cell_move(head, heading);
    const int tail = g.ring[(g.hp + g.len - 1) % SC];
    const bool eats = nh == g.apple;
    // every segment but the tail, which moves away unless the snake eats
    const bool hit = g.occ[nh] && (eats || nh != tail);
    __syncthreads();
    float r = 0.f;
    if (hit) {
        r = -1.f;
        new_game(g, w0, w1);
    } else {
        if (l == 0) {
            const int hp = (g.hp + SC - 1) % SC;
            if (!eats) g.occ[tail] = 0;
            g.ring[hp] = (int16_t)nh;
            g.occ[nh] = 1;
            g.hp = hp;
            g.heading = heading;
            if (eats) g.len = g.len + 1;
        }
        __syncthreads();
        if (eats) {
            r = 1.f;
            const int apple = place_apple(g, w1);
            __syncthreads();
            if (l == 0) g.apple = apple;
            __syncthreads();
        }
    }
    store_game(g, games + e);
    write_state(g, states + (size_t)e * 4 * FB, hit, kept, rp, e);
    if (l == 0) {
        reward[e] = r;
        terminal[e] = hit ? 1 : 0;
        if (rp.frames && rp.t >= 0) {
            const int64_t i = (int64_t)e * (rp.cap + 1) + rp.t % rp.cap;
            rp.action[i] = (uint8_t)a;
            rp.reward[i] = (int8_t)r;
            rp.terminal[i] = hit ? 1 : 0;
        }
    }
}

}  // namespace

bool replay_ok(const ReplayOut& rp) {
    if (!rp.frames) return true;
    return rp.action && rp.reward && rp.terminal && rp.cap >= 2 && rp.stride >= 4 * FB && rp.stride % 16 == 0 &&
           ((uintptr_t)rp.frames % 16) == 0;
}

}  // namespace dqn

using namespace dqn;

extern "C" {

int64_t snake_state_bytes(int32_t n_games) {
    if (n_games <= 0) return DQN_EINVAL;
    return (int64_t)n_games * DQN_SNAKE_STATE_BYTES;
}

int snake_reset(void* games, int32_t n_games, const uint64_t* draws, uint8_t* states,
                const dqn_replay_out* replay, void* stream) {
    if (!games || !draws || !states || n_games <= 0) return DQN_EINVAL;
    if (((uintptr_t)games % 16) || ((uintptr_t)states % 16)) return DQN_EINVAL;
    ReplayOut rp{};
    if (replay) rp = ReplayOut{replay->frames, replay->record_stride, replay->action, replay->reward,
                               replay->terminal, replay->capacity, -1};
    if (!replay_ok(rp)) return DQN_EINVAL;
    hipLaunchKernelGGL(snake_reset_kernel, dim3((unsigned)n_games), dim3(AW), 0, (hipStream_t)stream,
                       (SnakeDev*)games, draws, states, rp);
    return hipGetLastError() == hipSuccess ? DQN_OK : DQN_EHIP;
}

int snake_step(void* games, int32_t n_games, const int32_t* actions, const uint64_t* draws, uint8_t* states,
               float* reward_out, uint8_t* terminal_out, const dqn_replay_out* replay, int64_t t, void* stream) {
    if (!games || !actions || !draws || !states || !reward_out || !terminal_out || n_games <= 0) return DQN_EINVAL;
    if (((uintptr_t)games % 16) || ((uintptr_t)states % 16)) return DQN_EINVAL;
    ReplayOut rp{};
    if (replay) {
        if (t < 0) return DQN_EINVAL;
        rp = ReplayOut{replay->frames, replay->record_stride, replay->action, replay->reward, replay->terminal,
                       replay->capacity, t};
    }
    if (!replay_ok(rp)) return DQN_EINVAL;
    prof_mark_begin(DQN_K_SNAKE_STEP, (hipStream_t)stream);
    hipLaunchKernelGGL(snake_step_kernel, dim3((unsigned)n_games), dim3(AW), 0, (hipStream_t)stream,
                       (SnakeDev*)games, actions, draws, states, reward_out, terminal_out, rp);
    if (hipGetLastError() != hipSuccess) return DQN_EHIP;
    prof_mark_end(DQN_K_SNAKE_STEP, (hipStream_t)stream);
    return DQN_OK;
}

double dqn_anneal_epsilon(int64_t n, int64_t n_max, double eps_min, double eps_max) {
    double q = n_max > 0 ? (double)(n_max - n) / (double)n_max : 0.0;
    if (q < 0.0) q = 0.0;
    return (1.0 - q) * eps_min + q * eps_max;
}

}  // extern "C"

extern "C" int dqn_act(const dqn_net* net, const float* theta, void* games, int32_t n_games, uint8_t* states,
                       float epsilon, const uint64_t* eps_draws, const uint64_t* env_draws, int32_t* actions_out,
                       float* reward_out, uint8_t* terminal_out, const dqn_replay_out* replay, int64_t t,
                       void* ws, size_t ws_bytes, void* stream) {
    if (!games || !env_draws || !actions_out || !reward_out || !terminal_out || n_games <= 0) return DQN_EINVAL;
    if (((uintptr_t)games % 16) || (replay && t < 0)) return DQN_EINVAL;
    if (replay) {
        const ReplayOut rp{replay->frames, replay->record_stride, replay->action, replay->reward, replay->terminal,
                           replay->capacity, t};
        if (!replay_ok(rp)) return DQN_EINVAL;
    }
    const int rc = dqn_forward(net, theta, states, n_games, epsilon, eps_draws, nullptr, actions_out, ws, ws_bytes,
                               stream);
    if (rc != DQN_OK) return rc;
    return snake_step(games, n_games, actions_out, env_draws, states, reward_out, terminal_out, replay, t, stream);
}
