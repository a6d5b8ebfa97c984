// Preprocessing phi of raw RGB screens (Sec. III.A, Fig. 2) and the observe
// step of Alg. 1 for games whose screens come from outside the library
// ("observe frame x_{t+1}, preprocess, store the experience"): phi of each
// game's new screen goes into the newest slot of its four-frame state, and
// the state into the replay memory, in one launch.
//
// phi (readings in include/dqn_actor.h): gray = (299 R + 587 G + 114 B +
// 500) / 1000 per pixel, then the 84F x 84F window at (top, left) averaged
// over F x F blocks with rounding half up.  Integer arithmetic throughout,
// so results are exact.
//
// A workgroup owns a band of R output rows of one screen.  It stages the R*F
// source rows of the window in LDS with 16-byte loads over the aligned cover
// of each row (a row of the window starts at any byte), reduces them from
// LDS, assembles the band's bytes in LDS, and writes 16-byte vectors: the
// band of phi alone, or, for the observe step, the band of all four frames
// of the state (three kept frames shifted down by one, staged in LDS with
// the screen rows so that every read precedes every write) and the same
// band of the replay record, one vector per thread.
#include <cstdint>

#include "common.h"
#include "dqn_actor.h"
#include "dqn_profile.h"

namespace dqn {
namespace {

constexpr int OBW = 256;        // threads per workgroup
constexpr int OFB = 84 * 84;    // bytes per 84 x 84 frame
constexpr int MAX_F = 8;

struct ObsParams {
    const uint8_t* rgb;     // [n][h][w][3]
    int64_t frame_bytes;    // h * w * 3
    int64_t total_bytes;    // n * frame_bytes
    int64_t w3;             // w * 3
    int top, left, bands;
    // phi alone
    uint8_t* out;           // frame i at out + i * out_stride
    int64_t out_stride;
    // observe step
    uint8_t* states;        // [n][4][84][84]
    const int32_t* actions;
    const int8_t* rewards;
    const uint8_t* term;
    ReplayOut rp;
};

// Band height: a multiple of 4 so that a band of a frame is whole 16-byte
// vectors (R * 84 bytes), and small enough that the staged rows fit in LDS.
constexpr int band_rows(int f) { return f <= 3 ? 12 : 4; }
// 16-byte vectors of the aligned cover of a window row (84F * 3 bytes from
// any byte offset).
constexpr int row_vecs(int f) { return (252 * f + 30) / 16; }
constexpr int XCDS = 8;  // workgroups go to the chip's dies round-robin

__device__ __forceinline__ uint32_t gray(uint32_t r, uint32_t g, uint32_t b) {
    return (299u * r + 587u * g + 114u * b + 500u) / 1000u;
}

template <int F, bool OBSERVE>
__global__ __launch_bounds__(OBW) void observe_kernel(ObsParams p, int64_t n) {
    constexpr int R = band_rows(F);
    constexpr int RV = row_vecs(F);
    constexpr int ROWS = R * F;
    constexpr int BV = R * 84 / 16;            // 16-byte vectors per frame band
    constexpr int LOADS = (ROWS * RV + OBW - 1) / OBW;
    static_assert(4 * BV <= OBW, "one vector of the state band per thread");
    extern __shared__ __align__(16) uint4 s_rgb[];             // [ROWS][RV]
    uint8_t* s_new = (uint8_t*)(s_rgb + ROWS * RV);            // [R * 84]
    uint4* s_kept = s_rgb + ROWS * RV + BV;                    // [3][BV]

    // All bands of a game run on one die, so the 16-byte pieces of a cache
    // line that two bands write meet in the same L2.
    const int t = threadIdx.x;
    const int64_t slot = blockIdx.x / XCDS;
    const int64_t e = (slot / p.bands) * XCDS + blockIdx.x % XCDS;
    if (e >= n) return;  // whole workgroup
    const int band = (int)(slot % p.bands);
    const int y0 = band * R;
    const int64_t row0 = e * p.frame_bytes + (int64_t)(p.top + y0 * F) * p.w3 + (int64_t)p.left * 3;

    bool fresh = true;
    uint8_t* st = nullptr;
    uint4 kept = {0, 0, 0, 0};
    if constexpr (OBSERVE) {
        fresh = p.rp.t < 0 || p.term[e] != 0;
        st = p.states + e * 4 * OFB + y0 * 84;
        // the kept frames 1..3 of this band
        if (!fresh && t < 3 * BV) kept = ((const uint4*)(st + (t / BV + 1) * OFB))[t % BV];
    }

    // the aligned cover of every source row; a vector that reaches past the
    // end of the screens is read byte by byte
    uint4 v[LOADS];
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
        const int i = t + u * OBW;
        if (i < ROWS * RV) {
            const int r = i / RV, d = i - r * RV;
            const int64_t a = ((row0 + (int64_t)r * p.w3) & ~(int64_t)15) + 16 * d;
            if (a + 16 <= p.total_bytes) {
                v[u] = *(const uint4*)(p.rgb + a);
            } else {
                uint32_t w[4] = {0, 0, 0, 0};
                for (int b = 0; b < 16; ++b)
                    if (a + b < p.total_bytes) w[b >> 2] |= (uint32_t)p.rgb[a + b] << (8 * (b & 3));
                v[u] = uint4{w[0], w[1], w[2], w[3]};
            }
        }
    }
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
        const int i = t + u * OBW;
        if (i < ROWS * RV) s_rgb[i] = v[u];
    }
    if (OBSERVE && !fresh && t < 3 * BV) s_kept[t] = kept;
    __syncthreads();

    const uint8_t* s_bytes = (const uint8_t*)s_rgb;
    for (int o = t; o < R * 84; o += OBW) {
        const int yl = o / 84, x = o - yl * 84;
        uint32_t sum = 0;
#pragma unroll
        for (int dy = 0; dy < F; ++dy) {
            const int r = yl * F + dy;
            const int shift = (int)((row0 + (int64_t)r * p.w3) & 15);
            const uint8_t* px = s_bytes + r * RV * 16 + shift + 3 * F * x;
#pragma unroll
            for (int dx = 0; dx < F; ++dx) sum += gray(px[3 * dx], px[3 * dx + 1], px[3 * dx + 2]);
        }
        s_new[o] = (uint8_t)((sum + (F * F) / 2) / (F * F));
    }
    __syncthreads();

    if constexpr (!OBSERVE) {
        if (t < BV) ((uint4*)(p.out + e * p.out_stride + y0 * 84))[t] = ((const uint4*)s_new)[t];
    } else {
        // thread t: vector t % BV of frame t / BV of the state band; every
        // load of the band has landed in LDS before the first store
        if (t >= 4 * BV) return;
        const int k = t / BV, q = t - k * BV;
        const uint4 f = (fresh || k == 3) ? ((const uint4*)s_new)[q] : s_kept[t];
        ((uint4*)(st + k * OFB))[q] = f;
        if (p.rp.frames) {
            const int64_t base = e * (p.rp.cap + 1);
            const int64_t rslot = (p.rp.t + 1) % p.rp.cap;
            ((uint4*)(p.rp.frames + (base + rslot) * p.rp.stride + y0 * 84 + k * OFB))[q] = f;
            if (rslot == 0) ((uint4*)(p.rp.frames + (base + p.rp.cap) * p.rp.stride + y0 * 84 + k * OFB))[q] = f;
            if (band == 0 && t == 0 && p.rp.t >= 0) {
                const int64_t i = base + p.rp.t % p.rp.cap;
                p.rp.action[i] = (uint8_t)p.actions[e];
                p.rp.reward[i] = p.rewards[e];
                p.rp.terminal[i] = p.term[e] ? 1 : 0;
            }
        }
    }
}

template <int F, bool OBSERVE>
hipError_t observe_launch(ObsParams prm, int64_t n, hipStream_t st) {
    constexpr int R = band_rows(F);
    const size_t lds = (size_t)R * F * row_vecs(F) * 16 + (size_t)R * 84 + (size_t)3 * R * 84;
    auto kern = observe_kernel<F, OBSERVE>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    prm.bands = 84 / R;
    const int64_t blocks = (n + XCDS - 1) / XCDS * XCDS * prm.bands;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(OBW), lds, st, prm, n);
    return hipGetLastError();
}

template <bool OBSERVE>
hipError_t observe_dispatch(const ObsParams& prm, int f, int64_t n, hipStream_t st) {
    switch (f) {
        case 1: return observe_launch<1, OBSERVE>(prm, n, st);
        case 2: return observe_launch<2, OBSERVE>(prm, n, st);
        case 3: return observe_launch<3, OBSERVE>(prm, n, st);
        case 4: return observe_launch<4, OBSERVE>(prm, n, st);
        case 5: return observe_launch<5, OBSERVE>(prm, n, st);
        case 6: return observe_launch<6, OBSERVE>(prm, n, st);
        case 7: return observe_launch<7, OBSERVE>(prm, n, st);
        case 8: return observe_launch<8, OBSERVE>(prm, n, st);
        default: return hipErrorInvalidValue;
    }
}

// Shared checks of the screen geometry; fills the screen fields of prm.
int screen_args(const uint8_t* rgb, int64_t n, int32_t h, int32_t w, int32_t top, int32_t left, int32_t f,
                ObsParams& prm) {
    if ((!rgb && n > 0) || n < 0 || h < 1 || w < 1 || f < 1 || f > MAX_F || top < 0 || left < 0) return DQN_EINVAL;
    if ((int64_t)top + 84 * f > h || (int64_t)left + 84 * f > w) return DQN_EINVAL;
    if ((uintptr_t)rgb % 16) return DQN_EINVAL;
    const int64_t fb = (int64_t)h * w * 3;
    if (n > 0 && fb > INT64_MAX / n) return DQN_EINVAL;
    // one workgroup per band of a screen; the grid's thread count fits 32 bits
    if ((n + XCDS) * (84 / band_rows(f)) > (int64_t)(UINT32_MAX / OBW)) return DQN_EINVAL;
    prm.rgb = rgb;
    prm.frame_bytes = fb;
    prm.total_bytes = n * fb;
    prm.w3 = (int64_t)w * 3;
    prm.top = top;
    prm.left = left;
    return DQN_OK;
}

bool overlaps(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + (uintptr_t)b_bytes && y < x + (uintptr_t)a_bytes;
}

}  // namespace
}  // namespace dqn

using namespace dqn;

extern "C" int dqn_preprocess(const uint8_t* rgb, int64_t n, int32_t h, int32_t w, int32_t top, int32_t left,
                              int32_t factor, uint8_t* out, int64_t out_stride, void* stream) {
    ObsParams prm{};
    if (screen_args(rgb, n, h, w, top, left, factor, prm) != DQN_OK) return DQN_EINVAL;
    if ((!out && n > 0) || (uintptr_t)out % 16 || out_stride < OFB || out_stride % 16) return DQN_EINVAL;
    if (n == 0) return DQN_OK;
    if (out_stride > (INT64_MAX - OFB) / n) return DQN_EINVAL;
    if (overlaps(rgb, prm.total_bytes, out, (n - 1) * out_stride + OFB)) return DQN_EINVAL;
    prm.out = out;
    prm.out_stride = out_stride;
    prof_mark_begin(DQN_K_OBSERVE, (hipStream_t)stream);
    if (observe_dispatch<false>(prm, factor, n, (hipStream_t)stream) != hipSuccess) return DQN_EHIP;
    prof_mark_end(DQN_K_OBSERVE, (hipStream_t)stream);
    return DQN_OK;
}

extern "C" int dqn_observe(const uint8_t* rgb, int32_t n_games, int32_t h, int32_t w, int32_t top, int32_t left,
                           int32_t factor, const int32_t* actions, const int8_t* rewards, const uint8_t* terminal,
                           uint8_t* states, const dqn_replay_out* replay, int64_t t, void* stream) {
    ObsParams prm{};
    if (n_games <= 0 || t < -1) return DQN_EINVAL;
    if (screen_args(rgb, n_games, h, w, top, left, factor, prm) != DQN_OK) return DQN_EINVAL;
    if (!states || (uintptr_t)states % 16) return DQN_EINVAL;
    if (t >= 0 && !terminal) return DQN_EINVAL;
    if (t >= 0 && replay && (!actions || !rewards)) return DQN_EINVAL;
    if (overlaps(rgb, prm.total_bytes, states, (int64_t)n_games * 4 * OFB)) return DQN_EINVAL;
    ReplayOut rp{};
    if (replay) {
        rp = ReplayOut{replay->frames, replay->record_stride, replay->action, replay->reward, replay->terminal,
                       replay->capacity, t};
        if (!rp.frames || !replay_ok(rp)) return DQN_EINVAL;
    }
    rp.t = t;
    prm.states = states;
    prm.actions = actions;
    prm.rewards = rewards;
    prm.term = terminal;
    prm.rp = rp;
    prof_mark_begin(DQN_K_OBSERVE, (hipStream_t)stream);
    if (observe_dispatch<true>(prm, factor, n_games, (hipStream_t)stream) != hipSuccess) return DQN_EHIP;
    prof_mark_end(DQN_K_OBSERVE, (hipStream_t)stream);
    return DQN_OK;
}
