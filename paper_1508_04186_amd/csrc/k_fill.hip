// Seeded synthetic replay contents, written on the device: input generation
// for benchmarks and tests, not part of the method.  A stand-in for a replay
// memory filled with preprocessed game frames (Sec. III.A, Sec. III.C):
// 84 x 84 frames of a dark background (noise uniform on 0..8) with one to
// four bright rectangles (2..4 x 4..16, brightness 192..255) that move with a
// constant velocity in {-2..2}^2 and bounce off the borders; the stream is
// cut into segments of 100 frames, each drawing fresh rectangles.  Record i
// stacks stream frames i .. i+c-1.
//
// Every byte is a pure function of (seed, frame, pixel) through a counter
// hash: SplitMix64's output mix (Steele, Lea and Flood, OOPSLA 2014) of
// seed + golden_gamma * ((stream << 40) | counter), and a bounded draw in
// [0, n) is ((h >> 32) * n) >> 32.  Noise takes 16 bits per pixel, four
// pixels per hash of counter frame * 1764 + quad.  Segment g's rectangles use
// counters 64g (count - 1) and 64g + 1 + 8r + field for rectangle r (fields
// height, width, brightness, start row, start column, row and column
// velocity); where rectangles overlap the brightest wins.  Side fields:
// action = draw(H(3, i), A), reward = draw(H(4, i), 3) - 1, terminal iff the
// top 32 bits of H(5, i) are below floor(0.01 * 2^32).
//
// One workgroup per stream frame: it forms the frame's bytes four at a time
// and writes them to each of the (up to c) records that hold the frame.
#include "common.h"

namespace dqn {
namespace {

constexpr int FL_WG = 256;
constexpr int FL_SIDE = 84;
constexpr int FL_QUADS = FL_SIDE * FL_SIDE / 4;
constexpr uint64_t FL_RECT = 1, FL_NOISE = 2, FL_ACT = 3, FL_REW = 4, FL_TERM = 5;
constexpr uint64_t FL_TERM_BELOW = 42949672ull;

__device__ __forceinline__ uint64_t fl_hash(uint64_t seed, uint64_t stream, uint64_t i) {
    uint64_t z = seed + 0x9E3779B97F4A7C15ull * ((stream << 40) | i);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
__device__ __forceinline__ int fl_draw(uint64_t h, uint32_t n) { return (int)(((h >> 32) * (uint64_t)n) >> 32); }
// p folded into [0, L] (a ball bouncing between 0 and L)
__device__ __forceinline__ int fl_bounce(int64_t p, int64_t L) {
    if (L <= 0) return 0;
    const int64_t period = 2 * L;
    int64_t q = p % period;
    if (q < 0) q += period;
    return (int)(q > L ? period - q : q);
}

__global__ __launch_bounds__(FL_WG) void fill_frames_kernel(uint8_t* frames, int64_t stride, int64_t size, int c,
                                                             uint64_t seed) {
    __shared__ uint64_t s_h[29];
    __shared__ int s_rect[4][5];   // row, column, height, width, brightness
    __shared__ int s_n;
    const int tid = threadIdx.x;
    const int64_t t = blockIdx.x;
    const int64_t g = t / 100, tau = t - g * 100;
    const uint64_t base = (uint64_t)g * 64u;
    if (tid < 29) {
        const uint64_t ctr = tid == 0 ? base : base + 1u + (uint64_t)((tid - 1) / 7) * 8u + (uint64_t)((tid - 1) % 7);
        s_h[tid] = fl_hash(seed, FL_RECT, ctr);
    }
    __syncthreads();
    if (tid == 0) {
        const int n = 1 + fl_draw(s_h[0], 4);
        s_n = n;
        for (int r = 0; r < n; ++r) {
            const uint64_t* f = s_h + 1 + 7 * r;
            const int h = 2 + fl_draw(f[0], 3), w = 4 + fl_draw(f[1], 13), br = 192 + fl_draw(f[2], 64);
            const int y0 = fl_draw(f[3], (uint32_t)(FL_SIDE - h + 1)), x0 = fl_draw(f[4], (uint32_t)(FL_SIDE - w + 1));
            const int vy = fl_draw(f[5], 5) - 2, vx = fl_draw(f[6], 5) - 2;
            s_rect[r][0] = fl_bounce(y0 + (int64_t)vy * tau, FL_SIDE - h);
            s_rect[r][1] = fl_bounce(x0 + (int64_t)vx * tau, FL_SIDE - w);
            s_rect[r][2] = h;
            s_rect[r][3] = w;
            s_rect[r][4] = br;
        }
    }
    __syncthreads();
    const int n = s_n;
    for (int q = tid; q < FL_QUADS; q += FL_WG) {
        const uint64_t hn = fl_hash(seed, FL_NOISE, (uint64_t)t * FL_QUADS + (uint64_t)q);
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p = 4 * q + k, y = p / FL_SIDE, x = p - y * FL_SIDE;
            int v = (int)((((hn >> (16 * k)) & 0xffffu) * 9u) >> 16);
            for (int r = 0; r < n; ++r)
                if (y >= s_rect[r][0] && y < s_rect[r][0] + s_rect[r][2] && x >= s_rect[r][1] &&
                    x < s_rect[r][1] + s_rect[r][3])
                    v = (v < 192 || v < s_rect[r][4]) ? s_rect[r][4] : v;
            word |= (uint32_t)v << (8 * k);
        }
        // frame t is slot k of record t - k
        for (int k = 0; k < c; ++k) {
            const int64_t i = t - k;
            if (i >= 0 && i < size) *(uint32_t*)(frames + i * stride + (int64_t)k * FL_SIDE * FL_SIDE + 4 * q) = word;
        }
    }
}

__global__ void fill_side_kernel(uint8_t* action, int8_t* reward, uint8_t* terminal, int64_t size, int n_actions,
                                 uint64_t seed) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= size) return;
    action[i] = (uint8_t)fl_draw(fl_hash(seed, FL_ACT, (uint64_t)i), (uint32_t)n_actions);
    reward[i] = (int8_t)(fl_draw(fl_hash(seed, FL_REW, (uint64_t)i), 3) - 1);
    terminal[i] = (fl_hash(seed, FL_TERM, (uint64_t)i) >> 32) < FL_TERM_BELOW ? 1 : 0;
}

}  // namespace
}  // namespace dqn

using namespace dqn;

extern "C" int replay_fill_synthetic(const dqn_replay* replay, int32_t n_actions, uint64_t seed, void* stream) {
    if (!replay || !replay->frames || !replay->action || !replay->reward || !replay->terminal) return DQN_EINVAL;
    if (replay->h != FL_SIDE || replay->w != FL_SIDE || replay->c < 1 || replay->size < 1) return DQN_EINVAL;
    if (n_actions < 1 || n_actions > 256) return DQN_EINVAL;
    if ((uintptr_t)replay->frames % 16 || replay->record_stride % 16 ||
        replay->record_stride < (int64_t)replay->c * FL_SIDE * FL_SIDE)
        return DQN_EINVAL;
    const int64_t nframes = replay->size + replay->c - 1;
    if (nframes > 0x7fffffffLL) return DQN_EINVAL;
    hipLaunchKernelGGL(fill_frames_kernel, dim3((unsigned)nframes), dim3(FL_WG), 0, (hipStream_t)stream,
                       (uint8_t*)replay->frames, replay->record_stride, replay->size, replay->c, seed);
    if (hipGetLastError() != hipSuccess) return DQN_EHIP;
    const int64_t blocks = (replay->size + 255) / 256;
    hipLaunchKernelGGL(fill_side_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       (uint8_t*)replay->action, (int8_t*)replay->reward, (uint8_t*)replay->terminal, replay->size,
                       n_actions, seed);
    return hipGetLastError() == hipSuccess ? DQN_OK : DQN_EHIP;
}
