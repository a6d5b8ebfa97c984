/*
 * Seeded synthetic game frames for the replay memory.
 *
 * Input generation only: nothing here computes any part of the Q-learning
 * method.  Frames stand in for the paper's preprocessed 84x84 grayscale game
 * screens (Sec. III.A, Sec. V.A): a dark background with uniform noise in
 * 0..8 and one to four bright rectangles (2..4 rows by 4..16 columns,
 * brightness 192..255) that move with a constant velocity in {-2..2}^2 and
 * bounce off the borders.  Noise takes 16 hash bits per pixel, four pixels
 * per hash.  The frame stream is cut into segments of 100
 * frames; each segment draws fresh rectangles.
 *
 * Every byte is a pure function of (seed, frame index t, y, x), so any frame
 * can be regenerated without the rest of the stream.  The hash is SplitMix64's
 * output mix (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014) applied to seed + golden_gamma * counter.
 *
 * synth_side gives hashed side fields (action, reward, terminal) for the
 * same stream, the ones a device-filled replay holds.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC frames.c -o libframes.so
 */
#include <stdint.h>

#define FRAME_H 84
#define FRAME_W 84
#define SEGMENT 100
#define STREAM_RECT 1ull
#define STREAM_NOISE 2ull
#define STREAM_ACT 3ull
#define STREAM_REW 4ull
#define STREAM_TERM 5ull
#define TERM_BELOW 42949672ull   /* floor(0.01 * 2^32): P(terminal) = 0.01 */

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t synth_hash(uint64_t seed, uint64_t stream, uint64_t i) {
    return mix64(seed + 0x9E3779B97F4A7C15ull * ((stream << 40) | i));
}

/* Uniform integer in [0, n) from the top 32 bits of a hash value. */
static inline uint32_t bounded(uint64_t h, uint32_t n) {
    return (uint32_t)(((h >> 32) * (uint64_t)n) >> 32);
}

/* Fold p into [0, L] as a ball bouncing between 0 and L. */
static inline int reflect(int64_t p, int64_t L) {
    if (L <= 0) return 0;
    int64_t period = 2 * L;
    int64_t q = p % period;
    if (q < 0) q += period;
    if (q > L) q = period - q;
    return (int)q;
}

typedef struct { int y, x, h, w, bright; } rect_t;

static int segment_rects(uint64_t seed, int64_t t, rect_t* out) {
    int64_t g = t / SEGMENT;
    int64_t tau = t - g * SEGMENT;
    uint64_t base = (uint64_t)g * 64u;
    int n = 1 + (int)bounded(synth_hash(seed, STREAM_RECT, base), 4);
    for (int r = 0; r < n; ++r) {
        uint64_t f = base + 1u + (uint64_t)r * 8u;
        int h = 2 + (int)bounded(synth_hash(seed, STREAM_RECT, f + 0), 3);
        int w = 4 + (int)bounded(synth_hash(seed, STREAM_RECT, f + 1), 13);
        int br = 192 + (int)bounded(synth_hash(seed, STREAM_RECT, f + 2), 64);
        int y0 = (int)bounded(synth_hash(seed, STREAM_RECT, f + 3), (uint32_t)(FRAME_H - h + 1));
        int x0 = (int)bounded(synth_hash(seed, STREAM_RECT, f + 4), (uint32_t)(FRAME_W - w + 1));
        int vy = (int)bounded(synth_hash(seed, STREAM_RECT, f + 5), 5) - 2;
        int vx = (int)bounded(synth_hash(seed, STREAM_RECT, f + 6), 5) - 2;
        out[r].y = reflect(y0 + (int64_t)vy * tau, FRAME_H - h);
        out[r].x = reflect(x0 + (int64_t)vx * tau, FRAME_W - w);
        out[r].h = h;
        out[r].w = w;
        out[r].bright = br;
    }
    return n;
}

static void one_frame(uint64_t seed, int64_t t, uint8_t* dst) {
    /* background noise for every pixel, then the rectangles on top (the
     * brightest one wins where they overlap) */
    uint64_t quad0 = (uint64_t)t * (uint64_t)(FRAME_H * FRAME_W / 4);
    for (int q = 0; q < FRAME_H * FRAME_W / 4; ++q) {
        uint64_t h = synth_hash(seed, STREAM_NOISE, quad0 + (uint64_t)q);
        for (int k = 0; k < 4; ++k)   /* 16 bits per pixel -> uniform 0..8 */
            dst[4 * q + k] = (uint8_t)((((h >> (16 * k)) & 0xffffu) * 9u) >> 16);
    }
    rect_t rc[4];
    int n = segment_rects(seed, t, rc);
    for (int r = 0; r < n; ++r)
        for (int y = rc[r].y; y < rc[r].y + rc[r].h; ++y)
            for (int x = rc[r].x; x < rc[r].x + rc[r].w; ++x) {
                uint8_t* d = dst + y * FRAME_W + x;
                if (*d < 192 || *d < rc[r].bright) *d = (uint8_t)rc[r].bright;
            }
}

/* Writes frames t0 .. t0+count-1, each 84*84 bytes, back to back into out. */
void synth_frames(uint64_t seed, int64_t t0, int64_t count, uint8_t* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k)
        one_frame(seed, t0 + k, out + k * (int64_t)(FRAME_H * FRAME_W));
}

/* Hashed side fields of records i0 .. i0+count-1: action bounded(H(ACT, i),
 * n_actions), reward bounded(H(REW, i), 3) - 1, terminal iff the top 32
 * bits of H(TERM, i) are below TERM_BELOW. */
void synth_side(uint64_t seed, uint32_t n_actions, int64_t i0, int64_t count, uint8_t* action, int8_t* reward,
                uint8_t* terminal) {
    #pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < count; ++k) {
        const uint64_t i = (uint64_t)(i0 + k);
        action[k] = (uint8_t)bounded(synth_hash(seed, STREAM_ACT, i), n_actions);
        reward[k] = (int8_t)((int)bounded(synth_hash(seed, STREAM_REW, i), 3) - 1);
        terminal[k] = (synth_hash(seed, STREAM_TERM, i) >> 32) < TERM_BELOW ? 1 : 0;
    }
}
