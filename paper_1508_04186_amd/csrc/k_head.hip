// Output head of the Q-network and the TD step of Alg. 1, one workgroup per
// sample: reduce the fc1 split-K partials, add the bias and apply ReLU, run
// the linear output layer with a block reduction, then either
//   (td)  form y = r (terminal) or r + gamma * max_a' Q(s', a'; theta^-),
//         the residual delta = (Q(s, a) - y) / B, the per-sample loss term
//         and the fc1 pre-activation gradient delta * W2[a, :] * [z1 > 0];
//   (fwd) pick the greedy action (lowest index of the maximum) or, with
//         epsilon-greedy exploration, the caller-drawn random action.
// The finalize kernel then reduces everything that sums over samples or over
// wgrad chunks in a fixed order (no atomics), so results are deterministic.
#include <algorithm>

#include "common.h"

namespace dqn {
namespace {

constexpr int HT = 256;  // threads per head workgroup

// Sum of n strided values split over the 8 lanes of an aligned lane group:
// lane q of the group takes terms c = 16*(8*i + q) + u into partial sum
// u % 4 (missing tail terms count as +0), and the group combines its lanes'
// sums in a fixed butterfly order.  Every lane of the group gets the result.
__device__ __forceinline__ float sum_strided_x8(const float* __restrict__ x, int n, int64_t stride) {
    const int q = threadIdx.x & 7;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 16 * q; c < n; c += 128) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = (c + u < n) ? x[(int64_t)(c + u) * stride] : 0.f;
#pragma unroll
        for (int u = 0; u < 16; ++u) s[u & 3] += v[u];
    }
    float t = (s[0] + s[1]) + (s[2] + s[3]);
    t += __shfl_xor(t, 1, 64);
    t += __shfl_xor(t, 2, 64);
    t += __shfl_xor(t, 4, 64);
    return t;
}

// Block-wide sums of NV per-thread values; every thread gets the results.
// Wave sums first (by halving: per value the butterfly order of wave_sum,
// NV + 6 shuffles instead of 6 NV; batch 32, head 6.8 us, most of it the
// chain of 12 wave sums), then the four wave results in wave order.
template <int NV>
__device__ __forceinline__ void block_sums(float (&v)[NV], float* red /* [4][NV] */) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float s = halving_step<NV, 32>(v, lane);
    const int i = halving_index<NV>(lane);
    if (i >= 0) red[wave * NV + i] = s;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] = (red[k] + red[NV + k]) + (red[2 * NV + k] + red[3 * NV + k]);
}

// Sum of the ks split-K slices of NR rows of the fc1 partial sums
// (row r at fc1p + rows[r]*H, slice z at + z*slice).  Thread t adds, for the
// four hidden units 4q..4q+3 (q = t mod H/4), the slices congruent to
// t / (H/4) modulo G = 1024/H in increasing order, with up to 12 slices per
// row in flight; the G group sums are then added in group order through LDS.
// Thread t receives hidden units t + 256e in out[r][e].
template <int H, int NR>
__device__ __forceinline__ void reduce_slices(const float* __restrict__ fc1p, const int64_t (&rows)[NR],
                                              int ks, int64_t slice, float* red /* [NR][G][H] */,
                                              float (&out)[NR][H / HT]) {
    constexpr int Q = H / 4, G = HT / Q, U = 12;
    static_assert(HT % Q == 0, "hidden width must divide 1024");
    const int q = threadIdx.x % Q, sg = threadIdx.x / Q;
    f4 acc[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) acc[r] = f4{0.f, 0.f, 0.f, 0.f};
    for (int z0 = sg; z0 < ks; z0 += U * G) {
        f4 v[NR][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int z = z0 + u * G;
#pragma unroll
            for (int r = 0; r < NR; ++r)
                v[r][u] = z < ks ? *(const f4*)(fc1p + (int64_t)z * slice + rows[r] * H + 4 * q)
                                 : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < NR; ++r) acc[r] += v[r][u];
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) *(f4*)&red[(r * G + sg) * H + 4 * q] = acc[r];
    __syncthreads();
#pragma unroll
    for (int e = 0; e < H / HT; ++e) {
        const int h = threadIdx.x + HT * e;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            float x = red[(r * G) * H + h];
#pragma unroll
            for (int k = 1; k < G; ++k) x += red[(r * G + k) * H + h];
            out[r][e] = x;
        }
    }
}

template <int H, int A>
__global__ __launch_bounds__(HT) void head_td_kernel(HeadTdArgs p) {
    constexpr int E = H / HT;
    __shared__ __align__(16) float sred[2 * 1024];
    __shared__ float red[4 * 2 * A];
    const int j = blockIdx.x;
    const int B = p.B;
    const int64_t slice = (int64_t)2 * B * H;
    // Everything else this workgroup reads is loaded before the slice
    // reduction, so that all of it is in flight together.  An action outside
    // [0, A) is clamped so it can never select a row outside W2.
    const int act = min(max(p.action[j], 0), A - 1);
    const float r = p.reward[j];
    const bool term = p.terminal[j] != 0;
    float b1v[E], b1tv[E], w2[A][E], w2t[A][E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = threadIdx.x + HT * e;
        b1v[e] = p.b1[h];
        b1tv[e] = p.b1t[h];
#pragma unroll
        for (int k = 0; k < A; ++k) {
            w2[k][e] = p.W2[k * H + h];
            w2t[k][e] = p.W2t[k * H + h];
        }
    }
    float zs[E], hs[E], v[2 * A];
#pragma unroll
    for (int k = 0; k < 2 * A; ++k) v[k] = 0.f;
    float sums[2][E];
    const int64_t rows[2] = {j, B + j};
    reduce_slices<H, 2>(p.fc1p, rows, p.ks, slice, sred, sums);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        zs[e] = sums[0][e] + b1v[e];
        hs[e] = fmaxf(zs[e], 0.f);
        const float hn = fmaxf(sums[1][e] + b1tv[e], 0.f);
#pragma unroll
        for (int k = 0; k < A; ++k) {
            v[k] = fmaf(w2[k][e], hs[e], v[k]);
            v[A + k] = fmaf(w2t[k][e], hn, v[A + k]);
        }
    }
    block_sums<2 * A>(v, red);
    float m = v[A] + p.b2t[0];
#pragma unroll
    for (int k = 1; k < A; ++k) m = fmaxf(m, v[A + k] + p.b2t[k]);
    const float y = term ? r : fmaf(p.gamma, m, r);
    float qa = v[0] + p.b2[0];
#pragma unroll
    for (int k = 1; k < A; ++k) qa = (k == act) ? v[k] + p.b2[k] : qa;
    const float diff = qa - y;
    const float delta = diff / (float)B;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = threadIdx.x + HT * e;
        float wa = w2[0][e];
#pragma unroll
        for (int k = 1; k < A; ++k) wa = (k == act) ? w2[k][e] : wa;
        const float d = zs[e] > 0.f ? delta * wa : 0.f;
        p.h1s[(int64_t)j * H + h] = hs[e];
        p.dz1[(int64_t)j * H + h] = d;
        if (p.dz1h) p.dz1h[(int64_t)j * H + h] = (__bf16)d;
    }
    if (threadIdx.x == 0) {
        p.delta[j] = delta;
        p.lossj[j] = 0.5f * diff * diff / (float)B;
        if (p.y_out) p.y_out[j] = y;
    }
    if (p.q_out && threadIdx.x < A) {
        float q = v[0];
#pragma unroll
        for (int k = 1; k < A; ++k) q = (k == (int)threadIdx.x) ? v[k] : q;
        p.q_out[(int64_t)j * A + threadIdx.x] = q + p.b2[threadIdx.x];
    }
}


// The TD head for large batches: one wave per sample, lane l owning the
// hidden units 4l + 256e .. +3 (float4 loads and stores).  A workgroup first
// issues the loads of its first samples' fc1 slices, then stages both fc2
// weight sets in LDS, so the two are in flight together; slices are summed
// in slice order, KG of them loaded at once.  The 2A fc2 outputs of a sample are
// summed over the wave with halving_step; the maximum over a' and Q(s, a)
// are then read across lanes.  Same arithmetic per sample as head_td_kernel
// up to the association of the hidden-unit sums.
constexpr int kHeadWideWaves = 4;
template <int H, int A>
__global__ __launch_bounds__(64 * kHeadWideWaves) void head_td_wide_kernel(HeadTdArgs p) {
    constexpr int E = H / 256, KG = 4;
    static_assert(H % 256 == 0 && 2 * A <= 64, "head shape");
    extern __shared__ __align__(16) float s_w2[];   // [2][A][H]: W2, then W2t
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int B = p.B;
    const int64_t slice = (int64_t)2 * B * H;
    const int stride = gridDim.x * kHeadWideWaves;
    int j = blockIdx.x * kHeadWideWaves + w;
    f4 a[KG][E], b[KG][E];
    auto load_group = [&](int jj, int z0) {
#pragma unroll
        for (int g = 0; g < KG; ++g)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const bool ok = z0 + g < p.ks;
                const float* sl = p.fc1p + (int64_t)(z0 + g) * slice + 4 * lane + 256 * e;
                a[g][e] = ok ? *(const f4*)(sl + (int64_t)jj * H) : f4{0.f, 0.f, 0.f, 0.f};
                b[g][e] = ok ? *(const f4*)(sl + (int64_t)(B + jj) * H) : f4{0.f, 0.f, 0.f, 0.f};
            }
    };
    if (j < B) load_group(j, 0);
    for (int i = threadIdx.x; i < A * H / 4; i += 64 * kHeadWideWaves) {
        ((f4*)s_w2)[i] = ((const f4*)p.W2)[i];
        ((f4*)s_w2)[A * H / 4 + i] = ((const f4*)p.W2t)[i];
    }
    f4 b1v[E], b1tv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        b1v[e] = *(const f4*)(p.b1 + 4 * lane + 256 * e);
        b1tv[e] = *(const f4*)(p.b1t + 4 * lane + 256 * e);
    }
    const int my = halving_index<2 * A>(lane);
    const float b2my = my >= 0 && my < A ? p.b2[my] : 0.f;
    const float b2tmy = my >= A ? p.b2t[my - A] : 0.f;
    __syncthreads();
    const float* W2 = s_w2;
    const float* W2t = s_w2 + A * H;
    for (; j < B; j += stride) {
        if (j != blockIdx.x * kHeadWideWaves + w) load_group(j, 0);   // (beyond the first pass)
        f4 zs[E], zn[E];
#pragma unroll
        for (int e = 0; e < E; ++e) zs[e] = zn[e] = f4{0.f, 0.f, 0.f, 0.f};
        for (int z0 = 0;;) {
#pragma unroll
            for (int g = 0; g < KG; ++g)
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    zs[e] += a[g][e];
                    zn[e] += b[g][e];
                }
            z0 += KG;
            if (z0 >= p.ks) break;
            load_group(j, z0);
        }
        const int act = min(max(p.action[j], 0), A - 1);
        const float r = p.reward[j];
        const bool term = p.terminal[j] != 0;
        f4 hs[E];
        float v[2 * A];
#pragma unroll
        for (int k = 0; k < 2 * A; ++k) v[k] = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int h = 4 * lane + 256 * e;
            zs[e] += b1v[e];
            f4 hn;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                hs[e][c] = fmaxf(zs[e][c], 0.f);
                hn[c] = fmaxf(zn[e][c] + b1tv[e][c], 0.f);
            }
#pragma unroll
            for (int k = 0; k < A; ++k) {
                const f4 wk = *(const f4*)&W2[k * H + h];
                const f4 wt = *(const f4*)&W2t[k * H + h];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    v[k] = fmaf(wk[c], hs[e][c], v[k]);
                    v[A + k] = fmaf(wt[c], hn[c], v[A + k]);
                }
                // (keeps the compiler from hoisting every weight read at once)
                if (k % 4 == 3) __builtin_amdgcn_sched_barrier(0);
            }
        }
        const float sum = halving_step<2 * A, 32>(v, lane);
        // max over a' of Q(s', a'; theta^-): the lanes holding values A..2A-1
        float m = my >= A ? sum + b2tmy : -INFINITY;
#pragma unroll
        for (int msk = 32; msk >= 1; msk >>= 1) m = fmaxf(m, __shfl_xor(m, msk, 64));
        // Q(s, a): read from the lane holding value act
        const uint64_t at = __ballot(my == act);
        const float qa = __shfl(sum, __ffsll((unsigned long long)at) - 1, 64) + p.b2[act];
        const float y = term ? r : fmaf(p.gamma, m, r);
        const float diff = qa - y;
        const float delta = diff / (float)B;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int h = 4 * lane + 256 * e;
            const f4 wa = *(const f4*)&W2[act * H + h];
            f4 d;
#pragma unroll
            for (int c = 0; c < 4; ++c) d[c] = zs[e][c] > 0.f ? delta * wa[c] : 0.f;
            *(f4*)&p.h1s[(int64_t)j * H + h] = hs[e];
            *(f4*)&p.dz1[(int64_t)j * H + h] = d;
            if (p.dz1h) {
                uint32_t u[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) u[c] = __builtin_bit_cast(unsigned short, (__bf16)d[c]);
                *(uint2*)&p.dz1h[(int64_t)j * H + h] = uint2{u[0] | (u[1] << 16), u[2] | (u[3] << 16)};
            }
        }
        if (lane == 0) {
            p.delta[j] = delta;
            p.lossj[j] = 0.5f * diff * diff / (float)B;
            if (p.y_out) p.y_out[j] = y;
        }
        if (p.q_out && my >= 0 && my < A) p.q_out[(int64_t)j * A + my] = sum + b2my;
    }
}

template <int H, int A>
__global__ __launch_bounds__(HT) void head_fwd_kernel(HeadFwdArgs p) {
    constexpr int E = H / HT;
    __shared__ __align__(16) float sred[1024];
    __shared__ float red[4 * A];
    const int j = blockIdx.x;
    const int64_t slice = (int64_t)p.B * H;
    float v[A];
#pragma unroll
    for (int k = 0; k < A; ++k) v[k] = 0.f;
    float sums[1][E];
    const int64_t rows[1] = {j};
    reduce_slices<H, 1>(p.fc1p, rows, p.ks, slice, sred, sums);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = threadIdx.x + HT * e;
        const float hs = fmaxf(sums[0][e] + p.b1[h], 0.f);
#pragma unroll
        for (int k = 0; k < A; ++k) v[k] = fmaf(p.W2[k * H + h], hs, v[k]);
    }
    block_sums<A>(v, red);
    float q[A];
#pragma unroll
    for (int k = 0; k < A; ++k) q[k] = v[k] + p.b2[k];
    int best = 0;
    float bq = q[0];
#pragma unroll
    for (int k = 1; k < A; ++k)
        if (q[k] > bq) {
            bq = q[k];
            best = k;
        }
    if (p.thresh > 0) {
        const uint64_t w = p.draws[j];
        if ((w >> 32) < p.thresh) best = (int)(((w & 0xffffffffull) * (uint64_t)A) >> 32);
    }
    if (threadIdx.x == 0 && p.action_out) p.action_out[j] = best;
    if (p.q_out && threadIdx.x < A) {
        float o = q[0];
#pragma unroll
        for (int k = 1; k < A; ++k) o = (k == (int)threadIdx.x) ? q[k] : o;
        p.q_out[(int64_t)j * A + threadIdx.x] = o;
    }
}

// The forward head for large batches, laid out as head_td_wide_kernel: one
// wave per state, the A outputs summed over the wave by halving, then the
// greedy action (lowest index of the maximum, for finite Q) by a wave
// reduction over (value, index) pairs, replaced by the caller-drawn action
// where the state explores.
template <int H, int A>
__global__ __launch_bounds__(64 * kHeadWideWaves) void head_fwd_wide_kernel(HeadFwdArgs p) {
    constexpr int E = H / 256, KG = 4;
    static_assert(H % 256 == 0 && A <= 64, "head shape");
    extern __shared__ __align__(16) float s_w2[];   // [A][H]
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int B = p.B;
    const int64_t slice = (int64_t)B * H;
    const int stride = gridDim.x * kHeadWideWaves;
    const int j0 = blockIdx.x * kHeadWideWaves + w;
    f4 a[KG][E];
    auto load_group = [&](int jj, int z0) {
#pragma unroll
        for (int g = 0; g < KG; ++g)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float* sl = p.fc1p + (int64_t)(z0 + g) * slice + (int64_t)jj * H + 4 * lane + 256 * e;
                a[g][e] = z0 + g < p.ks ? *(const f4*)sl : f4{0.f, 0.f, 0.f, 0.f};
            }
    };
    if (j0 < B) load_group(j0, 0);
    for (int i = threadIdx.x; i < A * H / 4; i += 64 * kHeadWideWaves) ((f4*)s_w2)[i] = ((const f4*)p.W2)[i];
    f4 b1v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) b1v[e] = *(const f4*)(p.b1 + 4 * lane + 256 * e);
    const int my = halving_index<A>(lane);
    const float b2my = my >= 0 ? p.b2[my] : 0.f;
    __syncthreads();
    for (int j = j0; j < B; j += stride) {
        if (j != j0) load_group(j, 0);   // (beyond the first pass)
        f4 zs[E];
#pragma unroll
        for (int e = 0; e < E; ++e) zs[e] = f4{0.f, 0.f, 0.f, 0.f};
        for (int z0 = 0;;) {
#pragma unroll
            for (int g = 0; g < KG; ++g)
#pragma unroll
                for (int e = 0; e < E; ++e) zs[e] += a[g][e];
            z0 += KG;
            if (z0 >= p.ks) break;
            load_group(j, z0);
        }
        float v[A];
#pragma unroll
        for (int k = 0; k < A; ++k) v[k] = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int h = 4 * lane + 256 * e;
            f4 hs;
#pragma unroll
            for (int c = 0; c < 4; ++c) hs[c] = fmaxf(zs[e][c] + b1v[e][c], 0.f);
#pragma unroll
            for (int k = 0; k < A; ++k) {
                const f4 wk = *(const f4*)&s_w2[k * H + h];
#pragma unroll
                for (int c = 0; c < 4; ++c) v[k] = fmaf(wk[c], hs[c], v[k]);
                if (k % 8 == 7) __builtin_amdgcn_sched_barrier(0);
            }
        }
        const float q = halving_step<A, 32>(v, lane) + b2my;
        float bq = my >= 0 ? q : -INFINITY;
        int bi = my >= 0 ? my : A;
#pragma unroll
        for (int msk = 32; msk >= 1; msk >>= 1) {
            const float ov = __shfl_xor(bq, msk, 64);
            const int oi = __shfl_xor(bi, msk, 64);
            if (ov > bq || (ov == bq && oi < bi)) {
                bq = ov;
                bi = oi;
            }
        }
        int best = bi;
        if (p.thresh > 0) {
            const uint64_t d = p.draws[j];
            if ((d >> 32) < p.thresh) best = (int)(((d & 0xffffffffull) * (uint64_t)A) >> 32);
        }
        if (lane == 0 && p.action_out) p.action_out[j] = best;
        if (p.q_out && my >= 0) p.q_out[(int64_t)j * A + my] = q;
    }
}

// Each output's terms are summed in a fixed association, without atomics.
// Up to 128 samples, finalize_small_kernel below.  Above, two launches:
//  - sample_partials_kernel: for chunks of 32 samples, the chunk's sums of
//    the fc2 weight gradient (delta_j * h1[j][h] added to the sum of the
//    action j took), the fc1 bias gradient, the fc2 bias gradient and the
//    loss, into one partial-sum slot per chunk.  A workgroup takes 64 hidden
//    units of a chunk, so its loads are 256-byte rows;
//  - finalize_wide_kernel: four lanes per output (sixteen consecutive
//    outputs per wave, so every load is four 64-byte row pieces), lane q
//    summing slots q, q + 4, ... in order, then the four lane sums by a
//    butterfly: the conv weight and bias gradients over the wgrad
//    partial-sum slots, then the sample sums over the chunk slots.  With
//    one lane per output, 256 slots took eight dependent rounds of 32 loads.
//
// MODE < 0 stores the gradient; MODE = 0, 1, 2 applies update rule MODE to
// each parameter instead (fused parameter-server update), and the blocks
// from n_fin on update the fc1 weights from the gradient stored there.
template <int MODE>
__device__ __forceinline__ void emit(const FinalizeArgs& a, const PsUpdate& u, float* dst, float v) {
    if constexpr (MODE < 0) {
        *dst = v;
    } else {
        const int64_t off = dst - a.grad_base;
        float th = u.theta[off], sv = MODE != 0 ? u.state[off] : 0.f;
        ps_update<MODE>(th, sv, v, u.lr, u.decay, u.eps);
        u.theta[off] = th;
        if constexpr (MODE != 0) u.state[off] = sv;
    }
}

// The fc1 weights, four per thread: the gradient stored (MODE < 0, only
// with slices to add) or applied; with fc1w_part, the slices' sum in slice
// order.
template <int MODE>
__device__ __forceinline__ void apply_fc1w(const FinalizeArgs& a, const PsUpdate& u, int64_t i4) {
    if (i4 >= a.fc1w_count / 4) return;
    const int64_t off = a.fc1w_off + 4 * i4;
    f4 gv;
    if (a.fc1w_part) {
        gv = *(const f4*)(a.fc1w_part + 4 * i4);
        for (int z = 1; z < a.fc1w_slices; ++z) gv += *(const f4*)(a.fc1w_part + (int64_t)z * a.fc1w_count + 4 * i4);
        if constexpr (MODE < 0) {
            *(f4*)(const_cast<float*>(a.grad_base) + off) = gv;
            return;
        }
    } else {
        gv = *(const f4*)(a.grad_base + off);
    }
    if constexpr (MODE < 0) return;   // (no slices: the gradient is already in place)
    f4 th = *(const f4*)(u.theta + off);
    f4 sv = f4{0.f, 0.f, 0.f, 0.f};
    if constexpr (MODE != 0) sv = *(const f4*)(u.state + off);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float t = th[r], s = sv[r];
        ps_update<MODE>(t, s, gv[r], u.lr, u.decay, u.eps);
        th[r] = t;
        sv[r] = s;
    }
    *(f4*)(u.theta + off) = th;
    if constexpr (MODE != 0) *(f4*)(u.state + off) = sv;
}

// Actions outside [0, A) count as the nearest valid one, as in the head.
__device__ __forceinline__ int clamp_action(int a, int A) { return min(max(a, 0), A - 1); }

// The layout for small batches (up to 128 samples): eight lanes per output
// throughout, in segment order conv weights and biases, fc1 bias, fc2
// weights (per action and hidden unit, over the samples that took the
// action), fc2 bias, loss.  Measured faster than the wave-per-output sums at
// batch 32 (6.6 against 7.1 us under rocprofv3).
template <int MODE>
__global__ __launch_bounds__(256) void finalize_small_kernel(FinalizeArgs a, PsUpdate u, int n_fin) {
    if ((int)blockIdx.x >= n_fin) {   // (launched for MODE < 0 only with slices to add)
        apply_fc1w<MODE>(a, u, (int64_t)(blockIdx.x - n_fin) * 256 + threadIdx.x);
        return;
    }
    int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 3;
    const bool lead = (threadIdx.x & 7) == 0;
    for (int l = 0; l < a.n_conv; ++l) {
        if (i < a.wcount[l]) {
            const float v = sum_strided_x8(a.wpart[l] + i, a.chunks[l], a.wcount[l]);
            if (lead) emit<MODE>(a, u, a.gw[l] + i, v);
            return;
        }
        i -= a.wcount[l];
        if (i < a.cout[l]) {
            const float v = sum_strided_x8(a.bpart[l] + i, a.chunks[l], a.cout[l]);
            if (lead) emit<MODE>(a, u, a.gb[l] + i, v);
            return;
        }
        i -= a.cout[l];
    }
    if (i < a.H) {
        const float v = sum_strided_x8(a.dz1 + i, a.B, a.H);
        if (lead) emit<MODE>(a, u, a.g_b1 + i, v);
        return;
    }
    i -= a.H;
    if (i < (int64_t)a.A * a.H) {
        const int k = (int)(i / a.H), h = (int)(i - (int64_t)k * a.H);
        const int q = threadIdx.x & 7;
        float s0 = 0.f, s1 = 0.f;
        // every load issued before the action test that selects it (an index
        // past the batch reads sample j and is not added)
#pragma unroll 4
        for (int j = q; j < a.B; j += 16) {
            const int jb = j + 8 < a.B ? j + 8 : j;
            const int a0 = a.action[j], a1 = a.action[jb];
            const float d0 = a.delta[j], d1 = a.delta[jb];
            const float h0 = a.h1s[(int64_t)j * a.H + h], h1 = a.h1s[(int64_t)jb * a.H + h];
            const float t0 = clamp_action(a0, a.A) == k ? d0 * h0 : 0.f;
            const float t1 = (j + 8 < a.B && clamp_action(a1, a.A) == k) ? d1 * h1 : 0.f;
            s0 += t0;
            s1 += t1;
        }
        float t = s0 + s1;
        t += __shfl_xor(t, 1, 64);
        t += __shfl_xor(t, 2, 64);
        t += __shfl_xor(t, 4, 64);
        if (lead) emit<MODE>(a, u, a.g_W2 + i, t);
        return;
    }
    i -= (int64_t)a.A * a.H;
    if (i < a.A) {
        const int q = threadIdx.x & 7;
        float s = 0.f;
#pragma unroll 4
        for (int j = q; j < a.B; j += 8) {
            const int aj = a.action[j];
            const float dj = a.delta[j];
            s += clamp_action(aj, a.A) == (int)i ? dj : 0.f;
        }
        s += __shfl_xor(s, 1, 64);
        s += __shfl_xor(s, 2, 64);
        s += __shfl_xor(s, 4, 64);
        if (lead) emit<MODE>(a, u, a.g_b2 + i, s);
        return;
    }
    i -= a.A;
    if (i == 0) {
        const float v = sum_strided_x8(a.lossj, a.B, 1);
        if (lead) a.loss_out[0] = v;
    }
}

// Chunk c of 32 samples, hidden units 64 bx .. 64 bx + 63 (one per lane);
// wave w takes samples 32c + w + 4i in order, the four wave sums are added
// in wave order.  Block x = 0 also forms the chunk's fc2 bias gradient and
// loss (lane = sample, fixed butterfly).  Slot layout: fc2 weights [A][H],
// fc1 bias [H], fc2 bias [A], loss.
constexpr int SP_CHUNK = 32;
template <int A>
__global__ __launch_bounds__(256) void sample_partials_kernel(FinalizeArgs a) {
    __shared__ float red[4][A + 1][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int h = blockIdx.x * 64 + lane;
    const int c = blockIdx.y;
    const int j0 = c * SP_CHUNK, j1 = min(a.B, j0 + SP_CHUNK);
    const int64_t count = (int64_t)A * a.H + a.H + A + 1;
    float* slot = a.spart + (int64_t)c * count;
    float sw[A], sb = 0.f;
#pragma unroll
    for (int k = 0; k < A; ++k) sw[k] = 0.f;
    // Every load of the eight samples is issued before the first use (an
    // index past the chunk reads sample j0 and is not added), so the loads
    // are one round trip instead of eight dependent ones.
    constexpr int NS = SP_CHUNK / 4;
    int acts[NS];
    float dl[NS], hv[NS], zv[NS];
#pragma unroll
    for (int i = 0; i < NS; ++i) {
        const int j = j0 + w + 4 * i;
        const int jc = j < j1 ? j : j0;
        acts[i] = a.action[jc];
        dl[i] = a.delta[jc];
        hv[i] = a.h1s[(int64_t)jc * a.H + h];
        zv[i] = a.dz1[(int64_t)jc * a.H + h];
    }
#pragma unroll
    for (int i = 0; i < NS; ++i) {
        if (j0 + w + 4 * i < j1) {
            const int act = clamp_action(acts[i], A);
            const float d = dl[i] * hv[i];
#pragma unroll
            for (int k = 0; k < A; ++k) sw[k] += act == k ? d : 0.f;
            sb += zv[i];
        }
    }
#pragma unroll
    for (int k = 0; k < A; ++k) red[w][k][lane] = sw[k];
    red[w][A][lane] = sb;
    __syncthreads();
    if (w == 0) {
#pragma unroll
        for (int k = 0; k <= A; ++k) {
            const float v = ((red[0][k][lane] + red[1][k][lane]) + red[2][k][lane]) + red[3][k][lane];
            slot[(k < A ? (int64_t)k * a.H : (int64_t)A * a.H) + h] = v;
        }
    } else if (w == 1 && blockIdx.x == 0) {
        // the A fc2 bias sums and the loss (slot entries A*H + H + i, i <= A)
        // by halving over the wave: the same butterfly order per value as
        // A + 1 wave sums, in 22 shuffles instead of 114 (batch 256: this
        // kernel 7.9 us, most of it the chain of wave sums)
        const int j = j0 + lane;
        const bool v = lane < SP_CHUNK && j < j1;
        const int act = v ? clamp_action(a.action[j], A) : -1;
        const float d = v ? a.delta[j] : 0.f;
        float vals[A + 1];
#pragma unroll
        for (int k = 0; k < A; ++k) vals[k] = act == k ? d : 0.f;
        vals[A] = v ? a.lossj[j] : 0.f;
        const float t = halving_step<A + 1, 32>(vals, lane);
        const int i = halving_index<A + 1>(lane);
        if (i >= 0) slot[(int64_t)A * a.H + a.H + i] = t;
    }
}

constexpr int FW_U = 32;   // slots in flight per lane
constexpr int FW_L = 4;    // lanes per output
template <int MODE>
__global__ __launch_bounds__(256) void finalize_wide_kernel(FinalizeArgs a, PsUpdate u, int n_fin) {
    if ((int)blockIdx.x >= n_fin) {   // (launched for MODE < 0 only with slices to add)
        apply_fc1w<MODE>(a, u, (int64_t)(blockIdx.x - n_fin) * 256 + threadIdx.x);
        return;
    }
    // FW_L consecutive lanes share an output (a group exits or stays as one)
    const int ql = threadIdx.x & (FW_L - 1);
    int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) / FW_L;
    const float* part = nullptr;
    int64_t count = 0;
    int slots = 0;
    float* dst = nullptr;
    bool loss = false;
    for (int l = 0; l < a.n_conv && !part; ++l) {
        if (i < a.wcount[l]) {
            part = a.wpart[l] + i, count = a.wcount[l], slots = a.chunks[l], dst = a.gw[l] + i;
        } else if ((i -= a.wcount[l]) < a.cout[l]) {
            part = a.bpart[l] + i, count = a.cout[l], slots = a.chunks[l], dst = a.gb[l] + i;
        } else {
            i -= a.cout[l];
        }
    }
    if (!part) {
        const int64_t wh = (int64_t)a.A * a.H, cs = wh + a.H + a.A + 1;
        if (i >= cs) return;
        part = a.spart + i, count = cs, slots = a.schunks;
        if (i < wh) dst = a.g_W2 + i;
        else if (i < wh + a.H) dst = a.g_b1 + (i - wh);
        else if (i < wh + a.H + a.A) dst = a.g_b2 + (i - wh - a.H);
        else loss = true;
    }
    // lane ql of the group sums slots ql, ql + FW_L, ... in order; the
    // group's lane sums are then combined by a butterfly, which gives every
    // lane the same value (float addition is commutative)
    float s = 0.f;
    for (int q = ql; q < slots; q += FW_L * FW_U) {
        float v[FW_U];
#pragma unroll
        for (int e = 0; e < FW_U; ++e) {
            const int z = q + FW_L * e;
            v[e] = z < slots ? part[(int64_t)z * count] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < FW_U; ++e) s += v[e];
    }
    static_assert(FW_L == 4, "two butterfly steps");
    s += __shfl_xor(s, 1, 64);
    s += __shfl_xor(s, 2, 64);
    if (ql != 0) return;
    if (loss) a.loss_out[0] = s;
    else emit<MODE>(a, u, dst, s);
}

// From kHeadWideRows samples on, the wide heads (one wave per sample);
// below, one workgroup per sample is faster.
constexpr int kHeadWideRows = 128;
template <int H, int A>
hipError_t td_launch(const HeadTdArgs& a, hipStream_t st) {
    if (a.B >= kHeadWideRows) {
        for (const float* x : {a.fc1p, a.b1, a.b1t, a.W2, a.W2t, (const float*)a.h1s, (const float*)a.dz1})
            if ((uintptr_t)x & 15) return hipErrorInvalidValue;
        // one sample per wave; beyond 1024 workgroups the waves loop
        const int blocks = std::min(1024, (a.B + kHeadWideWaves - 1) / kHeadWideWaves);
        constexpr size_t lds = (size_t)2 * A * H * 4;
        auto kern = head_td_wide_kernel<H, A>;
        if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * kHeadWideWaves), lds, st, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((head_td_kernel<H, A>), dim3((unsigned)a.B), dim3(HT), 0, st, a);
    return hipGetLastError();
}

template <int H, int A>
hipError_t fwd_launch(const HeadFwdArgs& a, hipStream_t st) {
    if (a.B >= kHeadWideRows) {
        for (const float* x : {a.fc1p, a.b1, a.W2})
            if ((uintptr_t)x & 15) return hipErrorInvalidValue;
        const int blocks = std::min(1024, (a.B + kHeadWideWaves - 1) / kHeadWideWaves);
        constexpr size_t lds = (size_t)A * H * 4;
        auto kern = head_fwd_wide_kernel<H, A>;
        if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * kHeadWideWaves), lds, st, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((head_fwd_kernel<H, A>), dim3((unsigned)a.B), dim3(HT), 0, st, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_head_td(int H, int A, const HeadTdArgs& a, hipStream_t st) {
    if (H == 256 && A == 6) return td_launch<256, 6>(a, st);
    if (H == 512 && A == 18) return td_launch<512, 18>(a, st);
    return hipErrorInvalidValue;
}

hipError_t launch_head_fwd(int H, int A, const HeadFwdArgs& a, hipStream_t st) {
    if (H == 256 && A == 6) return fwd_launch<256, 6>(a, st);
    if (H == 512 && A == 18) return fwd_launch<512, 18>(a, st);
    return hipErrorInvalidValue;
}

template <int A>
hipError_t finalize_wide_launch(const FinalizeArgs& a, const PsUpdate* upd, hipStream_t st) {
    if (!a.spart || a.schunks != (a.B + SP_CHUNK - 1) / SP_CHUNK || a.H % 64) return hipErrorInvalidValue;
    hipLaunchKernelGGL(sample_partials_kernel<A>, dim3((unsigned)(a.H / 64), (unsigned)a.schunks), dim3(256), 0, st,
                       a);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    int64_t total = (int64_t)A * a.H + a.H + A + 1;
    for (int l = 0; l < a.n_conv; ++l) total += a.wcount[l] + a.cout[l];
    const int n_fin = (int)((total * FW_L + 255) / 256);
    if ((upd || a.fc1w_part) && (a.fc1w_off % 4 != 0 || a.fc1w_count % 4 != 0 || !a.grad_base))
        return hipErrorInvalidValue;
    const int n_w = upd || a.fc1w_part ? (int)((a.fc1w_count / 4 + 255) / 256) : 0;
    const dim3 grid((unsigned)(n_fin + n_w));
    if (!upd) {
        hipLaunchKernelGGL(finalize_wide_kernel<-1>, grid, dim3(256), 0, st, a, PsUpdate{}, n_fin);
        return hipGetLastError();
    }
    switch (upd->rule) {
        case 0: hipLaunchKernelGGL(finalize_wide_kernel<0>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        case 1: hipLaunchKernelGGL(finalize_wide_kernel<1>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        case 2: hipLaunchKernelGGL(finalize_wide_kernel<2>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t finalize_small_launch(const FinalizeArgs& a, const PsUpdate* upd, hipStream_t st) {
    int64_t total = a.H + (int64_t)a.A * a.H + a.A + 1;
    for (int l = 0; l < a.n_conv; ++l) total += a.wcount[l] + a.cout[l];
    const int n_fin = (int)((total * 8 + 255) / 256);
    if ((upd || a.fc1w_part) && (a.fc1w_off % 4 != 0 || a.fc1w_count % 4 != 0 || !a.grad_base))
        return hipErrorInvalidValue;
    const int n_w = upd || a.fc1w_part ? (int)((a.fc1w_count / 4 + 255) / 256) : 0;
    const dim3 grid((unsigned)(n_fin + n_w));
    if (!upd) {
        hipLaunchKernelGGL(finalize_small_kernel<-1>, grid, dim3(256), 0, st, a, PsUpdate{}, n_fin);
        return hipGetLastError();
    }
    switch (upd->rule) {
        case 0: hipLaunchKernelGGL(finalize_small_kernel<0>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        case 1: hipLaunchKernelGGL(finalize_small_kernel<1>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        case 2: hipLaunchKernelGGL(finalize_small_kernel<2>, grid, dim3(256), 0, st, a, *upd, n_fin); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeArgs& a, const PsUpdate* upd, hipStream_t st) {
    // up to 128 samples the eight-lane layout; above, chunk slots and a lane per output
    if (a.B <= 128) return finalize_small_launch(a, upd, st);
    if (a.A == 6) return finalize_wide_launch<6>(a, upd, st);
    if (a.A == 18) return finalize_wide_launch<18>(a, upd, st);
    return hipErrorInvalidValue;
}

}  // namespace dqn
