// Output head of the Q-network and the TD step of Alg. 1, one wave per
// sample: reduce the fc1 split-K partials, add the bias and apply ReLU, run
// the linear output layer, then either
//   (td)  form y = r (terminal) or r + gamma * max_a' Q(s', a'; theta^-),
//         the residual delta = (Q(s, a) - y) / B, the per-sample loss term
//         and the fc1 pre-activation gradient delta * W2[a, :] * [z1 > 0];
//   (fwd) pick the greedy action (lowest index of the maximum) or, with
//         epsilon-greedy exploration, the caller-drawn random action.
// The finalize kernel then reduces everything that sums over samples or over
// wgrad chunks in a fixed order (no atomics), so results are deterministic.
#include "common.h"

namespace dqn {
namespace {

template <int H, int A>
__global__ __launch_bounds__(256) void head_td_kernel(HeadTdArgs p) {
    constexpr int E = H / 64;
    const int lane = threadIdx.x & 63;
    const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= p.B) return;
    const int B = p.B;
    float zs[E], hs[E], hn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = lane + 64 * e;
        float a = 0.f, b = 0.f;
        for (int z = 0; z < p.ks; ++z) {
            a += p.fc1p[((size_t)z * 2 * B + j) * H + h];
            b += p.fc1p[((size_t)z * 2 * B + B + j) * H + h];
        }
        zs[e] = a + p.b1[h];
        hs[e] = fmaxf(zs[e], 0.f);
        hn[e] = fmaxf(b + p.b1t[h], 0.f);
    }
    float q[A], qn[A];
#pragma unroll
    for (int k = 0; k < A; ++k) {
        float a = 0.f, b = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int h = lane + 64 * e;
            a = fmaf(p.W2[k * H + h], hs[e], a);
            b = fmaf(p.W2t[k * H + h], hn[e], b);
        }
        q[k] = wave_sum(a) + p.b2[k];
        qn[k] = wave_sum(b) + p.b2t[k];
    }
    float m = qn[0];
#pragma unroll
    for (int k = 1; k < A; ++k) m = fmaxf(m, qn[k]);
    // An action outside [0, A) is clamped so it can never index outside W2.
    const int act = min(max(p.action[j], 0), A - 1);
    const float r = p.reward[j];
    const float y = p.terminal[j] ? r : fmaf(p.gamma, m, r);
    float qa = q[0];
#pragma unroll
    for (int k = 1; k < A; ++k) qa = (k == act) ? q[k] : qa;
    const float diff = qa - y;
    const float delta = diff / (float)B;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = lane + 64 * e;
        p.h1s[(size_t)j * H + h] = hs[e];
        p.dz1[(size_t)j * H + h] = zs[e] > 0.f ? delta * p.W2[act * H + h] : 0.f;
    }
    if (lane == 0) {
        p.delta[j] = delta;
        p.lossj[j] = 0.5f * diff * diff / (float)B;
        if (p.y_out) p.y_out[j] = y;
    }
    if (p.q_out && lane < A) {
        float v = q[0];
#pragma unroll
        for (int k = 1; k < A; ++k) v = (k == lane) ? q[k] : v;
        p.q_out[(size_t)j * A + lane] = v;
    }
}

template <int H, int A>
__global__ __launch_bounds__(256) void head_fwd_kernel(HeadFwdArgs p) {
    constexpr int E = H / 64;
    const int lane = threadIdx.x & 63;
    const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= p.B) return;
    float hs[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int h = lane + 64 * e;
        float a = 0.f;
        for (int z = 0; z < p.ks; ++z) a += p.fc1p[((size_t)z * p.B + j) * H + h];
        hs[e] = fmaxf(a + p.b1[h], 0.f);
    }
    float q[A];
#pragma unroll
    for (int k = 0; k < A; ++k) {
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) a = fmaf(p.W2[k * H + lane + 64 * e], hs[e], a);
        q[k] = wave_sum(a) + p.b2[k];
    }
    int best = 0;
    float bq = q[0];
#pragma unroll
    for (int k = 1; k < A; ++k)
        if (q[k] > bq) { bq = q[k]; best = k; }
    if (p.thresh > 0) {
        const uint64_t w = p.draws[j];
        if ((w >> 32) < p.thresh) best = (int)(((w & 0xffffffffull) * (uint64_t)A) >> 32);
    }
    if (lane == 0 && p.action_out) p.action_out[j] = best;
    if (p.q_out && lane < A) {
        float v = q[0];
#pragma unroll
        for (int k = 1; k < A; ++k) v = (k == lane) ? q[k] : v;
        p.q_out[(size_t)j * A + lane] = v;
    }
}

// One thread per output value; each sums its terms in a fixed order.
__global__ __launch_bounds__(256) void finalize_kernel(FinalizeArgs a) {
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (int l = 0; l < a.n_conv; ++l) {
        if (i < a.wcount[l]) {
            float s = 0.f;
            for (int c = 0; c < a.chunks[l]; ++c) s += a.wpart[l][(size_t)c * a.wcount[l] + i];
            a.gw[l][i] = s;
            return;
        }
        i -= a.wcount[l];
        if (i < a.cout[l]) {
            float s = 0.f;
            for (int c = 0; c < a.chunks[l]; ++c) s += a.bpart[l][(size_t)c * a.cout[l] + i];
            a.gb[l][i] = s;
            return;
        }
        i -= a.cout[l];
    }
    if (i < a.H) {
        float s = 0.f;
        for (int j = 0; j < a.B; ++j) s += a.dz1[(size_t)j * a.H + i];
        a.g_b1[i] = s;
        return;
    }
    i -= a.H;
    if (i < (int64_t)a.A * a.H) {
        const int k = (int)(i / a.H), h = (int)(i - (int64_t)k * a.H);
        float s = 0.f;
        for (int j = 0; j < a.B; ++j)
            if (a.action[j] == k) s = fmaf(a.delta[j], a.h1s[(size_t)j * a.H + h], s);
        a.g_W2[i] = s;
        return;
    }
    i -= (int64_t)a.A * a.H;
    if (i < a.A) {
        float s = 0.f;
        for (int j = 0; j < a.B; ++j)
            if (a.action[j] == (int)i) s += a.delta[j];
        a.g_b2[i] = s;
        return;
    }
    i -= a.A;
    if (i == 0) {
        float s = 0.f;
        for (int j = 0; j < a.B; ++j) s += a.lossj[j];
        a.loss_out[0] = s;
    }
}

template <int H, int A>
hipError_t td_launch(const HeadTdArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((head_td_kernel<H, A>), dim3((unsigned)((a.B + 3) / 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int H, int A>
hipError_t fwd_launch(const HeadFwdArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((head_fwd_kernel<H, A>), dim3((unsigned)((a.B + 3) / 4)), dim3(256), 0, st, a);
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

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t st) {
    int64_t total = a.H + (int64_t)a.A * a.H + a.A + 1;
    for (int l = 0; l < a.n_conv; ++l) total += a.wcount[l] + a.cout[l];
    hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace dqn
