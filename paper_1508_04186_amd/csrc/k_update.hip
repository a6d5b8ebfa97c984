// Parameter-server update (Alg. 2 RMSPROPUPDATE; gradient descent of
// Sec. III.B; AdaGrad named in Sec. IV.D.2): one streaming elementwise pass,
// four parameters per thread with 16-byte loads and stores.
#include "common.h"

namespace dqn {
namespace {

template <int RULE>
__global__ __launch_bounds__(256) void apply_kernel(const float* __restrict__ th_in,
                                                    float* th_out, float* state,
                                                    const float* __restrict__ g, int64_t n,
                                                    float lr, float decay, float eps) {
    const int64_t n4 = n / 4;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
        f4 th = ((const f4*)th_in)[i];
        f4 gv = ((const f4*)g)[i];
        f4 s = f4{0.f, 0.f, 0.f, 0.f};
        if constexpr (RULE != 0) s = ((const f4*)state)[i];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float t = th[r], sv = s[r];
            ps_update<RULE>(t, sv, gv[r], lr, decay, eps);
            th[r] = t;
            s[r] = sv;
        }
        ((f4*)th_out)[i] = th;
        if constexpr (RULE != 0) ((f4*)state)[i] = s;
    }
    // tail of n % 4 elements
    if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
        const int64_t i = n4 * 4 + threadIdx.x;
        float t = th_in[i], sv = RULE != 0 ? state[i] : 0.f;
        ps_update<RULE>(t, sv, g[i], lr, decay, eps);
        th_out[i] = t;
        if constexpr (RULE != 0) state[i] = sv;
    }
}

// Target-network refresh: dst <- src over n floats (a kernel rather than a
// runtime copy, so it records as an ordinary node under graph capture).
__global__ __launch_bounds__(256) void copy_kernel(const float* __restrict__ src,
                                                   float* __restrict__ dst, int64_t n) {
    const int64_t n4 = n / 4;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride)
        ((f4*)dst)[i] = ((const f4*)src)[i];
    if (blockIdx.x == 0 && threadIdx.x < (n & 3)) dst[n4 * 4 + threadIdx.x] = src[n4 * 4 + threadIdx.x];
}

}  // namespace

hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t st) {
    int64_t blocks = (n / 4 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, st, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_apply(int rule, const float* th_in, float* th_out, float* state, const float* g,
                        int64_t n, float lr, float decay, float eps, hipStream_t st) {
    int64_t n4 = n / 4;
    int64_t blocks = (n4 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    dim3 grid((unsigned)blocks), block(256);
    switch (rule) {
        case 0: hipLaunchKernelGGL(apply_kernel<0>, grid, block, 0, st, th_in, th_out, state, g, n, lr, decay, eps); break;
        case 1: hipLaunchKernelGGL(apply_kernel<1>, grid, block, 0, st, th_in, th_out, state, g, n, lr, decay, eps); break;
        case 2: hipLaunchKernelGGL(apply_kernel<2>, grid, block, 0, st, th_in, th_out, state, g, n, lr, decay, eps); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace dqn
