// Denominator checks for the roofline figures: a pure matrix-core loop (fp32
// v_mfma_f32_16x16x4_f32 or bf16 v_mfma_f32_16x16x32_bf16, the two MFMA
// forms the hot path uses) and a streaming copy.  The caller times each
// launch with events on the same stream and divides the known work by it.
#include "common.h"
#include "dqn_profile.h"

namespace dqn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int PK_WG = 256;
constexpr int PK_CHAINS = 4;   // independent accumulators per wave

// Every wave runs iters rounds of PK_CHAINS independent MFMAs on register
// operands; one float per workgroup is stored so nothing is eliminated.
template <bool BF16>
__global__ __launch_bounds__(PK_WG) void mfma_peak_kernel(int iters, float seed, float* out) {
    const int lane = threadIdx.x & 63;
    f4 acc[PK_CHAINS];
#pragma unroll
    for (int c = 0; c < PK_CHAINS; ++c) acc[c] = f4{0.f, 0.f, 0.f, 0.f};
    const float a = seed * (float)(lane + 1), b = seed * 0.5f;
    if constexpr (BF16) {
        bf16x8 av, bv;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            av[e] = (__bf16)(a + (float)e);
            bv[e] = (__bf16)(b - (float)e);
        }
        for (int i = 0; i < iters; ++i)
#pragma unroll
            for (int c = 0; c < PK_CHAINS; ++c)
                acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[c], 0, 0, 0);
    } else {
        for (int i = 0; i < iters; ++i)
#pragma unroll
            for (int c = 0; c < PK_CHAINS; ++c) acc[c] = mfma16x16x4(a, b, acc[c]);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < PK_CHAINS; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    s = wave_sum(s);
    if (threadIdx.x == 0) out[blockIdx.x] = s;
}

// dst = src over n16 16-byte vectors, grid-stride, PK_UNROLL loads in
// flight per thread before their stores.
constexpr int PK_UNROLL = 4;
__global__ __launch_bounds__(PK_WG) void stream_copy_kernel(const f4* __restrict__ src, f4* __restrict__ dst,
                                                            int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * PK_WG;
    int64_t i = (int64_t)blockIdx.x * PK_WG + threadIdx.x;
    for (; i + (PK_UNROLL - 1) * stride < n16; i += PK_UNROLL * stride) {
        f4 v[PK_UNROLL];
#pragma unroll
        for (int u = 0; u < PK_UNROLL; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
        for (int u = 0; u < PK_UNROLL; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
    }
    for (; i < n16; i += stride) dst[i] = src[i];
}

}  // namespace
}  // namespace dqn

using namespace dqn;

extern "C" {

int64_t dqn_profile_mfma_peak(int32_t dtype, int32_t workgroups, int32_t iters, float* out, void* stream) {
    if ((dtype != DQN_PEAK_FP32 && dtype != DQN_PEAK_BF16) || workgroups <= 0 || iters <= 0 || !out)
        return DQN_EINVAL;
    const hipStream_t st = (hipStream_t)stream;
    if (dtype == DQN_PEAK_BF16)
        hipLaunchKernelGGL(mfma_peak_kernel<true>, dim3((unsigned)workgroups), dim3(PK_WG), 0, st, iters, 0.25f, out);
    else
        hipLaunchKernelGGL(mfma_peak_kernel<false>, dim3((unsigned)workgroups), dim3(PK_WG), 0, st, iters, 0.25f, out);
    if (hipGetLastError() != hipSuccess) return DQN_EHIP;
    const int64_t per_mfma = dtype == DQN_PEAK_BF16 ? 16 * 16 * 32 * 2 : 16 * 16 * 4 * 2;
    return (int64_t)workgroups * (PK_WG / 64) * iters * PK_CHAINS * per_mfma;
}

int dqn_profile_stream_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream) {
    if (!src || !dst || bytes <= 0 || bytes % 16 != 0 || workgroups <= 0) return DQN_EINVAL;
    if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return DQN_EINVAL;
    const char* s = (const char*)src;
    const char* d = (const char*)dst;
    if (s < d + bytes && d < s + bytes) return DQN_EINVAL;
    hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)workgroups), dim3(PK_WG), 0, (hipStream_t)stream,
                       (const f4*)src, (f4*)dst, bytes / 16);
    return hipGetLastError() == hipSuccess ? DQN_OK : DQN_EHIP;
}

}  // extern "C"
