// Minibatch draw from the replay memory (Sec. III.C; Alg. 1): copy the
// stacked frames of records idx[j] and idx[j]+1 and the side fields of
// transition idx[j].  Pure HBM traffic: 16-byte loads and stores, one record
// row of 16-byte words per thread, records read once (non-temporal).
#include "common.h"

namespace dqn {
namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void gather_kernel(
    const uint8_t* __restrict__ frames, int64_t stride, int64_t words, const int64_t* __restrict__ idx,
    uint8_t* __restrict__ s, uint8_t* __restrict__ sn, const uint8_t* __restrict__ act,
    const int8_t* __restrict__ rew, const uint8_t* __restrict__ term, int32_t* __restrict__ a_out,
    float* __restrict__ r_out, uint8_t* __restrict__ t_out) {
    const int j = blockIdx.y;
    const int which = blockIdx.z;  // 0: s, 1: s_next
    const int64_t i = idx[j] + which;
    const u4* src = (const u4*)(frames + i * stride);
    u4* dst = (u4*)((which ? sn : s) + (size_t)j * words * 16);
    for (int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x; w < words; w += (int64_t)gridDim.x * 256)
        dst[w] = __builtin_nontemporal_load(src + w);
    if (which == 0 && blockIdx.x == 0 && threadIdx.x == 0) {
        const int64_t k = idx[j];
        if (a_out) a_out[j] = act[k];
        if (r_out) r_out[j] = (float)rew[k];
        if (t_out) t_out[j] = term[k];
    }
}

// Counts the indices outside [0, hi] into *bad: one workgroup walks the
// stream, wave counts by ballot, the four wave counts added through LDS and
// stored by one lane (no atomics).
__global__ __launch_bounds__(256) void validate_kernel(const int64_t* __restrict__ idx, int batch, int64_t hi,
                                                       int32_t* __restrict__ bad) {
    __shared__ int32_t wc[4];
    int32_t n = 0;
    for (int j0 = 0; j0 < batch; j0 += 256) {
        const int j = j0 + (int)threadIdx.x;
        const bool out = j < batch && (idx[j] < 0 || idx[j] > hi);
        n += __popcll(__ballot(out));
    }
    if ((threadIdx.x & 63) == 0) wc[threadIdx.x >> 6] = n;
    __syncthreads();
    if (threadIdx.x == 0) *bad = (wc[0] + wc[1]) + (wc[2] + wc[3]);
}

}  // namespace

hipError_t launch_validate(const int64_t* idx, int batch, int64_t hi, int32_t* bad, hipStream_t st) {
    hipLaunchKernelGGL(validate_kernel, dim3(1), dim3(256), 0, st, idx, batch, hi, bad);
    return hipGetLastError();
}

hipError_t launch_gather(const uint8_t* frames, int64_t stride, int64_t rec_bytes,
                         const uint8_t* act, const int8_t* rew, const uint8_t* term,
                         const int64_t* idx, int batch, uint8_t* s, uint8_t* sn, int32_t* a,
                         float* r, uint8_t* t, hipStream_t st) {
    const int64_t words = rec_bytes / 16;
    const unsigned bx = (unsigned)((words + 255) / 256);
    dim3 grid(bx, (unsigned)batch, sn ? 2u : 1u);
    hipLaunchKernelGGL(gather_kernel, grid, dim3(256), 0, st, frames, stride, words, idx, s, sn, act,
                       rew, term, a, r, t);
    return hipGetLastError();
}

}  // namespace dqn
