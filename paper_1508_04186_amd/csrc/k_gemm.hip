// Fully connected layer contractions on fp32 MFMA: fc1 forward (split-K,
// partial sums), fc1 weight gradient, and fc1 input gradient with the ReLU
// mask of the last conv layer fused in.  64x64 output tiles, k-steps of 16
// staged through LDS; four waves each own a 32x32 quadrant (2x2 MFMA tiles).
#include "common.h"

namespace dqn {
namespace {

constexpr int BM = 64, BN = 64, BK = 16, LDP = BM + 4;

// TA: A(m,k) = A[k*lda + m] else A[m*lda + k].
// TB: B(k,n) = B[n*ldb + k] else B[k*ldb + n].
template <bool TA, bool TB, bool MASK>
__global__ __launch_bounds__(256) void gemm_kernel(int M, int N, int K,
                                                   const float* __restrict__ A, int lda,
                                                   const float* __restrict__ Bm, int ldb,
                                                   float* __restrict__ C, int ldc, int kchunk,
                                                   int64_t c_slice,
                                                   const float* __restrict__ mask) {
    __shared__ __align__(16) float As[BK][LDP];
    __shared__ __align__(16) float Bs[BK][LDP];
    const int m0 = blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int z = blockIdx.z;
    const int kbeg = z * kchunk;
    const int kend = min(K, kbeg + kchunk);
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;

    f4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        // ---- A tile -> As[k][m]
        if constexpr (!TA) {
            const int row = t >> 2, kq = (t & 3) * 4;
            f4 v = f4{0.f, 0.f, 0.f, 0.f};
            if (m0 + row < M && k0 + kq < kend) v = *(const f4*)(A + (size_t)(m0 + row) * lda + k0 + kq);
            As[kq + 0][row] = v[0];
            As[kq + 1][row] = v[1];
            As[kq + 2][row] = v[2];
            As[kq + 3][row] = v[3];
        } else {
            const int kr = t >> 4, mq = (t & 15) * 4;
            f4 v = f4{0.f, 0.f, 0.f, 0.f};
            if (k0 + kr < kend && m0 + mq < M) v = *(const f4*)(A + (size_t)(k0 + kr) * lda + m0 + mq);
            *(f4*)&As[kr][mq] = v;
        }
        // ---- B tile -> Bs[k][n]
        if constexpr (!TB) {
            const int kr = t >> 4, nq = (t & 15) * 4;
            f4 v = f4{0.f, 0.f, 0.f, 0.f};
            if (k0 + kr < kend && n0 + nq < N) v = *(const f4*)(Bm + (size_t)(k0 + kr) * ldb + n0 + nq);
            *(f4*)&Bs[kr][nq] = v;
        } else {
            const int col = t >> 2, kq = (t & 3) * 4;
            f4 v = f4{0.f, 0.f, 0.f, 0.f};
            if (n0 + col < N && k0 + kq < kend) v = *(const f4*)(Bm + (size_t)(n0 + col) * ldb + k0 + kq);
            Bs[kq + 0][col] = v[0];
            Bs[kq + 1][col] = v[1];
            Bs[kq + 2][col] = v[2];
            Bs[kq + 3][col] = v[3];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK / 4; ++kk) {
            float a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = As[kk * 4 + g][wm + i * 16 + li];
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = Bs[kk * 4 + g][wn + j * 16 + li];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma16x16x4(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }

    float* Cz = C + (size_t)z * c_slice;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn + j * 16 + li;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm + i * 16 + 4 * g + r;
                if (m < M && n < N) {
                    float v = acc[i][j][r];
                    if constexpr (MASK) v = mask[(size_t)m * ldc + n] > 0.f ? v : 0.f;
                    Cz[(size_t)m * ldc + n] = v;
                }
            }
        }
}

}  // namespace

hipError_t launch_gemm(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B,
                       int ldb, float* C, int ldc, int kslices, int kchunk, int64_t c_slice,
                       const float* mask, hipStream_t st) {
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((N + BN - 1) / BN), (unsigned)kslices);
    dim3 block(256);
    switch (kind) {
        case GEMM_NT:
            hipLaunchKernelGGL((gemm_kernel<false, true, false>), grid, block, 0, st, M, N, K, A,
                               lda, B, ldb, C, ldc, kchunk, c_slice, (const float*)nullptr);
            break;
        case GEMM_TN:
            hipLaunchKernelGGL((gemm_kernel<true, false, false>), grid, block, 0, st, M, N, K, A,
                               lda, B, ldb, C, ldc, kchunk, c_slice, (const float*)nullptr);
            break;
        case GEMM_NN:
            if (mask)
                hipLaunchKernelGGL((gemm_kernel<false, false, true>), grid, block, 0, st, M, N, K,
                                   A, lda, B, ldb, C, ldc, kchunk, c_slice, mask);
            else
                hipLaunchKernelGGL((gemm_kernel<false, false, false>), grid, block, 0, st, M, N, K,
                                   A, lda, B, ldb, C, ldc, kchunk, c_slice, (const float*)nullptr);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace dqn
