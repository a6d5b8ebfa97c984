// Fully connected layer contractions on fp32 MFMA: fc1 forward (split-K,
// partial sums), fc1 weight gradient, and fc1 input gradient with the ReLU
// mask of the last conv layer fused in.  BMxBN output tiles (32 or 64 each),
// k-steps of BK (32, or 128 for long contractions so that fewer dependent
// global round trips are needed) staged through LDS, with the next step's
// global loads issued before the current step's MFMAs; four waves in a 2x2
// arrangement.
#include "common.h"

namespace dqn {
namespace {

// TA: A(m,k) = A[k*lda + m] else A[m*lda + k].
// TB: B(k,n) = B[n*ldb + k] else B[k*ldb + n].
template <int BM, int BN, int BK, bool TA, bool TB, bool MASK>
__global__ __launch_bounds__(256) void gemm_kernel(int M, int N, int K,
                                                   const float* __restrict__ A, int lda,
                                                   const float* __restrict__ Bm, int ldb,
                                                   float* __restrict__ C, int ldc, int kchunk,
                                                   int64_t c_slice,
                                                   const float* __restrict__ mask) {
    constexpr int TM = BM / 32, TN = BN / 32;     // MFMA tiles per wave
    constexpr int LDA = BM + 4, LDB = BN + 4;
    constexpr int AV = BM * BK / 4 / 256;         // float4 loads per thread per k-step
    constexpr int BV = BN * BK / 4 / 256;
    extern __shared__ __align__(16) float smem[];
    float (*As)[LDA] = (float (*)[LDA])smem;              // [BK][LDA]
    float (*Bs)[LDB] = (float (*)[LDB])(smem + BK * LDA); // [BK][LDB]
    const int m0 = blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int z = blockIdx.z;
    const int kbeg = z * kchunk;
    const int kend = min(K, kbeg + kchunk);
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * (BN / 2);

    f4 ra[AV], rb[BV];
    auto load = [&](int k0) {
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int e = t + 256 * v;
            f4 x = f4{0.f, 0.f, 0.f, 0.f};
            if constexpr (!TA) {  // rows of A, 4 consecutive k
                const int row = e / (BK / 4), kq = (e % (BK / 4)) * 4;
                if (m0 + row < M && k0 + kq < kend) x = *(const f4*)(A + (size_t)(m0 + row) * lda + k0 + kq);
            } else {              // k rows, 4 consecutive m
                const int kr = e / (BM / 4), mq = (e % (BM / 4)) * 4;
                if (k0 + kr < kend && m0 + mq < M) x = *(const f4*)(A + (size_t)(k0 + kr) * lda + m0 + mq);
            }
            ra[v] = x;
        }
#pragma unroll
        for (int v = 0; v < BV; ++v) {
            const int e = t + 256 * v;
            f4 x = f4{0.f, 0.f, 0.f, 0.f};
            if constexpr (!TB) {  // k rows, 4 consecutive n
                const int kr = e / (BN / 4), nq = (e % (BN / 4)) * 4;
                if (k0 + kr < kend && n0 + nq < N) x = *(const f4*)(Bm + (size_t)(k0 + kr) * ldb + n0 + nq);
            } else {              // columns n, 4 consecutive k
                const int col = e / (BK / 4), kq = (e % (BK / 4)) * 4;
                if (n0 + col < N && k0 + kq < kend) x = *(const f4*)(Bm + (size_t)(n0 + col) * ldb + k0 + kq);
            }
            rb[v] = x;
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            const int e = t + 256 * v;
            if constexpr (!TA) {
                const int row = e / (BK / 4), kq = (e % (BK / 4)) * 4;
#pragma unroll
                for (int q = 0; q < 4; ++q) As[kq + q][row] = ra[v][q];
            } else {
                const int kr = e / (BM / 4), mq = (e % (BM / 4)) * 4;
                *(f4*)&As[kr][mq] = ra[v];
            }
        }
#pragma unroll
        for (int v = 0; v < BV; ++v) {
            const int e = t + 256 * v;
            if constexpr (!TB) {
                const int kr = e / (BN / 4), nq = (e % (BN / 4)) * 4;
                *(f4*)&Bs[kr][nq] = rb[v];
            } else {
                const int col = e / (BK / 4), kq = (e % (BK / 4)) * 4;
#pragma unroll
                for (int q = 0; q < 4; ++q) Bs[kq + q][col] = rb[v][q];
            }
        }
    };

    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    if (kbeg < kend) load(kbeg);
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        store();
        __syncthreads();
        if (k0 + BK < kend) load(k0 + BK);   // in flight during the MFMAs below
#pragma unroll
        for (int kk = 0; kk < BK / 4; ++kk) {
            float a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[kk * 4 + g][wm + i * 16 + li];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[kk * 4 + g][wn + j * 16 + li];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x4(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }

    float* Cz = C + (size_t)z * c_slice;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
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

template <int BM, int BN, int BK, bool TA, bool TB, bool MASK>
hipError_t launch_tile(int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C,
                 int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                 hipStream_t st) {
    constexpr size_t lds = (size_t)BK * ((BM + 4) + (BN + 4)) * 4;
    auto kern = gemm_kernel<BM, BN, BK, TA, TB, MASK>;
    static bool granted = false;
    if (!granted) {
        if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
            hipSuccess)
            return hipErrorInvalidValue;
        granted = true;
    }
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((N + BN - 1) / BN), (unsigned)kslices);
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, st, M, N, K, A, lda, B, ldb, C, ldc, kchunk, c_slice,
                       mask);
    return hipGetLastError();
}

template <int BK, bool TA, bool TB, bool MASK>
hipError_t launch_bk(int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C,
               int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask, hipStream_t st) {
    // Narrow tiles when the output is small, so more workgroups run.
    const bool small_m = M <= 32;
    const long tiles64 = (long)((M + 63) / 64) * ((N + 63) / 64) * kslices;
    const bool small_n = tiles64 < 128 && N > 32;
    if (small_m && small_n)
        return launch_tile<32, 32, BK, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
    else if (small_m)
        return launch_tile<32, 64, BK, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
    else if (small_n)
        return launch_tile<64, 32, BK, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
    else
        return launch_tile<64, 64, BK, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
}

template <bool TA, bool TB, bool MASK>
hipError_t launch_shape(int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C,
                  int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                  hipStream_t st) {
    if (kchunk >= 128)
        return launch_bk<128, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
    else
        return launch_bk<32, TA, TB, MASK>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
}

}  // namespace

hipError_t launch_gemm(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B,
                       int ldb, float* C, int ldc, int kslices, int kchunk, int64_t c_slice,
                       const float* mask, hipStream_t st) {
    if (kchunk % 32 != 0) return hipErrorInvalidValue;
    switch (kind) {
        case GEMM_NT:
            return launch_shape<false, true, false>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, nullptr, st);
        case GEMM_TN:
            return launch_shape<true, false, false>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, nullptr, st);
        case GEMM_NN:
            if (mask)
                return launch_shape<false, false, true>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
            else
                return launch_shape<false, false, false>(M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, nullptr, st);
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace dqn
