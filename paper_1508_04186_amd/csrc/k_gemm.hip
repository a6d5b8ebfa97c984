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

struct GemmParams {
    int M, N, K;
    const float* A;
    int lda;
    const float* B;
    int ldb;
    float* C;
    int ldc, kchunk;
    int64_t c_slice;
    const float* mask;
};

// TA: A(m,k) = A[k*lda + m] else A[m*lda + k].
// TB: B(k,n) = B[n*ldb + k] else B[k*ldb + n].
// One BMxBN output tile (bx, by) of k-slice bz.
template <int BM, int BN, int BK, bool TA, bool TB, bool MASK>
__device__ __forceinline__ void gemm_body(const GemmParams& p, int bx, int by, int bz, float* smem) {
    const int M = p.M, N = p.N, K = p.K, lda = p.lda, ldb = p.ldb, ldc = p.ldc, kchunk = p.kchunk;
    const float* __restrict__ A = p.A;
    const float* __restrict__ Bm = p.B;
    float* __restrict__ C = p.C;
    const float* __restrict__ mask = p.mask;
    const int64_t c_slice = p.c_slice;
    constexpr int TM = BM / 32, TN = BN / 32;     // MFMA tiles per wave
    constexpr int LDA = BM + 4, LDB = BN + 4;
    constexpr int AV = BM * BK / 4 / 256;         // float4 loads per thread per k-step
    constexpr int BV = BN * BK / 4 / 256;
    float (*As)[LDA] = (float (*)[LDA])smem;              // [BK][LDA]
    float (*Bs)[LDB] = (float (*)[LDB])(smem + BK * LDA); // [BK][LDB]
    const int m0 = bx * BM;
    const int n0 = by * BN;
    const int z = bz;
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
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    extern __shared__ __align__(16) float smem[];
    gemm_body<BM, BN, BK, TA, TB, MASK>(p, blockIdx.x, blockIdx.y, blockIdx.z, smem);
}

// Two independent GEMMs in one launch (flattened block index; the first
// n1 = g1x*g1y*g1z blocks run GEMM 1).
template <int BM1, int BN1, int BK1, bool TA1, bool TB1, bool M1,
          int BM2, int BN2, int BK2, bool TA2, bool TB2, bool M2>
__global__ __launch_bounds__(256) void gemm_pair_kernel(GemmParams p1, int g1x, int g1y, GemmParams p2,
                                                        int g2x, int g2y, int n1) {
    extern __shared__ __align__(16) float smem[];
    int b = blockIdx.x;
    if (b < n1) {
        gemm_body<BM1, BN1, BK1, TA1, TB1, M1>(p1, b % g1x, (b / g1x) % g1y, b / (g1x * g1y), smem);
    } else {
        b -= n1;
        gemm_body<BM2, BN2, BK2, TA2, TB2, M2>(p2, b % g2x, (b / g2x) % g2y, b / (g2x * g2y), smem);
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
    const GemmParams p{M, N, K, A, lda, B, ldb, C, ldc, kchunk, c_slice, mask};
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, st, p);
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

// Tile configuration the single launches pick for a shape.
struct TileCfg {
    int bm, bn, bk;
};

TileCfg pick_tile(int M, int N, int kslices, int kchunk) {
    const bool small_m = M <= 32;
    const long tiles64 = (long)((M + 63) / 64) * ((N + 63) / 64) * kslices;
    const bool small_n = tiles64 < 128 && N > 32;
    return TileCfg{small_m ? 32 : 64, small_n ? 32 : 64, kchunk >= 128 ? 128 : 32};
}

template <int BM1, int BN1, int BK1, int BM2, int BN2, int BK2>
hipError_t pair_tn_nnmask(const GemmParams& w, const GemmParams& d, hipStream_t st) {
    auto kern = gemm_pair_kernel<BM1, BN1, BK1, true, false, false, BM2, BN2, BK2, false, false, true>;
    constexpr size_t l1 = (size_t)BK1 * ((BM1 + 4) + (BN1 + 4)) * 4;
    constexpr size_t l2 = (size_t)BK2 * ((BM2 + 4) + (BN2 + 4)) * 4;
    constexpr size_t lds = l1 > l2 ? l1 : l2;
    static bool granted = false;
    if (!granted) {
        if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
            hipSuccess)
            return hipErrorInvalidValue;
        granted = true;
    }
    const int g1x = (w.M + BM1 - 1) / BM1, g1y = (w.N + BN1 - 1) / BN1;
    const int g2x = (d.M + BM2 - 1) / BM2, g2y = (d.N + BN2 - 1) / BN2;
    const int n1 = g1x * g1y, n2 = g2x * g2y;
    hipLaunchKernelGGL(kern, dim3((unsigned)(n1 + n2)), dim3(256), lds, st, w, g1x, g1y, d, g2x, g2y, n1);
    return hipGetLastError();
}

}  // namespace

// The fc1 weight gradient (TN, one k-slice) and the masked fc1 input gradient
// (NN, one k-slice) in one launch when their tile configurations are one of
// the instantiated pairs; otherwise two launches.
hipError_t launch_gemm_wgrad_dgrad(int H, int F, int B, const float* dz1, const float* x,
                                   float* dW, const float* W, float* dx, hipStream_t st) {
    const int kw = (B + 31) / 32 * 32, kd = (H + 31) / 32 * 32;
    const GemmParams w{H, F, B, dz1, H, x, F, dW, F, kw, 0, nullptr};
    const GemmParams d{B, F, H, dz1, H, W, F, dx, F, kd, 0, x};
    const TileCfg cw = pick_tile(H, F, 1, kw), cd = pick_tile(B, F, 1, kd);
    if (cw.bm == 64 && cw.bn == 64 && cd.bk == 128) {
        if (cw.bk == 32 && cd.bm == 32 && cd.bn == 32) return pair_tn_nnmask<64, 64, 32, 32, 32, 128>(w, d, st);
        if (cw.bk == 32 && cd.bm == 64 && cd.bn == 32) return pair_tn_nnmask<64, 64, 32, 64, 32, 128>(w, d, st);
        if (cw.bk == 128 && cd.bm == 64 && cd.bn == 32) return pair_tn_nnmask<64, 64, 128, 64, 32, 128>(w, d, st);
        if (cw.bk == 128 && cd.bm == 64 && cd.bn == 64) return pair_tn_nnmask<64, 64, 128, 64, 64, 128>(w, d, st);
    }
    hipError_t e = launch_gemm(GEMM_TN, H, F, B, dz1, H, x, F, dW, F, 1, kw, 0, nullptr, st);
    if (e != hipSuccess) return e;
    return launch_gemm(GEMM_NN, B, F, H, dz1, H, W, F, dx, F, 1, kd, 0, x, st);
}

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
