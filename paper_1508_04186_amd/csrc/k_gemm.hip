// Fully connected layer contractions on fp32 MFMA: fc1 forward (split-K,
// partial sums), fc1 weight gradient, and fc1 input gradient with the ReLU
// mask of the last conv layer fused in.  BMxBN output tiles (32 or 64 each),
// k-steps of BK (32, or 128 for long contractions so that fewer dependent
// global round trips are needed) staged through LDS, with the next step's
// global loads issued before the current step's MFMAs; four waves in a 2x2
// arrangement.  The bf16-input variant rounds both staged operands to
// bfloat16 as it reads them and runs one v_mfma_f32_16x16x32_bf16 per 32
// k-values instead of eight fp32 steps.  The weight and input gradients
// take their output tiles in the XCD-contiguous order of xcd_tile (tiles
// sharing the column operand run on one XCD, so it is fetched into that
// XCD's L2 once), and so does the forward when its k-slices are many.
#include <algorithm>

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
//
// Each operand is staged in LDS in its global orientation, so global loads
// and LDS stores are both 16-byte vectors with no transposition:
//   k-contiguous operand (A without TA, B with TB): [mn][BK + 4]
//   mn-contiguous operand (A with TA, B without TB): [BK][MN + 16]
// The MFMA loop reads, per lane (li = lane % 16, g = lane / 16), element
// (mn0 + li, 4*kk + g).  With a row stride of 4 (mod 64) floats in the first
// layout and 16 (mod 64) in the second, the 64 lanes of one read hit 64
// distinct banks.
template <int BM, int BN, int BK, bool TA, bool TB>
struct GemmSmem {
    static constexpr int RA = TA ? BM + 16 : BK + 4;   // row stride of A's stage
    static constexpr int RB = TB ? BK + 4 : BN + 16;
    static constexpr int NA = TA ? BK * RA : BM * RA;  // floats
    static constexpr int NB = TB ? BN * RB : BK * RB;
    static constexpr size_t bytes = (size_t)(NA + NB) * 4;
};

template <int BM, int BN, int BK, bool TA, bool TB, bool MASK, bool BF16>
__device__ __forceinline__ void gemm_body(const GemmParams& p, int bx, int by, int bz, float* smem) {
    using SM = GemmSmem<BM, BN, BK, TA, TB>;
    const int M = p.M, N = p.N, K = p.K, lda = p.lda, ldb = p.ldb, ldc = p.ldc, kchunk = p.kchunk;
    const float* __restrict__ A = p.A;
    const float* __restrict__ Bm = p.B;
    float* __restrict__ C = p.C;
    const float* __restrict__ mask = p.mask;
    const int64_t c_slice = p.c_slice;
    constexpr int TM = BM / 32, TN = BN / 32;     // MFMA tiles per wave
    constexpr int AV = BM * BK / 4 / 256;         // float4 loads per thread per stage
    constexpr int BV = BN * BK / 4 / 256;
    static_assert(AV >= 1 && BV >= 1, "tile too small for 256 threads");
    float* As = smem;
    float* Bs = smem + SM::NA;
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
                *(f4*)&As[row * SM::RA + kq] = ra[v];
            } else {
                const int kr = e / (BM / 4), mq = (e % (BM / 4)) * 4;
                *(f4*)&As[kr * SM::RA + mq] = ra[v];
            }
        }
#pragma unroll
        for (int v = 0; v < BV; ++v) {
            const int e = t + 256 * v;
            if constexpr (!TB) {
                const int kr = e / (BN / 4), nq = (e % (BN / 4)) * 4;
                *(f4*)&Bs[kr * SM::RB + nq] = rb[v];
            } else {
                const int col = e / (BK / 4), kq = (e % (BK / 4)) * 4;
                *(f4*)&Bs[col * SM::RB + kq] = rb[v];
            }
        }
    };
    // Element (mn, k) of each stage.
    auto a_at = [&](int m, int k) { return TA ? As[k * SM::RA + m] : As[m * SM::RA + k]; };
    auto b_at = [&](int k, int n) { return TB ? Bs[n * SM::RB + k] : Bs[k * SM::RB + n]; };

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
        if constexpr (BF16) {
            // one bf16-input step per 32 k-values (bf16_operand's k order)
#pragma unroll
            for (int kb = 0; kb < BK / 32; ++kb) {
                bf16x8 a[TM], b[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    a[i] = bf16_operand([&](int k) { return a_at(wm + i * 16 + li, kb * 32 + k); }, g);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    b[j] = bf16_operand([&](int k) { return b_at(kb * 32 + k, wn + j * 16 + li); }, g);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32bf16(a[i], b[j], acc[i][j]);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < BK / 4; ++kk) {
                float a[TM], b[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) a[i] = a_at(wm + i * 16 + li, kk * 4 + g);
#pragma unroll
                for (int j = 0; j < TN; ++j) b[j] = b_at(kk * 4 + g, wn + j * 16 + li);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x4(a[i], b[j], acc[i][j]);
            }
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

template <int BM, int BN, int BK, bool TA, bool TB, bool MASK, bool BF16>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    extern __shared__ __align__(16) float smem[];
    const TileXYZ tile = !TA && TB ? fwd_tile_order() : xcd_tile<false>();
    gemm_body<BM, BN, BK, TA, TB, MASK, BF16>(p, tile.x, tile.y, tile.z, smem);
}

// Two forward GEMMs of one shape in one launch (the online network on s and
// the target network on s'): k-slices z < ks0 run p0, the rest p1.
template <int BM, int BN, int BK, bool BF16>
__global__ __launch_bounds__(256) void gemm_fwd2_kernel(GemmParams p0, GemmParams p1, int ks0) {
    extern __shared__ __align__(16) float smem[];
    const TileXYZ tile = fwd_tile_order();
    const int z = tile.z;
    if (z < ks0)
        gemm_body<BM, BN, BK, false, true, false, BF16>(p0, tile.x, tile.y, z, smem);
    else
        gemm_body<BM, BN, BK, false, true, false, BF16>(p1, tile.x, tile.y, z - ks0, smem);
}

template <int BM, int BN, int BK>
hipError_t launch_fwd2_tile(const GemmParams& p0, const GemmParams& p1, int kslices, hipStream_t st) {
    if (p0.kchunk % BK != 0) return hipErrorInvalidValue;
    constexpr size_t lds = GemmSmem<BM, BN, BK, false, true>::bytes;
    auto kern = gemm_fwd2_kernel<BM, BN, BK, false>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((p0.M + BM - 1) / BM), (unsigned)((p0.N + BN - 1) / BN), (unsigned)(2 * kslices));
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, st, p0, p1, kslices);
    return hipGetLastError();
}

// Two independent GEMMs in one launch (flattened block index; the first
// n1 = g1x*g1y*g1z blocks run GEMM 1).
template <int BM1, int BN1, int BK1, bool TA1, bool TB1, bool M1,
          int BM2, int BN2, int BK2, bool TA2, bool TB2, bool M2, bool BF16>
__global__ __launch_bounds__(256) void gemm_pair_kernel(GemmParams p1, int g1x, int g1y, GemmParams p2,
                                                        int g2x, int g2y, int n1) {
    extern __shared__ __align__(16) float smem[];
    int b = blockIdx.x;
    if (b < n1) {
        gemm_body<BM1, BN1, BK1, TA1, TB1, M1, BF16>(p1, b % g1x, (b / g1x) % g1y, b / (g1x * g1y), smem);
    } else {
        b -= n1;
        gemm_body<BM2, BN2, BK2, TA2, TB2, M2, BF16>(p2, b % g2x, (b / g2x) % g2y, b / (g2x * g2y), smem);
    }
}

template <int BM, int BN, int BK, bool TA, bool TB, bool MASK, bool BF16>
hipError_t launch_tile(int M, int N, int K, const float* A, int lda, const float* B, int ldb, float* C,
                       int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                       hipStream_t st) {
    if (kchunk % BK != 0) return hipErrorInvalidValue;
    constexpr size_t lds = GemmSmem<BM, BN, BK, TA, TB>::bytes;
    auto kern = gemm_kernel<BM, BN, BK, TA, TB, MASK, BF16>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((N + BN - 1) / BN), (unsigned)kslices);
    const GemmParams p{M, N, K, A, lda, B, ldb, C, ldc, kchunk, c_slice, mask};
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, st, p);
    return hipGetLastError();
}

// Tile shapes, from a sweep of dependent back-to-back launches over the fc
// shapes of both networks (batch 32 to 4096):
//   forward (NT, split-K): 32x32 up to 64 rows, 64x32 up to 1023 rows, 64x64
//     beyond; k-stages of 64 when the slices are long (kchunk >= 256);
//   weight gradient (TN): 32x32, k-stages of 32;
//   input gradient (NN, masked): 32x32, k-stages of 64 up to 64 rows.
struct TileCfg {
    int bm, bn, bk;
};

TileCfg fwd_tile(int M, int kchunk) {
    return TileCfg{M <= 64 ? 32 : 64, M >= 1024 ? 64 : 32, (kchunk >= 256 && kchunk % 64 == 0) ? 64 : 32};
}

TileCfg dgrad_tile(int M, int kchunk) { return TileCfg{32, 32, (M <= 64 && kchunk % 64 == 0) ? 64 : 32}; }

template <bool TA, bool TB, bool MASK, bool BF16>
hipError_t launch_cfg(TileCfg c, int M, int N, int K, const float* A, int lda, const float* B, int ldb,
                      float* C, int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                      hipStream_t st) {
#define DQN_TILE(TBM, TBN, TBK)                                                                     \
    if (c.bm == TBM && c.bn == TBN && c.bk == TBK)                                                  \
        return launch_tile<TBM, TBN, TBK, TA, TB, MASK, BF16>(M, N, K, A, lda, B, ldb, C, ldc, kslices, \
                                                        kchunk, c_slice, mask, st);
    if constexpr (!TA && TB) {  // forward
        DQN_TILE(32, 32, 32)
        DQN_TILE(32, 32, 64)
        DQN_TILE(64, 32, 32)
        DQN_TILE(64, 32, 64)
        DQN_TILE(64, 64, 32)
        DQN_TILE(64, 64, 64)
    } else if constexpr (TA && !TB) {  // weight gradient
        DQN_TILE(32, 32, 32)
    } else {  // input gradient
        DQN_TILE(32, 32, 32)
        DQN_TILE(32, 32, 64)
    }
#undef DQN_TILE
    return hipErrorInvalidValue;
}

template <int BK2, bool BF16>
hipError_t pair_tn_nnmask(const GemmParams& w, const GemmParams& d, hipStream_t st) {
    constexpr int BM = 32, BN = 32, BK1 = 32;
    auto kern = gemm_pair_kernel<BM, BN, BK1, true, false, false, BM, BN, BK2, false, false, true, BF16>;
    constexpr size_t l1 = GemmSmem<BM, BN, BK1, true, false>::bytes;
    constexpr size_t l2 = GemmSmem<BM, BN, BK2, false, false>::bytes;
    constexpr size_t lds = l1 > l2 ? l1 : l2;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    const int g1x = (w.M + BM - 1) / BM, g1y = (w.N + BN - 1) / BN;
    const int g2x = (d.M + BM - 1) / BM, g2y = (d.N + BN - 1) / BN;
    const int n1 = g1x * g1y, n2 = g2x * g2y;
    hipLaunchKernelGGL(kern, dim3((unsigned)(n1 + n2)), dim3(256), lds, st, w, g1x, g1y, d, g2x, g2y, n1);
    return hipGetLastError();
}

}  // namespace

void gemm_fwd_split(int rows, int N, int K, int* ks, int* kchunk) {
    if (rows >= kGemmX6MinRows) return gemm_fwd_split_x6(rows, N, K, ks, kchunk);
    // Enough k-slices that the launch has several hundred workgroups; the
    // head kernel sums the slices.  Past 256 output tiles the launch fills
    // the chip without splitting, and every slice would cost the head a
    // read of rows x N partial sums.
    const TileCfg c = fwd_tile(rows, 64);
    const long tiles = (long)((rows + c.bm - 1) / c.bm) * ((N + c.bn - 1) / c.bn);
    const int whole = (K + 63) / 64 * 64;
    const int kc = std::min(tiles <= 32 ? 64 : tiles <= 256 ? 256 : whole, whole);
    *kchunk = kc;
    *ks = (K + kc - 1) / kc;
}

// The fc1 weight gradient (TN, one k-slice) and the masked fc1 input gradient
// (NN, one k-slice) in one launch.
hipError_t launch_gemm_wgrad_dgrad(int H, int F, int B, const float* dz1, const float* x,
                                   float* dW, const float* W, float* dx, bool bf16, hipStream_t st) {
    const int kw = (B + 31) / 32 * 32, kd = (H + 31) / 32 * 32;
    const GemmParams w{H, F, B, dz1, H, x, F, dW, F, kw, 0, nullptr};
    const GemmParams d{B, F, H, dz1, H, W, F, dx, F, kd, 0, x};
    if (dgrad_tile(B, kd).bk == 64) return bf16 ? pair_tn_nnmask<64, true>(w, d, st) : pair_tn_nnmask<64, false>(w, d, st);
    return bf16 ? pair_tn_nnmask<32, true>(w, d, st) : pair_tn_nnmask<32, false>(w, d, st);
}

namespace {

template <bool BF16>
hipError_t launch_gemm_prec(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B,
                            int ldb, float* C, int ldc, int kslices, int kchunk, int64_t c_slice,
                            const float* mask, hipStream_t st) {
    switch (kind) {
        case GEMM_NT:
            return launch_cfg<false, true, false, BF16>(fwd_tile(M, kchunk), M, N, K, A, lda, B, ldb, C, ldc,
                                                        kslices, kchunk, c_slice, nullptr, st);
        case GEMM_TN:
            return launch_cfg<true, false, false, BF16>(TileCfg{32, 32, 32}, M, N, K, A, lda, B, ldb, C, ldc,
                                                        kslices, kchunk, c_slice, nullptr, st);
        case GEMM_NN:
            if (!mask) return hipErrorInvalidValue;
            return launch_cfg<false, false, true, BF16>(dgrad_tile(M, kchunk), M, N, K, A, lda, B, ldb, C,
                                                        ldc, kslices, kchunk, c_slice, mask, st);
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemm_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0, const float* A1,
                            const float* B1, float* C1, int lda, int ldb, int ldc, int kslices, int kchunk,
                            int64_t c_slice, bool bf16, bool x16, hipStream_t st) {
    if (kchunk % 32 != 0 || kslices <= 0 || (x16 && !bf16)) return hipErrorInvalidValue;
    if (bf16) return launch_gemm_bf16_fwd2(M, N, K, A0, B0, C0, A1, B1, C1, lda, ldb, ldc, kslices, kchunk,
                                           c_slice, x16, st);
    // (the split was chosen for the 2M rows of both sets: gemm_fwd_split)
    if (2 * M >= kGemmX6MinRows)
        return launch_gemm_x6_fwd2(M, N, K, A0, B0, C0, A1, B1, C1, lda, ldb, ldc, kslices, kchunk, c_slice, st);
    const GemmParams p0{M, N, K, A0, lda, B0, ldb, C0, ldc, kchunk, c_slice, nullptr};
    const GemmParams p1{M, N, K, A1, lda, B1, ldb, C1, ldc, kchunk, c_slice, nullptr};
    const TileCfg c = fwd_tile(M, kchunk);
#define DQN_TILE(TBM, TBN, TBK) \
    if (c.bm == TBM && c.bn == TBN && c.bk == TBK) return launch_fwd2_tile<TBM, TBN, TBK>(p0, p1, kslices, st);
    DQN_TILE(32, 32, 32)
    DQN_TILE(32, 32, 64)
    DQN_TILE(64, 32, 32)
    DQN_TILE(64, 32, 64)
    DQN_TILE(64, 64, 32)
    DQN_TILE(64, 64, 64)
#undef DQN_TILE
    return hipErrorInvalidValue;
}

hipError_t launch_gemm(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B,
                       int ldb, float* C, int ldc, int kslices, int kchunk, int64_t c_slice,
                       const float* mask, bool bf16, bool x16, hipStream_t st, bool a16) {
    if (kchunk % 32 != 0 || ((x16 || a16) && !bf16)) return hipErrorInvalidValue;
    if (bf16)
        return launch_gemm_bf16(kind, M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, x16, st, a16);
    // the batch is M of the forward and the input gradient, K of the weight gradient
    if ((kind == GEMM_TN ? K : M) >= kGemmX6MinRows)
        return launch_gemm_x6(kind, M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
    return launch_gemm_prec<false>(kind, M, N, K, A, lda, B, ldb, C, ldc, kslices, kchunk, c_slice, mask, st);
}

}  // namespace dqn
