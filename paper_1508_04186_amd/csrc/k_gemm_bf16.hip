// The fully connected layer contractions on bf16 MFMA (fc1 forward with
// split-K partial sums, fc1 weight gradient, fc1 input gradient with the
// ReLU mask of the last conv layer), fp32 accumulation, in two arithmetics:
//  - the bf16-input variant: both operands rounded to bfloat16
//    (nearest-even) as they are staged (PARTS = 1);
//  - float32: both operands split exactly into three bfloat16 planes
//    (hi + mid + lo, as the float32 convolutions) as they are staged, and
//    six products per 32 k-values (hi*hi, hi*mid, mid*hi, hi*lo, mid*mid,
//    lo*hi; the dropped pairs are below 2^-23 of the product), which keeps
//    float32 accuracy (PARTS = 3).
//
// BMxBN output tiles on WGM x WGN waves, each wave a block of 16x16
// v_mfma_f32_16x16x32_bf16 tiles, k-stages of BK.  Each operand is staged
// in LDS as bf16 rows of BK k-values, so that the eight k-values a lane
// feeds one MFMA are one 16-byte read.  The 16-byte chunks of a row are
// permuted by an XOR with a function of the row (lds_off): the 16 rows a
// lane group reads land in 16 distinct groups of four banks, and so do the
// rows of the 8-byte stores of a transposed stage (below), which with a
// padded row stride instead hit four banks sixteen times.  An operand
// contiguous along k in memory is loaded as float4s along k; one contiguous
// along m or n as 4x4 blocks (four k-rows of four values) transposed in
// registers (v_perm_b32 for bf16 values), so every LDS store is 8 bytes.
// A stage wholly inside the operands is loaded without per-value bounds
// tests.  The next stage's global loads are in flight during the current
// stage's MFMAs.  The tiles are large where the batch is (each operand is
// re-read once per tile of the other dimension, from L2), and the forward
// pass splits K so that the launch still covers the chip.  The weight and
// input gradients take their tiles in the XCD-contiguous order of xcd_tile,
// so that the tiles of one XCD share the column operand (the activations of
// the weight gradient, the weight columns of the input gradient), which is
// then fetched into each L2 once instead of once per XCD; the forward does
// so when its k-slices are many (fwd_tile_order).
#include <algorithm>
#include <initializer_list>
#include <type_traits>

#include "common.h"

namespace dqn {
namespace {

struct GemmBf16Params {
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

__device__ __forceinline__ uint2 pack4(f4 v) {
    const uint32_t a = __builtin_bit_cast(unsigned short, (__bf16)v[0]);
    const uint32_t b = __builtin_bit_cast(unsigned short, (__bf16)v[1]);
    const uint32_t c = __builtin_bit_cast(unsigned short, (__bf16)v[2]);
    const uint32_t d = __builtin_bit_cast(unsigned short, (__bf16)v[3]);
    return uint2{a | (b << 16), c | (d << 16)};
}

// The three exact bf16 planes of four floats, packed as pack4 does.
__device__ __forceinline__ void split4(f4 v, uint2& h, uint2& m, uint2& l) {
    uint32_t hh[4], mm[4], ll[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        __bf16 a, b, c;
        split3(v[i], a, b, c);
        hh[i] = __builtin_bit_cast(unsigned short, a);
        mm[i] = __builtin_bit_cast(unsigned short, b);
        ll[i] = __builtin_bit_cast(unsigned short, c);
    }
    h = uint2{hh[0] | (hh[1] << 16), hh[2] | (hh[3] << 16)};
    m = uint2{mm[0] | (mm[1] << 16), mm[2] | (mm[3] << 16)};
    l = uint2{ll[0] | (ll[1] << 16), ll[2] | (ll[3] << 16)};
}

// Offset (bf16 elements) of k-value k of row `row` in a stage of BK
// k-values per row: 16-byte chunk k/8 of the row is stored at chunk
// (k/8) xor f(row).  f takes the row's position within a 256-byte bank line
// (128/BK rows share one when BK < 128) and the row's block of 16, so that
// rows 16a..16a+15 (one MFMA operand read) and rows 4l+i, l = 0..15 (one
// transposed store) each cover distinct chunks of the bank line.
template <int BK>
__device__ __forceinline__ int lds_off(int row, int k) {
    constexpr int CH = BK / 8, RPL = BK >= 128 ? 1 : 128 / BK, FM = (CH < 16 ? CH : 16) - 1;
    const int f = ((row / RPL) ^ (row >> 4)) & FM;
    return row * BK + (((k >> 3) ^ f) << 3) + (k & 7);
}

// One operand's stage: ROWS rows (m or n) x BK k, staged by NT threads.
// KCONT: the operand is contiguous along k in memory (element (r, k) at
// src[r*ld + k]); otherwise along r (element (r, k) at src[k*ld + r]).
// SRC16: the operand holds bfloat16 values (moved as they are) instead of
// floats (rounded as they are staged).  PARTS = 3: floats split into three
// planes, plane pl at s + pl * ROWS * RS.
template <int ROWS, int BK, int NT, bool KCONT, bool SRC16 = false, int PARTS = 1>
struct Stage {
    static constexpr int KQ = BK / 4;                 // four-value groups along k per row
    static constexpr int NV = ROWS * BK / 4 / NT;     // four-value groups per thread
    static constexpr int RS = BK;                     // LDS row stride (bf16)
    static_assert(NV * NT * 4 == ROWS * BK && (KCONT || NV % 4 == 0), "stage split");
    using V = std::conditional_t<SRC16, uint2, f4>;
    V v[NV];
    __device__ __forceinline__ static V zero() {
        if constexpr (SRC16) return uint2{0u, 0u};
        else return f4{0.f, 0.f, 0.f, 0.f};
    }
    __device__ __forceinline__ static V at(const float* __restrict__ src, size_t off) {
        if constexpr (SRC16) return *(const uint2*)((const __bf16*)src + off);
        else return *(const f4*)(src + off);
    }
    __device__ __forceinline__ void load(const float* __restrict__ src, int ld, int r0, int rlim, int k0, int klim) {
        if (r0 + ROWS <= rlim && k0 + BK <= klim) load_body<false>(src, ld, r0, rlim, k0, klim);
        else load_body<true>(src, ld, r0, rlim, k0, klim);
    }
    // GUARD: values outside rows < rlim, k < klim read as zero
    template <bool GUARD>
    __device__ __forceinline__ void load_body(const float* __restrict__ src, int ld, int r0, int rlim, int k0,
                                              int klim) {
        const int t = threadIdx.x;
        if constexpr (KCONT) {
            // value group u: row rt + RP u, k-values kt .. kt+3
            static_assert(NT % KQ == 0, "rows per pass");
            constexpr int RP = NT / KQ;
            const int rt = t / KQ, kt = 4 * (t % KQ);
            const size_t off0 = (size_t)(r0 + rt) * ld + k0 + kt;
#pragma unroll
            for (int u = 0; u < NV; ++u) {
                if (!GUARD || (r0 + rt + RP * u < rlim && k0 + kt < klim))
                    v[u] = at(src, off0 + (size_t)(RP * u) * ld);
                else
                    v[u] = zero();
            }
        } else {
            // 4x4 block w: rows rt .. rt+3, k-rows kt + 4 RK w .. +3
            constexpr int RQ = ROWS / 4;
            static_assert(NT % RQ == 0, "blocks per pass");
            constexpr int RK = NT / RQ;
            const int rt = 4 * (t % RQ), kt = 4 * (t / RQ);
            const size_t off0 = (size_t)(k0 + kt) * ld + r0 + rt;
#pragma unroll
            for (int w = 0; w < NV / 4; ++w)
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (!GUARD || (k0 + kt + 4 * RK * w + u < klim && r0 + rt < rlim))
                        v[4 * w + u] = at(src, off0 + (size_t)(4 * RK * w + u) * ld);
                    else
                        v[4 * w + u] = zero();
                }
        }
    }
    // the four values x at row r, k-values k..k+3 of every plane
    __device__ __forceinline__ static void put(__bf16* s, int off, f4 x) {
        if constexpr (PARTS == 3) {
            uint2 h, m, l;
            split4(x, h, m, l);
            *(uint2*)&s[off] = h;
            *(uint2*)&s[off + ROWS * RS] = m;
            *(uint2*)&s[off + 2 * ROWS * RS] = l;
        } else {
            *(uint2*)&s[off] = pack4(x);
        }
    }
    __device__ __forceinline__ void store(__bf16* s) const {
        const int t = threadIdx.x;
        static_assert(PARTS == 1 || !SRC16, "the exact split takes float input");
        if constexpr (KCONT) {
#pragma unroll
            for (int u = 0; u < NV; ++u) {
                const int q = t + NT * u, r = q / KQ, k = 4 * (q % KQ);
                if constexpr (SRC16) *(uint2*)&s[lds_off<BK>(r, k)] = v[u];
                else put(s, lds_off<BK>(r, k), v[u]);
            }
        } else {
#pragma unroll
            for (int w = 0; w < NV / 4; ++w) {
                const int b = t + NT * w;
                const int r = 4 * (b % (ROWS / 4)), k = 4 * (b / (ROWS / 4));
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if constexpr (SRC16) {
                        // bf16 value i of four k-rows: halves of packed words picked by v_perm_b32
                        const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
                        const uint2 a = v[4 * w], b = v[4 * w + 1], c = v[4 * w + 2], d = v[4 * w + 3];
                        *(uint2*)&s[lds_off<BK>(r + i, k)] =
                            uint2{__builtin_amdgcn_perm(i < 2 ? b.x : b.y, i < 2 ? a.x : a.y, sel),
                                  __builtin_amdgcn_perm(i < 2 ? d.x : d.y, i < 2 ? c.x : c.y, sel)};
                    } else {
                        put(s, lds_off<BK>(r + i, k), f4{v[4 * w][i], v[4 * w + 1][i], v[4 * w + 2][i], v[4 * w + 3][i]});
                    }
                }
            }
        }
    }
};

// TA: A(m,k) = A[k*lda + m] else A[m*lda + k].
// TB: B(k,n) = B[n*ldb + k] else B[k*ldb + n].
// MASK: C(m,n) = 0 where mask[m*ldc + n] <= 0.
// A16, B16, M16: A, B or the mask hold bfloat16 values.
// PARTS: 1 (operands rounded) or 3 (exact split, six products); the stages
// live at As, Bs (PARTS planes each).
template <int BM, int BN, int BK, int WGM, int WGN, bool TA, bool TB, bool MASK, bool A16 = false, bool B16 = false,
          bool M16 = false, int PARTS = 1>
__device__ __forceinline__ void gemm_bf16_body(const GemmBf16Params& p, TileXYZ tile, int z, __bf16* As,
                                               __bf16* Bs) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int WTM = BM / WGM, WTN = BN / WGN;     // wave tile
    constexpr int TM = WTM / 16, TN = WTN / 16;       // MFMA tiles per wave
    constexpr int RS = BK;
    static_assert(BK % 32 == 0 && WTM % 16 == 0 && WTN % 16 == 0, "tile shape");
    const int m0 = tile.x * BM, n0 = tile.y * BN;
    const int kbeg = z * p.kchunk, kend = min(p.K, kbeg + p.kchunk);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave / WGN) * WTM, wn = (wave % WGN) * WTN;

    Stage<BM, BK, NT, !TA, A16, PARTS> sa;
    Stage<BN, BK, NT, TB, B16, PARTS> sb;
    f4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    if (kbeg < kend) {
        sa.load(p.A, p.lda, m0, p.M, kbeg, kend);
        sb.load(p.B, p.ldb, n0, p.N, kbeg, kend);
    }
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        sa.store(As);
        sb.store(Bs);
        __syncthreads();
        if (k0 + BK < kend) {   // in flight during the MFMAs below
            sa.load(p.A, p.lda, m0, p.M, k0 + BK, kend);
            sb.load(p.B, p.ldb, n0, p.N, k0 + BK, kend);
        }
#pragma unroll
        for (int kb = 0; kb < BK / 32; ++kb) {
            bf16x8 a[PARTS][TM], b[PARTS][TN];
#pragma unroll
            for (int pl = 0; pl < PARTS; ++pl) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    a[pl][i] = *(const bf16x8*)&As[pl * BM * RS + lds_off<BK>(wm + 16 * i + li, 32 * kb + 8 * g)];
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    b[pl][j] = *(const bf16x8*)&Bs[pl * BN * RS + lds_off<BK>(wn + 16 * j + li, 32 * kb + 8 * g)];
            }
            if constexpr (PARTS == 1) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32bf16(a[0][i], b[0][j], acc[i][j]);
            } else {
                // the six plane pairs (pa, pb), smallest first; each over all tiles
                constexpr int PA[6] = {2, 1, 0, 1, 0, 0}, PB[6] = {0, 1, 2, 0, 1, 0};
#pragma unroll
                for (int q = 0; q < 6; ++q)
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = mfma16x16x32bf16(a[PA[q]][i], b[PB[q]][j], acc[i][j]);
            }
        }
        __syncthreads();
    }

    // D[4g + r][li] of tile (i, j): row m0 + wm + 16i + 4g + r, column n0 + wn + 16j + li
    float* Cz = p.C + (size_t)z * p.c_slice;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + wn + 16 * j + li;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm + 16 * i + 4 * g + r;
                if (m < p.M && n < p.N) {
                    float v = acc[i][j][r];
                    if constexpr (MASK && M16) v = (float)((const __bf16*)p.mask)[(size_t)m * p.ldc + n] > 0.f ? v : 0.f;
                    else if constexpr (MASK) v = p.mask[(size_t)m * p.ldc + n] > 0.f ? v : 0.f;
                    Cz[(size_t)m * p.ldc + n] = v;
                }
            }
        }
}

template <int BM, int BN, int BK>
constexpr int gemm_lds_bf16(int parts) { return parts * (BM + BN) * BK; }   // bf16 elements

template <int BM, int BN, int BK, int WGM, int WGN, bool TA, bool TB, bool MASK, bool A16, bool B16, bool M16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_kernel(GemmBf16Params p) {
    __shared__ __align__(16) __bf16 As[BM * BK];
    __shared__ __align__(16) __bf16 Bs[BN * BK];
    const TileXYZ tile = !TA && TB ? fwd_tile_order() : xcd_tile<false>();
    gemm_bf16_body<BM, BN, BK, WGM, WGN, TA, TB, MASK, A16, B16, M16>(p, tile, tile.z, As, Bs);
}

// float32 operands, exact three-plane split (stages in dynamic LDS)
template <int BM, int BN, int BK, int WGM, int WGN, bool TA, bool TB, bool MASK>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_x6_kernel(GemmBf16Params p) {
    extern __shared__ __align__(16) __bf16 smem_x6[];
    const TileXYZ tile = !TA && TB ? fwd_tile_order() : xcd_tile<false>();
    gemm_bf16_body<BM, BN, BK, WGM, WGN, TA, TB, MASK, false, false, false, 3>(p, tile, tile.z, smem_x6,
                                                                              smem_x6 + 3 * BM * BK);
}

// Two forward contractions of one shape (the online network on s, the
// target network on s'): k-slices z < ks0 run p0, the rest p1.
template <int BM, int BN, int BK, int WGM, int WGN, bool A16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_fwd2_kernel(GemmBf16Params p0, GemmBf16Params p1,
                                                                       int ks0) {
    __shared__ __align__(16) __bf16 As[BM * BK];
    __shared__ __align__(16) __bf16 Bs[BN * BK];
    const TileXYZ tile = fwd_tile_order();
    const int z = tile.z;
    if (z < ks0)
        gemm_bf16_body<BM, BN, BK, WGM, WGN, false, true, false, A16>(p0, tile, z, As, Bs);
    else
        gemm_bf16_body<BM, BN, BK, WGM, WGN, false, true, false, A16>(p1, tile, z - ks0, As, Bs);
}

template <int BM, int BN, int BK, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_x6_fwd2_kernel(GemmBf16Params p0, GemmBf16Params p1, int ks0) {
    extern __shared__ __align__(16) __bf16 smem_x6[];
    __bf16* Bs = smem_x6 + 3 * BM * BK;
    const TileXYZ tile = fwd_tile_order();
    const int z = tile.z;
    if (z < ks0)
        gemm_bf16_body<BM, BN, BK, WGM, WGN, false, true, false, false, false, false, 3>(p0, tile, z, smem_x6, Bs);
    else
        gemm_bf16_body<BM, BN, BK, WGM, WGN, false, true, false, false, false, false, 3>(p1, tile, z - ks0, smem_x6,
                                                                                         Bs);
}

template <int BM, int BN, int BK, int WGM, int WGN, bool TA, bool TB, bool MASK>
hipError_t gemm_x6_launch(const GemmBf16Params& prm, int kslices, hipStream_t st) {
    const dim3 grid((unsigned)((prm.M + BM - 1) / BM), (unsigned)((prm.N + BN - 1) / BN), (unsigned)kslices);
    auto kern = gemm_x6_kernel<BM, BN, BK, WGM, WGN, TA, TB, MASK>;
    const size_t lds = (size_t)gemm_lds_bf16<BM, BN, BK>(3) * 2;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, grid, dim3(64 * WGM * WGN), lds, st, prm);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WGM, int WGN>
hipError_t gemm_x6_fwd2_launch(const GemmBf16Params& p0, const GemmBf16Params& p1, int kslices, hipStream_t st) {
    const dim3 grid((unsigned)((p0.M + BM - 1) / BM), (unsigned)((p0.N + BN - 1) / BN), (unsigned)(2 * kslices));
    auto kern = gemm_x6_fwd2_kernel<BM, BN, BK, WGM, WGN>;
    const size_t lds = (size_t)gemm_lds_bf16<BM, BN, BK>(3) * 2;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, grid, dim3(64 * WGM * WGN), lds, st, p0, p1, kslices);
    return hipGetLastError();
}

template <int BM, int BN, int BK, int WGM, int WGN>
hipError_t gemm_bf16_fwd2_launch(const GemmBf16Params& p0, const GemmBf16Params& p1, int kslices, bool a16,
                                 hipStream_t st) {
    const dim3 grid((unsigned)((p0.M + BM - 1) / BM), (unsigned)((p0.N + BN - 1) / BN), (unsigned)(2 * kslices));
    if (a16)
        hipLaunchKernelGGL((gemm_bf16_fwd2_kernel<BM, BN, BK, WGM, WGN, true>), grid, dim3(64 * WGM * WGN), 0, st, p0,
                           p1, kslices);
    else
        hipLaunchKernelGGL((gemm_bf16_fwd2_kernel<BM, BN, BK, WGM, WGN, false>), grid, dim3(64 * WGM * WGN), 0, st, p0,
                           p1, kslices);
    return hipGetLastError();
}

// x16: the activation operand (A of the forward, B of the weight gradient,
// the mask of the input gradient) holds bfloat16 values.  a16: A of the
// weight or input gradient (the pre-activation gradient) holds bfloat16
// values.
template <int BM, int BN, int BK, int WGM, int WGN, bool TA, bool TB, bool MASK>
hipError_t gemm_bf16_launch(const GemmBf16Params& prm, int kslices, bool x16, hipStream_t st, bool a16 = false) {
    const dim3 grid((unsigned)((prm.M + BM - 1) / BM), (unsigned)((prm.N + BN - 1) / BN), (unsigned)kslices);
    constexpr bool FWD = !TA && TB && !MASK, WGR = TA && !TB && !MASK;
    if (a16) {
        if constexpr (WGR || MASK) {
            if (x16)
                hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, TA, TB, MASK, true, WGR, MASK>), grid,
                                   dim3(64 * WGM * WGN), 0, st, prm);
            else
                hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, TA, TB, MASK, true, false, false>), grid,
                                   dim3(64 * WGM * WGN), 0, st, prm);
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (x16)
        hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, TA, TB, MASK, FWD, WGR, MASK>), grid,
                           dim3(64 * WGM * WGN), 0, st, prm);
    else
        hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, BK, WGM, WGN, TA, TB, MASK, false, false, false>), grid,
                           dim3(64 * WGM * WGN), 0, st, prm);
    return hipGetLastError();
}

// Forward and input-gradient tiles: 128x256 and 128x128 from kBf16BigRows
// rows on (fewer re-reads of the operands), else 64x64 (more workgroups).
constexpr int kBf16BigRows = 1024;

}  // namespace

void gemm_fwd_split_bf16(int rows, int N, int K, int* ks, int* kchunk) {
    const bool big = rows >= kBf16BigRows;
    const int bm = big ? 128 : 64, bn = big ? 256 : 64;
    const long tiles = (long)((rows + bm - 1) / bm) * ((N + bn - 1) / bn);
    const int steps = (K + 63) / 64;                       // 64-wide k-steps
    const long target = big ? 256 : 768;                   // workgroups: one (large tiles) or three per CU
    const int want = (int)std::min<long>(steps, std::max<long>(1, (target + tiles - 1) / tiles));
    *kchunk = (steps + want - 1) / want * 64;
    *ks = (K + *kchunk - 1) / *kchunk;
}

// The float32 forward's split (from kGemmX6MinRows rows): 128x256 tiles
// from kBf16BigRows rows, else 64x64, and enough k-slices (of a multiple of
// 64) for about 256 workgroups (the head sums the slices).  (128x128 tiles
// in two slices instead of four, batch 2,048: 85 -> 94 us, a forward-only
// batch of 8,192: 165 -> 188 us.)
void gemm_fwd_split_x6(int rows, int N, int K, int* ks, int* kchunk) {
    const bool big = rows >= kBf16BigRows;
    const int bm = big ? 128 : 64, bn = big ? 256 : 64;
    const long tiles = (long)((rows + bm - 1) / bm) * ((N + bn - 1) / bn);
    const int steps = (K + 63) / 64;
    const int want = (int)std::min<long>(steps, std::max<long>(1, (256 + tiles - 1) / tiles));
    *kchunk = (steps + want - 1) / want * 64;
    *ks = (K + *kchunk - 1) / *kchunk;
}

hipError_t launch_gemm_x6_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0, const float* A1,
                               const float* B1, float* C1, int lda, int ldb, int ldc, int kslices, int kchunk,
                               int64_t c_slice, hipStream_t st) {
    if (M <= 0 || N <= 0 || K <= 0 || kslices <= 0 || kchunk % 32 != 0 || K % 4) return hipErrorInvalidValue;
    for (const float* x : {A0, B0, A1, B1})
        if ((uintptr_t)x % 16) return hipErrorInvalidValue;
    if (lda % 4 || ldb % 4) return hipErrorInvalidValue;
    const GemmBf16Params p0{M, N, K, A0, lda, B0, ldb, C0, ldc, kchunk, c_slice, nullptr};
    const GemmBf16Params p1{M, N, K, A1, lda, B1, ldb, C1, ldc, kchunk, c_slice, nullptr};
    if (M >= kBf16BigRows) return gemm_x6_fwd2_launch<128, 256, 32, 2, 4>(p0, p1, kslices, st);
    return gemm_x6_fwd2_launch<64, 64, 64, 2, 2>(p0, p1, kslices, st);
}

hipError_t launch_gemm_x6(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B, int ldb,
                          float* C, int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                          hipStream_t st) {
    if (M <= 0 || N <= 0 || K <= 0 || kslices <= 0 || kchunk % 32 != 0) return hipErrorInvalidValue;
    if ((uintptr_t)A % 16 || (uintptr_t)B % 16 || lda % 4 || ldb % 4) return hipErrorInvalidValue;
    const GemmBf16Params prm{M, N, K, A, lda, B, ldb, C, ldc, kchunk, c_slice, mask};
    switch (kind) {
        case GEMM_NT:
            if (mask || K % 4) return hipErrorInvalidValue;
            if (M >= kBf16BigRows) return gemm_x6_launch<128, 256, 32, 2, 4, false, true, false>(prm, kslices, st);
            return gemm_x6_launch<64, 64, 64, 2, 2, false, true, false>(prm, kslices, st);
        case GEMM_TN:   // (the output is hidden x flat: 64x64 tiles, or 128x128 over k-slices)
            if (mask || M % 4 || N % 4) return hipErrorInvalidValue;
            if (kslices >= 2) return gemm_x6_launch<128, 128, 64, 2, 4, true, false, false>(prm, kslices, st);
            return gemm_x6_launch<64, 64, 64, 2, 2, true, false, false>(prm, kslices, st);
        case GEMM_NN:
            if (!mask || K % 4 || N % 4) return hipErrorInvalidValue;
            return gemm_x6_launch<64, 64, 64, 2, 2, false, false, true>(prm, kslices, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_bf16_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0,
                                 const float* A1, const float* B1, float* C1, int lda, int ldb, int ldc,
                                 int kslices, int kchunk, int64_t c_slice, bool x16, hipStream_t st) {
    if (M <= 0 || N <= 0 || K <= 0 || kslices <= 0 || kchunk % 32 != 0 || K % 4) return hipErrorInvalidValue;
    for (const float* x : {A0, B0, A1, B1})
        if ((uintptr_t)x % 16) return hipErrorInvalidValue;
    if (lda % 4 || ldb % 4) return hipErrorInvalidValue;
    const GemmBf16Params p0{M, N, K, A0, lda, B0, ldb, C0, ldc, kchunk, c_slice, nullptr};
    const GemmBf16Params p1{M, N, K, A1, lda, B1, ldb, C1, ldc, kchunk, c_slice, nullptr};
    if (M >= kBf16BigRows) return gemm_bf16_fwd2_launch<128, 256, 64, 2, 4>(p0, p1, kslices, x16, st);
    return gemm_bf16_fwd2_launch<64, 64, 128, 2, 2>(p0, p1, kslices, x16, st);
}

hipError_t launch_gemm_bf16(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B, int ldb,
                            float* C, int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                            bool x16, hipStream_t st, bool a16) {
    if (M <= 0 || N <= 0 || K <= 0 || kslices <= 0 || kchunk % 32 != 0) return hipErrorInvalidValue;
    if ((uintptr_t)A % 16 || (uintptr_t)B % 16 || lda % 4 || ldb % 4) return hipErrorInvalidValue;
    const GemmBf16Params prm{M, N, K, A, lda, B, ldb, C, ldc, kchunk, c_slice, mask};
    if (a16 && kind == GEMM_NT) return hipErrorInvalidValue;
    switch (kind) {
        case GEMM_NT:
            if (K % 4) return hipErrorInvalidValue;
            if (M >= kBf16BigRows) return gemm_bf16_launch<128, 256, 64, 2, 4, false, true, false>(prm, kslices, x16, st);
            return gemm_bf16_launch<64, 64, 128, 2, 2, false, true, false>(prm, kslices, x16, st);
        case GEMM_TN:
            if (M % 4 || N % 4) return hipErrorInvalidValue;
            return gemm_bf16_launch<64, 64, 128, 2, 2, true, false, false>(prm, kslices, x16, st, a16);
        case GEMM_NN:
            if (!mask || K % 4 || N % 4) return hipErrorInvalidValue;
            if (M >= kBf16BigRows)
                return gemm_bf16_launch<128, 128, 64, 2, 4, false, false, true>(prm, kslices, x16, st, a16);
            return gemm_bf16_launch<64, 64, 128, 2, 2, false, false, true>(prm, kslices, x16, st, a16);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn
