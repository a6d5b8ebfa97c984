// Forward convolution of the fp32 conv layers (Sec. III.A) at large batch as
// an implicit GEMM over all samples at once: M = output pixels of every
// sample (flattened, so a 7x7 or 9x9 map wastes no MFMA rows), N = output
// channels, K = cin*k*k in the weights' own [o][c][ky][kx] order.  A 64x64
// output tile per workgroup, four waves of 32x32 (four independent MFMA
// accumulators each); the A tile is gathered from the NCHW input (an
// im2col row per pixel, built on the fly) and the B tile read from the
// weight rows, both into k-contiguous LDS rows padded to 4 floats mod 64
// (conflict-free MFMA reads), with the next k-stage's loads in flight
// during the current stage's MFMAs.  Bias + ReLU epilogue.  Samples below
// n_a use weight set a, the rest set b; no tile straddles the two.
#include <algorithm>

#include "common.h"

namespace dqn {
namespace {

constexpr int IG_WG = 256;
constexpr int IG_BM = 64, IG_BN = 64, IG_BK = 32;
constexpr int IG_LD = IG_BK + 4;  // = 4 mod 64 after the 64-row stride math below

// One 32-deep k-stage of a wave's TMxTN block of 16x16 MFMA tiles, both
// operands staged k-contiguous as [row][IG_LD] fp32 (A rows wm + 16i + li,
// B rows wn + 16j + li): eight fp32 steps, or with BF16 one bf16-input step
// on the values rounded to bfloat16 (bf16_operand's k order).
template <int TM, int TN, bool BF16>
__device__ __forceinline__ void mfma_stage(f4 (&acc)[TM][TN], const float* As, const float* Bs, int wm, int wn,
                                           int li, int g) {
    if constexpr (BF16) {
        bf16x8 a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const float* r = As + (wm + i * 16 + li) * IG_LD;
            a[i] = bf16_operand([&](int k) { return r[k]; }, g);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const float* r = Bs + (wn + j * 16 + li) * IG_LD;
            b[j] = bf16_operand([&](int k) { return r[k]; }, g);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x32bf16(a[i], b[j], acc[i][j]);
    } else {
#pragma unroll
        for (int kk = 0; kk < IG_BK / 4; ++kk) {
            float a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) a[i] = As[(wm + i * 16 + li) * IG_LD + kk * 4 + g];
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = Bs[(wn + j * 16 + li) * IG_LD + kk * 4 + g];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = mfma16x16x4(a[i], b[j], acc[i][j]);
        }
    }
}

struct IgemmFwdParams {
    const float* in;       // [n][cin][ih][iw]
    int n, n_a;
    int tiles_a;           // M-tiles of the first weight set
    const float *w_a, *b_a, *w_b, *b_b;
    float* out;            // [n][cout][oh][ow]
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool BF16>
__global__ __launch_bounds__(IG_WG) void conv_igemm_fwd_kernel(IgemmFwdParams p) {
    constexpr int P = OH * OW;
    constexpr int KK = K * K;
    constexpr int KT = CIN * KK;                 // contraction length
    static_assert(KT % IG_BK == 0, "whole k-stages");
    static_assert(COUT % IG_BN == 0, "whole N-tiles");
    __shared__ __align__(16) float As[IG_BM * IG_LD];
    __shared__ __align__(16) float Bs[IG_BN * IG_LD];

    // tile -> weight set and first pixel (global pixel index over samples)
    const int nt = blockIdx.x % (COUT / IG_BN);
    int mt = blockIdx.x / (COUT / IG_BN);
    const bool second = mt >= p.tiles_a;
    const int m_lo = second ? p.n_a * P : 0;             // first pixel of this set
    const int m_hi = second ? p.n * P : p.n_a * P;       // end of this set
    if (second) mt -= p.tiles_a;
    const int m0 = m_lo + mt * IG_BM;
    const int n0 = nt * IG_BN;
    const float* __restrict__ W = second ? p.w_b : p.w_a;
    const float* __restrict__ bias = second ? p.b_b : p.b_a;

    const int t = threadIdx.x;
    // A loads: thread t gathers pixel m0 + t/4, k = k0 + 8*(t%4) .. +7
    const int am = t >> 2, ak = (t & 3) * 8;
    const int gm = m0 + am;
    const bool avalid = gm < m_hi;
    const int gmc = avalid ? gm : m_lo;
    const int sn = gmc / P, pp = gmc - sn * P;
    const int oy = pp / OW, ox = pp - oy * OW;
    const float* __restrict__ abase = p.in + (size_t)sn * CIN * IH * IW + (S * oy) * IW + S * ox;
    // B loads: thread t reads row o = n0 + t/4, k = k0 + 8*(t%4) .. +7 (two float4)
    const float* __restrict__ bbase = W + (size_t)(n0 + am) * KT + ak;

    float ra[8];
    f4 rb[2];
    auto load = [&](int k0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int k = k0 + ak + e;
            const int c = k / KK, r = k - c * KK;
            const int ky = r / K, kx = r - ky * K;
            ra[e] = avalid ? abase[c * IH * IW + ky * IW + kx] : 0.f;
        }
        rb[0] = *(const f4*)(bbase + k0);
        rb[1] = *(const f4*)(bbase + k0 + 4);
    };
    auto store = [&]() {
        *(f4*)&As[am * IG_LD + ak] = f4{ra[0], ra[1], ra[2], ra[3]};
        *(f4*)&As[am * IG_LD + ak + 4] = f4{ra[4], ra[5], ra[6], ra[7]};
        *(f4*)&Bs[am * IG_LD + ak] = rb[0];
        *(f4*)&Bs[am * IG_LD + ak + 4] = rb[1];
    };

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
    f4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    load(0);
    for (int k0 = 0; k0 < KT; k0 += IG_BK) {
        store();
        __syncthreads();
        if (k0 + IG_BK < KT) load(k0 + IG_BK);   // in flight during the MFMAs below
        mfma_stage<2, 2, BF16>(acc, As, Bs, wm, wn, li, g);
        __syncthreads();
    }

    // D[4g + r][li] of tile (i, j): pixel m0 + wm + 16i + 4g + r, channel
    // n0 + wn + 16j + li.
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int o = n0 + wn + j * 16 + li;
        const float bo = bias[o];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm + i * 16 + 4 * g + r;
                if (m < m_hi) {
                    const int s2 = m / P, q = m - s2 * P;
                    p.out[((size_t)s2 * COUT + o) * P + q] = fmaxf(acc[i][j][r] + bo, 0.f);
                }
            }
    }
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool BF16>
hipError_t igemm_launch(const float* in, int n_a, int n, const float* w_a, const float* b_a,
                        const float* w_b, const float* b_b, float* out, hipStream_t st) {
    constexpr int P = OH * OW;
    if (((uintptr_t)w_a & 15) || ((uintptr_t)w_b & 15)) return hipErrorInvalidValue;
    const long tiles_a = ((long)n_a * P + IG_BM - 1) / IG_BM;
    const long tiles_b = ((long)(n - n_a) * P + IG_BM - 1) / IG_BM;
    const long blocks = (tiles_a + tiles_b) * (COUT / IG_BN);
    if (blocks <= 0 || blocks > 0x7fffffffL || (long)n * P > 0x7fffffffL) return hipErrorInvalidValue;
    IgemmFwdParams prm{in, n, n_a, (int)tiles_a, w_a, b_a, w_b, b_b, out};
    hipLaunchKernelGGL((conv_igemm_fwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW, BF16>), dim3((unsigned)blocks),
                       dim3(IG_WG), 0, st, prm);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Input gradient as an implicit GEMM per stride phase (py, px): input pixels
// (S*qy + py, S*qx + px) of every sample (M), input channels (N), and the
// contraction over (ty, tx, o) with ky = py + S*ty, kx = px + S*tx, so no
// MFMA multiplies a structural zero:
//   din[n][c][y][x] = [h_in > 0] * sum W[o][c][ky][kx] * dz[n][o][qy-ty][qx-tx]
// (dz taken as 0 outside the output map).  64 x BN tiles, k-stages of 32.
struct IgemmDgradParams {
    const float* dz;     // [n][cout][oh][ow]
    const float* w;      // [cout][cin][k][k]
    const float* h_in;   // [n][cin][ih][iw] (ReLU mask)
    float* din;          // [n][cin][ih][iw]
    int n, mtiles;       // samples; M-tiles per phase
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int BN, bool BF16>
__global__ __launch_bounds__(IG_WG) void conv_igemm_dgrad_kernel(IgemmDgradParams p) {
    static_assert(K % S == 0 && IH % S == 0 && IW % S == 0, "phases must tile the input");
    constexpr int T = K / S;
    constexpr int QH = IH / S, QW = IW / S, QP = QH * QW;
    constexpr int KT = COUT * T * T;
    constexpr int TN = BN / 32;                       // MFMA N-tiles per wave
    static_assert(KT % IG_BK == 0 && CIN % BN == 0 && (BN == 32 || BN == 64), "tile shape");
    __shared__ __align__(16) float As[IG_BM * IG_LD];
    __shared__ __align__(16) float Bs[BN * IG_LD];

    int b = blockIdx.x;
    const int nt = b % (CIN / BN);
    b /= (CIN / BN);
    const int mt = b % p.mtiles;
    const int ph = b / p.mtiles;
    const int py = ph / S, px = ph - (ph / S) * S;
    const int m0 = mt * IG_BM, c0 = nt * BN;
    const int mcount = p.n * QP;

    const int t = threadIdx.x;
    // The contraction runs over k = tap * COUT + o (tap = ty*T + tx), so a
    // k-stage of 32 lies within one tap and a thread's 8 values are 8
    // consecutive output channels: each address is a per-thread base plus a
    // compile-time stride.
    static_assert(COUT % IG_BK == 0, "a k-stage lies within one tap");
    // A: thread t gathers phase pixel m0 + t/4, channels o0 + 8*(t%4) .. +7
    const int am = t >> 2, ak = (t & 3) * 8;
    const int gm = m0 + am;
    const bool avalid = gm < mcount;
    const int gmc = avalid ? gm : 0;
    const int sn = gmc / QP, q = gmc - sn * QP;
    const int qy = q / QW, qx = q - (q / QW) * QW;
    const float* __restrict__ dzn = p.dz + (size_t)sn * COUT * OH * OW + (size_t)ak * OH * OW;
    // B: thread t (t < 4*BN) gathers channel c0 + t/4 of the same 8 k
    const bool bthread = t < 4 * BN;
    const float* __restrict__ wc =
        p.w + (size_t)ak * CIN * K * K + (size_t)(c0 + (bthread ? am : 0)) * K * K + py * K + px;

    float ra[8], rb[8];
    auto load = [&](int k0) {
        const int tap = k0 / COUT, ob = k0 - tap * COUT;
        const int ty = tap / T, tx = tap - ty * T;
        const int y = qy - ty, x = qx - tx;
        const bool av = avalid && y >= 0 && y < OH && x >= 0 && x < OW;
        const float* ap = dzn + (size_t)ob * OH * OW + (av ? y * OW + x : 0);
        const float* bp = wc + (size_t)ob * CIN * K * K + (S * ty) * K + S * tx;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            ra[e] = av ? ap[e * OH * OW] : 0.f;
            rb[e] = bthread ? bp[e * CIN * K * K] : 0.f;
        }
    };
    auto store = [&]() {
        *(f4*)&As[am * IG_LD + ak] = f4{ra[0], ra[1], ra[2], ra[3]};
        *(f4*)&As[am * IG_LD + ak + 4] = f4{ra[4], ra[5], ra[6], ra[7]};
        if (bthread) {
            *(f4*)&Bs[am * IG_LD + ak] = f4{rb[0], rb[1], rb[2], rb[3]};
            *(f4*)&Bs[am * IG_LD + ak + 4] = f4{rb[4], rb[5], rb[6], rb[7]};
        }
    };

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave >> 1) * 32, wn = (wave & 1) * (BN / 2);
    f4 acc[2][TN];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    load(0);
    for (int k0 = 0; k0 < KT; k0 += IG_BK) {
        store();
        __syncthreads();
        if (k0 + IG_BK < KT) load(k0 + IG_BK);
        mfma_stage<2, TN, BF16>(acc, As, Bs, wm, wn, li, g);
        __syncthreads();
    }

#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int c = c0 + wn + j * 16 + li;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm + i * 16 + 4 * g + r;
                if (m < mcount) {
                    const int s2 = m / QP, q2 = m - s2 * QP;
                    const int y = S * (q2 / QW) + py, x = S * (q2 % QW) + px;
                    const size_t idx = (((size_t)s2 * CIN + c) * IH + y) * IW + x;
                    p.din[idx] = p.h_in[idx] > 0.f ? acc[i][j][r] : 0.f;
                }
            }
    }
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int BN, bool BF16>
hipError_t igemm_dgrad_launch(const float* dz, const float* w, const float* h_in, float* din, int n,
                              hipStream_t st) {
    constexpr int QP = (IH / S) * (IW / S);
    const long mtiles = ((long)n * QP + IG_BM - 1) / IG_BM;
    const long blocks = (long)S * S * mtiles * (CIN / BN);
    if (n <= 0 || blocks > 0x7fffffffL || (long)n * QP > 0x7fffffffL) return hipErrorInvalidValue;
    IgemmDgradParams prm{dz, w, h_in, din, n, (int)mtiles};
    hipLaunchKernelGGL((conv_igemm_dgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, BN, BF16>), dim3((unsigned)blocks),
                       dim3(IG_WG), 0, st, prm);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient as an implicit GEMM: M = output channels, N = weight
// columns (c, ky, kx), contraction over the output pixels of every sample,
// split into chunks of `chunk` pixels (one partial-sum slot each, written
// without atomics and reduced later in a fixed order).  A = dz rows, B =
// im2col of the layer input (bytes scaled by in_scale at the end for the
// network input).  64x64 tiles (BM = 32 when cout is 32), k-stages of 32
// pixels; workgroups of the first N-tile also sum dz per channel (the bias
// gradient partials).
struct IgemmWgradParams {
    const void* in;      // [n][cin][ih][iw], bytes or floats
    const int64_t* idx;  // bytes from replay records: sample j is record idx[j] (NULL: dense)
    int64_t in_stride;   // bytes between samples (records)
    const float* dz;     // [n][cout][oh][ow]
    float* wpart;        // [chunks][cout][cin*k*k]
    float* bpart;        // [chunks][cout]
    float in_scale;
    int n, chunk, chunks;
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8, int BM, bool BF16>
__global__ __launch_bounds__(IG_WG) void conv_igemm_wgrad_kernel(IgemmWgradParams p) {
    constexpr int P = OH * OW;
    constexpr int KK = K * K, KT = CIN * KK;
    constexpr int TM = BM / 32;                       // MFMA M-tiles per wave
    static_assert(KT % IG_BN == 0 && COUT % BM == 0 && (BM == 32 || BM == 64), "tile shape");
    __shared__ __align__(16) float As[BM * IG_LD];
    __shared__ __align__(16) float Bs[IG_BN * IG_LD];

    int b = blockIdx.x;
    const int nt = b % (KT / IG_BN);
    b /= (KT / IG_BN);
    const int mt = b % (COUT / BM);
    const int ch = b / (COUT / BM);
    const int o0 = mt * BM, k0c = nt * IG_BN;
    const int pix0 = ch * p.chunk;
    const int pix1 = min(p.n * P, pix0 + p.chunk);

    const int t = threadIdx.x;
    // A thread loads one pixel of the stage (pix = t % 32) for 8 tile rows
    // (group t / 32): rows are output channels for A and weight columns for
    // B, so the pixel is decoded once per stage and each value's address is
    // a per-thread base plus a fixed offset.
    const int pix = t & 31, grp = t >> 5;
    const bool athread = grp < BM / 8;
    int boff[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int kc = k0c + grp * 8 + e;
        const int c = kc / KK, r = kc - c * KK;
        const int ky = r / K, kx = r - ky * K;
        boff[e] = (c * IH + ky) * IW + kx;           // element offset within a sample
    }
    const float* __restrict__ dzo = p.dz + (size_t)(o0 + (athread ? grp * 8 : 0)) * P;

    float ra[8], rb[8];
    auto load = [&](int s0) {
        const int m = s0 + pix;
        const bool v = m < pix1;
        const int mc = v ? m : pix0;
        const int sn = mc / P, q = mc - sn * P;
        const int oy = q / OW, ox = q - oy * OW;
        const float* ap = dzo + (size_t)sn * COUT * P + q;
        const int64_t rec = p.idx ? p.idx[sn] : sn;
        const int pofs = (S * oy) * IW + S * ox;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            ra[e] = (athread && v) ? ap[e * P] : 0.f;
            if constexpr (U8) {
                const unsigned char* src = (const unsigned char*)p.in + rec * p.in_stride + pofs;
                rb[e] = v ? (float)src[boff[e]] : 0.f;
            } else {
                const float* src = (const float*)((const char*)p.in + rec * p.in_stride) + pofs;
                rb[e] = v ? src[boff[e]] : 0.f;
            }
        }
    };
    float bsum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    auto store = [&]() {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (athread) {
                As[(grp * 8 + e) * IG_LD + pix] = ra[e];
                if (nt == 0) bsum[e] += ra[e];
            }
            Bs[(grp * 8 + e) * IG_LD + pix] = rb[e];
        }
    };

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int wm = (wave >> 1) * (BM / 2), wn = (wave & 1) * 32;
    f4 acc[TM][2];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    load(pix0);
    for (int s0 = pix0; s0 < pix1; s0 += IG_BK) {
        store();
        __syncthreads();
        if (s0 + IG_BK < pix1) load(s0 + IG_BK);
        mfma_stage<TM, 2, BF16>(acc, As, Bs, wm, wn, li, g);
        __syncthreads();
    }

    // D[4g + r][li] of tile (i, j): channel o0 + wm + 16i + 4g + r, column
    // k0c + wn + 16j + li.
    float* wp = p.wpart + (size_t)ch * COUT * KT;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                wp[(size_t)(o0 + wm + i * 16 + 4 * g + r) * KT + k0c + wn + j * 16 + li] = acc[i][j][r] * p.in_scale;
    if (nt == 0) {
        // bias partial: the 32 pixel lanes of each row group combine their
        // sums in a fixed butterfly order
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float v = bsum[e];
#pragma unroll
            for (int m = 1; m < 32; m <<= 1) v += __shfl_xor(v, m, 64);
            if (athread && pix == 0) p.bpart[(size_t)ch * COUT + o0 + grp * 8 + e] = v;
        }
    }
}

// Pixels per weight-gradient chunk for n samples: enough chunks for about 512
// workgroups, whole k-stages.
template <int CIN, int K, int COUT, int P, int BM>
int igemm_wgrad_chunk(int n) {
    const long tiles = (long)(COUT / BM) * (CIN * K * K / IG_BN);
    const long want = std::max<long>(1, 512 / tiles);
    const long npix = (long)n * P;
    long chunk = (npix + want - 1) / want;
    chunk = (chunk + IG_BK - 1) / IG_BK * IG_BK;
    return (int)std::max<long>(chunk, IG_BK);
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8, int BM, bool BF16>
hipError_t igemm_wgrad_launch(const ConvIn& in, const float* dz, int n, float* wpart, float* bpart,
                              float in_scale, hipStream_t st) {
    constexpr int P = OH * OW;
    if (n <= 0 || (long)n * P > 0x7fffffffL || in.off != 0) return hipErrorInvalidValue;
    const int chunk = igemm_wgrad_chunk<CIN, K, COUT, P, BM>(n);
    const int chunks = (int)(((long)n * P + chunk - 1) / chunk);
    const long blocks = (long)chunks * (COUT / BM) * (CIN * K * K / IG_BN);
    IgemmWgradParams prm{in.base, in.idx, in.stride, dz, wpart, bpart, in_scale, n, chunk, chunks};
    hipLaunchKernelGGL((conv_igemm_wgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8, BM, BF16>), dim3((unsigned)blocks),
                       dim3(IG_WG), 0, st, prm);
    return hipGetLastError();
}

}  // namespace

bool conv_igemm_fwd_supported(ConvId id) { return id == CONV_L2 || id == CONV_L3; }

hipError_t launch_conv_igemm_fwd(ConvId id, const float* in, int n_a, int n, const float* w_a,
                                 const float* b_a, const float* w_b, const float* b_b, float* out,
                                 bool bf16, bool in16, bool out16, const float* pk_a, const float* pk_b,
                                 hipStream_t st) {
    if (conv_fwd_cl_use(id, n, bf16))
        return launch_conv_fwd_cl(id, in, n_a, n, w_a, b_a, w_b, b_b, out, bf16, in16, out16, pk_a, pk_b, st);
    if (in16 || out16 || pk_a || pk_b) return hipErrorInvalidValue;   // only through the kernel above
    switch (id) {
        case CONV_L2:
            return bf16 ? igemm_launch<32, 20, 20, 64, 4, 2, 9, 9, true>(in, n_a, n, w_a, b_a, w_b, b_b, out, st)
                        : igemm_launch<32, 20, 20, 64, 4, 2, 9, 9, false>(in, n_a, n, w_a, b_a, w_b, b_b, out, st);
        case CONV_L3:
            return bf16 ? igemm_launch<64, 9, 9, 64, 3, 1, 7, 7, true>(in, n_a, n, w_a, b_a, w_b, b_b, out, st)
                        : igemm_launch<64, 9, 9, 64, 3, 1, 7, 7, false>(in, n_a, n, w_a, b_a, w_b, b_b, out, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_igemm_dgrad(ConvId id, const float* dz, const float* w, const float* h_in, float* din,
                                   int n, bool bf16, hipStream_t st) {
    switch (id) {
        case CONV_L2:
            return bf16 ? igemm_dgrad_launch<32, 20, 20, 64, 4, 2, 9, 9, 32, true>(dz, w, h_in, din, n, st)
                        : igemm_dgrad_launch<32, 20, 20, 64, 4, 2, 9, 9, 32, false>(dz, w, h_in, din, n, st);
        case CONV_L3:
            return bf16 ? igemm_dgrad_launch<64, 9, 9, 64, 3, 1, 7, 7, 64, true>(dz, w, h_in, din, n, st)
                        : igemm_dgrad_launch<64, 9, 9, 64, 3, 1, 7, 7, 64, false>(dz, w, h_in, din, n, st);
        default: return hipErrorInvalidValue;
    }
}

int conv_igemm_wgrad_chunks(ConvId id, int n) {
    int chunk, p;
    switch (id) {
        case CONV_L1: chunk = igemm_wgrad_chunk<4, 8, 32, 400, 32>(n); p = 400; break;
        case CONV_L2: chunk = igemm_wgrad_chunk<32, 4, 64, 81, 64>(n); p = 81; break;
        case CONV_L3: chunk = igemm_wgrad_chunk<64, 3, 64, 49, 64>(n); p = 49; break;
        default: return -1;
    }
    return (int)(((long)n * p + chunk - 1) / chunk);
}

hipError_t launch_conv_igemm_wgrad(ConvId id, const ConvIn& in, const float* dz, int n, float* wpart,
                                   float* bpart, float in_scale, bool bf16, hipStream_t st) {
#define DQN_WG(CIN, IH, IW, COUT, K, S, OH, OW, U8, BM)                                                      \
    return bf16 ? igemm_wgrad_launch<CIN, IH, IW, COUT, K, S, OH, OW, U8, BM, true>(in, dz, n, wpart, bpart,  \
                                                                                     in_scale, st)           \
                : igemm_wgrad_launch<CIN, IH, IW, COUT, K, S, OH, OW, U8, BM, false>(in, dz, n, wpart, bpart, \
                                                                                      in_scale, st)
    switch (id) {
        case CONV_L1: DQN_WG(4, 84, 84, 32, 8, 4, 20, 20, true, 32);
        case CONV_L2: DQN_WG(32, 20, 20, 64, 4, 2, 9, 9, false, 64);
        case CONV_L3: DQN_WG(64, 9, 9, 64, 3, 1, 7, 7, false, 64);
        default: return hipErrorInvalidValue;
    }
#undef DQN_WG
}

}  // namespace dqn
