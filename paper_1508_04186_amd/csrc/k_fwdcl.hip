// Forward convolution + bias + ReLU of the large network's conv2 and conv3
// (Sec. III.A) in the bf16-input variant at large batch: bf16 operands,
// fp32 accumulation, fp32 activations in and out.
//
// A workgroup (eight waves, one per compute unit) runs a run of samples with
// the layer's weights held in registers as bf16 MFMA operands: wave (nt, mh)
// owns output-channel tile nt (16 channels, about 70 registers of weights)
// and half of the sample's 16-pixel M-tiles.  Each sample's input is staged
// in LDS as bf16, channels-last, so that the eight k-values a lane feeds one
// v_mfma_f32_16x16x32_bf16 (eight consecutive input channels at one pixel of
// one filter tap) are one 16-byte LDS read, issued two k-steps ahead of its
// MFMA.  The k order of a step is (tap, 32 channels).  The staged pixels are
// laid out as the float32 kernel's (FwdX6Geom::slot: stride-2 rows and
// columns split by parity, rows at a pitch of OH + 16 slots, an odd number
// of 16-byte chunks per pixel), so that the reads of 16 consecutive output
// pixels hit 16 distinct groups of four banks; a sample is staged as items
// of eight channels at one pixel, one 16-byte store each.  A round takes SPR
// samples; the next round's input is read from HBM into registers during
// the current round's MFMAs, and the output maps are assembled in LDS and
// written as whole 16-byte vectors.  Weights reach the registers through
// LDS: coalesced loads, converted to bf16 and stored in the order the lanes
// read them.
#include <algorithm>
#include <initializer_list>
#include <type_traits>

#include "common.h"

namespace dqn {
namespace {

constexpr int FC_WG = 512;               // eight waves: 4 output-channel tiles x 2 M-halves
constexpr int FC_TARGET_BLOCKS = 256;   // one workgroup per compute unit

template <int CIN, int IH, int K, int S, int OH, int SPR>
struct FwdClGeom {
    static constexpr int COUT = 64;
    static constexpr int P = OH * OH;                   // output pixels
    static constexpr int MT = (P + 15) / 16;            // M-tiles per sample
    static constexpr int MPW = MT / 2;                  // M-tiles per wave
    static constexpr int KK = K * K;                    // taps
    static constexpr int CH = CIN / 32;                 // k-steps per tap
    static constexpr int KS = KK * CH;                  // k-steps
    static constexpr int KT = CIN * KK;                 // contraction length
    static constexpr int IP = IH * IH;                  // input pixels
    static constexpr int PSB = CIN * 2 + 16;            // LDS bytes per staged pixel (16-byte multiple)
    static constexpr int RP = OH + 16;                  // row pitch (slots): RP = OH (mod 16)
    static constexpr int SLOTS = IH * RP;
    static constexpr int IN = CIN * IP;                 // input floats per sample
    static constexpr int OUTF = COUT * P;               // output floats per sample
    static constexpr int LDS_MAIN = SPR * (SLOTS * PSB + OUTF * 4);
    static constexpr int LDS_W = COUT * KT * 2;         // all weights as bf16 operands
    static constexpr int WPER = COUT * KT / 4 / FC_WG;  // weight float4s per thread
    static_assert(COUT * KT % (4 * FC_WG) == 0, "whole weight float4s per thread");
    static constexpr int LDS = LDS_MAIN > LDS_W ? LDS_MAIN : LDS_W;
    static_assert(MT % 2 == 0 && CIN % 32 == 0, "geometry");
    static_assert(OUTF % 4 == 0 && KT % 4 == 0 && PSB % 16 == 0 && (PSB / 16) % 2 == 1, "vector widths");
    static_assert(S == 1 || (S == 2 && IH % 2 == 0 && IH / 2 <= RP), "stride-phase layout");
    static_assert(RP >= IH, "row pitch");
    // slot of input pixel (y, x); slot(S oy + ky, S ox + kx) = slot(ky, kx) + oy RP + ox
    __host__ __device__ static constexpr int slot(int y, int x) {
        return S == 2 ? ((y & 1) * (IH / 2) + (y >> 1)) * RP + (x & 1) * (IH / 2) + (x >> 1) : y * RP + x;
    }
};

struct FwdClParams {
    const float* in;           // [n][cin][ih][ih] (bfloat16 values when in16)
    float* out;                // [n][64][oh][oh] (bfloat16 values when out16)
    const float *w_a, *b_a, *w_b, *b_b;
    int n, n_a, g_a, spg;      // blocks [0, g_a) take samples [0, n_a), the rest [n_a, n); runs of spg
    const float *wpk_a, *wpk_b;  // w_a, w_b in per-lane order (weight_repack's forward jobs), or NULL
};

// PK: the weights from wpk_a / wpk_b (weight_repack: per-lane order, rounded)
template <int CIN, int IH, int K, int S, int OH, int SPR, bool IN16, bool OUT16, bool PK>
__global__ __launch_bounds__(FC_WG) void conv_fwd_cl_kernel(FwdClParams p) {
    using G = FwdClGeom<CIN, IH, K, S, OH, SPR>;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_in = smem;                                  // [SPR][SLOTS][PSB] bf16, channels-last
    float* s_out = (float*)(smem + SPR * G::SLOTS * G::PSB);     // [SPR][64][P]
    __bf16* s_w = (__bf16*)smem;                                 // [4][KS][64][8] bf16 (weights, before the samples)
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int nt = wave & 3, mh = wave >> 2;   // output channels 16nt .. 16nt+15

    const bool second = (int)blockIdx.x >= p.g_a;
    const int blk = second ? (int)blockIdx.x - p.g_a : (int)blockIdx.x;
    const int first = second ? p.n_a : 0;
    const int end = second ? p.n : p.n_a;
    const int j_lo = first + blk * p.spg;
    const int j_hi = min(end, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // whole workgroup
    const float* __restrict__ W = second ? p.w_b : p.w_a;
    const float* __restrict__ bias = second ? p.b_b : p.b_a;

    // SPR samples per round: sample j + s of the round is read into
    // registers (hv) and staged into s_in buffer s, as items of eight
    // channels 8cg .. 8cg+7: bfloat16 input with an even pixel count
    // (conv2's) is read as 32-bit words of two pixels of one channel, an item
    // covering pixels 2w, 2w+1 (split by v_perm_b32, moved bit for bit);
    // otherwise an item is one pixel, its eight values read one by one
    // (bfloat16 moved as they are, floats rounded as they are staged).
    constexpr bool PAIRS16 = IN16 && G::IP % 2 == 0;
    constexpr int NPIX = PAIRS16 ? G::IP / 2 : G::IP;   // items per channel group
    constexpr int ITEMS = (CIN / 8) * NPIX;
    constexpr int IPER = (ITEMS + FC_WG - 1) / FC_WG;
    uint32_t hv[SPR][IPER][8];
    auto fetch = [&](int j) {
#pragma unroll
        for (int s = 0; s < SPR; ++s) {
            if (j + s >= j_hi) break;
            const float* x = p.in + (size_t)(j + s) * G::IN;
            const unsigned short* xh = (const unsigned short*)p.in + (size_t)(j + s) * G::IN;
#pragma unroll
            for (int u = 0; u < IPER; ++u) {
                const int q = t + u * FC_WG;
                if (q < ITEMS) {
                    const int cg = q / NPIX, w = q - cg * NPIX;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        if constexpr (PAIRS16) hv[s][u][e] = ((const uint32_t*)xh)[(8 * cg + e) * (G::IP / 2) + w];
                        else if constexpr (IN16) hv[s][u][e] = xh[(8 * cg + e) * G::IP + w];
                        else hv[s][u][e] = __builtin_bit_cast(uint32_t, x[(8 * cg + e) * G::IP + w]);
                    }
                }
            }
        }
    };
    auto stage = [&](int j) {
#pragma unroll
        for (int s = 0; s < SPR; ++s) {
            if (j + s >= j_hi) break;
#pragma unroll
            for (int u = 0; u < IPER; ++u) {
                const int q = t + u * FC_WG;
                if (q < ITEMS) {
                    const int cg = q / NPIX, w = q - cg * NPIX;
                    const uint32_t* h = hv[s][u];
                    unsigned char* base = s_in + s * G::SLOTS * G::PSB + 16 * cg;
                    if constexpr (PAIRS16) {
                        const int pix = 2 * w, y = pix / IH, x = pix - y * IH;   // x even: x + 1 on the same row
                        uint4 a, b;
                        a.x = __builtin_amdgcn_perm(h[1], h[0], 0x05040100u);
                        a.y = __builtin_amdgcn_perm(h[3], h[2], 0x05040100u);
                        a.z = __builtin_amdgcn_perm(h[5], h[4], 0x05040100u);
                        a.w = __builtin_amdgcn_perm(h[7], h[6], 0x05040100u);
                        b.x = __builtin_amdgcn_perm(h[1], h[0], 0x07060302u);
                        b.y = __builtin_amdgcn_perm(h[3], h[2], 0x07060302u);
                        b.z = __builtin_amdgcn_perm(h[5], h[4], 0x07060302u);
                        b.w = __builtin_amdgcn_perm(h[7], h[6], 0x07060302u);
                        *(uint4*)(base + G::slot(y, x) * G::PSB) = a;
                        *(uint4*)(base + G::slot(y, x + 1) * G::PSB) = b;
                    } else {
                        const int y = w / IH, x = w - y * IH;
                        uint32_t k[4];
#pragma unroll
                        for (int e2 = 0; e2 < 4; ++e2) {
                            uint32_t lo, hi;
                            if constexpr (IN16) {
                                lo = h[2 * e2];
                                hi = h[2 * e2 + 1];
                            } else {
                                lo = __builtin_bit_cast(unsigned short, (__bf16)__builtin_bit_cast(float, h[2 * e2]));
                                hi = __builtin_bit_cast(unsigned short, (__bf16)__builtin_bit_cast(float, h[2 * e2 + 1]));
                            }
                            k[e2] = lo | (hi << 16);
                        }
                        *(uint4*)(base + G::slot(y, x) * G::PSB) = uint4{k[0], k[1], k[2], k[3]};
                    }
                }
            }
        }
    };
    fetch(j_lo);  // in flight while the weights are loaded

    // Weights: from the per-lane copy (PK), or every thread converts its
    // share of W (coalesced float4s) to bf16 and stores each value where the
    // lane that feeds it to the MFMAs reads it: lane (li, g) of the wave
    // owning N-tile nt holds, at k-step ks, W[o][c][tap] for o = 16nt + li,
    // tap = ks / CH, c = 32 (ks % CH) + 8g + e in element e, at
    // s_w[((nt KS + ks) 64 + lane) 8 + e].
    bf16x8 wv[G::KS];
    if constexpr (PK) {
        const bf16x8* wp = (const bf16x8*)(second ? p.wpk_b : p.wpk_a);
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks) wv[ks] = wp[(nt * G::KS + ks) * 64 + lane];
    } else {
        f4 wr[G::WPER];
#pragma unroll
        for (int u = 0; u < G::WPER; ++u) wr[u] = ((const f4*)W)[t + u * FC_WG];
#pragma unroll
        for (int u = 0; u < G::WPER; ++u) {
            const int q = t + u * FC_WG;
            const int o = (4 * q) / G::KT, k0 = 4 * q - o * G::KT;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int k = k0 + v, c = k / G::KK, tap = k - c * G::KK;
                const int ks = tap * G::CH + c / 32, ln = (o & 15) + 16 * ((c & 31) >> 3);
                s_w[(((o >> 4) * G::KS + ks) * 64 + ln) * 8 + (c & 7)] = (__bf16)wr[u][v];
            }
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks) wv[ks] = *(const bf16x8*)&s_w[((nt * G::KS + ks) * 64 + lane) * 8];
    }
    const float bo = bias[16 * nt + li];

    // byte offset in s_in of the lane's first input pixel for each of its
    // M-tiles (rows past the map read pixel 0; their results are dropped)
    int pb[G::MPW];
#pragma unroll
    for (int i = 0; i < G::MPW; ++i) {
        const int pp = 16 * (mh * G::MPW + i) + li;
        const int pc = pp < G::P ? pp : 0;
        const int oy = pc / OH, ox = pc - oy * OH;
        pb[i] = (oy * G::RP + ox) * G::PSB + 16 * g;
    }

    for (int j = j_lo; j < j_hi; j += SPR) {
        __syncthreads();  // weight staging, or the previous round's reads of s_in / s_out, done
        stage(j);
        __syncthreads();
        if (j + SPR < j_hi) fetch(j + SPR);
        // (the MFMAs of a sample past j_hi read stale LDS; their results are not written)
        f4 acc[SPR][G::MPW];
#pragma unroll
        for (int s = 0; s < SPR; ++s)
#pragma unroll
            for (int i = 0; i < G::MPW; ++i) acc[s][i] = f4{0.f, 0.f, 0.f, 0.f};
        // The A operands of step ks + AHEAD are read while step ks multiplies
        // (LDS latency covered by AHEAD steps of MFMAs).
        constexpr int AHEAD = 2;
        auto a_addr = [&](int ks, int s, int i) {
            const int tap = ks / G::CH;
            return s_in + s * G::SLOTS * G::PSB + pb[i] + G::slot(tap / K, tap % K) * G::PSB + 64 * (ks % G::CH);
        };
        bf16x8 abuf[AHEAD + 1][SPR][G::MPW];
#pragma unroll
        for (int d = 0; d < AHEAD; ++d)
#pragma unroll
            for (int s = 0; s < SPR; ++s)
#pragma unroll
                for (int i = 0; i < G::MPW; ++i) abuf[d][s][i] = *(const bf16x8*)a_addr(d, s, i);
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks) {
            if (ks + AHEAD < G::KS) {
#pragma unroll
                for (int s = 0; s < SPR; ++s)
#pragma unroll
                    for (int i = 0; i < G::MPW; ++i)
                        abuf[(ks + AHEAD) % (AHEAD + 1)][s][i] = *(const bf16x8*)a_addr(ks + AHEAD, s, i);
            }
#pragma unroll
            for (int s = 0; s < SPR; ++s)
#pragma unroll
                for (int i = 0; i < G::MPW; ++i)
                    acc[s][i] = mfma16x16x32bf16(abuf[ks % (AHEAD + 1)][s][i], wv[ks], acc[s][i]);
            __builtin_amdgcn_sched_barrier(0);  // keep the reads of later steps where they are
        }
        // D[4g + r][li] of an M-tile: pixel 16 mt + 4g + r, channel 16nt + li
#pragma unroll
        for (int s = 0; s < SPR; ++s)
#pragma unroll
            for (int i = 0; i < G::MPW; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int pp = 16 * (mh * G::MPW + i) + 4 * g + r;
                    if (pp < G::P) s_out[(s * G::COUT + 16 * nt + li) * G::P + pp] = fmaxf(acc[s][i][r] + bo, 0.f);
                }
        __syncthreads();
        const int ns = min(SPR, j_hi - j);
        if constexpr (OUT16) {
            bf16x4* dst = (bf16x4*)((__bf16*)p.out + (size_t)j * G::OUTF);
            for (int q = t; q < ns * G::OUTF / 4; q += FC_WG) {
                const f4 v = ((const f4*)s_out)[q];
                dst[q] = bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            }
        } else {
            f4* dst = (f4*)(p.out + (size_t)j * G::OUTF);
            for (int q = t; q < ns * G::OUTF / 4; q += FC_WG) dst[q] = ((const f4*)s_out)[q];
        }
    }
}

template <int CIN, int IH, int K, int S, int OH, int SPR>
hipError_t fwd_cl_launch(const float* in, int n_a, int n, const float* w_a, const float* b_a, const float* w_b,
                         const float* b_b, float* out, bool in16, bool out16, const float* pk_a, const float* pk_b,
                         hipStream_t st) {
    using G = FwdClGeom<CIN, IH, K, S, OH, SPR>;
    if (n <= 0 || n_a < 0 || n_a > n) return hipErrorInvalidValue;
    if (((uintptr_t)w_a & 15) || ((uintptr_t)w_b & 15) || ((uintptr_t)out & 15)) return hipErrorInvalidValue;
    // the packed weights: both sets or neither, 16-byte aligned
    if (!pk_a != !pk_b || ((uintptr_t)pk_a & 15) || ((uintptr_t)pk_b & 15)) return hipErrorInvalidValue;
    const int spg = std::max(1, (n + FC_TARGET_BLOCKS - 1) / FC_TARGET_BLOCKS);
    const int g_a = (n_a + spg - 1) / spg, g_b = (n - n_a + spg - 1) / spg;
    const FwdClParams prm{in, out, w_a, b_a, w_b, b_b, n, n_a, g_a, spg, pk_a, pk_b};
    auto go = [&](auto kern) -> hipError_t {
        if (!allow_lds((const void*)kern, G::LDS)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)(g_a + g_b)), dim3(FC_WG), G::LDS, st, prm);
        return hipGetLastError();
    };
    if (pk_a) {   // (the TD step's bf16 activations)
        if (in16 && out16) return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, true, true, true>);
        if (in16) return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, true, false, true>);
        return hipErrorInvalidValue;
    }
    if (in16 && out16) return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, true, true, false>);
    if (in16) return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, true, false, false>);
    if (out16) return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, false, true, false>);
    return go(conv_fwd_cl_kernel<CIN, IH, K, S, OH, SPR, false, false, false>);
}

// The float32 variant on bf16 MFMA: every float32 operand is split exactly
// into three bfloat16 terms, x = hi + mid + lo (8 significand bits each), and
// a k-step multiplies the six pairs whose product is at least 2^-16 of
// hi*hi: hi*hi, hi*mid, mid*hi, hi*lo, mid*mid, lo*hi.  The products of 8-bit
// significands are exact and accumulate in float32; the two dropped pairs
// are below 2^-23 of the product, the size of a float32 rounding, so the
// sums keep float32 accuracy at six v_mfma_f32_16x16x32_bf16 per 32 k-values
// (2.7x the matrix rate of eight v_mfma_f32_16x16x4_f32).
//
// Eight waves per workgroup, one workgroup per compute unit: wave (nt, kh)
// owns output channels 16nt .. 16nt+15 and half kh of the k-steps (k order
// (tap, 32 channels), as the bf16 variant), holding those weights' three
// planes in registers (96 or 108), for every M-tile of the sample.  Each
// sample's input is split into three bf16 planes staged channels-last in LDS
// (one 16-byte read per operand and plane, free of bank conflicts: see
// FwdX6Geom::slot); the two halves' sums meet in LDS
// at the end of the sample, where bias and ReLU are applied and the output
// map is assembled and written as 16-byte vectors.  The next sample's input
// is read into registers during the MFMAs.
template <int CIN, int IH, int K, int S, int OH>
struct FwdX6Geom {
    static constexpr int COUT = 64;
    static constexpr int P = OH * OH;
    static constexpr int MT = (P + 15) / 16;            // M-tiles per sample (all in every wave)
    static constexpr int KK = K * K;
    static constexpr int CH = CIN / 32;                 // k-steps per tap
    static constexpr int KS = KK * CH;                  // k-steps
    static constexpr int KSH = KS / 2;                  // per half
    static constexpr int IP = IH * IH;
    static constexpr int PSB = CIN * 2 + 16;            // bytes per staged pixel and plane
    // Staged pixel order: stride 2 splits rows and columns by parity, so the
    // input pixels of consecutive output pixels are consecutive slots; rows
    // at a pitch of RP slots, RP = OH (mod 16), so the slots of any 16
    // consecutive output pixels are 16 consecutive values mod 16, and with
    // PSB / 16 odd a lane group's 16-byte reads hit 16 distinct groups of
    // four banks.
    static constexpr int RP = OH + 16;
    static constexpr int SLOTS = IH * RP;
    static constexpr int PLANE = SLOTS * PSB;
    static constexpr int IN = CIN * IP;
    static constexpr int ITEMS = (CIN / 8) * IP;        // (8-channel group, pixel) items
    static constexpr int IPER = (ITEMS + FC_WG - 1) / FC_WG;
    static constexpr int OUTF = COUT * P;
    static constexpr int PART = 4 * MT * 64 * 16;       // half-sums of the kh = 1 waves (bytes)
    static constexpr int LDS = 3 * PLANE;
    static_assert(KS % 2 == 0 && CIN % 32 == 0 && PSB % 16 == 0 && (PSB / 16) % 2 == 1 && OUTF % 4 == 0, "geometry");
    static_assert(S == 1 || (S == 2 && IH % 2 == 0 && IH / 2 <= RP), "stride-phase layout");
    static_assert(RP >= IH && (RP - OH) % 16 == 0, "row pitch");
    static_assert(PART + OUTF * 4 <= LDS, "half-sums and output map fit in the input planes");
    // slot of input pixel (y, x); slot(S oy + ky, S ox + kx) = slot(ky, kx) + oy RP + ox
    __host__ __device__ static constexpr int slot(int y, int x) {
        return S == 2 ? ((y & 1) * (IH / 2) + (y >> 1)) * RP + (x & 1) * (IH / 2) + (x >> 1) : y * RP + x;
    }
};


template <int CIN, int IH, int K, int S, int OH, bool PK>   // PK: weight planes from wpk_a / wpk_b
__global__ __launch_bounds__(FC_WG) void conv_fwd_x6_kernel(FwdClParams p) {
    using G = FwdX6Geom<CIN, IH, K, S, OH>;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_in = smem;                                     // [3][IP][PSB] bf16 planes
    f4* s_part = (f4*)smem;                                         // [4][MT][64] (after the MFMAs)
    float* s_out = (float*)(smem + G::PART);                        // [64][P]     (after the MFMAs)
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int nt = wave & 3, kh = wave >> 2;

    const bool second = (int)blockIdx.x >= p.g_a;
    const int blk = second ? (int)blockIdx.x - p.g_a : (int)blockIdx.x;
    const int first = second ? p.n_a : 0;
    const int end = second ? p.n : p.n_a;
    const int j_lo = first + blk * p.spg;
    const int j_hi = min(end, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // whole workgroup
    const float* __restrict__ bias = second ? p.b_b : p.b_a;

    // input items (8 channels at one pixel) of the next sample, in registers
    float v[G::IPER][8];
    auto fetch = [&](int j) {
        const float* x = p.in + (size_t)j * G::IN;
#pragma unroll
        for (int u = 0; u < G::IPER; ++u) {
            const int q = t + u * FC_WG;
            if (q < G::ITEMS) {
                const int cg = q / G::IP, pix = q - cg * G::IP;
#pragma unroll
                for (int e = 0; e < 8; ++e) v[u][e] = x[(8 * cg + e) * G::IP + pix];
            }
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int u = 0; u < G::IPER; ++u) {
            const int q = t + u * FC_WG;
            if (q < G::ITEMS) {
                const int cg = q / G::IP, pix = q - cg * G::IP;
                const int y = pix / IH, x = pix - y * IH;
                bf16x8 h, m, l;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    __bf16 a, b, c;
                    split3(v[u][e], a, b, c);
                    h[e] = a;
                    m[e] = b;
                    l[e] = c;
                }
                unsigned char* d = s_in + G::slot(y, x) * G::PSB + 16 * cg;
                *(bf16x8*)d = h;
                *(bf16x8*)(d + G::PLANE) = m;
                *(bf16x8*)(d + 2 * G::PLANE) = l;
            }
        }
    };
    fetch(j_lo);

    // weights: lane (li, g) of wave (nt, kh) at its k-step s holds, in plane
    // pl, W[16nt + li][32 cb + 8g + e][tap] split, with ks = kh KSH + s,
    // tap = ks / CH, cb = ks % CH
    bf16x8 wv[3][G::KSH];
    if constexpr (PK) {
        const bf16x8* wp = (const bf16x8*)(second ? p.wpk_b : p.wpk_a);
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
#pragma unroll
            for (int s = 0; s < G::KSH; ++s) wv[pl][s] = wp[X6FwdPack<CIN, G::KK>::index(pl, nt, kh, s, lane)];
    } else {
        const float* __restrict__ W = second ? p.w_b : p.w_a;
        const float* wr = W + (size_t)(16 * nt + li) * CIN * G::KK;
#pragma unroll
        for (int s = 0; s < G::KSH; ++s) {
            const int ks = kh * G::KSH + s, tap = ks / G::CH, cb = ks % G::CH;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                __bf16 a, b, c;
                split3(wr[(32 * cb + 8 * g + e) * G::KK + tap], a, b, c);
                wv[0][s][e] = a;
                wv[1][s][e] = b;
                wv[2][s][e] = c;
            }
        }
    }
    const float bo = bias[16 * nt + li];

    // byte offset in a plane of the lane's first input pixel for each M-tile
    // (rows past the map read pixel 0; their results are dropped)
    int pb[G::MT];
#pragma unroll
    for (int i = 0; i < G::MT; ++i) {
        const int pp = 16 * i + li;
        const int pc = pp < G::P ? pp : 0;
        const int oy = pc / OH, ox = pc - oy * OH;
        pb[i] = (oy * G::RP + ox) * G::PSB + 16 * g;
    }

    // the k-steps of half KH: per step, the three planes of every M-tile's A
    // operand, then the six products, each over all M-tiles (independent chains)
    auto half = [&](auto khc, f4* acc) {
        constexpr int KH = decltype(khc)::value;
#pragma unroll
        for (int s = 0; s < G::KSH; ++s) {
            const int ks = KH * G::KSH + s, tap = ks / G::CH, cb = ks % G::CH;
            const int off = G::slot(tap / K, tap % K) * G::PSB + 64 * cb;
            bf16x8 a[3][G::MT];
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
#pragma unroll
                for (int i = 0; i < G::MT; ++i) a[pl][i] = *(const bf16x8*)(s_in + pl * G::PLANE + pb[i] + off);
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[2][i], wv[0][s], acc[i]);   // lo*hi
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[1][i], wv[1][s], acc[i]);   // mid*mid
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wv[2][s], acc[i]);   // hi*lo
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[1][i], wv[0][s], acc[i]);   // mid*hi
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wv[1][s], acc[i]);   // hi*mid
#pragma unroll
            for (int i = 0; i < G::MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wv[0][s], acc[i]);   // hi*hi
        }
    };

    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the previous sample's reads of s_out are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        f4 acc[G::MT];
#pragma unroll
        for (int i = 0; i < G::MT; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        if (kh == 0)
            half(std::integral_constant<int, 0>{}, acc);
        else
            half(std::integral_constant<int, 1>{}, acc);
        __syncthreads();  // every wave's reads of the planes are done
        if (kh == 1) {
#pragma unroll
            for (int i = 0; i < G::MT; ++i) s_part[(nt * G::MT + i) * 64 + lane] = acc[i];
        }
        __syncthreads();
        if (kh == 0) {
            // D[4g + r][li] of M-tile i: pixel 16 i + 4g + r, channel 16nt + li
#pragma unroll
            for (int i = 0; i < G::MT; ++i) {
                const f4 o = s_part[(nt * G::MT + i) * 64 + lane];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int pp = 16 * i + 4 * g + r;
                    if (pp < G::P) s_out[(16 * nt + li) * G::P + pp] = fmaxf((acc[i][r] + o[r]) + bo, 0.f);
                }
            }
        }
        __syncthreads();
        f4* dst = (f4*)(p.out + (size_t)j * G::OUTF);
        for (int q = t; q < G::OUTF / 4; q += FC_WG) dst[q] = ((const f4*)s_out)[q];
    }
}

template <int CIN, int IH, int K, int S, int OH>
hipError_t fwd_x6_launch(const float* in, int n_a, int n, const float* w_a, const float* b_a, const float* w_b,
                         const float* b_b, float* out, const float* pk_a, const float* pk_b, hipStream_t st) {
    using G = FwdX6Geom<CIN, IH, K, S, OH>;
    if (n <= 0 || n_a < 0 || n_a > n || ((uintptr_t)out & 15) || (!pk_a != !pk_b)) return hipErrorInvalidValue;
    if (pk_a && (((uintptr_t)pk_a & 15) || ((uintptr_t)pk_b & 15))) return hipErrorInvalidValue;
    const int spg = std::max(1, (n + FC_TARGET_BLOCKS - 1) / FC_TARGET_BLOCKS);
    const int g_a = (n_a + spg - 1) / spg, g_b = (n - n_a + spg - 1) / spg;
    const FwdClParams prm{in, out, w_a, b_a, w_b, b_b, n, n_a, g_a, spg, pk_a, pk_b};
    auto go = [&](auto kern) -> hipError_t {
        if (!allow_lds((const void*)kern, G::LDS)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)(g_a + g_b)), dim3(FC_WG), G::LDS, st, prm);
        return hipGetLastError();
    };
    return pk_a ? go(conv_fwd_x6_kernel<CIN, IH, K, S, OH, true>) : go(conv_fwd_x6_kernel<CIN, IH, K, S, OH, false>);
}

}  // namespace

bool conv_fwd_cl_use(ConvId id, int n, bool bf16) {
    return (id == CONV_L2 || id == CONV_L3) && n >= kFwdClMinRows;
}

hipError_t launch_conv_fwd_cl(ConvId id, const float* in, int n_a, int n, const float* w_a, const float* b_a,
                              const float* w_b, const float* b_b, float* out, bool bf16, bool in16, bool out16,
                              const float* pk_a, const float* pk_b, hipStream_t st) {
    if (!bf16 && (in16 || out16)) return hipErrorInvalidValue;   // bf16 activations: the bf16 variant only
    switch (id) {
        case CONV_L2:
            return bf16 ? fwd_cl_launch<32, 20, 4, 2, 9, 1>(in, n_a, n, w_a, b_a, w_b, b_b, out, in16, out16, pk_a, pk_b,
                                                            st)
                        : fwd_x6_launch<32, 20, 4, 2, 9>(in, n_a, n, w_a, b_a, w_b, b_b, out, pk_a, pk_b, st);
        case CONV_L3:
            return bf16 ? fwd_cl_launch<64, 9, 3, 1, 7, 1>(in, n_a, n, w_a, b_a, w_b, b_b, out, in16, out16, pk_a, pk_b,
                                                           st)
                        : fwd_x6_launch<64, 9, 3, 1, 7>(in, n_a, n, w_a, b_a, w_b, b_b, out, pk_a, pk_b, st);
        default: return hipErrorInvalidValue;
    }
}

int64_t fwd_x6_pack_floats(ConvId id) {
    // bf16x8 vectors (4 floats each) of the three planes
    return id == CONV_L2 ? 4 * X6FwdPack<32, 16>::VECS : 4 * X6FwdPack<64, 9>::VECS;
}


}  // namespace dqn
