// Input gradients of the large network's second and third convolutions at
// large batch, masked by the ReLU mask of the layer below.
//
// conv2 (32 -> 64 channels, 4x4 stride 2, 20x20 -> 9x9) by stride phase
// (py, px): input pixel (2qy + py, 2qx + px), qy, qx in [0, 10), receives
//   din = [h_in > 0] * sum_{o, ty, tx} W[o][c][py + 2ty][px + 2tx] * dz[o][qy - ty][qx - tx]
// with dz = 0 outside the 9x9 map, so no product multiplies a structural
// zero of the strided kernel.  conv3 (64 -> 64, 3x3 stride 1, 9x9 -> 7x7):
//   din[c][y][x] = [h_in > 0] * sum_{o, ky, kx} W[o][c][ky][kx] * dz[o][y - ky][x - kx].
//
// A workgroup walks a group of samples, one per round, its eight waves
// holding slices of the weights in registers for the whole launch (the B
// operand of every k-step).  A sample's dz is staged in LDS channels-last
// with a zero border, so the A operand of a pixel and tap sits at a per-lane
// base plus a compile-time offset and needs no bounds test; the sample's
// whole input gradient is assembled in LDS and written with 16-byte stores,
// masked by the ReLU mask read into registers at the start of the round, and
// the next sample's dz is read into registers while the current one is
// computed.  The bf16-input variant rounds operands to bf16
// (conv2_dgrad_cl_kernel, conv3_dgrad_cl_kernel); the float32 kernels split
// them exactly into three bf16 terms (conv2_dgrad_x6_kernel,
// conv3_dgrad_x6_kernel).
#include <algorithm>
#include <initializer_list>
#include <type_traits>

#include "common.h"

namespace dqn {
namespace {

constexpr int D2_WG = 512;
constexpr int D2_CIN = 32, D2_IH = 20, D2_COUT = 64, D2_OH = 9, D2_K = 4;
constexpr int D2_Q = 10;                       // phase grid side
constexpr int D2_QP = D2_Q * D2_Q;             // phase pixels per sample
constexpr int D2_MT = (D2_QP + 15) / 16;       // M-tiles per phase (7)
constexpr int D2_DZ = D2_COUT * D2_OH * D2_OH; // dz floats per sample (5,184)
constexpr int D2_IN = D2_CIN * D2_IH * D2_IH;  // input-gradient floats per sample (12,800)
constexpr int D2_KT = D2_COUT * 4;             // contraction length (o, tap): 256
constexpr int D2_OUT4 = (D2_IN / 4 + D2_WG - 1) / D2_WG;  // float4 of din per thread (7)
static_assert(D2_IN % 4 == 0, "whole float4 rows");

struct Dgrad2Params {
    const float* dz;    // [n][64][9][9]
    const float* w;     // [64][32][4][4]
    const float* h_in;  // [n][32][20][20] (bfloat16 values when h16)
    float* din;         // [n][32][20][20]
    int n, spg;         // samples, samples per workgroup
    const float* wpk;   // the weights in per-lane order (weight_repack), or NULL
    __bf16* din16;      // conv2 bf16 kernel: when set, din is written here rounded to bfloat16 instead,
    float* bpart;       // ... and the workgroup's per-channel sums of the float32 din to bpart[block][32]
};

// Four consecutive values of the layer input h_in (the ReLU mask source) at
// element offset off (a multiple of 4): floats, or, with H16 (h_in holds
// bfloat16), the raw 16-bit values, tested only where the mask is applied so
// that nothing waits for the load before then.
template <bool H16>
struct Mask4 {
    f4 v;
    __device__ void load(const Dgrad2Params& p, size_t off) { v = *(const f4*)(p.h_in + off); }
    __device__ bool pos(int k) const { return v[k] > 0.f; }
};
template <>
struct Mask4<true> {
    uint2 v;
    __device__ void load(const Dgrad2Params& p, size_t off) { v = *(const uint2*)((const __bf16*)p.h_in + off); }
    __device__ bool pos(int k) const {   // > 0: sign clear, nonzero, not a NaN (bits 0x0001..0x7f80)
        const uint32_t w = k < 2 ? v.x : v.y;
        const uint32_t b = (w >> (16 * (k & 1))) & 0xffffu;
        return b - 1u < 0x7f80u;
    }
};

// conv2 with dz staged as bf16 (the bf16-input variant),
// channels-last: slot sigma(y, x) = 10 (y + 1) + x + 1 of the zero-bordered
// 10-wide map (rows -1 .. 10; a row's column 9 is the next row's column -1)
// holds dz[o][y][x] for the 64 channels o, 144 bytes per slot.  The eight
// k-values a lane feeds one v_mfma_f32_16x16x32_bf16 are then eight
// consecutive channels at one slot: one 16-byte read at a per-lane base and
// a compile-time tap offset, issued two k-steps ahead of its MFMA.  k-step
// s: tap s / 2, channels 32 (s % 2) + 8g + e in element e of lane group g
// (the weights in registers follow the same order).  The input gradient is
// assembled in LDS channel by channel at a row stride of D2_CS = 402 floats:
// a stride of 400 (16 mod 32 banks) put the 16 channels of one store on two
// banks (16-way conflicts), 402 spreads them (at most 4-way); rows then start
// 8-byte aligned and the read-out takes a float4 as two 8-byte reads.
constexpr int D2C_SLOTS = 132;                 // sigma of every read: 0 .. 122
constexpr int D2C_PSB = 144;                   // bytes per slot: 64 bf16 + 16
static_assert(D2C_PSB % 16 == 0 && D2C_PSB >= 2 * D2_COUT && (D2C_PSB / 16) % 2 == 1, "slot size");
constexpr int D2_CS = D2_IH * D2_IH + 2;       // LDS row stride of the assembled input gradient (floats)

// A sample's dz [64][OH][OH] staged channels-last (144-byte slots, slot
// RW (oy + R0) + ox + C0 for pixel (oy, ox)) as items of CPI channels at
// one pixel: one 2*CPI-byte store per item and plane, consecutive lanes at
// consecutive slots (9 chunks of 16 bytes apart).  Items of eight channels
// store without bank conflicts and of four with at most two-way ones, where
// 4-byte stores of channel pairs at that stride conflicted four to eight
// ways; four channels keep fewer values in registers (for the float32 conv2
// kernel's budget).  PLANES = 1: rounded to bf16; 3: the exact split, plane
// pl at + pl * plane bytes.
template <int OH, int RW, int R0, int C0, int PLANES, int CPI = 8>
struct DzStage {
    static_assert(CPI == 4 || CPI == 8, "item width");
    static constexpr int P = OH * OH, ITEMS = (D2_COUT / CPI) * P, IPER = (ITEMS + D2_WG - 1) / D2_WG;
    using V = std::conditional_t<CPI == 8, bf16x8, bf16x4>;
    float v[IPER][CPI];
    __device__ __forceinline__ void fetch(const float* src, int t) {
#pragma unroll
        for (int u = 0; u < IPER; ++u) {
            const int q2 = t + u * D2_WG;
            if (q2 < ITEMS) {
                const int og = q2 / P, q = q2 - og * P;
#pragma unroll
                for (int e = 0; e < CPI; ++e) v[u][e] = src[(CPI * og + e) * P + q];
            }
        }
    }
    __device__ __forceinline__ void stage(unsigned char* s_cl, int t, int plane_bytes) const {
#pragma unroll
        for (int u = 0; u < IPER; ++u) {
            const int q2 = t + u * D2_WG;
            if (q2 < ITEMS) {
                const int og = q2 / P, q = q2 - og * P, oy = q / OH, ox = q - oy * OH;
                unsigned char* d = s_cl + (RW * (oy + R0) + ox + C0) * 144 + 2 * CPI * og;
                V h, m, l;
#pragma unroll
                for (int e = 0; e < CPI; ++e) {
                    if constexpr (PLANES == 3) {
                        __bf16 a, b, c;
                        split3(v[u][e], a, b, c);
                        h[e] = a;
                        m[e] = b;
                        l[e] = c;
                    } else {
                        h[e] = (__bf16)v[u][e];
                    }
                }
                *(V*)d = h;
                if constexpr (PLANES == 3) {
                    *(V*)(d + plane_bytes) = m;
                    *(V*)(d + 2 * plane_bytes) = l;
                }
            }
        }
    }
};

// Float4 e4 of the input gradient (pixels 4k .. 4k+3 of channel c) from the
// LDS assembly above (rows at a stride of D2_CS floats, 8-byte aligned).
__device__ __forceinline__ f4 d2_din4(const float* s_din, int e4) {
    constexpr int CP = D2_IH * D2_IH;
    const int ch = e4 / (CP / 4);
    const float* r = s_din + ch * D2_CS + (4 * e4 - ch * CP);
    const float2 a = *(const float2*)r, b = *(const float2*)(r + 2);
    return f4{a.x, a.y, b.x, b.y};
}

template <bool H16, bool PK>   // PK: bf16 weight operands from p.wpk (weight_repack)
__global__ __launch_bounds__(D2_WG) void conv2_dgrad_cl_kernel(Dgrad2Params p) {
    __shared__ __align__(16) unsigned char s_cl[D2C_SLOTS * D2C_PSB];
    __shared__ __align__(16) float s_din[D2_CIN * D2_CS];
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int ph = wave >> 1, nt = wave & 1;   // phase; N-tile
    const int py = ph >> 1, px = ph & 1;

    for (int e = t; e < D2C_SLOTS * D2C_PSB / 16; e += D2_WG) ((uint4*)s_cl)[e] = uint4{0u, 0u, 0u, 0u};

    const int j_lo = blockIdx.x * p.spg;
    const int j_hi = min(p.n, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // uniform

    constexpr int KS = D2_KT / 32;
    const int c = nt * 16 + li;
    bf16x8 wreg[KS];
    if constexpr (PK) {
#pragma unroll
        for (int s = 0; s < KS; ++s) wreg[s] = ((const bf16x8*)p.wpk)[((size_t)wave * KS + s) * 64 + lane];
    } else {
        const float* wc = p.w + (size_t)c * D2_K * D2_K + py * D2_K + px;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int o = 32 * (s % 2) + 8 * g + e;
                wreg[s][e] = (__bf16)wc[(size_t)o * D2_CIN * D2_K * D2_K + 2 * ty * D2_K + 2 * tx];
            }
        }
    }
    // byte base of each M-tile's slot for this lane: phase pixel m = 16 mt + li
    int base[D2_MT];
#pragma unroll
    for (int i = 0; i < D2_MT; ++i) {
        const int m = i * 16 + li, qy = m / D2_Q, qx = m - qy * D2_Q;
        base[i] = (D2_Q * (qy + 1) + qx + 1) * D2C_PSB + 16 * g;
    }

    DzStage<D2_OH, D2_Q, 1, 1, 1> dzs;
    auto fetch = [&](int j) { dzs.fetch(p.dz + (size_t)j * D2_DZ, t); };
    auto stage = [&]() { dzs.stage(s_cl, t, 0); };

    float bsum[D2_OUT4];
#pragma unroll
    for (int u = 0; u < D2_OUT4; ++u) bsum[u] = 0.f;
    fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous round's LDS reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);  // in flight during this sample's MFMAs
        // this sample's ReLU mask, for the write-out below
        const size_t o0 = (size_t)j * D2_IN;
        Mask4<H16> mreg[D2_OUT4];
#pragma unroll
        for (int u = 0; u < D2_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D2_IN / 4) mreg[u].load(p, o0 + 4 * e4);
        }

        f4 acc[D2_MT];
#pragma unroll
        for (int i = 0; i < D2_MT; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        constexpr int AHEAD = 2;
        auto a_at = [&](int s, int i) {
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
            return *(const bf16x8*)(s_cl + base[i] - (D2_Q * ty + tx) * D2C_PSB + 64 * (s % 2));
        };
        bf16x8 abuf[AHEAD + 1][D2_MT];
#pragma unroll
        for (int d = 0; d < AHEAD; ++d)
#pragma unroll
            for (int i = 0; i < D2_MT; ++i) abuf[d][i] = a_at(d, i);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            if (s + AHEAD < KS) {
#pragma unroll
                for (int i = 0; i < D2_MT; ++i) abuf[(s + AHEAD) % (AHEAD + 1)][i] = a_at(s + AHEAD, i);
            }
#pragma unroll
            for (int i = 0; i < D2_MT; ++i) acc[i] = mfma16x16x32bf16(abuf[s % (AHEAD + 1)][i], wreg[s], acc[i]);
            __builtin_amdgcn_sched_barrier(0);
        }

#pragma unroll
        for (int i = 0; i < D2_MT; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = i * 16 + 4 * g + r;
                if (m < D2_QP) {
                    const int qy = m / D2_Q, qx = m - qy * D2_Q;
                    s_din[c * D2_CS + (2 * qy + py) * D2_IH + 2 * qx + px] = acc[i][r];
                }
            }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < D2_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D2_IN / 4) {
                const f4 d = d2_din4(s_din, e4);
                f4 o;
#pragma unroll
                for (int k = 0; k < 4; ++k) o[k] = mreg[u].pos(k) ? d[k] : 0.f;
                if (p.din16) {
                    bsum[u] += (o[0] + o[1]) + (o[2] + o[3]);
                    uint32_t hb[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) hb[k] = __builtin_bit_cast(unsigned short, (__bf16)o[k]);
                    *(uint2*)(p.din16 + o0 + 4 * e4) = uint2{hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16)};
                } else {
                    *(f4*)(p.din + o0 + 4 * e4) = o;
                }
            }
        }
    }
    if (p.din16) {
        // channel c's sum over its 100 float4 groups (400 pixels), each
        // summed over this workgroup's samples in sample order: four lanes
        // take 25 consecutive groups each, then ((l0 + l1) + (l2 + l3))
        __syncthreads();
#pragma unroll
        for (int u = 0; u < D2_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D2_IN / 4) s_din[e4] = bsum[u];
        }
        __syncthreads();
        constexpr int G = D2_IH * D2_IH / 4, GL = G / 4;
        static_assert(G % 4 == 0 && 4 * D2_CIN <= D2_WG, "four lanes per channel");
        if (t < 4 * D2_CIN) {
            const float* src = s_din + (t >> 2) * G + (t & 3) * GL;
            float sum = 0.f;
            for (int q = 0; q < GL; ++q) sum += src[q];
            sum += __shfl_xor(sum, 1, 64);
            sum += __shfl_xor(sum, 2, 64);
            if ((t & 3) == 0) p.bpart[(size_t)blockIdx.x * D2_CIN + (t >> 2)] = sum;
        }
    }
}

// ---------------------------------------------------------------------------
// conv3 geometry.
constexpr int D3_CIN = 64, D3_IH = 9, D3_COUT = 64, D3_OH = 7, D3_K = 3;
constexpr int D3_P = D3_IH * D3_IH;            // input pixels per sample (81)
constexpr int D3_MT = (D3_P + 15) / 16;        // M-tiles (6)
constexpr int D3_TPW = D3_MT / 2;              // M-tiles per wave (3)
constexpr int D3_DZ = D3_COUT * D3_OH * D3_OH; // dz floats per sample (3,136)
constexpr int D3_IN = D3_CIN * D3_P;           // input-gradient floats per sample (5,184)
constexpr int D3_KT = D3_COUT * D3_K * D3_K;   // contraction length (tap, o): 576
constexpr int D3_OUT4 = (D3_IN / 4 + D2_WG - 1) / D2_WG;
static_assert(D3_MT % 2 == 0 && D3_IN % 4 == 0, "tile split and float4 rows");

// conv3 with dz staged channels-last as bf16 (the bf16-input variant; eight
// waves of (N-tile, half of the six M-tiles)): slot
// sigma = 9 (y + 2) + x + 2 of the zero-bordered map (two zero rows above
// and below, columns 7 and 8 of a row zero, two lead slots) holds dz[o][y][x]
// for the 64 channels, 144 bytes per slot; pixel m reads tap (ky, kx) at
// slot m + 20 - 9ky - kx.  k-step s: tap s / 2, channels 32 (s % 2) + 8g + e.
constexpr int D3C_SLOTS = 120;                 // every read: slot 0 .. 115
constexpr int D3C_PSB = 144;

template <bool H16, bool PK>   // PK: bf16 weight operands from p.wpk (weight_repack)
__global__ __launch_bounds__(D2_WG) void conv3_dgrad_cl_kernel(Dgrad2Params p) {
    __shared__ __align__(16) unsigned char s_cl[D3C_SLOTS * D3C_PSB];
    __shared__ __align__(16) float s_din[D3_IN];
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int nt = wave & 3, mh = wave >> 2;   // N-tile; half of the M-tiles

    for (int e = t; e < D3C_SLOTS * D3C_PSB / 16; e += D2_WG) ((uint4*)s_cl)[e] = uint4{0u, 0u, 0u, 0u};

    const int j_lo = blockIdx.x * p.spg;
    const int j_hi = min(p.n, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // uniform

    constexpr int KS = D3_KT / 32;
    const int c = nt * 16 + li;
    bf16x8 wreg[KS];
    if constexpr (PK) {
#pragma unroll
        for (int s = 0; s < KS; ++s) wreg[s] = ((const bf16x8*)p.wpk)[((size_t)nt * KS + s) * 64 + lane];
    } else {
        const float* wc = p.w + (size_t)c * D3_K * D3_K;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int tap = s / 2;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int o = 32 * (s % 2) + 8 * g + e;
                wreg[s][e] = (__bf16)wc[(size_t)o * D3_CIN * D3_K * D3_K + tap];
            }
        }
    }
    int base[D3_TPW];
#pragma unroll
    for (int i = 0; i < D3_TPW; ++i) base[i] = ((mh * D3_TPW + i) * 16 + li + 20) * D3C_PSB + 16 * g;

    DzStage<D3_OH, D3_IH, 2, 2, 1> dzs;
    auto fetch = [&](int j) { dzs.fetch(p.dz + (size_t)j * D3_DZ, t); };
    auto stage = [&]() { dzs.stage(s_cl, t, 0); };

    fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        const size_t o0 = (size_t)j * D3_IN;
        Mask4<H16> mreg[D3_OUT4];
#pragma unroll
        for (int u = 0; u < D3_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D3_IN / 4) mreg[u].load(p, o0 + 4 * e4);
        }

        f4 acc[D3_TPW];
#pragma unroll
        for (int i = 0; i < D3_TPW; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        constexpr int AHEAD = 2;
        auto a_at = [&](int s, int i) {
            const int tap = s / 2, ky = tap / 3, kx = tap % 3;
            return *(const bf16x8*)(s_cl + base[i] - (D3_IH * ky + kx) * D3C_PSB + 64 * (s % 2));
        };
        bf16x8 abuf[AHEAD + 1][D3_TPW];
#pragma unroll
        for (int d = 0; d < AHEAD; ++d)
#pragma unroll
            for (int i = 0; i < D3_TPW; ++i) abuf[d][i] = a_at(d, i);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            if (s + AHEAD < KS) {
#pragma unroll
                for (int i = 0; i < D3_TPW; ++i) abuf[(s + AHEAD) % (AHEAD + 1)][i] = a_at(s + AHEAD, i);
            }
#pragma unroll
            for (int i = 0; i < D3_TPW; ++i) acc[i] = mfma16x16x32bf16(abuf[s % (AHEAD + 1)][i], wreg[s], acc[i]);
            __builtin_amdgcn_sched_barrier(0);
        }

#pragma unroll
        for (int i = 0; i < D3_TPW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = (mh * D3_TPW + i) * 16 + 4 * g + r;
                if (m < D3_P) s_din[c * D3_P + m] = acc[i][r];
            }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < D3_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D3_IN / 4) {
                const f4 d = *(const f4*)(s_din + 4 * e4);
                f4 o;
#pragma unroll
                for (int q = 0; q < 4; ++q) o[q] = mreg[u].pos(q) ? d[q] : 0.f;
                *(f4*)(p.din + o0 + 4 * e4) = o;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// The float32 input gradients on bf16 MFMA with exact three-term splits (the
// arithmetic of the float32 forward, conv_fwd_x6_kernel: six products per 32
// k-values, float32 accuracy): dz is split into three bf16 planes staged in
// the slot layouts of the bf16 kernels above, the weights' three planes sit
// in registers, loaded in per-lane order from the step's repack (or split
// in the kernel).  Plane pl of the packed weights: element
// ((pl W + w) KS + s) 64 + lane for wave (or N-tile) w and k-step s, in the
// bf16 kernels' k order.
//
// conv2: waves are (phase, N-tile) pairs as in conv2_dgrad_cl_kernel (8
// k-steps of 32: 96 registers of weights); the seven M-tiles of a phase run
// in two groups (4, then 3) to bound the operand registers.
constexpr int X2_KS = D2_KT / 32;              // 8
constexpr int X3_KS = D3_KT / 32;              // 18 (9 per half)
constexpr int X2_LDS = 3 * D2C_SLOTS * D2C_PSB;
constexpr int X3_LDS = 3 * D3C_SLOTS * D3C_PSB;

template <bool PK>
__global__ __launch_bounds__(D2_WG) void conv2_dgrad_x6_kernel(Dgrad2Params p) {
    __shared__ __align__(16) unsigned char s_cl[X2_LDS];     // [3][slots][144]
    __shared__ __align__(16) float s_din[D2_CIN * D2_CS];
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int ph = wave >> 1, nt = wave & 1;
    const int py = ph >> 1, px = ph & 1;
    constexpr int PL = D2C_SLOTS * D2C_PSB;

    for (int e = t; e < X2_LDS / 16; e += D2_WG) ((uint4*)s_cl)[e] = uint4{0u, 0u, 0u, 0u};

    const int j_lo = blockIdx.x * p.spg;
    const int j_hi = min(p.n, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // uniform

    const int c = nt * 16 + li;
    bf16x8 wreg[3][X2_KS];
    if constexpr (PK) {
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
#pragma unroll
            for (int s = 0; s < X2_KS; ++s)
                wreg[pl][s] = ((const bf16x8*)p.wpk)[((size_t)(pl * 8 + wave) * X2_KS + s) * 64 + lane];
    } else {
        const float* wc = p.w + (size_t)c * D2_K * D2_K + py * D2_K + px;
#pragma unroll
        for (int s = 0; s < X2_KS; ++s) {
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int o = 32 * (s % 2) + 8 * g + e;
                __bf16 a, b, d;
                split3(wc[(size_t)o * D2_CIN * D2_K * D2_K + 2 * ty * D2_K + 2 * tx], a, b, d);
                wreg[0][s][e] = a;
                wreg[1][s][e] = b;
                wreg[2][s][e] = d;
            }
        }
    }
    int base[D2_MT];
#pragma unroll
    for (int i = 0; i < D2_MT; ++i) {
        const int m = i * 16 + li, qy = m / D2_Q, qx = m - qy * D2_Q;
        base[i] = (D2_Q * (qy + 1) + qx + 1) * D2C_PSB + 16 * g;
    }

    DzStage<D2_OH, D2_Q, 1, 1, 3, 4> dzs;   // (four channels an item: the register budget)
    auto fetch = [&](int j) { dzs.fetch(p.dz + (size_t)j * D2_DZ, t); };
    auto stage = [&]() { dzs.stage(s_cl, t, PL); };

    // M-tiles [I0, I0 + NI): per k-step the three planes of their A operands,
    // then the six products, each over the group's tiles
    auto group = [&](auto i0c, auto nic, f4* acc) {
        constexpr int I0 = decltype(i0c)::value, NI = decltype(nic)::value;
#pragma unroll
        for (int s = 0; s < X2_KS; ++s) {
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
            const int off = -(D2_Q * ty + tx) * D2C_PSB + 64 * (s % 2);
            bf16x8 a[3][NI];
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
#pragma unroll
                for (int i = 0; i < NI; ++i) a[pl][i] = *(const bf16x8*)(s_cl + pl * PL + base[I0 + i] + off);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[2][i], wreg[0][s], acc[I0 + i]);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[1][i], wreg[1][s], acc[I0 + i]);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[0][i], wreg[2][s], acc[I0 + i]);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[1][i], wreg[0][s], acc[I0 + i]);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[0][i], wreg[1][s], acc[I0 + i]);
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[I0 + i] = mfma16x16x32bf16(a[0][i], wreg[0][s], acc[I0 + i]);
        }
    };

    fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous round's LDS reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);  // in flight during this sample's MFMAs
        const size_t o0 = (size_t)j * D2_IN;
        Mask4<false> mreg[D2_OUT4];
#pragma unroll
        for (int u = 0; u < D2_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D2_IN / 4) mreg[u].load(p, o0 + 4 * e4);
        }
        f4 acc[D2_MT];
#pragma unroll
        for (int i = 0; i < D2_MT; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        group(std::integral_constant<int, 0>{}, std::integral_constant<int, 4>{}, acc);
        group(std::integral_constant<int, 4>{}, std::integral_constant<int, D2_MT - 4>{}, acc);
#pragma unroll
        for (int i = 0; i < D2_MT; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = i * 16 + 4 * g + r;
                if (m < D2_QP) {
                    const int qy = m / D2_Q, qx = m - qy * D2_Q;
                    s_din[c * D2_CS + (2 * qy + py) * D2_IH + 2 * qx + px] = acc[i][r];
                }
            }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < D2_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D2_IN / 4) {
                const f4 d = d2_din4(s_din, e4);
                f4 o;
#pragma unroll
                for (int k = 0; k < 4; ++k) o[k] = mreg[u].pos(k) ? d[k] : 0.f;
                *(f4*)(p.din + o0 + 4 * e4) = o;
            }
        }
    }
}

// conv3: waves are (N-tile, half of the 18 k-steps) pairs (108 registers of
// weights) over all six M-tiles; the second half's sums reach the first
// half's waves through LDS.
template <bool PK>
__global__ __launch_bounds__(D2_WG) void conv3_dgrad_x6_kernel(Dgrad2Params p) {
    __shared__ __align__(16) unsigned char s_cl[X3_LDS];     // [3][slots][144]
    __shared__ __align__(16) float s_din[D3_IN];
    __shared__ f4 s_part[4 * D3_MT * 64];                     // the k-half 1 waves' sums
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int nt = wave & 3, kh = wave >> 2;
    constexpr int PL = D3C_SLOTS * D3C_PSB;
    constexpr int KSH = X3_KS / 2;

    for (int e = t; e < X3_LDS / 16; e += D2_WG) ((uint4*)s_cl)[e] = uint4{0u, 0u, 0u, 0u};

    const int j_lo = blockIdx.x * p.spg;
    const int j_hi = min(p.n, j_lo + p.spg);
    if (j_lo >= j_hi) return;  // uniform

    const int c = nt * 16 + li;
    bf16x8 wreg[3][KSH];
    if constexpr (PK) {
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
#pragma unroll
            for (int s = 0; s < KSH; ++s)
                wreg[pl][s] = ((const bf16x8*)p.wpk)[((size_t)(pl * 4 + nt) * X3_KS + kh * KSH + s) * 64 + lane];
    } else {
        const float* wc = p.w + (size_t)c * D3_K * D3_K;
#pragma unroll
        for (int s = 0; s < KSH; ++s) {
            const int ks = kh * KSH + s, tap = ks / 2;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int o = 32 * (ks % 2) + 8 * g + e;
                __bf16 a, b, d;
                split3(wc[(size_t)o * D3_CIN * D3_K * D3_K + tap], a, b, d);
                wreg[0][s][e] = a;
                wreg[1][s][e] = b;
                wreg[2][s][e] = d;
            }
        }
    }
    int base[D3_MT];
#pragma unroll
    for (int i = 0; i < D3_MT; ++i) base[i] = (i * 16 + li + 20) * D3C_PSB + 16 * g;

    DzStage<D3_OH, D3_IH, 2, 2, 3> dzs;
    auto fetch = [&](int j) { dzs.fetch(p.dz + (size_t)j * D3_DZ, t); };
    auto stage = [&]() { dzs.stage(s_cl, t, PL); };
    auto half = [&](auto khc, f4* acc) {
        constexpr int KH = decltype(khc)::value;
#pragma unroll
        for (int s = 0; s < KSH; ++s) {
            const int ks = KH * KSH + s, tap = ks / 2, ky = tap / 3, kx = tap % 3;
            const int off = -(D3_IH * ky + kx) * D3C_PSB + 64 * (ks % 2);
            bf16x8 a[3][D3_MT];
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
#pragma unroll
                for (int i = 0; i < D3_MT; ++i) a[pl][i] = *(const bf16x8*)(s_cl + pl * PL + base[i] + off);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[2][i], wreg[0][s], acc[i]);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[1][i], wreg[1][s], acc[i]);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wreg[2][s], acc[i]);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[1][i], wreg[0][s], acc[i]);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wreg[1][s], acc[i]);
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) acc[i] = mfma16x16x32bf16(a[0][i], wreg[0][s], acc[i]);
        }
    };

    fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous round's LDS reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        const size_t o0 = (size_t)j * D3_IN;
        Mask4<false> mreg[D3_OUT4];
#pragma unroll
        for (int u = 0; u < D3_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D3_IN / 4) mreg[u].load(p, o0 + 4 * e4);
        }
        f4 acc[D3_MT];
#pragma unroll
        for (int i = 0; i < D3_MT; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        if (kh == 0)
            half(std::integral_constant<int, 0>{}, acc);
        else
            half(std::integral_constant<int, 1>{}, acc);
        if (kh == 1) {
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) s_part[(nt * D3_MT + i) * 64 + lane] = acc[i];
        }
        __syncthreads();
        if (kh == 0) {
            // D[4g + r][li] of tile i: pixel m, channel c
#pragma unroll
            for (int i = 0; i < D3_MT; ++i) {
                const f4 o = s_part[(nt * D3_MT + i) * 64 + lane];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = i * 16 + 4 * g + r;
                    if (m < D3_P) s_din[c * D3_P + m] = acc[i][r] + o[r];
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < D3_OUT4; ++u) {
            const int e4 = t + u * D2_WG;
            if (e4 < D3_IN / 4) {
                const f4 d = *(const f4*)(s_din + 4 * e4);
                f4 o;
#pragma unroll
                for (int q = 0; q < 4; ++q) o[q] = mreg[u].pos(q) ? d[q] : 0.f;
                *(f4*)(p.din + o0 + 4 * e4) = o;
            }
        }
    }
}

// The weights of the large network's conv2/conv3 input-gradient kernels in
// the order their lanes load them into registers, so that every load of a
// wave is one contiguous row instead of a gather of scattered words: one
// 8-value bf16 vector per element, element ((w KS + s) 64 + lane) holding
// wave w's k-step s, w over the 8 (phase, N-tile) waves of conv2 (KS = 8) or
// the 4 N-tiles of conv3 (KS = 18), values W[o][c][tap] as the kernels read;
// the float32 kernels' copies hold the three planes of the exact split one
// after another.  Job j of the launch (blockIdx.y) writes one copy; a NULL
// output skips it.  Jobs 4 to 7: the bf16-input forward's weights of
// conv2 and conv3 for both weight sets, vector (nt KS + ks) 64 + lane
// holding W[16nt + li][32 (ks % CH) + 8g + q][ks / CH] rounded (CH = cin /
// 32, KS = taps * CH), as its kernel reads them.  Jobs 8 to 11: the float32
// forward's three planes of the same weights (X6FwdPack), in the same
// launch (a launch of its own had cost 4.4 us at batch 2,048).
template <int CIN, int KK>
__device__ __forceinline__ void fwd_bf16_pack_job(const float* w, void* out, int e) {
    constexpr int CH = CIN / 32, KS = KK * CH;
    if (!out || e >= 4 * KS * 64) return;
    const int lane = e & 63, ks = (e >> 6) % KS, nt = (e >> 6) / KS;
    const int li = lane & 15, g = lane >> 4, tap = ks / CH, cb = ks % CH;
    const float* wr = w + (size_t)(16 * nt + li) * CIN * KK;
    bf16x8 v;
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = (__bf16)wr[(32 * cb + 8 * g + q) * KK + tap];
    ((bf16x8*)out)[e] = v;
}

__global__ __launch_bounds__(256) void weight_repack_kernel(WeightRepack r) {
    const int e = blockIdx.x * 256 + threadIdx.x;
    const int job = blockIdx.y;
    if (job >= 4) {
        switch (job) {
            case 4: fwd_bf16_pack_job<D2_CIN, D2_K * D2_K>(r.w2a, r.f2a, e); break;
            case 5: fwd_bf16_pack_job<D3_CIN, D3_K * D3_K>(r.w3a, r.f3a, e); break;
            case 6: fwd_bf16_pack_job<D2_CIN, D2_K * D2_K>(r.w2b, r.f2b, e); break;
            case 7: fwd_bf16_pack_job<D3_CIN, D3_K * D3_K>(r.w3b, r.f3b, e); break;
            case 8: x6_fwd_pack_job<D2_CIN, D2_K * D2_K>(r.w2a, r.p2a, e); break;
            case 9: x6_fwd_pack_job<D3_CIN, D3_K * D3_K>(r.w3a, r.p3a, e); break;
            case 10: x6_fwd_pack_job<D2_CIN, D2_K * D2_K>(r.w2b, r.p2b, e); break;
            default: x6_fwd_pack_job<D3_CIN, D3_K * D3_K>(r.w3b, r.p3b, e); break;
        }
        return;
    }
    if (job == 0) {   // conv2 input gradient, bf16 operands: one 8-value vector per thread
        constexpr int KS2 = D2_KT / 32;
        if (r.h2 && e < 8 * KS2 * 64) {
            const int lane = e & 63, s = (e >> 6) % KS2, wave = (e >> 6) / KS2;
            const int li = lane & 15, g = lane >> 4, ph = wave >> 1, nt = wave & 1;
            const int py = ph >> 1, px = ph & 1, c = nt * 16 + li;
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int o = 32 * (s % 2) + 8 * g + q;
                v[q] = (__bf16)r.w2a[(size_t)o * D2_CIN * D2_K * D2_K + (size_t)c * D2_K * D2_K +
                                     (py + 2 * ty) * D2_K + px + 2 * tx];
            }
            ((bf16x8*)r.h2)[e] = v;
        }
    } else if (job == 1) {   // conv3 input gradient, bf16 operands
        constexpr int KS3 = D3_KT / 32;
        if (r.h3 && e < 4 * KS3 * 64) {
            const int lane = e & 63, s = (e >> 6) % KS3, nt = (e >> 6) / KS3;
            const int li = lane & 15, g = lane >> 4, c = nt * 16 + li;
            const int tap = s / 2;
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int o = 32 * (s % 2) + 8 * g + q;
                v[q] = (__bf16)r.w3a[(size_t)o * D3_CIN * D3_K * D3_K + (size_t)c * D3_K * D3_K + tap];
            }
            ((bf16x8*)r.h3)[e] = v;
        }
    } else if (job == 2) {   // conv2 float32 input gradient: plane pl of the split, as job 0
        if (r.x2 && e < 3 * 8 * X2_KS * 64) {
            const int lane = e & 63, s = (e >> 6) % X2_KS, wave = ((e >> 6) / X2_KS) % 8, pl = (e >> 6) / (8 * X2_KS);
            const int li = lane & 15, g = lane >> 4, ph = wave >> 1, nt = wave & 1;
            const int py = ph >> 1, px = ph & 1, c = nt * 16 + li;
            const int tap = s / 2, ty = tap >> 1, tx = tap & 1;
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int o = 32 * (s % 2) + 8 * g + q;
                __bf16 a, b, d;
                split3(r.w2a[(size_t)o * D2_CIN * D2_K * D2_K + (size_t)c * D2_K * D2_K + (py + 2 * ty) * D2_K + px +
                             2 * tx], a, b, d);
                v[q] = pl == 0 ? a : pl == 1 ? b : d;
            }
            ((bf16x8*)r.x2)[e] = v;
        }
    } else {   // job 3: conv3 float32 input gradient, as job 1
        if (r.x3 && e < 3 * 4 * X3_KS * 64) {
            const int lane = e & 63, s = (e >> 6) % X3_KS, nt = ((e >> 6) / X3_KS) % 4, pl = (e >> 6) / (4 * X3_KS);
            const int li = lane & 15, g = lane >> 4, c = nt * 16 + li;
            const int tap = s / 2;
            bf16x8 v;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int o = 32 * (s % 2) + 8 * g + q;
                __bf16 a, b, d;
                split3(r.w3a[(size_t)o * D3_CIN * D3_K * D3_K + (size_t)c * D3_K * D3_K + tap], a, b, d);
                v[q] = pl == 0 ? a : pl == 1 ? b : d;
            }
            ((bf16x8*)r.x3)[e] = v;
        }
    }
}

}  // namespace

// floats of the larger copy of a layer (the float32 planes: 4 floats per bf16x8)
int64_t weight_repack_floats(ConvId id) { return id == CONV_L2 ? 4 * 3 * 8 * X2_KS * 64 : 4 * 3 * 4 * X3_KS * 64; }

hipError_t launch_weight_repack(const WeightRepack& r, hipStream_t st) {
    for (const void* q : {r.h2, r.h3, r.x2, r.x3, r.f2a, r.f3a, r.f2b, r.f3b, r.p2a, r.p3a, r.p2b, r.p3b})
        if ((uintptr_t)q & 15) return hipErrorInvalidValue;
    if ((r.f2b && !r.w2b) || (r.f3b && !r.w3b) || (r.p2b && !r.w2b) || (r.p3b && !r.w3b)) return hipErrorInvalidValue;
    // every copy has at most 3 * 4 * 18 * 64 = 13,824 vectors; the forward's
    // jobs only when one of their outputs is set
    static_assert(X6FwdPack<D2_CIN, D2_K * D2_K>::VECS <= 13824 && X6FwdPack<D3_CIN, D3_K * D3_K>::VECS <= 13824 &&
                      3 * 8 * X2_KS * 64 <= 13824 && 3 * 4 * X3_KS * 64 <= 13824,
                  "copies within the grid");
    const bool x6 = r.p2a || r.p3a || r.p2b || r.p3b;
    const bool fwd = r.f2a || r.f3a || r.f2b || r.f3b;
    hipLaunchKernelGGL(weight_repack_kernel, dim3(13824 / 256, x6 ? 12 : fwd ? 8 : 4), dim3(256), 0, st, r);
    return hipGetLastError();
}

hipError_t launch_conv3_dgrad(const float* dz, const float* w, const float* h_in, float* din, int n, bool bf16,
                              bool h16, const float* wpk, hipStream_t st) {
    if (n <= 0 || ((uintptr_t)h_in & 15) || ((uintptr_t)din & 15) || (h16 && !bf16)) return hipErrorInvalidValue;
    const int spg = std::max(1, (n + 255) / 256);
    const int blocks = (n + spg - 1) / spg;
    const Dgrad2Params prm{dz, w, h_in, din, n, spg, wpk};
    const dim3 grid((unsigned)blocks), blk(D2_WG);
    if (bf16 && h16 && wpk) hipLaunchKernelGGL((conv3_dgrad_cl_kernel<true, true>), grid, blk, 0, st, prm);
    else if (bf16 && h16) hipLaunchKernelGGL((conv3_dgrad_cl_kernel<true, false>), grid, blk, 0, st, prm);
    else if (bf16 && wpk) hipLaunchKernelGGL((conv3_dgrad_cl_kernel<false, true>), grid, blk, 0, st, prm);
    else if (bf16) hipLaunchKernelGGL((conv3_dgrad_cl_kernel<false, false>), grid, blk, 0, st, prm);
    else if (prm.wpk) hipLaunchKernelGGL(conv3_dgrad_x6_kernel<true>, grid, blk, 0, st, prm);
    else hipLaunchKernelGGL(conv3_dgrad_x6_kernel<false>, grid, blk, 0, st, prm);
    return hipGetLastError();
}

int conv2_dgrad_phase_blocks(int n) {
    const int spg = std::max(1, (n + 255) / 256);
    return (n + spg - 1) / spg;
}

hipError_t launch_conv2_dgrad_phase(const float* dz, const float* w, const float* h_in, float* din, int n,
                                    bool bf16, bool h16, const float* wpk, hipStream_t st, __bf16* din16,
                                    float* bpart) {
    if (n <= 0 || ((uintptr_t)h_in & 15) || (h16 && !bf16)) return hipErrorInvalidValue;
    if (din16 ? (!bf16 || !bpart || ((uintptr_t)din16 & 15)) : ((uintptr_t)din & 15)) return hipErrorInvalidValue;
    // about one workgroup per CU, one sample per round
    const int spg = std::max(1, (n + 255) / 256);
    const int blocks = (n + spg - 1) / spg;
    const Dgrad2Params prm{dz, w, h_in, din, n, spg, wpk, din16, bpart};
    const dim3 grid((unsigned)blocks), blk(D2_WG);
    if (bf16 && h16 && wpk) hipLaunchKernelGGL((conv2_dgrad_cl_kernel<true, true>), grid, blk, 0, st, prm);
    else if (bf16 && h16) hipLaunchKernelGGL((conv2_dgrad_cl_kernel<true, false>), grid, blk, 0, st, prm);
    else if (bf16 && wpk) hipLaunchKernelGGL((conv2_dgrad_cl_kernel<false, true>), grid, blk, 0, st, prm);
    else if (bf16) hipLaunchKernelGGL((conv2_dgrad_cl_kernel<false, false>), grid, blk, 0, st, prm);
    else if (prm.wpk) hipLaunchKernelGGL(conv2_dgrad_x6_kernel<true>, grid, blk, 0, st, prm);
    else hipLaunchKernelGGL(conv2_dgrad_x6_kernel<false>, grid, blk, 0, st, prm);
    return hipGetLastError();
}

}  // namespace dqn
