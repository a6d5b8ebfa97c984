// Weight and bias gradients of the large network's conv2 and conv3 at large
// batch: dW[o][c][ky][kx] = sum over samples and output pixels p of
// dz[o][p] * in[c][S*oy + ky][S*ox + kx], db[o] = sum dz[o][p].
//
// A workgroup owns every output of the layer (64 x cin*k*k) for a run of
// samples and keeps them in registers across the samples; it writes one
// partial-sum slot at the end, which the finalize kernel reduces in a fixed
// order (no atomics).  For conv3 up to 256 samples (MS = 2) two workgroups
// share a slot, each owning 32 of the 64 output channels for a run of two
// samples: as many workgroups, half the partial-sum bytes written here and
// read back by the finalize kernel (batch 256: conv3 17.1 -> 15.9 us,
// finalize 27.5 -> 27.4; conv2's input is 2.5 times conv3's, and staging it
// twice per workgroup cost more than its halved slots saved).  Per sample, dz and the layer input are staged in LDS
// (the next sample's values read into registers during the MFMAs); the
// contraction runs over the output pixels.  Eight waves: (half of the four
// M-tiles of output channels, or one of the workgroup's two M-tiles when
// MS = 2) x (quarter of the weight columns).  A operand
// dz[o][p]: row stride = 4 (mod 16) floats so the 64 lanes of a read hit 64
// banks; pixels past the map are zero in the stage, so their products
// vanish.  B operand in[c][S*oy + ky][S*ox + kx]: a per-lane column base
// plus a per-step pixel base.  Both precisions: fp32 MFMA (pixel 4s + g in
// step s), or the bf16-input variant (pixel 32s + 4e + g in element e).
// Below, the kernels that stage row segments (every MFMA operand one
// 16-byte LDS read): the bf16-input variant's with bfloat16 activations, and
// the float32 one from 256 samples on bf16 MFMA with the exact three-plane
// split (batch 2,048: conv2 108.6 -> 90.6 us, conv3 73.0 -> 49.3 us).
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace dqn {
namespace {

constexpr int WR_WG = 512;

template <int CIN, int IH, int K, int S, int OH>
struct WgradGeom {
    static constexpr int COUT = 64;
    static constexpr int P = OH * OH;                   // output pixels per sample
    static constexpr int KT = CIN * K * K;              // weight columns
    static constexpr int NTT = KT / 16;                 // N-tiles
    static constexpr int NPW = NTT / 4;                 // N-tiles per wave
    static constexpr int PSTEP32 = (P + 31) / 32;       // bf16 steps
    static constexpr int DCS = ((PSTEP32 * 32 + 3) / 4 | 1) * 4;  // dz row stride: an odd multiple of 4, >= padded pixels
    static constexpr int ICS = IH * IH;                 // input channel stride in LDS
    static constexpr int DZ = COUT * P;                 // dz floats per sample
    static constexpr int IN = CIN * IH * IH;            // input floats per sample
    static constexpr int PER_DZ = (DZ + WR_WG - 1) / WR_WG;
    static constexpr int PER_IN = (IN + WR_WG - 1) / WR_WG;
    static constexpr int LDS = COUT * DCS + IN;         // floats
    static_assert(NTT % 4 == 0, "whole N-tiles per wave");
    static_assert(DCS >= PSTEP32 * 32 && (DCS / 4) % 2 == 1, "dz row stride");
};

struct WgradRegParams {
    const float* in;    // [n][cin][ih][ih] (bfloat16 values when in16)
    const float* dz;    // [n][64][oh][oh]
    float* wpart;       // [slots][64][cin*k*k]
    float* bpart;       // [slots][64]
    int n, spg;         // samples; samples per workgroup (slot)
};

template <int CIN, int IH, int K, int S, int OH, bool BF16, int MS, bool IN16>
__global__ __launch_bounds__(WR_WG) void conv_wgrad_reg_kernel(WgradRegParams p) {
    using G = WgradGeom<CIN, IH, K, S, OH>;
    static_assert(MS == 1 || MS == 2, "one or two workgroups per slot");
    constexpr int MT = 2 / MS;           // M-tiles (16 output channels) per wave
    extern __shared__ __align__(16) float smem[];
    float* s_dz = smem;                  // [64][DCS]
    float* s_in = smem + G::COUT * G::DCS;  // [CIN][IH*IH]
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int mh = wave >> 2, ng = wave & 3;   // N-tiles ng*NPW ...
    const int slot = blockIdx.x / MS, half = blockIdx.x % MS;
    // M-tile of accumulator m: 2mh + m (MS = 1), or 2half + mh (MS = 2)
    auto mtile = [&](int m) { return MS == 1 ? 2 * mh + m : 2 * half + mh; };

    for (int e = t; e < G::COUT * G::DCS; e += WR_WG) s_dz[e] = 0.f;

    const int j_lo = slot * p.spg;
    const int j_hi = min(p.n, j_lo + p.spg);

    // column bases: column n = c*K*K + ky*K + kx of N-tile (ng*NPW + i)
    int cb[G::NPW];
#pragma unroll
    for (int i = 0; i < G::NPW; ++i) {
        const int n = (ng * G::NPW + i) * 16 + li;
        const int c = n / (K * K), r = n - c * (K * K);
        cb[i] = c * G::ICS + (r / K) * IH + (r % K);
    }
    // pixel bases of the steps (pixels past the map read pixel 0: their dz is 0)
    constexpr int NPB = BF16 ? G::PSTEP32 * 8 : (G::P + 3) / 4;
    int pb[NPB];
#pragma unroll
    for (int q = 0; q < NPB; ++q) {
        const int pix = BF16 ? 32 * (q / 8) + 4 * (q % 8) + g : 4 * q + g;
        const int pc = pix < G::P ? pix : 0;
        pb[q] = (S * (pc / OH)) * IH + S * (pc % OH);
    }
    int arow[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) arow[m] = (mtile(m) * 16 + li) * G::DCS + g;

    f4 acc[MT][G::NPW];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i) acc[m][i] = f4{0.f, 0.f, 0.f, 0.f};
    float bsum = 0.f;

    // bfloat16 input (IN16) is read as 32-bit words of two values
    static_assert(G::IN % 2 == 0, "whole words of bfloat16 input");
    constexpr int PER_IN2 = (G::IN / 2 + WR_WG - 1) / WR_WG;
    float vdz[G::PER_DZ], vin[IN16 ? 1 : G::PER_IN];
    uint32_t vin2[IN16 ? PER_IN2 : 1];
    auto fetch = [&](int j) {
        const float* dzj = p.dz + (size_t)j * G::DZ;
        const float* inj = p.in + (size_t)j * G::IN;
        const uint32_t* inw = (const uint32_t*)((const __bf16*)p.in + (size_t)j * G::IN);
#pragma unroll
        for (int u = 0; u < G::PER_DZ; ++u) {
            const int e = t + u * WR_WG;
            vdz[u] = e < G::DZ ? dzj[e] : 0.f;
        }
        if constexpr (IN16) {
#pragma unroll
            for (int u = 0; u < PER_IN2; ++u) {
                const int e = t + u * WR_WG;
                vin2[u] = e < G::IN / 2 ? inw[e] : 0u;
            }
        } else {
#pragma unroll
            for (int u = 0; u < G::PER_IN; ++u) {
                const int e = t + u * WR_WG;
                vin[u] = e < G::IN ? inj[e] : 0.f;
            }
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int u = 0; u < G::PER_DZ; ++u) {
            const int e = t + u * WR_WG;
            if (e < G::DZ) {
                const int o = e / G::P;
                s_dz[o * G::DCS + e - o * G::P] = vdz[u];
            }
        }
        if constexpr (IN16) {   // a bfloat16 is the top half of the float it stands for
#pragma unroll
            for (int u = 0; u < PER_IN2; ++u) {
                const int e = t + u * WR_WG;
                if (e < G::IN / 2) {
                    s_in[2 * e] = __builtin_bit_cast(float, vin2[u] << 16);
                    s_in[2 * e + 1] = __builtin_bit_cast(float, vin2[u] & 0xffff0000u);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < G::PER_IN; ++u) {
                const int e = t + u * WR_WG;
                if (e < G::IN) s_in[e] = vin[u];
            }
        }
    };

    if (j_lo < j_hi) fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous sample's reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        // Opaque per-sample copies of the column bases: the column + pixel
        // sums are then formed inside the loop instead of being hoisted out
        // of it (NPW x NPB live registers).
#pragma unroll
        for (int i = 0; i < G::NPW; ++i) asm volatile("" : "+v"(cb[i]));
        if (half == 0 && t < G::COUT) {
            const float* row = s_dz + t * G::DCS;
            float s0 = 0.f, s1 = 0.f;
            for (int q = 0; q + 1 < G::P; q += 2) {
                s0 += row[q];
                s1 += row[q + 1];
            }
            if (G::P & 1) s0 += row[G::P - 1];
            bsum += s0 + s1;
        }
        if constexpr (BF16) {
#pragma unroll
            for (int st = 0; st < G::PSTEP32; ++st) {
                bf16x8 a[MT], b[G::NPW];
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int e = 0; e < 8; ++e) a[m][e] = (__bf16)s_dz[arow[m] + 32 * st + 4 * e];
#pragma unroll
                for (int i = 0; i < G::NPW; ++i)
#pragma unroll
                    for (int e = 0; e < 8; ++e) b[i][e] = (__bf16)s_in[cb[i] + pb[st * 8 + e]];
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int i = 0; i < G::NPW; ++i) acc[m][i] = mfma16x16x32bf16(a[m], b[i], acc[m][i]);
            }
        } else {
#pragma unroll
            for (int st = 0; st < NPB; ++st) {
                float a[MT], b[G::NPW];
#pragma unroll
                for (int m = 0; m < MT; ++m) a[m] = s_dz[arow[m] + 4 * st];
#pragma unroll
                for (int i = 0; i < G::NPW; ++i) b[i] = s_in[cb[i] + pb[st]];
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int i = 0; i < G::NPW; ++i) acc[m][i] = mfma16x16x4(a[m], b[i], acc[m][i]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }

    // D[4g + r][li] of tile (m, i): channel mtile(m)*16 + 4g + r, column (ng*NPW + i)*16 + li
    if (j_lo >= j_hi) return;  // uniform; padding slot of nothing
    float* wp = p.wpart + (size_t)slot * G::COUT * G::KT;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                wp[(size_t)(mtile(m) * 16 + 4 * g + r) * G::KT + (ng * G::NPW + i) * 16 + li] = acc[m][i][r];
    if (half == 0 && t < G::COUT) p.bpart[(size_t)slot * G::COUT + t] = bsum;
}

// The bf16-input variant with bfloat16 layer input (the TD step's
// activations from 128 samples), one workgroup per slot: operands staged so
// that every MFMA operand is one 16-byte LDS read (the kernel above gathers
// eight scalar words per operand and converts them in the MFMA loop).  The
// contraction over a sample's output pixels runs in segments of eight: a
// row segment is pixels ox = 0..7 of one output row (conv3's rows of seven
// end in a zero of dz), and conv2's ninth column (ox = 8) forms one segment
// over rows 0..7 and one for row 8; k-step st takes segments 4 st + g (lane
// group g), a ninth segment of zeros pads the last step.  Per sample dz is
// staged as bfloat16 [o][segment][8] (the pixel order above) and the input
// as row segments: for channel c, input row y and kernel column kx, the
// eight values in[c][y][S e + kx], e = 0..7, which are the B operand of
// weight column (c, ky, kx) for output row (y - ky) / S; conv2's
// ninth-column segments in[c][2e + ky][16 + kx] are staged apart.  The bias
// sums come from the float32 dz: per (channel, output row) sums in LDS,
// added in row order.
template <int CIN, int IH, int K, int S, int OH>
struct SegGeom {
    static constexpr int COUT = 64, P = OH * OH, KT = CIN * K * K, NTT = KT / 16, NPW = NTT / 4;
    static constexpr bool COL9 = OH > 8;                   // a ninth output column (conv2)
    static constexpr int NROW = OH;                        // row segments
    static constexpr int NSEG = COL9 ? OH + 2 : OH;        // with the ninth column's two
    static constexpr int STEPS = (NSEG + 3) / 4;           // k-steps of four segments
    static constexpr int DZS = 4 * STEPS * 8 + 8;          // dz row stride (bf16; an odd number of 16-byte chunks)
    static constexpr int RSEG = CIN * IH * K * 8;          // [c][y][kx][8]
    static constexpr int CSEG = COL9 ? CIN * K * K * 8 : 0;   // [c][ky][kx][8]: rows 0..7, and row 8 (element 0)
    static constexpr int O_CSEG = RSEG, O_CSEG2 = O_CSEG + CSEG, O_ZERO = O_CSEG2 + CSEG, O_DZ = O_ZERO + 8;
    static constexpr int LDS16 = O_DZ + COUT * DZS;        // bf16 elements
    static constexpr int LDS = LDS16 * 2 + COUT * OH * 4;  // bytes, with the dz row sums
    static constexpr int DZ_ITEMS = COUT * OH, IN_ITEMS = CIN * IH;   // (o, output row), (c, input row)
    static constexpr int DZ_PER = (DZ_ITEMS + WR_WG - 1) / WR_WG, IN_PER = (IN_ITEMS + WR_WG - 1) / WR_WG;
    static constexpr int RW = COL9 ? IH / 2 : IH;          // words (conv2) or values (conv3) read per input row
    static_assert(NTT % 4 == 0 && (DZS / 8) % 2 == 1 && OH <= 9 && (S == 1 || (S == 2 && IH == 20 && K == 4 && OH == 9)),
                  "the large network's conv2 and conv3");
    static_assert(S == 2 || (IH == 9 && K == 3 && OH == 7), "conv3 geometry");
};

template <int CIN, int IH, int K, int S, int OH>
__global__ __launch_bounds__(WR_WG) void conv_wgrad_seg_kernel(WgradRegParams p) {
    using G = SegGeom<CIN, IH, K, S, OH>;
    extern __shared__ __align__(16) float smem[];
    __bf16* s16 = (__bf16*)smem;
    float* s_bs = smem + G::LDS16 / 2;                  // [64][OH] row sums of dz (after the bf16 region)
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int mh = wave >> 2, ng = wave & 3;

    // zero segments, and the dz slots no pixel writes, stay zero
    for (int e = t; e < (G::LDS16 - G::O_CSEG2) / 8; e += WR_WG)
        *(uint4*)(s16 + G::O_CSEG2 + 8 * e) = uint4{0u, 0u, 0u, 0u};

    const int slot = blockIdx.x;
    const int j_lo = slot * p.spg, j_hi = min(p.n, j_lo + p.spg);

    // B operand bases of the lane's column in each N-tile
    int rbase[G::NPW], cbase[G::NPW];
#pragma unroll
    for (int i = 0; i < G::NPW; ++i) {
        const int n = (ng * G::NPW + i) * 16 + li;
        const int c = n / (K * K), r = n - c * (K * K), ky = r / K, kx = r - ky * K;
        rbase[i] = ((c * IH + ky) * K + kx) * 8;
        cbase[i] = G::O_CSEG + ((c * K + ky) * K + kx) * 8;
    }
    // segment s of column base i: its B operand's element offset
    auto boff = [&](int s, int i) -> int {
        if (s < G::NROW) return rbase[i] + S * s * K * 8;
        if (G::COL9 && s == G::NROW) return cbase[i];
        if (G::COL9 && s == G::NROW + 1) return cbase[i] + G::CSEG;
        return G::O_ZERO;
    };
    int arow[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) arow[m] = G::O_DZ + ((2 * mh + m) * 16 + li) * G::DZS + 8 * g;

    f4 acc[2][G::NPW];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i) acc[m][i] = f4{0.f, 0.f, 0.f, 0.f};
    float bsum = 0.f;

    // next sample in registers: dz rows (o, oy) and input rows (c, y)
    float vdz[G::DZ_PER][OH];
    uint32_t vin[G::IN_PER][G::RW];
    auto fetch = [&](int j) {
        const float* dzj = p.dz + (size_t)j * G::COUT * G::P;
        const __bf16* inj = (const __bf16*)p.in + (size_t)j * CIN * IH * IH;
#pragma unroll
        for (int u = 0; u < G::DZ_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::DZ_ITEMS) {
#pragma unroll
                for (int x = 0; x < OH; ++x) vdz[u][x] = dzj[q * OH + x];
            }
        }
#pragma unroll
        for (int u = 0; u < G::IN_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::IN_ITEMS) {
                if constexpr (G::COL9) {   // 20 values, 8-byte aligned: ten words of two
                    const uint2* w = (const uint2*)(inj + q * IH);
#pragma unroll
                    for (int d = 0; d < G::RW / 2; ++d) {
                        const uint2 v = w[d];
                        vin[u][2 * d] = v.x;
                        vin[u][2 * d + 1] = v.y;
                    }
                } else {                   // 9 values, 2-byte aligned
                    const unsigned short* w = (const unsigned short*)(inj + q * IH);
#pragma unroll
                    for (int x = 0; x < IH; ++x) vin[u][x] = w[x];
                }
            }
        }
    };
    auto bits = [](float f) -> uint32_t { return __builtin_bit_cast(unsigned short, (__bf16)f); };
    auto stage = [&]() {
#pragma unroll
        for (int u = 0; u < G::DZ_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::DZ_ITEMS) {
                const int o = q / OH, oy = q - o * OH;
                uint32_t w[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t lo = 2 * k < OH ? bits(vdz[u][2 * k]) : 0u;
                    const uint32_t hi = 2 * k + 1 < OH ? bits(vdz[u][2 * k + 1]) : 0u;
                    w[k] = lo | (hi << 16);
                }
                __bf16* row = s16 + G::O_DZ + o * G::DZS;
                *(uint4*)(row + 8 * oy) = uint4{w[0], w[1], w[2], w[3]};
                if constexpr (G::COL9) {   // ox = 8: segment NROW (rows 0..7) or NROW + 1 (row 8)
                    *(unsigned short*)(row + (oy < 8 ? 8 * G::NROW + oy : 8 * (G::NROW + 1))) = (unsigned short)bits(vdz[u][8]);
                }
                float rs = 0.f;
#pragma unroll
                for (int x = 0; x < OH; ++x) rs += vdz[u][x];
                s_bs[q] = rs;
            }
        }
#pragma unroll
        for (int u = 0; u < G::IN_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::IN_ITEMS) {
                const int c = q / IH, y = q - c * IH;
                __bf16* seg = s16 + (c * IH + y) * K * 8;
                const uint32_t* w = vin[u];
                if constexpr (G::COL9) {
                    // words w_i = (x_2i, x_2i+1); kx even: x_{2e + kx} = lo(w_{e + kx/2}), odd: hi(...)
#pragma unroll
                    for (int kx = 0; kx < 4; ++kx) {
                        const int d = kx >> 1;
                        const uint32_t sel = (kx & 1) ? 0x07060302u : 0x05040100u;
                        uint4 v;
                        v.x = __builtin_amdgcn_perm(w[d + 1], w[d + 0], sel);
                        v.y = __builtin_amdgcn_perm(w[d + 3], w[d + 2], sel);
                        v.z = __builtin_amdgcn_perm(w[d + 5], w[d + 4], sel);
                        v.w = __builtin_amdgcn_perm(w[d + 7], w[d + 6], sel);
                        *(uint4*)(seg + kx * 8) = v;
                    }
                    // ninth column: x_{16 + kx} to segment (c, ky, kx) element (y - ky) / 2 for ky of y's parity
#pragma unroll
                    for (int kx = 0; kx < 4; ++kx) {
                        const unsigned short v = (unsigned short)(w[8 + (kx >> 1)] >> (16 * (kx & 1)));
#pragma unroll
                        for (int kp = 0; kp < 2; ++kp) {
                            const int ky = (y & 1) + 2 * kp, e2 = y - ky;
                            if (e2 >= 0 && e2 <= 16) {
                                const int e = e2 / 2;
                                __bf16* cs = s16 + G::O_CSEG + ((c * K + ky) * K + kx) * 8;
                                *(unsigned short*)(e < 8 ? cs + e : cs + G::CSEG) = v;
                            }
                        }
                    }
                } else {
#pragma unroll
                    for (int kx = 0; kx < K; ++kx) {
                        uint32_t v[4];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int x0 = 2 * k + kx, x1 = x0 + 1;
                            v[k] = (x0 < IH ? w[x0] : 0u) | ((x1 < IH ? w[x1] : 0u) << 16);
                        }
                        *(uint4*)(seg + kx * 8) = uint4{v[0], v[1], v[2], v[3]};
                    }
                }
            }
        }
    };

    if (j_lo < j_hi) fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous sample's reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        if (t < G::COUT) {
#pragma unroll
            for (int oy = 0; oy < OH; ++oy) bsum += s_bs[t * OH + oy];
        }
#pragma unroll
        for (int st = 0; st < G::STEPS; ++st) {
            bf16x8 a[2], b[G::NPW];
#pragma unroll
            for (int m = 0; m < 2; ++m) a[m] = *(const bf16x8*)(s16 + arow[m] + 32 * st);
#pragma unroll
            for (int i = 0; i < G::NPW; ++i) b[i] = *(const bf16x8*)(s16 + boff(4 * st + g, i));
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int i = 0; i < G::NPW; ++i) acc[m][i] = mfma16x16x32bf16(a[m], b[i], acc[m][i]);
        }
    }

    // D[4g + r][li] of tile (m, i): channel (2mh + m)*16 + 4g + r, column (ng*NPW + i)*16 + li
    if (j_lo >= j_hi) return;  // uniform; padding slot of nothing
    float* wp = p.wpart + (size_t)slot * G::COUT * G::KT;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                wp[(size_t)((2 * mh + m) * 16 + 4 * g + r) * G::KT + (ng * G::NPW + i) * 16 + li] = acc[m][i][r];
    if (t < G::COUT) p.bpart[(size_t)slot * G::COUT + t] = bsum;
}

// The float32 weight gradient on bf16 MFMA (from kWgradX6MinRows samples):
// dz and the layer input split exactly into three bfloat16 planes as they
// are staged (split3, hi + mid + lo), each plane in the segment layout of
// conv_wgrad_seg_kernel, and per k-step the six products of planes whose
// product is at least 2^-16 of hi*hi (as the float32 forward), which keeps
// float32 accuracy.  The fp32-MFMA kernel above is bound by the fp32 matrix
// rate (87-90% of its cycles busy at batch 2,048); six bf16 products take
// half that time at the measured rates.  Three planes of conv2's row
// segments do not fit in LDS with all 32 input channels: its workgroups
// take NSPLIT = 2 halves of them, two workgroups per slot (each staging the
// whole dz), which also halves the slots for the finalize to read.  The
// bias sums come from the float32 dz, as in the kernel above.
template <int CIN, int IH, int K, int S, int OH, int NSPLIT>
struct SegX6Geom {
    static constexpr int COUT = 64, P = OH * OH, KK = K * K;
    static constexpr int CW = CIN / NSPLIT;                // input channels per workgroup
    static constexpr int KT = CW * KK, KTF = CIN * KK;     // weight columns: the workgroup's, the layer's
    static constexpr int NTT = KT / 16, NPW = NTT / 4;
    static constexpr bool COL9 = OH > 8;
    static constexpr int NROW = OH;
    static constexpr int NSEG = COL9 ? OH + 2 : OH;
    static constexpr int STEPS = (NSEG + 3) / 4;
    static constexpr int DZS = 4 * STEPS * 8 + 8;           // dz row stride (bf16; an odd number of 16-byte chunks)
    static constexpr int RSEG = CW * IH * K * 8;           // [c][y][kx][8]
    static constexpr int CSEG = COL9 ? CW * KK * 8 : 0;    // [c][ky][kx][8]: rows 0..7, and row 8 (element 0)
    static constexpr int O_CSEG = RSEG, O_CSEG2 = O_CSEG + CSEG, O_ZERO = O_CSEG2 + CSEG, O_DZ = O_ZERO + 8;
    static constexpr int PLANE = O_DZ + COUT * DZS;        // bf16 elements per plane
    static constexpr int LDS = 3 * PLANE * 2 + COUT * OH * 4;   // bytes, with the dz row sums
    static constexpr int DZ_ITEMS = COUT * OH, IN_ITEMS = CW * IH;   // (o, output row), (c, input row)
    static constexpr int DZ_PER = (DZ_ITEMS + WR_WG - 1) / WR_WG, IN_PER = (IN_ITEMS + WR_WG - 1) / WR_WG;
    static_assert(CIN % NSPLIT == 0 && NTT % 4 == 0 && (DZS / 8) % 2 == 1 && PLANE % 8 == 0 && OH <= 9 &&
                      (S == 1 || (S == 2 && IH == 20 && K == 4 && OH == 9)) && (S == 2 || (IH == 9 && K == 3 && OH == 7)),
                  "the large network's conv2 and conv3");
};

template <int CIN, int IH, int K, int S, int OH, int NSPLIT>
__global__ __launch_bounds__(WR_WG) void conv_wgrad_seg_x6_kernel(WgradRegParams p) {
    using G = SegX6Geom<CIN, IH, K, S, OH, NSPLIT>;
    extern __shared__ __align__(16) float smem[];
    __bf16* s16 = (__bf16*)smem;                        // three planes of PLANE elements
    float* s_bs = smem + 3 * G::PLANE / 2;              // [64][OH] row sums of dz
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int mh = wave >> 2, ng = wave & 3;
    const int slot = blockIdx.x / NSPLIT, part = blockIdx.x % NSPLIT;
    const int c0 = part * G::CW;                        // the workgroup's first input channel

    // zero segments, and the dz slots no pixel writes, stay zero in every plane
#pragma unroll
    for (int pl = 0; pl < 3; ++pl)
        for (int e = t; e < (G::PLANE - G::O_CSEG2) / 8; e += WR_WG)
            *(uint4*)(s16 + pl * G::PLANE + G::O_CSEG2 + 8 * e) = uint4{0u, 0u, 0u, 0u};

    const int j_lo = slot * p.spg, j_hi = min(p.n, j_lo + p.spg);

    // B operand bases of the lane's column (of the workgroup's columns) in each N-tile
    int rbase[G::NPW], cbase[G::NPW];
#pragma unroll
    for (int i = 0; i < G::NPW; ++i) {
        const int n = (ng * G::NPW + i) * 16 + li;
        const int c = n / G::KK, r = n - c * G::KK, ky = r / K, kx = r - ky * K;
        rbase[i] = ((c * IH + ky) * K + kx) * 8;
        cbase[i] = G::O_CSEG + ((c * K + ky) * K + kx) * 8;
    }
    auto boff = [&](int sg, int i) -> int {
        if (sg < G::NROW) return rbase[i] + S * sg * K * 8;
        if (G::COL9 && sg == G::NROW) return cbase[i];
        if (G::COL9 && sg == G::NROW + 1) return cbase[i] + G::CSEG;
        return G::O_ZERO;
    };
    int arow[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) arow[m] = G::O_DZ + ((2 * mh + m) * 16 + li) * G::DZS + 8 * g;

    f4 acc[2][G::NPW];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i) acc[m][i] = f4{0.f, 0.f, 0.f, 0.f};
    float bsum = 0.f;

    // next sample in registers: dz rows (o, oy) and the workgroup's input rows (c, y)
    float vdz[G::DZ_PER][OH];
    float vin[G::IN_PER][IH];
    auto fetch = [&](int j) {
        const float* dzj = p.dz + (size_t)j * G::COUT * G::P;
        const float* inj = p.in + ((size_t)j * CIN + c0) * IH * IH;
#pragma unroll
        for (int u = 0; u < G::DZ_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::DZ_ITEMS) {
#pragma unroll
                for (int x = 0; x < OH; ++x) vdz[u][x] = dzj[q * OH + x];
            }
        }
#pragma unroll
        for (int u = 0; u < G::IN_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::IN_ITEMS) {
                if constexpr (IH % 4 == 0) {   // 16-byte aligned rows
                    const f4* w = (const f4*)(inj + q * IH);
#pragma unroll
                    for (int d = 0; d < IH / 4; ++d) {
                        const f4 v = w[d];
#pragma unroll
                        for (int e = 0; e < 4; ++e) vin[u][4 * d + e] = v[e];
                    }
                } else {
#pragma unroll
                    for (int x = 0; x < IH; ++x) vin[u][x] = inj[q * IH + x];
                }
            }
        }
    };
    // the three planes' bits of a value
    auto split_bits = [](float f, uint32_t (&b)[3]) {
        __bf16 h, m, l;
        split3(f, h, m, l);
        b[0] = __builtin_bit_cast(unsigned short, h);
        b[1] = __builtin_bit_cast(unsigned short, m);
        b[2] = __builtin_bit_cast(unsigned short, l);
    };
    auto stage = [&]() {
#pragma unroll
        for (int u = 0; u < G::DZ_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::DZ_ITEMS) {
                const int o = q / OH, oy = q - o * OH;
                uint32_t hb[OH][3];
#pragma unroll
                for (int x = 0; x < OH; ++x) split_bits(vdz[u][x], hb[x]);
#pragma unroll
                for (int pl = 0; pl < 3; ++pl) {
                    uint32_t w[4];
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const uint32_t lo = 2 * k < OH ? hb[2 * k][pl] : 0u;
                        const uint32_t hi = 2 * k + 1 < OH ? hb[2 * k + 1][pl] : 0u;
                        w[k] = lo | (hi << 16);
                    }
                    __bf16* row = s16 + pl * G::PLANE + G::O_DZ + o * G::DZS;
                    *(uint4*)(row + 8 * oy) = uint4{w[0], w[1], w[2], w[3]};
                    if constexpr (G::COL9)   // ox = 8: segment NROW (rows 0..7) or NROW + 1 (row 8)
                        *(unsigned short*)(row + (oy < 8 ? 8 * G::NROW + oy : 8 * (G::NROW + 1))) =
                            (unsigned short)hb[8][pl];
                }
                float rs = 0.f;
#pragma unroll
                for (int x = 0; x < OH; ++x) rs += vdz[u][x];
                s_bs[q] = rs;
            }
        }
#pragma unroll
        for (int u = 0; u < G::IN_PER; ++u) {
            const int q = t + u * WR_WG;
            if (q < G::IN_ITEMS) {
                const int c = q / IH, y = q - c * IH;
                uint32_t hb[IH][3];
#pragma unroll
                for (int x = 0; x < IH; ++x) split_bits(vin[u][x], hb[x]);
#pragma unroll
                for (int pl = 0; pl < 3; ++pl) {
                    __bf16* seg = s16 + pl * G::PLANE + (c * IH + y) * K * 8;
                    if constexpr (G::COL9) {
                        // words w_i = (x_2i, x_2i+1); kx even: x_{2e + kx} = lo(w_{e + kx/2}), odd: hi(...)
                        uint32_t w[IH / 2];
#pragma unroll
                        for (int d = 0; d < IH / 2; ++d) w[d] = hb[2 * d][pl] | (hb[2 * d + 1][pl] << 16);
#pragma unroll
                        for (int kx = 0; kx < 4; ++kx) {
                            const int d = kx >> 1;
                            const uint32_t sel = (kx & 1) ? 0x07060302u : 0x05040100u;
                            uint4 v;
                            v.x = __builtin_amdgcn_perm(w[d + 1], w[d + 0], sel);
                            v.y = __builtin_amdgcn_perm(w[d + 3], w[d + 2], sel);
                            v.z = __builtin_amdgcn_perm(w[d + 5], w[d + 4], sel);
                            v.w = __builtin_amdgcn_perm(w[d + 7], w[d + 6], sel);
                            *(uint4*)(seg + kx * 8) = v;
                        }
                        // ninth column: x_{16 + kx} to segment (c, ky, kx) element (y - ky) / 2 for ky of y's parity
#pragma unroll
                        for (int kx = 0; kx < 4; ++kx) {
                            const unsigned short v = (unsigned short)hb[16 + kx][pl];
#pragma unroll
                            for (int kp = 0; kp < 2; ++kp) {
                                const int ky = (y & 1) + 2 * kp, e2 = y - ky;
                                if (e2 >= 0 && e2 <= 16) {
                                    const int e = e2 / 2;
                                    __bf16* cs = s16 + pl * G::PLANE + G::O_CSEG + ((c * K + ky) * K + kx) * 8;
                                    *(unsigned short*)(e < 8 ? cs + e : cs + G::CSEG) = v;
                                }
                            }
                        }
                    } else {
#pragma unroll
                        for (int kx = 0; kx < K; ++kx) {
                            uint32_t v[4];
#pragma unroll
                            for (int k = 0; k < 4; ++k) {
                                const int x0 = 2 * k + kx, x1 = x0 + 1;
                                v[k] = (x0 < IH ? hb[x0][pl] : 0u) | ((x1 < IH ? hb[x1][pl] : 0u) << 16);
                            }
                            *(uint4*)(seg + kx * 8) = uint4{v[0], v[1], v[2], v[3]};
                        }
                    }
                }
            }
        }
    };

    if (j_lo < j_hi) fetch(j_lo);
    for (int j = j_lo; j < j_hi; ++j) {
        __syncthreads();  // the zero fill, or the previous sample's reads, are done
        stage();
        __syncthreads();
        if (j + 1 < j_hi) fetch(j + 1);
        if (part == 0 && t < G::COUT) {
#pragma unroll
            for (int oy = 0; oy < OH; ++oy) bsum += s_bs[t * OH + oy];
        }
#pragma unroll
        for (int st = 0; st < G::STEPS; ++st) {
            bf16x8 a[3][2];
#pragma unroll
            for (int pl = 0; pl < 3; ++pl)
#pragma unroll
                for (int m = 0; m < 2; ++m) a[pl][m] = *(const bf16x8*)(s16 + pl * G::PLANE + arow[m] + 32 * st);
            // the six plane pairs (dz plane, input plane), smallest first
            constexpr int PA[6] = {2, 1, 0, 1, 0, 0}, PB[6] = {0, 1, 2, 0, 1, 0};
            if constexpr (G::NPW <= 4) {
                // each pair over every tile: 2 NPW independent chains between dependent MFMAs
                // (conv2, batch 2,048: 94.8 -> 90.6 us; conv3's nine N-tiles so took 256
                // VGPRs and 48.8 -> 50.0 us)
                bf16x8 b[3][G::NPW];
#pragma unroll
                for (int pl = 0; pl < 3; ++pl)
#pragma unroll
                    for (int i = 0; i < G::NPW; ++i)
                        b[pl][i] = *(const bf16x8*)(s16 + pl * G::PLANE + boff(4 * st + g, i));
#pragma unroll
                for (int q = 0; q < 6; ++q)
#pragma unroll
                    for (int i = 0; i < G::NPW; ++i)
#pragma unroll
                        for (int m = 0; m < 2; ++m)
                            acc[m][i] = mfma16x16x32bf16(a[PA[q]][m], b[PB[q]][i], acc[m][i]);
            } else {
#pragma unroll
                for (int i = 0; i < G::NPW; ++i) {
                    bf16x8 b[3];
#pragma unroll
                    for (int pl = 0; pl < 3; ++pl)
                        b[pl] = *(const bf16x8*)(s16 + pl * G::PLANE + boff(4 * st + g, i));
#pragma unroll
                    for (int q = 0; q < 6; ++q)
#pragma unroll
                        for (int m = 0; m < 2; ++m) acc[m][i] = mfma16x16x32bf16(a[PA[q]][m], b[PB[q]], acc[m][i]);
                }
            }
        }
    }

    // D[4g + r][li] of tile (m, i): channel (2mh + m)*16 + 4g + r, column c0*KK + (ng*NPW + i)*16 + li
    if (j_lo >= j_hi) return;  // uniform; padding slot of nothing
    float* wp = p.wpart + (size_t)slot * G::COUT * G::KTF + c0 * G::KK;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int i = 0; i < G::NPW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                wp[(size_t)((2 * mh + m) * 16 + 4 * g + r) * G::KTF + (ng * G::NPW + i) * 16 + li] = acc[m][i][r];
    if (part == 0 && t < G::COUT) p.bpart[(size_t)slot * G::COUT + t] = bsum;
}

// Up to 256 samples: two samples per slot, a slot's two workgroups taking
// half of the output channels each; above, one workgroup per slot and
// enough samples per slot that there are at most 256 slots.
constexpr bool kSplitConv2 = false, kSplitConv3 = true;   // layers whose slots split up to 256 samples
int wgrad_reg_ms(int cin, int n) { return n <= 256 && (cin == 32 ? kSplitConv2 : kSplitConv3) ? 2 : 1; }
int wgrad_reg_spg(int cin, int n) { return wgrad_reg_ms(cin, n) == 2 ? 2 : std::max(1, (n + 255) / 256); }

// The float32 six-product kernel: from kWgradX6MinRows samples; conv2's
// slots of two workgroups; enough samples per slot for about 256
// workgroups.  (At batch 256: conv2 19.6 -> 15.1 us, conv3 14.7 -> 12.1 us,
// the finalize +1.8 us for conv3's 256 slots instead of 128.)
constexpr int kWgradX6MinRows = 256;
bool wgrad_x6(bool bf16, int n) { return !bf16 && n >= kWgradX6MinRows; }
int wgrad_x6_nsplit(int cin) { return cin == 32 ? 2 : 1; }
int wgrad_x6_spg(int cin, int n) { return std::max(1, (n * wgrad_x6_nsplit(cin) + 255) / 256); }

template <int CIN, int IH, int K, int S, int OH>
hipError_t wgrad_reg_launch(const float* in, const float* dz, int n, float* wpart, float* bpart, bool bf16,
                            bool in16, hipStream_t st) {
    using G = WgradGeom<CIN, IH, K, S, OH>;
    if (n <= 0) return hipErrorInvalidValue;
    if (in16 && !bf16) return hipErrorInvalidValue;
    if (wgrad_x6(bf16, n)) {
        constexpr int NS = CIN == 32 ? 2 : 1;
        using XG = SegX6Geom<CIN, IH, K, S, OH, NS>;
        const int spg = wgrad_x6_spg(CIN, n);
        const WgradRegParams prm{in, dz, wpart, bpart, n, spg};
        auto kern = conv_wgrad_seg_x6_kernel<CIN, IH, K, S, OH, NS>;
        if (!allow_lds((const void*)kern, XG::LDS)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)((n + spg - 1) / spg * NS)), dim3(WR_WG), XG::LDS, st, prm);
        return hipGetLastError();
    }
    const int spg = wgrad_reg_spg(CIN, n), ms = wgrad_reg_ms(CIN, n);
    const int blocks = (n + spg - 1) / spg * ms;
    const WgradRegParams prm{in, dz, wpart, bpart, n, spg};
    constexpr size_t lds = (size_t)G::LDS * 4;
    auto go = [&](auto kern) -> hipError_t {
        if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(WR_WG), lds, st, prm);
        return hipGetLastError();
    };
    if (ms == 2) {
        if (in16) return go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, true, 2, true>);
        return bf16 ? go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, true, 2, false>)
                    : go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, false, 2, false>);
    }
    if (in16) {   // (row segments staged once: batch 2,048, conv2 42 -> 36 us, conv3 32 -> 23 us)
        using SG = SegGeom<CIN, IH, K, S, OH>;
        auto kern = conv_wgrad_seg_kernel<CIN, IH, K, S, OH>;
        if (!allow_lds((const void*)kern, SG::LDS)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(WR_WG), SG::LDS, st, prm);
        return hipGetLastError();
    }
    return bf16 ? go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, true, 1, false>)
                : go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, false, 1, false>);
}

}  // namespace

int conv_wgrad_reg_slots(ConvId id, int n, bool bf16) {
    if (id != CONV_L2 && id != CONV_L3) return -1;
    const int cin = id == CONV_L2 ? 32 : 64;
    const int spg = wgrad_x6(bf16, n) ? wgrad_x6_spg(cin, n) : wgrad_reg_spg(cin, n);
    return (n + spg - 1) / spg;
}

hipError_t launch_conv_wgrad_reg(ConvId id, const float* in, const float* dz, int n, float* wpart, float* bpart,
                                 bool bf16, bool in16, hipStream_t st) {
    switch (id) {
        case CONV_L2: return wgrad_reg_launch<32, 20, 4, 2, 9>(in, dz, n, wpart, bpart, bf16, in16, st);
        case CONV_L3: return wgrad_reg_launch<64, 9, 3, 1, 7>(in, dz, n, wpart, bpart, bf16, in16, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn
