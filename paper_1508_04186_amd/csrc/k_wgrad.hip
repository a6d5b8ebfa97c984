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

// Up to 256 samples: two samples per slot, a slot's two workgroups taking
// half of the output channels each; above, one workgroup per slot and
// enough samples per slot that there are at most 256 slots.
constexpr bool kSplitConv2 = false, kSplitConv3 = true;   // layers whose slots split up to 256 samples
int wgrad_reg_ms(int cin, int n) { return n <= 256 && (cin == 32 ? kSplitConv2 : kSplitConv3) ? 2 : 1; }
int wgrad_reg_spg(int cin, int n) { return wgrad_reg_ms(cin, n) == 2 ? 2 : std::max(1, (n + 255) / 256); }

template <int CIN, int IH, int K, int S, int OH>
hipError_t wgrad_reg_launch(const float* in, const float* dz, int n, float* wpart, float* bpart, bool bf16,
                            bool in16, hipStream_t st) {
    using G = WgradGeom<CIN, IH, K, S, OH>;
    if (n <= 0) return hipErrorInvalidValue;
    const int spg = wgrad_reg_spg(CIN, n), ms = wgrad_reg_ms(CIN, n);
    const int blocks = (n + spg - 1) / spg * ms;
    if (in16 && !bf16) return hipErrorInvalidValue;
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
    if (in16) return go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, true, 1, true>);
    return bf16 ? go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, true, 1, false>)
                : go(conv_wgrad_reg_kernel<CIN, IH, K, S, OH, false, 1, false>);
}

}  // namespace

int conv_wgrad_reg_slots(ConvId id, int n) {
    if (id != CONV_L2 && id != CONV_L3) return -1;
    const int spg = wgrad_reg_spg(id == CONV_L2 ? 32 : 64, n);
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
