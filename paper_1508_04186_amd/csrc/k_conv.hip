// Convolution layers of the Q-network (Sec. III.A): forward with fused
// bias + ReLU, weight/bias gradient, and input gradient with the ReLU mask of
// the layer below fused in.  All three are implicit GEMMs on fp32 MFMA
// (v_mfma_f32_16x16x4_f32) with every operand staged in LDS: a workgroup
// copies its weights once (padded so the 16 lanes of an MFMA row and the 4
// lane groups fall in distinct banks) and the input rows it needs (16-byte
// loads where aligned), then runs its MFMA loop from LDS only.
// Activations are NCHW float32; the network input is bytes.

#include "conv_body.h"

namespace dqn {
namespace {

// LDS row strides for a weight block [o][c][k*k]: c stride = 16 mod 64,
// o stride = 1 mod 64, so lane (li, g) -> bank li + 16 g is conflict-free.
template <int CIN, int K>
struct WLayout {
    static constexpr int KK = K * K;
    static constexpr int RC = ((KK + 47) / 64) * 64 + 16;   // >= KK, = 16 mod 64
    static constexpr int RO = ((CIN * RC) / 64) * 64 + 65;  // > CIN*RC, = 1 mod 64
};

// Stage weight rows o in [o0, o0+CO) of W[COUT][CIN][K][K] into the padded
// LDS layout, reading 16 bytes at a time (the block is contiguous and k*k is
// a multiple of 4, or the scalar path is taken), 16 loads in flight.
template <int CIN, int K, int CO>
__device__ __forceinline__ void stage_weights(float* __restrict__ sw, const float* __restrict__ W, int o0) {
    using L = WLayout<CIN, K>;
    constexpr int NW = CIN * K * K;
    constexpr int U = 16;
    const float* src = W + (size_t)o0 * NW;
    if constexpr (L::KK % 4 == 0) {
        if (((uintptr_t)src & 15) == 0) {
            constexpr int NV = CO * NW / 4;
            for (int base = threadIdx.x; base < NV; base += U * WG) {
                f4 v[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int e = base + u * WG;
                    if (e < NV) v[u] = ((const f4*)src)[e];
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int e = (base + u * WG) * 4;
                    if (e < CO * NW) {
                        const int o = e / NW, r = e - o * NW;
                        const int c = r / L::KK, k = r - c * L::KK;
                        float* d = sw + o * L::RO + c * L::RC + k;
                        d[0] = v[u][0];
                        d[1] = v[u][1];
                        d[2] = v[u][2];
                        d[3] = v[u][3];
                    }
                }
            }
            return;
        }
    }
    for (int base = threadIdx.x; base < CO * NW; base += U * WG) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * WG;
            if (e < CO * NW) v[u] = src[e];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * WG;
            if (e < CO * NW) {
                const int o = e / NW, r = e - o * NW;
                const int c = r / L::KK, k = r - c * L::KK;
                sw[o * L::RO + c * L::RC + k] = v[u];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Forward.  GEMM view per sample: M = output pixels (oh*ow), N = cout,
// K = cin*k*k.  A workgroup owns a run of 16-pixel M-tiles, a block of CO
// output channels and a run of samples; it stages the weights once and, per
// sample, the input rows its pixels read.  Each wave computes whole M-tiles
// across the CO/16 N-tiles.  Contraction order: lane group g = lane/16 takes
// channel 4*cb + g; MFMA steps walk (cb, ky, kx).
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8, int CO>
__global__ __launch_bounds__(WG) void conv_fwd_kernel(
    ConvIn in_a, ConvIn in_b, int n_a, int n_total,
    const float* __restrict__ w_a, const float* __restrict__ bias_a,
    const float* __restrict__ w_b, const float* __restrict__ bias_b,
    float* __restrict__ out, int mt_per_wg, int spw, int in_rows_max, float in_scale,
    SideFields side) {
    using L = WLayout<CIN, K>;
    constexpr int P = OH * OW;
    constexpr int MT = (P + 15) / 16;
    constexpr int NT = CO / 16;
    constexpr int CB = CIN / 4;
    constexpr int ESZ = U8 ? 1 : 4;
    constexpr int COB = COUT / CO;
    extern __shared__ __align__(16) unsigned char smem[];
    float* sw = (float*)smem;                                       // [CO][RO]
    unsigned char* sin = smem + ((CO * L::RO * 4 + 15) / 16) * 16;  // [CIN][rows][IW]

    const int groups = (MT + mt_per_wg - 1) / mt_per_wg;
    int b = blockIdx.x;
    const int grp = b % groups;
    b /= groups;
    const int cob = b % COB;
    b /= COB;
    const int n0 = b * spw;
    const int n1 = min(n_total, n0 + spw);
    const int o0 = cob * CO;
    const int mt0 = grp * mt_per_wg;
    const int mt1 = min(MT, mt0 + mt_per_wg);
    const int p0 = mt0 * 16;
    const int p1 = min(P, mt1 * 16);
    const int oy0 = p0 / OW;
    const int oy1 = (p1 - 1) / OW;
    const int iy0 = oy0 * S;
    const int rows = (oy1 - oy0) * S + K;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    if (side.idx && blockIdx.x == 0) {
        for (int j = threadIdx.x; j < side.batch; j += WG) {
            const int64_t i = side.idx[j];
            side.a_out[j] = side.action[i];
            side.r_out[j] = (float)side.reward[i];
            side.t_out[j] = side.terminal[i];
        }
    }

    int staged_w = -1;  // which weight set is in LDS: 0 = a, 1 = b
    for (int n = n0; n < n1; ++n) {
        const int second = n >= n_a ? 1 : 0;
        const int ns = second ? n - n_a : n;
        const unsigned char* src = sample_ptr(second ? in_b : in_a, ns);
        __syncthreads();  // previous sample's reads are done
        if (staged_w != second) {
            stage_weights<CIN, K, CO>(sw, second ? w_b : w_a, o0);
            staged_w = second;
        }
        stage_rows(sin, in_rows_max * IW * ESZ, src + (size_t)iy0 * IW * ESZ, (int64_t)IH * IW * ESZ,
                   CIN, rows * IW * ESZ);
        __syncthreads();
        const float* bias = second ? bias_b : bias_a;
        const int row_elems = in_rows_max * IW;

        for (int mt = mt0 + wave; mt < mt1; mt += 4) {
            const int p = mt * 16 + li;
            const int pc = p < P ? p : P - 1;
            const int oy = pc / OW, ox = pc - (pc / OW) * OW;
            const float amask = p < P ? 1.f : 0.f;
            f4 acc[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
            for (int cb = 0; cb < CB; ++cb) {
                const int c = cb * 4 + g;
#pragma unroll
                for (int ky = 0; ky < K; ++ky) {
                    float a[K];
                    const int row = S * oy + ky - iy0;
                    if constexpr (U8) {
                        const unsigned char* base = sin + c * row_elems + row * IW + S * ox;
#pragma unroll
                        for (int q = 0; q < K / 4; ++q) {
                            const uint32_t wv = *(const uint32_t*)(base + 4 * q);
                            a[4 * q + 0] = (float)(wv & 0xffu) * amask;
                            a[4 * q + 1] = (float)((wv >> 8) & 0xffu) * amask;
                            a[4 * q + 2] = (float)((wv >> 16) & 0xffu) * amask;
                            a[4 * q + 3] = (float)(wv >> 24) * amask;
                        }
                    } else {
                        const float* base = (const float*)sin + c * row_elems + row * IW + S * ox;
#pragma unroll
                        for (int kx = 0; kx < K; ++kx) a[kx] = base[kx] * amask;
                    }
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const float* wp = sw + (t * 16 + li) * L::RO + c * L::RC + ky * K;
#pragma unroll
                        for (int kx = 0; kx < K; ++kx) acc[t] = mfma16x16x4(a[kx], wp[kx], acc[t]);
                    }
                }
            }
            // Epilogue: lane holds pixels mt*16 + 4g + r of channel o0 + t*16 + li.
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int o = o0 + t * 16 + li;
                const float bo = bias[o];
                float* dst = out + ((size_t)n * COUT + o) * P;
                const int pb = mt * 16 + 4 * g;
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[t][r] * in_scale + bo, 0.f);
                if constexpr (P % 4 == 0) {
                    if (pb < P) *(f4*)(dst + pb) = f4{v[0], v[1], v[2], v[3]};
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (pb + r < P) dst[pb + r] = v[r];
                }
            }
        }
    }
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
__global__ __launch_bounds__(WG) void conv_wgrad_kernel(WgradParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    conv_wgrad_body<CIN, IH, IW, COUT, K, S, OH, OW, U8>(p, blockIdx.x, smem);
}

// ---------------------------------------------------------------------------
// Input gradient (transposed convolution), split into stride phases so no
// MFMA multiplies a structural zero: input pixel (S*qy + py, S*qx + px)
// receives W[o][c][py + S*ty][px + S*tx] * dz[o][qy - ty][qx - tx] for taps
// ty, tx < K/S.  GEMM view per (sample, phase): M = phase pixels, N = cin,
// contraction over (o, ty, tx).  dz is staged in LDS with a zero border, and
// the phase's weight taps for a block of CI input channels as [tap][o][c].
struct DgradParams {
    const float* dz;
    const float* W;
    const float* h_in;
    float* din;
    int mt_per_wg;
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
__device__ __forceinline__ void conv_dgrad_body(const DgradParams& p, int bid, unsigned char* smem) {
    const float* __restrict__ dz = p.dz;
    const float* __restrict__ W = p.W;
    const float* __restrict__ h_in = p.h_in;
    float* __restrict__ din = p.din;
    const int mt_per_wg = p.mt_per_wg;
    static_assert(K % S == 0, "phase decomposition needs k divisible by stride");
    constexpr int T = K / S;
    constexpr int TT = T * T;
    constexpr int QHM = (IH + S - 1) / S;
    constexpr int QWM = (IW + S - 1) / S;
    constexpr int PH = QHM + T - 1;
    constexpr int PW = QWM + T - 1;
    constexpr int NT = CI / 16;
    constexpr int OB = COUT / 4;
    constexpr int CIB = CIN / CI;
    constexpr int RCW = CI + 1;   // LDS row stride of the [tap][o][c] weight slice
    constexpr int MTM = (QHM * QWM + 15) / 16;
    float* s_dz = (float*)smem;                 // [COUT][PH][PW]
    float* s_w = s_dz + COUT * PH * PW;         // [TT][COUT][RCW]

    const int groups = (MTM + mt_per_wg - 1) / mt_per_wg;
    int b = bid;
    const int grp = b % groups;
    b /= groups;
    const int cib = b % CIB;
    b /= CIB;
    const int ph = b % (S * S);
    const int n = b / (S * S);
    const int py = ph / S, px = ph - (ph / S) * S;
    const int QH = (IH - py + S - 1) / S;
    const int QW = (IW - px + S - 1) / S;
    const int QP = QH * QW;
    const int MTq = (QP + 15) / 16;
    const int mt0 = grp * mt_per_wg;
    const int mt1 = min(MTq, mt0 + mt_per_wg);
    if (mt0 >= mt1) return;  // uniform across the workgroup
    const int c0 = cib * CI;

    // The first UW weight-tap values per thread are loaded before dz is
    // staged, so both sets of loads are in flight together.
    const float* dzn = dz + (size_t)n * COUT * OH * OW;
    constexpr int NWT = TT * COUT * CI;
    constexpr int UW = 8, UD = 16;
    auto w_load = [&](int base, float (&v)[UW]) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int e = base + u * WG;
            const int c = e % CI;
            const int r = e / CI;
            const int o = r % COUT;
            const int tap = r / COUT;
            const int ty = tap / T, tx = tap - (tap / T) * T;
            v[u] = e < NWT ? W[(((size_t)o * CIN + c0 + c) * K + py + S * ty) * K + px + S * tx] : 0.f;
        }
    };
    auto w_store = [&](int base, const float (&v)[UW]) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int e = base + u * WG;
            if (e < NWT) s_w[(e / CI) * RCW + e % CI] = v[u];
        }
    };
    float wv0[UW];
    w_load(threadIdx.x, wv0);
    for (int base = threadIdx.x; base < COUT * PH * PW; base += UD * WG) {
        float v[UD];
#pragma unroll
        for (int u = 0; u < UD; ++u) {
            const int e = base + u * WG;
            const int o = e / (PH * PW);
            const int r = e - o * (PH * PW);
            const int yy = r / PW, xx = r - (r / PW) * PW;
            const int y = yy - (T - 1), x = xx - (T - 1);
            v[u] = (e < COUT * PH * PW && y >= 0 && y < OH && x >= 0 && x < OW)
                       ? dzn[(o * OH + y) * OW + x] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < UD; ++u) {
            const int e = base + u * WG;
            if (e < COUT * PH * PW) s_dz[e] = v[u];
        }
    }
    w_store(threadIdx.x, wv0);
    for (int base = threadIdx.x + UW * WG; base < NWT; base += UW * WG) {
        float v[UW];
        w_load(base, v);
        w_store(base, v);
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    for (int mt = mt0 + wave; mt < mt1; mt += 4) {
        const int q = mt * 16 + li;
        const int qc = q < QP ? q : QP - 1;
        const int qy = qc / QW, qx = qc - (qc / QW) * QW;
        const float amask = q < QP ? 1.f : 0.f;
        f4 acc[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
        for (int ob = 0; ob < OB; ++ob) {
            const int o = ob * 4 + g;
#pragma unroll
            for (int ty = 0; ty < T; ++ty)
#pragma unroll
                for (int tx = 0; tx < T; ++tx) {
                    const float a = s_dz[(o * PH + qy - ty + T - 1) * PW + qx - tx + T - 1] * amask;
                    const float* wrow = s_w + ((ty * T + tx) * COUT + o) * RCW;
#pragma unroll
                    for (int t = 0; t < NT; ++t) acc[t] = mfma16x16x4(a, wrow[t * 16 + li], acc[t]);
                }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int c = c0 + t * 16 + li;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int qq = mt * 16 + 4 * g + r;
                if (qq < QP) {
                    const int qyy = qq / QW, qxx = qq - (qq / QW) * QW;
                    const size_t idx = ((size_t)n * CIN + c) * IH * IW + (S * qyy + py) * IW + S * qxx + px;
                    din[idx] = h_in[idx] > 0.f ? acc[t][r] : 0.f;
                }
            }
        }
    }
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
__global__ __launch_bounds__(WG) void conv_dgrad_kernel(DgradParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    conv_dgrad_body<CIN, IH, IW, COUT, K, S, OH, OW, CI>(p, blockIdx.x, smem);
}

// Weight gradient and input gradient of one layer in a single launch: both
// read the same dz and are independent, so at small batch one launch keeps
// more of the chip busy than two in sequence.  Blocks [0, n_w) run the
// weight gradient, the rest the input gradient.
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
__global__ __launch_bounds__(WG) void conv_bwd_kernel(WgradParams w, DgradParams d, int n_w) {
    extern __shared__ __align__(16) unsigned char smem[];
    if ((int)blockIdx.x < n_w)
        conv_wgrad_body<CIN, IH, IW, COUT, K, S, OH, OW, false>(w, blockIdx.x, smem);
    else
        conv_dgrad_body<CIN, IH, IW, COUT, K, S, OH, OW, CI>(d, blockIdx.x - n_w, smem);
}

// ---------------------------------------------------------------------------
// Host-side launch shapes.

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8, int CO>
hipError_t fwd_launch(const ConvIn& in_a, const ConvIn& in_b, int n_a, int n, const float* w_a,
                      const float* b_a, const float* w_b, const float* b_b, float* out,
                      float in_scale, const SideFields* side, hipStream_t st) {
    using L = WLayout<CIN, K>;
    constexpr int P = OH * OW;
    constexpr int MT = (P + 15) / 16;
    constexpr int ESZ = U8 ? 1 : 4;
    constexpr int COB = COUT / CO;
    // Small batches: one M-tile per wave and one sample per workgroup, for
    // parallelism; large batches: whole samples and several per workgroup,
    // so the weight staging is amortised.
    const long tiles = (long)n * MT * COB;
    int mt_per_wg, spw;
    if (tiles >= 8L * 1024 * 4) {
        mt_per_wg = MT;
        spw = 4;
    } else if (tiles >= 2L * 1024 * 4) {
        mt_per_wg = MT;
        spw = 1;
    } else {
        mt_per_wg = 4;
        spw = 1;
    }
    if (mt_per_wg > MT) mt_per_wg = MT;
    const int groups = (MT + mt_per_wg - 1) / mt_per_wg;
    int max_rows = 0;
    for (int gi = 0; gi < groups; ++gi) {
        const int p0 = gi * mt_per_wg * 16;
        const int p1 = std::min(P, (gi + 1) * mt_per_wg * 16);
        max_rows = std::max(max_rows, ((p1 - 1) / OW - p0 / OW) * S + K);
    }
    // keep each channel's staged rows 16-byte aligned
    while ((max_rows * IW * ESZ) % 16 != 0) ++max_rows;
    const size_t w_bytes = ((size_t)CO * L::RO * 4 + 15) / 16 * 16;
    const size_t lds = w_bytes + (size_t)CIN * max_rows * IW * ESZ;
    auto kern = conv_fwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8, CO>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    const int nblk = (n + spw - 1) / spw;
    SideFields none{};
    hipLaunchKernelGGL(kern, dim3((unsigned)(nblk * COB * groups)), dim3(WG), lds, st, in_a, in_b, n_a,
                       n, w_a, b_a, w_b, b_b, out, mt_per_wg, spw, max_rows, in_scale,
                       side ? *side : none);
    return hipGetLastError();
}


// Launch parameters of a layer's input gradient for `batch` samples.
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
DgradParams dgrad_params(const float* dz, const float* w, const float* h_in, float* din, int batch,
                         int* blocks, size_t* lds) {
    constexpr int QP = ((IH + S - 1) / S) * ((IW + S - 1) / S);
    constexpr int MTM = (QP + 15) / 16;
    constexpr int CIB = CIN / CI;
    constexpr int T = K / S;
    constexpr int PH = (IH + S - 1) / S + T - 1;
    constexpr int PW = (IW + S - 1) / S + T - 1;
    const long wgs = (long)batch * S * S * CIB;
    const int mt_per_wg = wgs >= 1024 ? MTM : 4;
    const int groups = (MTM + mt_per_wg - 1) / mt_per_wg;
    *lds = ((size_t)COUT * PH * PW + (size_t)T * T * COUT * (CI + 1)) * 4;
    *blocks = (int)(wgs * groups);
    return DgradParams{dz, w, h_in, din, mt_per_wg};
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
hipError_t wgrad_launch(const ConvIn& in, const float* dz, int batch, float* wpart, float* bpart,
                        float in_scale, hipStream_t st) {
    int blocks;
    size_t lds;
    const WgradParams p = wgrad_params<CIN, IH, IW, COUT, K, S, OH, OW, U8>(in, dz, batch, wpart, bpart,
                                                                         in_scale, &blocks, &lds);
    auto kern = conv_wgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(WG), lds, st, p);
    return hipGetLastError();
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
hipError_t dgrad_launch(const float* dz, const float* w, const float* h_in, float* din, int batch,
                        hipStream_t st) {
    int blocks;
    size_t lds;
    const DgradParams p = dgrad_params<CIN, IH, IW, COUT, K, S, OH, OW, CI>(dz, w, h_in, din, batch,
                                                                         &blocks, &lds);
    auto kern = conv_dgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, CI>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(WG), lds, st, p);
    return hipGetLastError();
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, int CI>
hipError_t bwd_launch(const ConvIn& in, const float* dz, int batch, float* wpart, float* bpart,
                      const float* w, const float* h_in, float* din, hipStream_t st) {
    int bw, bd;
    size_t lw, ld;
    const WgradParams pw = wgrad_params<CIN, IH, IW, COUT, K, S, OH, OW, false>(in, dz, batch, wpart,
                                                                             bpart, 1.f, &bw, &lw);
    const DgradParams pd = dgrad_params<CIN, IH, IW, COUT, K, S, OH, OW, CI>(dz, w, h_in, din, batch,
                                                                          &bd, &ld);
    const size_t lds = std::max(lw, ld);
    auto kern = conv_bwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW, CI>;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, dim3((unsigned)(bw + bd)), dim3(WG), lds, st, pw, pd, bw);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_fwd(ConvId id, const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                           const float* w_a, const float* b_a, const float* w_b, const float* b_b,
                           float* out, float in_scale, const SideFields* side, hipStream_t st) {
    switch (id) {
        case CONV_S1: return fwd_launch<4, 84, 84, 16, 8, 4, 20, 20, true, 16>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, side, st);
        case CONV_S2: return fwd_launch<16, 20, 20, 32, 4, 2, 9, 9, false, 32>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, side, st);
        case CONV_L1: return fwd_launch<4, 84, 84, 32, 8, 4, 20, 20, true, 32>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, side, st);
        case CONV_L2: return fwd_launch<32, 20, 20, 64, 4, 2, 9, 9, false, 32>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, side, st);
        case CONV_L3: return fwd_launch<64, 9, 9, 64, 3, 1, 7, 7, false, 16>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, side, st);
        default: return hipErrorInvalidValue;
    }
}

int conv_wgrad_chunks(ConvId id, int batch) {
    WgradShape w;
    switch (id) {
        case CONV_S1: w = wgrad_shape(batch, wgrad_groups<4, 84, 84, 16, 8, 4, 20, 20>(), 20); break;
        case CONV_S2: w = wgrad_shape(batch, wgrad_groups<16, 20, 20, 32, 4, 2, 9, 9>(), 9); break;
        case CONV_L1: w = wgrad_shape(batch, wgrad_groups<4, 84, 84, 32, 8, 4, 20, 20>(), 20); break;
        case CONV_L2: w = wgrad_shape(batch, wgrad_groups<32, 20, 20, 64, 4, 2, 9, 9>(), 9); break;
        case CONV_L3: w = wgrad_shape(batch, wgrad_groups<64, 9, 9, 64, 3, 1, 7, 7>(), 7); break;
        default: return -1;
    }
    return w.chunks * w.rb;
}

hipError_t launch_conv_wgrad(ConvId id, const ConvIn& in, const float* dz, int batch, float* wpart,
                             float* bpart, float in_scale, hipStream_t st) {
    switch (id) {
        case CONV_S1: return wgrad_launch<4, 84, 84, 16, 8, 4, 20, 20, true>(in, dz, batch, wpart, bpart, in_scale, st);
        case CONV_S2: return wgrad_launch<16, 20, 20, 32, 4, 2, 9, 9, false>(in, dz, batch, wpart, bpart, in_scale, st);
        case CONV_L1: return wgrad_launch<4, 84, 84, 32, 8, 4, 20, 20, true>(in, dz, batch, wpart, bpart, in_scale, st);
        case CONV_L2: return wgrad_launch<32, 20, 20, 64, 4, 2, 9, 9, false>(in, dz, batch, wpart, bpart, in_scale, st);
        case CONV_L3: return wgrad_launch<64, 9, 9, 64, 3, 1, 7, 7, false>(in, dz, batch, wpart, bpart, in_scale, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_conv_dgrad(ConvId id, const float* dz, const float* w, const float* h_in,
                             float* din, int batch, hipStream_t st) {
    switch (id) {
        case CONV_S2: return dgrad_launch<16, 20, 20, 32, 4, 2, 9, 9, 16>(dz, w, h_in, din, batch, st);
        case CONV_L2: return dgrad_launch<32, 20, 20, 64, 4, 2, 9, 9, 16>(dz, w, h_in, din, batch, st);
        case CONV_L3: return dgrad_launch<64, 9, 9, 64, 3, 1, 7, 7, 16>(dz, w, h_in, din, batch, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn

namespace dqn {

hipError_t launch_conv_bwd(ConvId id, const ConvIn& in, const float* dz, int batch, float* wpart,
                           float* bpart, const float* w, const float* h_in, float* din,
                           hipStream_t st) {
    switch (id) {
        case CONV_S2: return bwd_launch<16, 20, 20, 32, 4, 2, 9, 9, 16>(in, dz, batch, wpart, bpart, w, h_in, din, st);
        case CONV_L2: return bwd_launch<32, 20, 20, 64, 4, 2, 9, 9, 16>(in, dz, batch, wpart, bpart, w, h_in, din, st);
        case CONV_L3: return bwd_launch<64, 9, 9, 64, 3, 1, 7, 7, 16>(in, dz, batch, wpart, bpart, w, h_in, din, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn
