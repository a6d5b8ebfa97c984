// Convolution layers of the Q-network (Sec. III.A): forward with fused
// bias + ReLU, weight/bias gradient, and input gradient with the ReLU mask of
// the layer below fused in.  All three are implicit GEMMs on fp32 MFMA
// (v_mfma_f32_16x16x4_f32) with LDS-staged operands.  Activations are NCHW
// float32; the network input is bytes.
#include "common.h"

namespace dqn {
namespace {

constexpr int WG = 256;  // 4 waves

// ---------------------------------------------------------------------------
// Forward.  GEMM view per sample: M = output pixels (oh*ow), N = cout,
// K = cin*k*k.  A workgroup takes one sample and a run of 16-pixel M-tiles;
// it stages the input rows those pixels read into LDS (all channels) and each
// wave computes whole M-tiles across all N-tiles.  Contraction order: lane
// group g = lane/16 takes channel 4*cb + g; MFMA steps walk (cb, ky, kx), so a
// lane reads k consecutive input columns per (c, ky).
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
__global__ __launch_bounds__(WG) void conv_fwd_kernel(
    const void* __restrict__ in_a, const void* __restrict__ in_b, int n_a,
    const float* __restrict__ w_a, const float* __restrict__ bias_a,
    const float* __restrict__ w_b, const float* __restrict__ bias_b,
    float* __restrict__ out, int mt_per_wg, float in_scale) {
    constexpr int P = OH * OW;
    constexpr int MT = (P + 15) / 16;
    constexpr int NT = COUT / 16;
    constexpr int CB = CIN / 4;
    constexpr int ESZ = U8 ? 1 : 4;
    extern __shared__ __align__(16) unsigned char smem[];

    const int groups = (MT + mt_per_wg - 1) / mt_per_wg;
    const int n = blockIdx.x / groups;
    const int grp = blockIdx.x - n * groups;
    const int mt0 = grp * mt_per_wg;
    const int mt1 = min(MT, mt0 + mt_per_wg);
    const int p0 = mt0 * 16;
    const int p1 = min(P, mt1 * 16);
    const int oy0 = p0 / OW;
    const int oy1 = (p1 - 1) / OW;
    const int iy0 = oy0 * S;
    const int rows = (oy1 - oy0) * S + K;

    const bool second = n >= n_a;
    const int ns = second ? n - n_a : n;
    const unsigned char* src = (const unsigned char*)(second ? in_b : in_a) +
                               (size_t)ns * CIN * IH * IW * ESZ;
    const float* W = second ? w_b : w_a;
    const float* bias = second ? bias_b : bias_a;

    // Stage rows [iy0, iy0+rows) of every channel, as 32-bit words.
    {
        const int words_per_ch = rows * IW * ESZ / 4;
        const int total = CIN * words_per_ch;
        const uint32_t* s32 = (const uint32_t*)src;
        uint32_t* d32 = (uint32_t*)smem;
        for (int e = threadIdx.x; e < total; e += WG) {
            int c = e / words_per_ch;
            int r = e - c * words_per_ch;
            d32[e] = s32[(c * IH * IW + iy0 * IW) * ESZ / 4 + r];
        }
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

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
                    const unsigned char* base = smem + (c * rows + row) * IW + S * ox;
#pragma unroll
                    for (int q = 0; q < K / 4; ++q) {
                        uint32_t wv = *(const uint32_t*)(base + 4 * q);
                        a[4 * q + 0] = (float)(wv & 0xffu) * amask;
                        a[4 * q + 1] = (float)((wv >> 8) & 0xffu) * amask;
                        a[4 * q + 2] = (float)((wv >> 16) & 0xffu) * amask;
                        a[4 * q + 3] = (float)(wv >> 24) * amask;
                    }
                } else {
                    const float* base = (const float*)smem + (c * rows + row) * IW + S * ox;
#pragma unroll
                    for (int kx = 0; kx < K; ++kx) a[kx] = base[kx] * amask;
                }
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const float* wp = W + (((t * 16 + li) * CIN + c) * K + ky) * K;
                    float b[K];
#pragma unroll
                    for (int kx = 0; kx < K; ++kx) b[kx] = __ldg(wp + kx);
#pragma unroll
                    for (int kx = 0; kx < K; ++kx) acc[t] = mfma16x16x4(a[kx], b[kx], acc[t]);
                }
            }
        }
        // Epilogue: lane holds pixels mt*16 + 4g + r of channel t*16 + li.
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int o = t * 16 + li;
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

// ---------------------------------------------------------------------------
// Weight gradient.  GEMM view: M = cout, N = cin*k*k (the W layout), the
// contraction runs over every output pixel of every sample.  A workgroup owns
// a chunk of samples and 4*NTW N-tiles; per sample it stages the input and
// dz into LDS and accumulates in registers.  Partial sums per chunk are
// written without atomics and reduced later in a fixed order.
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8, int NTW>
__global__ __launch_bounds__(WG) void conv_wgrad_kernel(
    const void* __restrict__ in, const float* __restrict__ dz, int batch, int spc,
    float* __restrict__ wpart, float* __restrict__ bpart, float in_scale) {
    constexpr int P = OH * OW;
    constexpr int PP = (P + 3) / 4 * 4;
    constexpr int NCOL = CIN * K * K;
    constexpr int NTT = NCOL / 16;
    constexpr int GROUPS = NTT / (4 * NTW);
    constexpr int MT = COUT / 16;
    constexpr int ESZ = U8 ? 1 : 4;
    constexpr int IN_BYTES = CIN * IH * IW * ESZ;
    constexpr int IN_BYTES_PAD = (IN_BYTES + 15) / 16 * 16;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* s_in = smem;
    float* s_dz = (float*)(smem + IN_BYTES_PAD);       // [COUT][PP]
    int* s_pix = (int*)(s_dz + COUT * PP);              // [PP]

    const int chunk = blockIdx.x / GROUPS;
    const int grp = blockIdx.x - chunk * GROUPS;
    const int j0 = chunk * spc;
    const int j1 = min(batch, j0 + spc);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    for (int p = threadIdx.x; p < PP; p += WG) {
        int oy = p / OW, ox = p - (p / OW) * OW;
        s_pix[p] = p < P ? (S * oy * IW + S * ox) : 0;
    }
    int koff[NTW];
#pragma unroll
    for (int u = 0; u < NTW; ++u) {
        const int col = (grp * 4 * NTW + wave + 4 * u) * 16 + li;
        const int c = col / (K * K);
        const int ky = (col / K) % K;
        const int kx = col % K;
        koff[u] = c * IH * IW + ky * IW + kx;
    }

    f4 acc[MT][NTW];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int u = 0; u < NTW; ++u) acc[m][u] = f4{0.f, 0.f, 0.f, 0.f};
    float bacc = 0.f;

    for (int j = j0; j < j1; ++j) {
        __syncthreads();
        {
            const uint32_t* s32 = (const uint32_t*)((const unsigned char*)in + (size_t)j * IN_BYTES);
            uint32_t* d32 = (uint32_t*)s_in;
            for (int e = threadIdx.x; e < IN_BYTES / 4; e += WG) d32[e] = s32[e];
            const float* dzj = dz + (size_t)j * COUT * P;
            for (int e = threadIdx.x; e < COUT * PP; e += WG) {
                int o = e / PP, p = e - (e / PP) * PP;
                s_dz[e] = p < P ? dzj[o * P + p] : 0.f;
            }
        }
        __syncthreads();
        if (grp == 0 && threadIdx.x < COUT) {
            const float* row = s_dz + threadIdx.x * PP;
            float s = 0.f;
            for (int p = 0; p < P; ++p) s += row[p];
            bacc += s;
        }
        for (int st = 0; st < PP / 4; ++st) {
            const int p = st * 4 + g;
            const int po = s_pix[p];
            float a[MT], b[NTW];
#pragma unroll
            for (int m = 0; m < MT; ++m) a[m] = s_dz[(m * 16 + li) * PP + p];
#pragma unroll
            for (int u = 0; u < NTW; ++u) {
                if constexpr (U8) b[u] = (float)s_in[koff[u] + po];
                else b[u] = ((const float*)s_in)[koff[u] + po];
            }
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int u = 0; u < NTW; ++u) acc[m][u] = mfma16x16x4(a[m], b[u], acc[m][u]);
        }
    }
    // D[4g + r][li] of tile (m, u): o = m*16 + 4g + r, col = tile col + li.
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int u = 0; u < NTW; ++u) {
            const int col = (grp * 4 * NTW + wave + 4 * u) * 16 + li;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int o = m * 16 + 4 * g + r;
                wpart[((size_t)chunk * COUT + o) * NCOL + col] = acc[m][u][r] * in_scale;
            }
        }
    if (grp == 0 && threadIdx.x < COUT) bpart[(size_t)chunk * COUT + threadIdx.x] = bacc;
}

// ---------------------------------------------------------------------------
// Input gradient (transposed convolution), split into stride phases so no
// MFMA multiplies a structural zero: input pixel (S*qy + py, S*qx + px)
// receives W[o][c][py + S*ty][px + S*tx] * dz[o][qy - ty][qx - tx] for taps
// ty, tx < K/S.  GEMM view per (sample, phase): M = phase pixels, N = cin,
// contraction over (o, ty, tx).  dz is staged in LDS with a zero border.
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
__global__ __launch_bounds__(WG) void conv_dgrad_kernel(
    const float* __restrict__ dz, const float* __restrict__ W, const float* __restrict__ h_in,
    float* __restrict__ din) {
    static_assert(K % S == 0, "phase decomposition needs k divisible by stride");
    constexpr int T = K / S;
    constexpr int QHM = (IH + S - 1) / S;
    constexpr int QWM = (IW + S - 1) / S;
    constexpr int PH = QHM + T - 1;
    constexpr int PW = QWM + T - 1;
    constexpr int NT = CIN / 16;
    constexpr int OB = COUT / 4;
    __shared__ float s_dz[COUT * PH * PW];

    const int n = blockIdx.x / (S * S);
    const int ph = blockIdx.x - n * (S * S);
    const int py = ph / S, px = ph - (ph / S) * S;
    const int QH = (IH - py + S - 1) / S;
    const int QW = (IW - px + S - 1) / S;
    const int QP = QH * QW;
    const int MTq = (QP + 15) / 16;

    const float* dzn = dz + (size_t)n * COUT * OH * OW;
    for (int e = threadIdx.x; e < COUT * PH * PW; e += WG) {
        int o = e / (PH * PW);
        int r = e - o * (PH * PW);
        int yy = r / PW, xx = r - (r / PW) * PW;
        int y = yy - (T - 1), x = xx - (T - 1);
        s_dz[e] = (y >= 0 && y < OH && x >= 0 && x < OW) ? dzn[(o * OH + y) * OW + x] : 0.f;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    for (int mt = wave; mt < MTq; mt += 4) {
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
                    const int ky = py + S * ty, kx = px + S * tx;
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const float b = __ldg(W + (((size_t)o * CIN + t * 16 + li) * K + ky) * K + kx);
                        acc[t] = mfma16x16x4(a, b, acc[t]);
                    }
                }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int c = t * 16 + li;
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

// ---------------------------------------------------------------------------

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
hipError_t fwd_launch(const void* in_a, const void* in_b, int n_a, int n, const float* w_a,
                      const float* b_a, const float* w_b, const float* b_b, float* out,
                      float in_scale, hipStream_t st) {
    constexpr int P = OH * OW;
    constexpr int MT = (P + 15) / 16;
    constexpr int ESZ = U8 ? 1 : 4;
    // Small batches: one M-tile per wave for parallelism; large batches: a
    // longer run of tiles per workgroup to amortise the input staging.
    int mt_per_wg = ((long)n * MT >= 4L * 4096) ? MT : 4;
    if (mt_per_wg > MT) mt_per_wg = MT;
    const int groups = (MT + mt_per_wg - 1) / mt_per_wg;
    int max_rows = 0;
    for (int gi = 0; gi < groups; ++gi) {
        int p0 = gi * mt_per_wg * 16;
        int p1 = std::min(P, (gi + 1) * mt_per_wg * 16);
        int rows = ((p1 - 1) / OW - p0 / OW) * S + K;
        max_rows = std::max(max_rows, rows);
    }
    size_t lds = (size_t)CIN * max_rows * IW * ESZ;
    lds = (lds + 15) / 16 * 16;
    auto kern = conv_fwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8>;
    if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds) != hipSuccess)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_fwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8>),
                       dim3((unsigned)(n * groups)), dim3(WG), lds, st, in_a, in_b, n_a, w_a, b_a,
                       w_b, b_b, out, mt_per_wg, in_scale);
    return hipGetLastError();
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
constexpr int wgrad_groups() {
    return (CIN * K * K / 16) / 4;  // NTW = 1
}

int target_chunks(int batch, int groups) {
    int c = (1024 + groups - 1) / groups;
    if (c > batch) c = batch;
    if (c < 1) c = 1;
    // chunk = ceil(batch / c) samples; recompute the chunk count from it
    int spc = (batch + c - 1) / c;
    return (batch + spc - 1) / spc;
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
hipError_t wgrad_launch(const void* in, const float* dz, int batch, float* wpart, float* bpart,
                        float in_scale, hipStream_t st) {
    constexpr int GROUPS = wgrad_groups<CIN, IH, IW, COUT, K, S, OH, OW>();
    constexpr int P = OH * OW;
    constexpr int PP = (P + 3) / 4 * 4;
    constexpr int ESZ = U8 ? 1 : 4;
    constexpr int IN_BYTES_PAD = (CIN * IH * IW * ESZ + 15) / 16 * 16;
    const int chunks = target_chunks(batch, GROUPS);
    const int spc = (batch + chunks - 1) / chunks;
    size_t lds = IN_BYTES_PAD + (size_t)COUT * PP * 4 + PP * 4;
    auto kern = conv_wgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8, 1>;
    if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds) != hipSuccess)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL((conv_wgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW, U8, 1>),
                       dim3((unsigned)(chunks * GROUPS)), dim3(WG), lds, st, in, dz, batch, spc,
                       wpart, bpart, in_scale);
    return hipGetLastError();
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
hipError_t dgrad_launch(const float* dz, const float* w, const float* h_in, float* din, int batch,
                        hipStream_t st) {
    hipLaunchKernelGGL((conv_dgrad_kernel<CIN, IH, IW, COUT, K, S, OH, OW>),
                       dim3((unsigned)(batch * S * S)), dim3(WG), 0, st, dz, w, h_in, din);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_fwd(ConvId id, const void* in_a, const void* in_b, int n_a, int n,
                           const float* w_a, const float* b_a, const float* w_b, const float* b_b,
                           float* out, float in_scale, hipStream_t st) {
    switch (id) {
        case CONV_S1: return fwd_launch<4, 84, 84, 16, 8, 4, 20, 20, true>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, st);
        case CONV_S2: return fwd_launch<16, 20, 20, 32, 4, 2, 9, 9, false>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, st);
        case CONV_L1: return fwd_launch<4, 84, 84, 32, 8, 4, 20, 20, true>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, st);
        case CONV_L2: return fwd_launch<32, 20, 20, 64, 4, 2, 9, 9, false>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, st);
        case CONV_L3: return fwd_launch<64, 9, 9, 64, 3, 1, 7, 7, false>(in_a, in_b, n_a, n, w_a, b_a, w_b, b_b, out, in_scale, st);
        default: return hipErrorInvalidValue;
    }
}

int conv_wgrad_chunks(ConvId id, int batch) {
    switch (id) {
        case CONV_S1: return target_chunks(batch, wgrad_groups<4, 84, 84, 16, 8, 4, 20, 20>());
        case CONV_S2: return target_chunks(batch, wgrad_groups<16, 20, 20, 32, 4, 2, 9, 9>());
        case CONV_L1: return target_chunks(batch, wgrad_groups<4, 84, 84, 32, 8, 4, 20, 20>());
        case CONV_L2: return target_chunks(batch, wgrad_groups<32, 20, 20, 64, 4, 2, 9, 9>());
        case CONV_L3: return target_chunks(batch, wgrad_groups<64, 9, 9, 64, 3, 1, 7, 7>());
        default: return -1;
    }
}

hipError_t launch_conv_wgrad(ConvId id, const void* in, const float* dz, int batch, float* wpart,
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
        case CONV_S2: return dgrad_launch<16, 20, 20, 32, 4, 2, 9, 9>(dz, w, h_in, din, batch, st);
        case CONV_L2: return dgrad_launch<32, 20, 20, 64, 4, 2, 9, 9>(dz, w, h_in, din, batch, st);
        case CONV_L3: return dgrad_launch<64, 9, 9, 64, 3, 1, 7, 7>(dz, w, h_in, din, batch, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn
