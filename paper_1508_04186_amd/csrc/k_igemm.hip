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
#include "common.h"

namespace dqn {
namespace {

constexpr int IG_WG = 256;
constexpr int IG_BM = 64, IG_BN = 64, IG_BK = 32;
constexpr int IG_LD = IG_BK + 4;  // = 4 mod 64 after the 64-row stride math below

struct IgemmFwdParams {
    const float* in;       // [n][cin][ih][iw]
    int n, n_a;
    int tiles_a;           // M-tiles of the first weight set
    const float *w_a, *b_a, *w_b, *b_b;
    float* out;            // [n][cout][oh][ow]
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
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
#pragma unroll
        for (int kk = 0; kk < IG_BK / 4; ++kk) {
            float a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = As[(wm + i * 16 + li) * IG_LD + kk * 4 + g];
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = Bs[(wn + j * 16 + li) * IG_LD + kk * 4 + g];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma16x16x4(a[i], b[j], acc[i][j]);
        }
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

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
hipError_t igemm_launch(const float* in, int n_a, int n, const float* w_a, const float* b_a,
                        const float* w_b, const float* b_b, float* out, hipStream_t st) {
    constexpr int P = OH * OW;
    if (((uintptr_t)w_a & 15) || ((uintptr_t)w_b & 15)) return hipErrorInvalidValue;
    const long tiles_a = ((long)n_a * P + IG_BM - 1) / IG_BM;
    const long tiles_b = ((long)(n - n_a) * P + IG_BM - 1) / IG_BM;
    const long blocks = (tiles_a + tiles_b) * (COUT / IG_BN);
    if (blocks <= 0 || blocks > 0x7fffffffL || (long)n * P > 0x7fffffffL) return hipErrorInvalidValue;
    IgemmFwdParams prm{in, n, n_a, (int)tiles_a, w_a, b_a, w_b, b_b, out};
    hipLaunchKernelGGL((conv_igemm_fwd_kernel<CIN, IH, IW, COUT, K, S, OH, OW>), dim3((unsigned)blocks),
                       dim3(IG_WG), 0, st, prm);
    return hipGetLastError();
}

}  // namespace

bool conv_igemm_fwd_supported(ConvId id) { return id == CONV_L2 || id == CONV_L3; }

hipError_t launch_conv_igemm_fwd(ConvId id, const float* in, int n_a, int n, const float* w_a,
                                 const float* b_a, const float* w_b, const float* b_b, float* out,
                                 hipStream_t st) {
    switch (id) {
        case CONV_L2: return igemm_launch<32, 20, 20, 64, 4, 2, 9, 9>(in, n_a, n, w_a, b_a, w_b, b_b, out, st);
        case CONV_L3: return igemm_launch<64, 9, 9, 64, 3, 1, 7, 7>(in, n_a, n, w_a, b_a, w_b, b_b, out, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace dqn
