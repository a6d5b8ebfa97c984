// Convolution building blocks shared by the per-layer kernels and the fused
// small-network kernels: row staging into LDS, and the weight-gradient body
// with its host-side launch shape.  Everything here has internal linkage in
// each translation unit that includes it.
#pragma once

#include <algorithm>

#include "common.h"

namespace dqn {
namespace {

constexpr int WG = 256;  // 4 waves

// Stage CH rows of `bytes` bytes each from global (row c at src + c*sstride)
// into LDS (row c at dst + c*dstride).  16-byte accesses when every address
// is 16-byte aligned, else 4-byte; each thread issues up to U loads before
// its first LDS store, so the copies of all rows are in flight together.
template <int U = 16>
__device__ __forceinline__ void stage_rows(unsigned char* __restrict__ dst, int dstride,
                                           const unsigned char* __restrict__ src, int64_t sstride,
                                           int ch, int bytes) {
    const bool v16 = ((((uintptr_t)src | (uintptr_t)dst | (uintptr_t)sstride | (uintptr_t)dstride |
                        (uintptr_t)bytes) & 15) == 0);
    if (v16) {
        const int per = bytes / 16, n = ch * per;
        for (int base = threadIdx.x; base < n; base += U * WG) {
            f4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int i = base + u * WG;
                if (i < n) {
                    const int c = i / per, r = i - c * per;
                    v[u] = *(const f4*)(src + c * sstride + 16 * r);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int i = base + u * WG;
                if (i < n) {
                    const int c = i / per, r = i - c * per;
                    *(f4*)(dst + c * dstride + 16 * r) = v[u];
                }
            }
        }
    } else {
        const int per = bytes / 4, n = ch * per;
        for (int base = threadIdx.x; base < n; base += U * WG) {
            uint32_t v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int i = base + u * WG;
                if (i < n) {
                    const int c = i / per, r = i - c * per;
                    v[u] = *(const uint32_t*)(src + c * sstride + 4 * r);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int i = base + u * WG;
                if (i < n) {
                    const int c = i / per, r = i - c * per;
                    *(uint32_t*)(dst + c * dstride + 4 * r) = v[u];
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Weight gradient.  GEMM view: M = cout, N = cin*k*k (the W layout), the
// contraction runs over every output pixel of every sample.  A workgroup
// owns (a chunk of samples, a block of output rows, 4 N-tiles); per sample it
// stages the input rows and the dz rows of its block, then accumulates in
// registers.  Partial sums per (chunk, row block) are written without atomics
// and reduced later in a fixed order.
struct WgradParams {
    ConvIn in;
    const float* dz;
    int batch, spc, rows_per_blk, in_rows_max, pix_pad;
    float* wpart;
    float* bpart;
    float in_scale;
};

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
__device__ __forceinline__ void conv_wgrad_body(const WgradParams& p, int bid, unsigned char* smem) {
    const ConvIn& in = p.in;
    const float* __restrict__ dz = p.dz;
    const int batch = p.batch, spc = p.spc, rows_per_blk = p.rows_per_blk;
    const int in_rows_max = p.in_rows_max, pix_pad = p.pix_pad;
    float* __restrict__ wpart = p.wpart;
    float* __restrict__ bpart = p.bpart;
    const float in_scale = p.in_scale;
    constexpr int P = OH * OW;
    constexpr int NCOL = CIN * K * K;
    constexpr int NTT = NCOL / 16;
    constexpr int GROUPS = NTT / 4;
    constexpr int MT = COUT / 16;
    constexpr int ESZ = U8 ? 1 : 4;
    const int RB = (OH + rows_per_blk - 1) / rows_per_blk;
    const int in_bytes = ((CIN * in_rows_max * IW * ESZ + 15) / 16) * 16;
    unsigned char* s_in = smem;
    float* s_dz = (float*)(smem + in_bytes);          // [COUT][pix_pad]
    int* s_pix = (int*)(s_dz + COUT * pix_pad);       // [pix_pad]

    int b = bid;
    const int grp = b % GROUPS;
    b /= GROUPS;
    const int rb = b % RB;
    const int chunk = b / RB;
    const int j0 = chunk * spc;
    const int j1 = min(batch, j0 + spc);
    const int oy0 = rb * rows_per_blk;
    const int oy1 = min(OH, oy0 + rows_per_blk);      // exclusive
    const int pbeg = oy0 * OW;
    const int npix = (oy1 - oy0) * OW;
    const int iy0 = oy0 * S;
    const int rows = (oy1 - 1 - oy0) * S + K;
    const int row_elems = in_rows_max * IW;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;

    for (int q = threadIdx.x; q < pix_pad; q += WG) {
        const int p = pbeg + q;
        const int oy = p / OW, ox = p - (p / OW) * OW;
        s_pix[q] = q < npix ? (S * (oy - oy0) * IW + S * ox) : 0;
    }
    const int col = (grp * 4 + wave) * 16 + li;
    const int kc = col / (K * K);
    const int kyy = (col / K) % K;
    const int kxx = col % K;
    const int koff = kc * row_elems + kyy * IW + kxx;

    f4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = f4{0.f, 0.f, 0.f, 0.f};
    float bacc = 0.f;

    for (int j = j0; j < j1; ++j) {
        __syncthreads();
        {
            // The first U dz values per thread are loaded before the input
            // rows are staged, so both sets of loads are in flight together.
            const float* dzj = dz + (size_t)j * COUT * P + pbeg;
            constexpr int U = 8;
            auto dz_load = [&](int base, float (&v)[U]) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int e = base + u * WG;
                    const int o = e / pix_pad, q = e - o * pix_pad;
                    v[u] = (e < COUT * pix_pad && q < npix) ? dzj[(size_t)o * P + q] : 0.f;
                }
            };
            auto dz_store = [&](int base, const float (&v)[U]) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int e = base + u * WG;
                    if (e < COUT * pix_pad) s_dz[e] = v[u];
                }
            };
            float v0[U];
            dz_load(threadIdx.x, v0);
            const unsigned char* src = sample_ptr(in, j);
            stage_rows<8>(s_in, row_elems * ESZ, src + (size_t)iy0 * IW * ESZ, (int64_t)IH * IW * ESZ, CIN,
                          rows * IW * ESZ);
            dz_store(threadIdx.x, v0);
            for (int base = threadIdx.x + U * WG; base < COUT * pix_pad; base += U * WG) {
                float v[U];
                dz_load(base, v);
                dz_store(base, v);
            }
        }
        __syncthreads();
        if (grp == 0 && threadIdx.x < COUT) {
            const float* row = s_dz + threadIdx.x * pix_pad;
            float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
            for (int q = 0; q < pix_pad; q += 4) {
                s0 += row[q];
                s1 += row[q + 1];
                s2 += row[q + 2];
                s3 += row[q + 3];
            }
            bacc += (s0 + s1) + (s2 + s3);
        }
        for (int st = 0; st < pix_pad / 4; ++st) {
            const int q = st * 4 + g;
            float bv;
            if constexpr (U8) bv = (float)s_in[koff + s_pix[q]];
            else bv = ((const float*)s_in)[koff + s_pix[q]];
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = mfma16x16x4(s_dz[(m * 16 + li) * pix_pad + q], bv, acc[m]);
        }
    }
    // D[4g + r][li] of tile m: o = m*16 + 4g + r, weight column col.
    const int slot = chunk * RB + rb;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int o = m * 16 + 4 * g + r;
            wpart[((size_t)slot * COUT + o) * NCOL + col] = acc[m][r] * in_scale;
        }
    if (grp == 0 && threadIdx.x < COUT) bpart[(size_t)slot * COUT + threadIdx.x] = bacc;
}

// wgrad launch shape: (chunks, row blocks); partial slots = chunks * row blocks.
struct WgradShape {
    int chunks, spc, rows_per_blk, rb;
};

WgradShape wgrad_shape(int batch, int groups, int oh) {
    WgradShape w;
    // Row blocks only when the batch alone cannot fill the chip.
    int rb = 1;
    if ((long)batch * groups < 512) {
        rb = (int)std::min<long>(oh, (512 + (long)batch * groups - 1) / ((long)batch * groups));
    }
    w.rows_per_blk = (oh + rb - 1) / rb;
    w.rb = (oh + w.rows_per_blk - 1) / w.rows_per_blk;
    int c = (1024 + groups * w.rb - 1) / (groups * w.rb);
    c = std::max(1, std::min(c, batch));
    w.spc = (batch + c - 1) / c;
    w.chunks = (batch + w.spc - 1) / w.spc;
    return w;
}

template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW>
constexpr int wgrad_groups() {
    return (CIN * K * K / 16) / 4;
}

// Launch parameters of a layer's weight gradient for `batch` samples.
template <int CIN, int IH, int IW, int COUT, int K, int S, int OH, int OW, bool U8>
WgradParams wgrad_params(const ConvIn& in, const float* dz, int batch, float* wpart, float* bpart,
                         float in_scale, int* blocks, size_t* lds) {
    constexpr int GROUPS = wgrad_groups<CIN, IH, IW, COUT, K, S, OH, OW>();
    constexpr int ESZ = U8 ? 1 : 4;
    const WgradShape w = wgrad_shape(batch, GROUPS, OH);
    int in_rows_max = (w.rows_per_blk - 1) * S + K;
    while ((in_rows_max * IW * ESZ) % 16 != 0) ++in_rows_max;
    const int pix_pad = (w.rows_per_blk * OW + 3) / 4 * 4;
    const size_t in_bytes = ((size_t)CIN * in_rows_max * IW * ESZ + 15) / 16 * 16;
    *lds = in_bytes + (size_t)COUT * pix_pad * 4 + (size_t)pix_pad * 4;
    *blocks = w.chunks * w.rb * GROUPS;
    return WgradParams{in, dz, batch, w.spc, w.rows_per_blk, in_rows_max, pix_pad, wpart, bpart,
                       in_scale};
}

}  // namespace
}  // namespace dqn
