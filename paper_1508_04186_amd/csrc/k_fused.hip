// The two convolution layers of the small Q-network (Sec. III.A: 16 filters
// 8x8 stride 4 on the 4x84x84 byte input, then 32 filters 4x4 stride 2, each
// with ReLU) in one launch, for small batches where the layers are latency
// bound.  A workgroup owns one sample and a band of three conv2 output rows:
// it stages the 36 input rows the band needs, both layers' weights and
// biases (all loads in flight together), computes the 8 conv1 rows the band
// reads into LDS, writes the conv1 rows it owns, then computes its conv2
// rows.  Bands overlap by two conv1 rows, which are computed twice and
// written once.
//
// conv1 runs on bf16 MFMA (v_mfma_f32_16x16x32_bf16) without loss of fp32
// accuracy: the input bytes are exact in bf16, each fp32 weight w is split
// exactly into three bf16 terms w = hi + mid + lo (8 significand bits each),
// and each byte x term product is exact in fp32, so the three MFMAs per
// k-step accumulate the same products an fp32 contraction would, in fp32.
// conv2 runs on fp32 MFMA with the contraction order of the per-layer kernel.
//
// The backward counterpart runs, in one launch, the conv2 weight gradient
// (the per-layer body) and, per (sample, band of conv1 rows), the conv2 input
// gradient for those rows with conv1's ReLU mask applied, kept in LDS, and
// the conv1 weight and bias partial sums over those rows (bands of 4 conv1
// rows here: the backward per row is heavier than the forward's).
#include <initializer_list>

#include "conv_body.h"

namespace dqn {
namespace {


// Small-network geometry.
constexpr int C0 = 4, H0 = 84;                   // input channels, side
constexpr int C1 = 16, K1 = 8, S1 = 4, H1 = 20;  // conv1
constexpr int C2 = 32, K2 = 4, S2 = 2, H2 = 9;   // conv2
constexpr int R2 = 3;                            // conv2 rows per band
constexpr int NBAND = H2 / R2;
constexpr int R1 = (R2 - 1) * S2 + K2;           // conv1 rows per band (8)
constexpr int R0 = (R1 - 1) * S1 + K1;           // input rows per band (36)
constexpr int KW1 = C0 * K1 * K1;                // conv1 contraction length (256)
constexpr int RS1 = KW1 + 8;                     // bf16 row stride of a split conv1 weight row
constexpr int A1C = R1 * H1 + 16;                // float stride between conv1 channels in LDS
constexpr int KK2 = K2 * K2;
constexpr int RC2 = 16;                          // conv2 weight LDS layout: [o][c][ky*kx]
constexpr int RO2 = (C1 * RC2 / 64) * 64 + 65;  // = 1 mod 64: conflict-free B reads
static_assert(H2 % R2 == 0, "bands must tile the conv2 rows");
static_assert(R1 * H1 % 16 == 0, "conv1 band must be whole M-tiles");

// LDS carve (bytes).
constexpr int OFF_IN = 0;                                  // bf16 [C0][R0][H0]
constexpr int OFF_W1 = OFF_IN + C0 * R0 * H0 * 2;          // bf16 [3][C1][RS1]
constexpr int OFF_A1 = OFF_W1 + 3 * C1 * RS1 * 2;          // f32 [C1][A1C]
constexpr int OFF_W2 = OFF_A1 + C1 * A1C * 4;              // f32 [C2][RO2]
constexpr int OFF_B = OFF_W2 + C2 * RO2 * 4;               // f32 b1[C1], b2[C2]
constexpr int LDS_BYTES = OFF_B + (C1 + C2) * 4;
static_assert(OFF_W1 % 16 == 0 && OFF_A1 % 16 == 0 && OFF_W2 % 16 == 0 && OFF_B % 16 == 0, "alignment");


struct FusedFwdParams {
    ConvIn in_a, in_b;
    int n_a, n;
    const float *w1_a, *b1_a, *w2_a, *b2_a;  // samples < n_a
    const float *w1_b, *b1_b, *w2_b, *b2_b;  // samples >= n_a
    float* act1;                             // [n][C1][H1][H1]
    float* act2;                             // [n][C2][H2][H2]
    SideFields side;
};

__global__ __launch_bounds__(WG) void conv_s12_fwd_kernel(FusedFwdParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    __bf16* s_in = (__bf16*)(smem + OFF_IN);
    __bf16* s_w1 = (__bf16*)(smem + OFF_W1);
    float* s_a1 = (float*)(smem + OFF_A1);
    float* s_w2 = (float*)(smem + OFF_W2);
    float* s_b = (float*)(smem + OFF_B);

    const int band = blockIdx.x % NBAND;
    const int n = blockIdx.x / NBAND;
    const bool second = n >= p.n_a;
    const unsigned char* src = sample_ptr(second ? p.in_b : p.in_a, second ? n - p.n_a : n);
    const float* w1 = second ? p.w1_b : p.w1_a;
    const float* w2 = second ? p.w2_b : p.w2_a;
    const float* b1 = second ? p.b1_b : p.b1_a;
    const float* b2 = second ? p.b2_b : p.b2_a;
    const int t = threadIdx.x;

    // side fields of the transitions (block 0), in stages around the work
    const bool side_on = p.side.idx && blockIdx.x == 0;
    SideCopy side;
    side.begin(p.side, side_on, t);

    // ---- staging: every global load of the workgroup is issued before the
    // first LDS store.  Input rows [band*R2*S2*S1, +R0) of each channel are
    // contiguous (R0*H0 bytes, 16-byte aligned); weights are contiguous.
    constexpr int IN_V = C0 * R0 * H0 / 16;    // 16-byte units of input
    constexpr int IN_PER = (IN_V + WG - 1) / WG;
    constexpr int W1_V = C1 * KW1 / 4;
    constexpr int W1_PER = W1_V / WG;
    constexpr int W2_V = C2 * C1 * KK2 / 4;
    constexpr int W2_PER = W2_V / WG;
    static_assert((C0 * R0 * H0) % 16 == 0 && (R0 * H0) % 16 == 0, "input rows must be whole 16-byte units");
    static_assert(W1_V % WG == 0 && W2_V % WG == 0, "weights must split evenly over the workgroup");
    const int iy0 = band * R2 * S2 * S1;
    f4 vin[IN_PER], vw1[W1_PER], vw2[W2_PER];
#pragma unroll
    for (int u = 0; u < IN_PER; ++u) {
        const int e = t + u * WG;
        if (e < IN_V) {
            const int c = e / (R0 * H0 / 16), r = e - c * (R0 * H0 / 16);
            vin[u] = *(const f4*)(src + (size_t)c * H0 * H0 + (size_t)iy0 * H0 + 16 * r);
        }
    }
#pragma unroll
    for (int u = 0; u < W1_PER; ++u) vw1[u] = ((const f4*)w1)[t + u * WG];
#pragma unroll
    for (int u = 0; u < W2_PER; ++u) vw2[u] = ((const f4*)w2)[t + u * WG];
    float bias = 0.f;
    if (t < C1) bias = b1[t];
    else if (t < C1 + C2) bias = b2[t - C1];

    // input bytes -> bf16 (exact), same [c][row][x] order
#pragma unroll
    for (int u = 0; u < IN_PER; ++u) {
        const int e = t + u * WG;
        if (e < IN_V) {
            union { f4 v; unsigned char b[16]; } q;
            q.v = vin[u];
            bf16x8 lo8, hi8;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                lo8[i] = (__bf16)(float)q.b[i];
                hi8[i] = (__bf16)(float)q.b[8 + i];
            }
            *(bf16x8*)(s_in + 16 * e) = lo8;
            *(bf16x8*)(s_in + 16 * e + 8) = hi8;
        }
    }
    // conv1 weights -> three bf16 planes [part][o][k]
#pragma unroll
    for (int u = 0; u < W1_PER; ++u) {
        const int e = t + u * WG;
        const int o = (4 * e) / KW1, k = (4 * e) % KW1;
        bf16x4 h, m, l;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            __bf16 hi, mid, lo;
            split3(vw1[u][i], hi, mid, lo);
            h[i] = hi;
            m[i] = mid;
            l[i] = lo;
        }
        *(bf16x4*)(s_w1 + (0 * C1 + o) * RS1 + k) = h;
        *(bf16x4*)(s_w1 + (1 * C1 + o) * RS1 + k) = m;
        *(bf16x4*)(s_w1 + (2 * C1 + o) * RS1 + k) = l;
    }
    // conv2 weights -> padded [o][c][ky*kx]
#pragma unroll
    for (int u = 0; u < W2_PER; ++u) {
        const int e = t + u * WG;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int f = 4 * e + i;
            const int o = f / (C1 * KK2), r = f - o * (C1 * KK2);
            const int c = r / KK2, k = r - c * KK2;
            s_w2[o * RO2 + c * RC2 + k] = vw2[u][i];
        }
    }
    if (t < C1 + C2) s_b[t] = bias;
    __syncthreads();
    side.fetch(p.side, side_on, t);   // in flight during conv1 (a barrier waits for loads)

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;

    // ---- conv1: band-local pixels 16*mt + li (row = p / H1, x = p % H1),
    // contraction k = c*64 + ky*8 + kx; k-step kb covers c = kb/2 and
    // ky = 4*(kb%2) + g, kx = 0..7 in lane group g.  Wave w owns M-tiles
    // w, w+4, w+8 (below MT1) and runs them together, so their accumulator
    // chains are independent and share the B operands.
    const int y1 = band * R2 * S2;             // first conv1 row of the band
    const int own0 = band == 0 ? 0 : y1 + (K2 - S2);
    const int own1 = band == NBAND - 1 ? H1 : y1 + R2 * S2 + (K2 - S2);
    constexpr int MT1 = R1 * H1 / 16;
    constexpr int TPW = (MT1 + 3) / 4;         // M-tiles per wave, at most
    float* a1g = p.act1 + (size_t)n * C1 * H1 * H1;
    {
        // Every wave runs TPW tiles; a wave with fewer repeats its last one
        // and discards the copy, so the loop has no per-tile branches.
        const int ntile = (MT1 - wave + 3) / 4;  // this wave's tiles (uniform)
        int abase[TPW];
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const int mt = wave + 4 * min(i, ntile - 1);
            const int pa = mt * 16 + li;
            const int ra = pa / H1, xa = pa - ra * H1;
            abase[i] = S1 * ra * H0 + S1 * xa;
        }
        f4 acc[TPW];
#pragma unroll
        for (int i = 0; i < TPW; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        // operands of k-step kb; the next step's are loaded before this
        // step's MFMAs issue
        auto load_a = [&](int kb, bf16x8 (&a)[TPW]) {
            const int c = kb >> 1, ky = (kb & 1) * 4 + g;
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                const __bf16* ap = s_in + (c * R0 + ky) * H0 + abase[i];
                const bf16x4 a0 = *(const bf16x4*)ap;
                const bf16x4 a1 = *(const bf16x4*)(ap + 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[i][q] = a0[q];
                    a[i][4 + q] = a1[q];
                }
            }
        };
        auto load_b = [&](int kb, bf16x8 (&b)[3]) {
#pragma unroll
            for (int part = 0; part < 3; ++part)
                b[part] = *(const bf16x8*)(s_w1 + (part * C1 + li) * RS1 + kb * 32 + 8 * g);
        };
        bf16x8 a[2][TPW], b[2][3];
        load_a(0, a[0]);
        load_b(0, b[0]);
#pragma unroll
        for (int kb = 0; kb < KW1 / 32; ++kb) {
            const int cur = kb & 1;
            if (kb + 1 < KW1 / 32) {
                load_a(kb + 1, a[cur ^ 1]);
                load_b(kb + 1, b[cur ^ 1]);
            }
#pragma unroll
            for (int part = 0; part < 3; ++part)
#pragma unroll
                for (int i = 0; i < TPW; ++i) acc[i] = mfma16x16x32bf16(a[cur][i], b[cur][part], acc[i]);
        }
        // lane holds pixels 16*mt + 4g + r (one row: H1 is a multiple of 4)
        // of channel o = li
        const float bo = s_b[li];
        constexpr float inv255 = (float)(1.0 / 255.0);
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            if (i < ntile) {
                const int pb = (wave + 4 * i) * 16 + 4 * g;
                const int rb = pb / H1, xb = pb - rb * H1;
                f4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[i][r] * inv255 + bo, 0.f);
                *(f4*)(s_a1 + li * A1C + rb * H1 + xb) = v;
                const int yg = y1 + rb;
                if (yg >= own0 && yg < own1) *(f4*)(a1g + ((size_t)li * H1 + yg) * H1 + xb) = v;
            }
        }
    }
    __syncthreads();

    // ---- conv2: wave w takes input channels 4w..4w+3 (lane group g takes
    // channel 4w + g) for both M-tiles (band-local pixels) and both N-tiles,
    // four independent accumulators; steps walk (ky, kx).  The four waves'
    // partial sums are then added in wave order through LDS (the input tile
    // is no longer needed).
    {
        constexpr int P2 = R2 * H2;
        constexpr int MT2 = (P2 + 15) / 16, NT2 = C2 / 16;
        static_assert(C1 / 4 == 4, "one channel block per wave");
        static_assert(MT2 * NT2 * 4 * 64 * 4 * 4 <= C0 * R0 * H0 * 2, "partials must fit the input tile");
        int arow[MT2];
        float amask[MT2];
#pragma unroll
        for (int m = 0; m < MT2; ++m) {
            const int pp = m * 16 + li;
            const int pc = pp < P2 ? pp : P2 - 1;
            const int oy = pc / H2, ox = pc - (pc / H2) * H2;
            arow[m] = S2 * oy * H1 + S2 * ox;
            amask[m] = pp < P2 ? 1.f : 0.f;
        }
        const int c = wave * 4 + g;
        f4 acc[MT2][NT2];
#pragma unroll
        for (int m = 0; m < MT2; ++m)
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) acc[m][nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ky = 0; ky < K2; ++ky) {
#pragma unroll
            for (int kx = 0; kx < K2; ++kx) {
                float a[MT2], b[NT2];
#pragma unroll
                for (int m = 0; m < MT2; ++m) a[m] = s_a1[c * A1C + arow[m] + ky * H1 + kx] * amask[m];
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) b[nt] = s_w2[(nt * 16 + li) * RO2 + c * RC2 + ky * K2 + kx];
#pragma unroll
                for (int m = 0; m < MT2; ++m)
#pragma unroll
                    for (int nt = 0; nt < NT2; ++nt) acc[m][nt] = mfma16x16x4(a[m], b[nt], acc[m][nt]);
            }
        }
        f4* part = (f4*)(smem + OFF_IN);  // [wave][m][nt][lane]
#pragma unroll
        for (int m = 0; m < MT2; ++m)
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) part[((wave * MT2 + m) * NT2 + nt) * 64 + lane] = acc[m][nt];
        __syncthreads();
        // thread t finishes (m, nt) tile t / 64 for lane t % 64
        {
            const int tile = t >> 6, ln = t & 63;
            const int m = tile / NT2, nt = tile - m * NT2;
            f4 sum = part[((0 * MT2 + m) * NT2 + nt) * 64 + ln];
#pragma unroll
            for (int w = 1; w < 4; ++w) sum += part[((w * MT2 + m) * NT2 + nt) * 64 + ln];
            const int o = nt * 16 + (ln & 15);
            const float bo = s_b[C1 + o];
            float* a2 = p.act2 + ((size_t)n * C2 + o) * H2 * H2 + band * R2 * H2;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int q = m * 16 + 4 * (ln >> 4) + r;
                if (q < P2) a2[q] = fmaxf(sum[r] + bo, 0.f);
            }
        }
        static_assert(MT2 * NT2 * 64 == WG, "one thread per output lane of the band");
    }
    side.end(p.side, side_on, t, WG);
}

// ---------------------------------------------------------------------------
// Backward: bands of NRMAX conv1 rows (a partition of the 20 rows; even row
// counts and band starts keep every stride phase aligned to the band).
constexpr int NRMAX = 4;                 // conv1 rows per backward band
constexpr int NBB = H1 / NRMAX;          // backward bands per sample
static_assert(H1 % NRMAX == 0 && NRMAX % 2 == 0, "backward bands must tile the conv1 rows in pairs");
constexpr int T2 = K2 / S2;              // taps per stride phase and axis (2)
constexpr int NZR = NRMAX / 2 + 1;       // staged conv2-gradient rows
constexpr int NZC = H2 + 2;              // staged conv2-gradient columns (zero border)
constexpr int RCW = C1 + 1;              // row stride of the [tap][o][c] conv2 weight slice
constexpr int LD1 = NRMAX * H1 + 4;      // row stride of the conv1 gradient tile (= 36 mod 64)
constexpr int RIN = (NRMAX - 1) * S1 + K1;  // staged input rows per channel

constexpr int BOFF_DZ = 0;                                  // f32 [C2][NZR][NZC]
constexpr int BOFF_W = BOFF_DZ + C2 * NZR * NZC * 4;        // f32 [KK2][C2][RCW]
constexpr int BOFF_MASK = BOFF_W + KK2 * C2 * RCW * 4;      // f32 [C1][NRMAX*H1]
constexpr int BOFF_D1 = BOFF_MASK + C1 * NRMAX * H1 * 4;    // f32 [C1][LD1]
constexpr int BOFF_IN = BOFF_D1 + C1 * LD1 * 4;             // u8 [C0][RIN][H0]
constexpr int B_LDS = BOFF_IN + C0 * RIN * H0;
static_assert(BOFF_MASK % 16 == 0 && BOFF_IN % 16 == 0, "alignment");

struct S1BwdParams {
    ConvIn in;            // network input of the B samples (bytes)
    const float* dz2;     // gradient at conv2's pre-activation [B][C2][H2][H2]
    const float* w2;      // conv2 weights [C2][C1][K2][K2]
    const float* act1;    // conv1 output [B][C1][H1][H1] (its ReLU mask)
    float* wpart1;        // conv1 weight partial sums [B*NBB][C1][KW1]
    float* bpart1;        // conv1 bias partial sums [B*NBB][C1]
    float in_scale;
};

// One (sample j, band) of the conv1 side of the backward pass.
__device__ __forceinline__ void s1_bwd_body(const S1BwdParams& p, int bid, unsigned char* smem) {
    float* s_dz = (float*)(smem + BOFF_DZ);
    float* s_w = (float*)(smem + BOFF_W);
    float* s_mask = (float*)(smem + BOFF_MASK);
    float* s_d1 = (float*)(smem + BOFF_D1);
    unsigned char* s_in = smem + BOFF_IN;

    const int band = bid % NBB;
    const int j = bid / NBB;
    const int y0 = band * NRMAX, y1 = y0 + NRMAX;
    const int nr = NRMAX;                    // owned rows
    const int npx = nr * H1;
    const int oyb = y0 / 2 - 1;              // conv2-gradient row of staged row 0
    const int t = threadIdx.x;

    // ---- staging, all loads in flight before the first LDS store
    constexpr int NDZ = C2 * NZR * NZC;
    constexpr int UDZ = (NDZ + WG - 1) / WG;
    constexpr int W2V = C2 * C1 * KK2 / 4;
    constexpr int UW = W2V / WG;
    constexpr int MV = C1 * NRMAX * H1 / 4;  // 16-byte units of the mask rows, at most
    constexpr int UM = (MV + WG - 1) / WG;
    constexpr int IV = C0 * RIN * H0 / 16;   // 16-byte units of the input rows, at most
    constexpr int UI = (IV + WG - 1) / WG;
    static_assert(W2V % WG == 0, "conv2 weights must split evenly");
    const float* dzj = p.dz2 + (size_t)j * C2 * H2 * H2;
    float vdz[UDZ];
#pragma unroll
    for (int u = 0; u < UDZ; ++u) {
        const int e = t + u * WG;
        const int o = e / (NZR * NZC), r = e - o * (NZR * NZC);
        const int oy = oyb + r / NZC, ox = r % NZC - 1;
        vdz[u] = (e < NDZ && oy >= 0 && oy < H2 && ox >= 0 && ox < H2) ? dzj[(o * H2 + oy) * H2 + ox] : 0.f;
    }
    f4 vw[UW];
#pragma unroll
    for (int u = 0; u < UW; ++u) vw[u] = ((const f4*)p.w2)[t + u * WG];
    const int mv = C1 * nr * H1 / 4;
    const float* a1j = p.act1 + (size_t)j * C1 * H1 * H1 + y0 * H1;
    f4 vm[UM];
#pragma unroll
    for (int u = 0; u < UM; ++u) {
        const int e = t + u * WG;
        if (e < mv) {
            const int c = e / (nr * H1 / 4), r = e - c * (nr * H1 / 4);
            vm[u] = *(const f4*)(a1j + (size_t)c * H1 * H1 + 4 * r);
        }
    }
    const int rin = (nr - 1) * S1 + K1;      // input rows for the owned conv1 rows
    const int iv = C0 * rin * H0 / 16;
    const unsigned char* src = sample_ptr(p.in, j) + (size_t)S1 * y0 * H0;
    f4 vi[UI];
#pragma unroll
    for (int u = 0; u < UI; ++u) {
        const int e = t + u * WG;
        if (e < iv) {
            const int c = e / (rin * H0 / 16), r = e - c * (rin * H0 / 16);
            vi[u] = *(const f4*)(src + (size_t)c * H0 * H0 + 16 * r);
        }
    }
#pragma unroll
    for (int u = 0; u < UDZ; ++u) {
        const int e = t + u * WG;
        if (e < NDZ) s_dz[e] = vdz[u];
    }
#pragma unroll
    for (int u = 0; u < UW; ++u) {
        const int e = t + u * WG;  // W2[o][c][ky][kx..kx+3], kx = 0
        const int o = e / (C1 * K2), r = e - o * (C1 * K2);
        const int c = r / K2, ky = r - c * K2;
#pragma unroll
        for (int kx = 0; kx < K2; ++kx) s_w[((ky * K2 + kx) * C2 + o) * RCW + c] = vw[u][kx];
    }
#pragma unroll
    for (int u = 0; u < UM; ++u) {
        const int e = t + u * WG;
        if (e < mv) {
            const int c = e / (nr * H1 / 4), r = e - c * (nr * H1 / 4);
            *(f4*)(s_mask + c * NRMAX * H1 + 4 * r) = vm[u];
        }
    }
#pragma unroll
    for (int u = 0; u < UI; ++u) {
        const int e = t + u * WG;
        if (e < iv) {
            const int c = e / (rin * H0 / 16), r = e - c * (rin * H0 / 16);
            *(f4*)(s_in + c * RIN * H0 + 16 * r) = vi[u];
        }
    }
    __syncthreads();

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;

    // ---- conv1 input gradient by stride phase (py, px): owned pixels
    // (y0 + py + 2*qr, px + 2*qc) receive W2[o][c][py+2ty][px+2tx] *
    // dz2[o][y/2 - ty][qc - tx]; contraction over (o, ty, tx), lane group g
    // taking o = 4*ob + g.  M = phase pixels, N = the 16 conv1 channels.
    // Tiles (phase, M-tile) tt = wave + 4i are run together by wave `wave`,
    // so their accumulator chains are independent.
    {
        constexpr int NRP = NRMAX / 2;
        constexpr int PP = NRP * (H1 / 2);      // pixels per phase
        constexpr int MTP = (PP + 15) / 16;
        constexpr int TW = MTP;                 // tiles per wave (4 phases x MTP / 4 waves)
        int zoff[TW], py[TW], px[TW];
        float amask[TW];
#pragma unroll
        for (int i = 0; i < TW; ++i) {
            const int tt = wave + 4 * i;
            const int ph = tt / MTP, mt = tt - ph * MTP;
            py[i] = ph >> 1;
            px[i] = ph & 1;
            const int q = mt * 16 + li;
            const int qv = q < PP ? q : PP - 1;
            const int qr = qv / (H1 / 2), qc = qv - qr * (H1 / 2);
            zoff[i] = (qr + 1) * NZC + qc + 1;
            amask[i] = q < PP ? 1.f : 0.f;
        }
        f4 acc[TW];
#pragma unroll
        for (int i = 0; i < TW; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        // Per (tile, tap) base addresses, fixed for the loop: inside it, the
        // output-channel step ob only adds compile-time offsets (the LDS
        // reads' immediate offsets).
        constexpr int NTAP = T2 * T2;
        int zb[TW][NTAP], wb[TW][NTAP];
#pragma unroll
        for (int i = 0; i < TW; ++i)
#pragma unroll
            for (int ty = 0; ty < T2; ++ty)
#pragma unroll
                for (int tx = 0; tx < T2; ++tx) {
                    const int tap = (py[i] + S2 * ty) * K2 + px[i] + S2 * tx;
                    zb[i][ty * T2 + tx] = g * NZR * NZC + zoff[i] - ty * NZC - tx;
                    wb[i][ty * T2 + tx] = (tap * C2 + g) * RCW + li;
                }
        // Double-buffered operands; the scheduling barriers keep the next
        // step's LDS reads ahead of this step's MFMAs (one wave per SIMD
        // has nothing else to hide LDS latency with).
        float a[2][TW][NTAP], b[2][TW][NTAP];
        auto load = [&](int ob, float (&av)[TW][NTAP], float (&bv)[TW][NTAP]) {
#pragma unroll
            for (int i = 0; i < TW; ++i)
#pragma unroll
                for (int k = 0; k < NTAP; ++k) {
                    av[i][k] = s_dz[zb[i][k] + ob * 4 * NZR * NZC];
                    bv[i][k] = s_w[wb[i][k] + ob * 4 * RCW];
                }
        };
        load(0, a[0], b[0]);
#pragma unroll
        for (int ob = 0; ob < C2 / 4; ++ob) {
            const int cur = ob & 1;
            if (ob + 1 < C2 / 4) load(ob + 1, a[cur ^ 1], b[cur ^ 1]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int k = 0; k < NTAP; ++k)
#pragma unroll
                for (int i = 0; i < TW; ++i) acc[i] = mfma16x16x4(a[cur][i][k] * amask[i], b[cur][i][k], acc[i]);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int i = 0; i < TW; ++i) {
            const int tt = wave + 4 * i;
            const int mt = tt - (tt / MTP) * MTP;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int qq = mt * 16 + 4 * g + r;
                if (qq < PP) {
                    const int lp = (py[i] + 2 * (qq / (H1 / 2))) * H1 + px[i] + 2 * (qq % (H1 / 2));
                    s_d1[li * LD1 + lp] = s_mask[li * NRMAX * H1 + lp] > 0.f ? acc[i][r] : 0.f;
                }
            }
        }
        static_assert(4 * MTP % 4 == 0, "phase tiles split evenly over the waves");
    }
    __syncthreads();

    // ---- conv1 weight gradient over the owned pixels: M = 16 output
    // channels, N = 256 weight columns (c, ky, kx), contraction over pixels
    // (lane group g takes pixel 4*st + g).  Wave w owns N-tiles w + 4i.
    const int slot = j * NBB + band;
    {
        constexpr int NTW = KW1 / 16 / 4;      // N-tiles per wave
        int koff[NTW];
#pragma unroll
        for (int i = 0; i < NTW; ++i) {
            const int col = (wave + 4 * i) * 16 + li;
            const int c = col / (K1 * K1), ky = (col / K1) % K1, kx = col % K1;
            koff[i] = c * RIN * H0 + ky * H0 + kx;
        }
        f4 acc[NTW];
#pragma unroll
        for (int i = 0; i < NTW; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
        // Pixel step st covers band pixels 4*st .. 4*st+3 (one per lane
        // group g), all in conv1 row (4*st)/H1 since H1 is a multiple of 4:
        // the addresses are a per-lane base plus compile-time offsets.
        constexpr int NST = NRMAX * H1 / 4;
        static_assert(H1 % 4 == 0, "a pixel step stays in one row");
        const int abase = li * LD1 + g;
        int bbase[NTW];
#pragma unroll
        for (int i = 0; i < NTW; ++i) bbase[i] = koff[i] + S1 * g;
#pragma unroll
        for (int st = 0; st < NST; ++st) {
            const int y = (4 * st) / H1, x0 = (4 * st) % H1;
            const float a = s_d1[abase + 4 * st];
            float b[NTW];
#pragma unroll
            for (int i = 0; i < NTW; ++i) b[i] = (float)s_in[bbase[i] + S1 * y * H0 + S1 * x0];
#pragma unroll
            for (int i = 0; i < NTW; ++i) acc[i] = mfma16x16x4(a, b[i], acc[i]);
        }
#pragma unroll
        for (int i = 0; i < NTW; ++i) {
            const int col = (wave + 4 * i) * 16 + li;
#pragma unroll
            for (int r = 0; r < 4; ++r)
                p.wpart1[((size_t)slot * C1 + 4 * g + r) * KW1 + col] = acc[i][r] * p.in_scale;
        }
    }
    if (t < C1) {
        const float* row = s_d1 + t * LD1;
        float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
        for (int q = 0; q < npx; q += 4) {
            s0 += row[q];
            s1 += row[q + 1];
            s2 += row[q + 2];
            s3 += row[q + 3];
        }
        p.bpart1[(size_t)slot * C1 + t] = (s0 + s1) + (s2 + s3);
    }
}

// Blocks [0, n_b) run the conv1 side (the longer per-block work, so it is
// dispatched first), the rest conv2's weight gradient.
__global__ __launch_bounds__(WG) void conv_s12_bwd_kernel(WgradParams w, S1BwdParams b, int n_b) {
    extern __shared__ __align__(16) unsigned char smem[];
    if ((int)blockIdx.x < n_b)
        s1_bwd_body(b, blockIdx.x, smem);
    else
        conv_wgrad_body<C1, H1, H1, C2, K2, S2, H2, H2, false>(w, blockIdx.x - n_b, smem);
}

}  // namespace

bool conv_s12_fwd_supported(ConvId c1, ConvId c2) { return c1 == CONV_S1 && c2 == CONV_S2; }

bool conv_s12_fwd_aligned(const ConvIn& in) {
    return ((uintptr_t)in.base & 15) == 0 && (in.stride & 15) == 0;
}

hipError_t launch_conv_s12_fwd(const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                               const float* w1_a, const float* b1_a, const float* w2_a,
                               const float* b2_a, const float* w1_b, const float* b1_b,
                               const float* w2_b, const float* b2_b, float* act1, float* act2,
                               const SideFields* side, hipStream_t st) {
    if (n <= 0 || !conv_s12_fwd_aligned(in_a) || !conv_s12_fwd_aligned(in_b)) return hipErrorInvalidValue;
    for (const float* w : {w1_a, w2_a, w1_b, w2_b})
        if (((uintptr_t)w & 15) != 0) return hipErrorInvalidValue;
    auto kern = conv_s12_fwd_kernel;
    if (!allow_lds((const void*)kern, LDS_BYTES)) return hipErrorInvalidValue;
    FusedFwdParams p{in_a, in_b, n_a, n, w1_a, b1_a, w2_a, b2_a, w1_b, b1_b, w2_b, b2_b,
                     act1, act2, side ? *side : SideFields{}};
    hipLaunchKernelGGL(kern, dim3((unsigned)(n * NBAND)), dim3(WG), LDS_BYTES, st, p);
    return hipGetLastError();
}

int conv_s12_bwd_slots(int batch) { return batch * NBB; }

hipError_t launch_conv_s12_bwd(const ConvIn& in, const float* act1, const float* dz2, const float* w2,
                               int batch, float* wpart2, float* bpart2, float* wpart1, float* bpart1,
                               hipStream_t st) {
    if (batch <= 0 || !conv_s12_fwd_aligned(in) || ((uintptr_t)w2 & 15) != 0 || ((uintptr_t)act1 & 15) != 0)
        return hipErrorInvalidValue;
    int n_w;
    size_t lw;
    const ConvIn in2{act1, nullptr, (int64_t)C1 * H1 * H1 * 4, 0};
    const WgradParams wp = wgrad_params<C1, H1, H1, C2, K2, S2, H2, H2, false>(in2, dz2, batch, wpart2, bpart2,
                                                                               1.f, &n_w, &lw);
    const S1BwdParams bp{in, dz2, w2, act1, wpart1, bpart1, (float)(1.0 / 255.0)};
    const size_t lds = std::max(lw, (size_t)B_LDS);
    auto kern = conv_s12_bwd_kernel;
    if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, dim3((unsigned)(n_w + batch * NBB)), dim3(WG), lds, st, wp, bp, batch * NBB);
    return hipGetLastError();
}

}  // namespace dqn

// ---------------------------------------------------------------------------
// conv1 forward on byte input (4 channels 84x84, 8x8 stride 4 -> 20x20) for
// many samples: a workgroup splits its weights into three bf16 planes once
// (exact, as above; PARTS = 3), or rounds them to one bf16 plane (the
// bf16-input variant; PARTS = 1), then walks its samples with the next
// sample's bytes loaded into registers while the current one is computed.
// Each sample is staged in LDS already converted to bfloat16 (exact for
// bytes), once per byte, so an A operand (eight consecutive bytes of one
// input row) is two 8-byte LDS reads; converting in the MFMA loop had
// converted every byte four times (the 8x8 windows at stride 4 overlap) and
// left the loop bound by that VALU work.  Eight waves, one workgroup per
// compute unit; M-tile (16 pixels) m goes to wave m mod 8, and each wave runs
// its M-tiles for every N-tile as independent accumulator chains.
namespace dqn {
namespace {

constexpr int U8F_WG = 512;

struct U8FwdParams {
    ConvIn in_a, in_b;
    int n_a, n, spb, blocks_a;   // samples per workgroup; workgroups of set a
    const float *w_a, *b_a, *w_b, *b_b;
    float* out;                  // [n][COUT][20][20], bfloat16 values when out16
    SideFields side;
};

constexpr size_t u8f_lds(int cout, int parts) {
    return (size_t)C0 * H0 * H0 * 2 + (size_t)parts * cout * RS1 * 2 + (size_t)cout * 4;
}

template <int COUT, int PARTS, bool OUT16>
__global__ __launch_bounds__(U8F_WG) void conv1_u8_fwd_kernel(U8FwdParams p) {
    constexpr int REC = C0 * H0 * H0;            // bytes per sample (28,224)
    constexpr int RV = REC / 16;                 // 16-byte units (1,764)
    constexpr int RPER = (RV + U8F_WG - 1) / U8F_WG;   // per thread (4)
    constexpr int NT = COUT / 16;
    constexpr int MT = H1 * H1 / 16;             // 25 M-tiles per sample
    constexpr int NW = U8F_WG / 64;              // waves (8)
    constexpr int MPW = (MT + NW - 1) / NW;      // M-tiles per wave, at most (4)
    constexpr int PL = COUT * RS1;               // bf16 per weight plane
    static_assert(REC % 16 == 0 && (H1 * H1) % 16 == 0 && (H0 * 2) % 8 == 0, "whole tiles, 8-byte rows");
    extern __shared__ __align__(16) unsigned char smem[];
    __bf16* s_in = (__bf16*)smem;                // bf16 [REC]
    __bf16* s_w = s_in + REC;                    // bf16 [PARTS][COUT][RS1]
    float* s_b = (float*)(s_w + PARTS * PL);
    static_assert(PARTS == 1 || PARTS == 3, "exact split or bf16 rounding");

    const bool second = (int)blockIdx.x >= p.blocks_a;
    const int blk = second ? (int)blockIdx.x - p.blocks_a : (int)blockIdx.x;
    const int j0 = (second ? p.n_a : 0) + blk * p.spb;
    const int j1 = min(second ? p.n : p.n_a, j0 + p.spb);
    const float* W = second ? p.w_b : p.w_a;
    const float* bias = second ? p.b_b : p.b_a;
    const int t = threadIdx.x;

    // side fields of the transitions (block 0, which always has samples),
    // in stages around the work
    const bool side_on = p.side.idx && blockIdx.x == 0;
    SideCopy side;
    side.begin(p.side, side_on, t);
    if (j0 >= j1) {  // uniform
        side.fetch(p.side, side_on, t);
        side.end(p.side, side_on, t, U8F_WG);
        return;
    }

    auto sample_src = [&](int j) -> const f4* {
        return (const f4*)(j < p.n_a ? sample_ptr(p.in_a, j) : sample_ptr(p.in_b, j - p.n_a));
    };
    uint4 vin[RPER];
    auto load_in = [&](int j) {
        const uint4* src = (const uint4*)sample_src(j);
#pragma unroll
        for (int u = 0; u < RPER; ++u) {
            const int e = t + u * U8F_WG;
            if (e < RV) vin[u] = src[e];
        }
    };
    // sixteen bytes -> sixteen bf16 (the upper halves of the exact floats)
    auto store_in = [&]() {
#pragma unroll
        for (int u = 0; u < RPER; ++u) {
            const int e = t + u * U8F_WG;
            if (e < RV) {
                const uint32_t w[4] = {vin[u].x, vin[u].y, vin[u].z, vin[u].w};
                uint32_t h[8];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t f0 = __builtin_bit_cast(uint32_t, (float)(w[q] & 0xffu));
                    const uint32_t f1 = __builtin_bit_cast(uint32_t, (float)((w[q] >> 8) & 0xffu));
                    const uint32_t f2 = __builtin_bit_cast(uint32_t, (float)((w[q] >> 16) & 0xffu));
                    const uint32_t f3 = __builtin_bit_cast(uint32_t, (float)(w[q] >> 24));
                    h[2 * q] = __builtin_amdgcn_perm(f1, f0, 0x07060302u);
                    h[2 * q + 1] = __builtin_amdgcn_perm(f3, f2, 0x07060302u);
                }
                uint4* d = (uint4*)(s_in + 16 * e);
                d[0] = uint4{h[0], h[1], h[2], h[3]};
                d[1] = uint4{h[4], h[5], h[6], h[7]};
            }
        }
    };

    // weights -> PARTS bf16 planes [part][o][k] (exact split, or rounding); bias
    load_in(j0);
    for (int e = t; e < COUT * KW1 / 4; e += U8F_WG) {
        const f4 w = ((const f4*)W)[e];
        const int o = (4 * e) / KW1, k = (4 * e) % KW1;
        bf16x4 h, m, l;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            __bf16 hi, mid, lo;
            split3(w[i], hi, mid, lo);
            h[i] = hi;
            m[i] = mid;
            l[i] = lo;
        }
        *(bf16x4*)(s_w + 0 * PL + o * RS1 + k) = h;
        if constexpr (PARTS == 3) {
            *(bf16x4*)(s_w + 1 * PL + o * RS1 + k) = m;
            *(bf16x4*)(s_w + 2 * PL + o * RS1 + k) = l;
        }
    }
    if (t < COUT) s_b[t] = bias[t];
    side.fetch(p.side, side_on, t);   // in flight during the first sample

    const int lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;
    const int ntile = (MT - wave + NW - 1) / NW;  // this wave's M-tiles (uniform)
    int abase[MPW];
#pragma unroll
    for (int i = 0; i < MPW; ++i) {
        const int mt = wave + NW * min(i, ntile - 1);
        const int pa = mt * 16 + li;
        const int ra = pa / H1, xa = pa - ra * H1;
        abase[i] = S1 * ra * H0 + S1 * xa;
    }
    constexpr float inv255 = (float)(1.0 / 255.0);

    for (int j = j0; j < j1; ++j) {
        store_in();
        __syncthreads();
        if (j + 1 < j1) load_in(j + 1);          // in flight during this sample
        f4 acc[MPW][NT];
#pragma unroll
        for (int i = 0; i < MPW; ++i)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[i][nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KW1 / 32; ++kb) {
            const int c = kb >> 1, ky = (kb & 1) * 4 + g;
            bf16x8 b[NT][PARTS];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int part = 0; part < PARTS; ++part)
                    b[nt][part] = *(const bf16x8*)(s_w + part * PL + (nt * 16 + li) * RS1 + kb * 32 + 8 * g);
#pragma unroll
            for (int i = 0; i < MPW; ++i) {
                if (i < ntile) {
                    // bytes (c, 4 ra + ky, 4 xa .. 4 xa + 7) as bf16: two 8-byte reads
                    const __bf16* ap = s_in + (c * H0 + ky) * H0 + abase[i];
                    const uint2 lo = *(const uint2*)ap, hi = *(const uint2*)(ap + 4);
                    const bf16x8 a = __builtin_bit_cast(bf16x8, uint4{lo.x, lo.y, hi.x, hi.y});
#pragma unroll
                    for (int part = 0; part < PARTS; ++part)
#pragma unroll
                        for (int nt = 0; nt < NT; ++nt) acc[i][nt] = mfma16x16x32bf16(a, b[nt][part], acc[i][nt]);
                }
            }
        }
        // lane holds pixels 16*mt + 4g + r of channel nt*16 + li
        float* oj = p.out + (size_t)j * COUT * H1 * H1;
#pragma unroll
        for (int i = 0; i < MPW; ++i) {
            if (i < ntile) {
                const int pb = (wave + NW * i) * 16 + 4 * g;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    const int o = nt * 16 + li;
                    const float bo = s_b[o];
                    f4 v;
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[i][nt][r] * inv255 + bo, 0.f);
                    if constexpr (OUT16) {
                        bf16x4 h;
#pragma unroll
                        for (int r = 0; r < 4; ++r) h[r] = (__bf16)v[r];
                        *(bf16x4*)((__bf16*)p.out + ((size_t)j * COUT + o) * H1 * H1 + pb) = h;
                    } else {
                        *(f4*)(oj + (size_t)o * H1 * H1 + pb) = v;
                    }
                }
            }
        }
        __syncthreads();  // all reads of s_in done before the next sample is stored
    }
    side.end(p.side, side_on, t, U8F_WG);
}

}  // namespace

bool conv1_u8_fwd_supported(ConvId id) { return id == CONV_L1 || id == CONV_S1; }

hipError_t launch_conv1_u8_fwd(ConvId id, const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                               const float* w_a, const float* b_a, const float* w_b, const float* b_b,
                               float* out, const SideFields* side, bool bf16, bool out16, hipStream_t st) {
    if (n <= 0 || n_a < 0 || n_a > n || !conv_s12_fwd_aligned(in_a) || !conv_s12_fwd_aligned(in_b) ||
        ((uintptr_t)w_a & 15) || ((uintptr_t)w_b & 15) || ((uintptr_t)out & 15) || (out16 && !bf16))
        return hipErrorInvalidValue;
    // about 256 workgroups (one per compute unit): a run of samples each, so
    // the weight split is amortized
    const int spb = std::max(1, (n + 255) / 256);
    const int blocks_a = (n_a + spb - 1) / spb, blocks_b = (n - n_a + spb - 1) / spb;
    U8FwdParams prm{in_a, in_b, n_a, n, spb, blocks_a, w_a, b_a, w_b, b_b, out, side ? *side : SideFields{}};
    const dim3 grid((unsigned)std::max(1, blocks_a + blocks_b));
    auto go = [&](auto kern, int cout, int parts) -> hipError_t {
        const size_t lds = u8f_lds(cout, parts);
        if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, grid, dim3(U8F_WG), lds, st, prm);
        return hipGetLastError();
    };
    if (id == CONV_L1) {
        if (out16) return go(conv1_u8_fwd_kernel<32, 1, true>, 32, 1);
        return bf16 ? go(conv1_u8_fwd_kernel<32, 1, false>, 32, 1) : go(conv1_u8_fwd_kernel<32, 3, false>, 32, 3);
    }
    if (id == CONV_S1 && !out16)
        return bf16 ? go(conv1_u8_fwd_kernel<16, 1, false>, 16, 1) : go(conv1_u8_fwd_kernel<16, 3, false>, 16, 3);
    return hipErrorInvalidValue;
}

}  // namespace dqn

// ---------------------------------------------------------------------------
// conv1 weight/bias gradient on byte input for many samples:
//   dW[o][c][ky][kx] = (1/255) sum over samples and pixels (y, x) of
//                      dz[o][y][x] * byte[c][4y + ky][4x + kx],  db[o] = sum dz.
// One workgroup of eight waves per compute unit owns all COUT x 256 outputs
// for a run of samples (one partial-sum slot).  The contraction over pixels
// runs on v_mfma_f32_16x16x32_bf16: the bytes are exact in bfloat16, and dz
// is split exactly into three bfloat16 planes (hi + mid + lo; PARTS = 3), so
// the three products per step are those of the float32 dz; the bf16-input
// variant rounds dz to one plane (PARTS = 1).  Per sample, dz is staged as
// the planes [part][o][pixel] and the bytes as phases
// [c][row][kx][i] = byte[c][row][4i + kx] (i < 20), so that four pixels
// (y, x..x+3) of one row are 8 contiguous bytes of a plane and one 4-byte
// word of a phase row.  Lane group g of k-step st takes pixels 32 st + 8 g + e
// (e < 8), two groups of four within rows; pixels 400..415 of the last step
// are zero in the planes.  Wave w owns N-tiles (weight columns) 2w, 2w+1 and
// every M-tile (output channel block); the next sample's dz and bytes are
// read into registers during the current sample's MFMAs.  With one dz plane
// (the bf16-input variant) the phases are staged already converted to
// bfloat16 (two bytes an entry, 105 KB), so a B operand is two 8-byte reads;
// with three the LDS holds only the bytes, converted as they are read.  The
// pixel-group offsets of a lane are formed once, and each k-step's operands
// are read while the previous step multiplies.
namespace dqn {
namespace {

constexpr int UW_WG = 512;                      // eight waves
constexpr int UW_TARGET_BLOCKS = 256;           // one workgroup per compute unit
constexpr int UW_P = H1 * H1;                   // 400 pixels
constexpr int UW_LDZ = 424;                     // bf16 plane row stride (848 B: 16-byte reads conflict-free)
constexpr int UW_STEPS = (UW_P + 31) / 32;      // 13 k-steps of 32 pixels
constexpr int UW_PHROW = 8 * H1;                // phase bytes per (channel, row): 8 kx x 20
constexpr int UW_PH = C0 * H0 * UW_PHROW;       // 53,760 bytes
constexpr int UW_ITEMS = C0 * H0 * 5;           // (channel, row, 16-byte column block) items
constexpr int UW_IPER = (UW_ITEMS + UW_WG - 1) / UW_WG;
static_assert(32 * UW_STEPS <= UW_LDZ && UW_P % 4 == 0 && H1 % 4 == 0, "pixel groups of four within rows");

// (phase entries of two bytes with one plane: bfloat16)
constexpr size_t uw_lds(int cout, int parts) { return (size_t)parts * cout * UW_LDZ * 2 + (size_t)UW_PH * (parts == 1 ? 2 : 1); }

struct U8WgradParams {
    ConvIn in;            // network input (bytes)
    const float* dz;      // [n][COUT][20][20] (bfloat16 values with DZ16)
    int n, spb;
    float* wpart;         // [blocks][COUT][256]
    float* bpart;         // [blocks][COUT]
    float in_scale;
};

// DZ16: dz arrives rounded to bfloat16 (bf16-input variant) and is staged as
// it is; the bias partial sums then come from dz's producer.
template <int COUT, int PARTS, bool DZ16 = false>
__global__ __launch_bounds__(UW_WG) void conv1_u8_wgrad_kernel(U8WgradParams p) {
    constexpr int MT = COUT / 16;
    constexpr int RPW = COUT / 8;                      // dz rows staged per wave
    constexpr int CPR = UW_P / 4;                      // four-value chunks per dz row (100)
    static_assert(PARTS == 1 || PARTS == 3, "exact split or bf16 rounding");
    static_assert(!DZ16 || PARTS == 1, "bfloat16 dz is one plane");
    static_assert(KW1 == 16 * 16 && COUT % 16 == 0, "16 N-tiles of weight columns, 2 per wave");
    constexpr bool PH16 = PARTS == 1;      // phases staged as bfloat16
    constexpr int PHB = PH16 ? 2 : 1;      // bytes per phase entry
    extern __shared__ __align__(16) unsigned char smem[];
    __bf16* s_dz = (__bf16*)smem;                                   // [PARTS][COUT][UW_LDZ]
    unsigned char* s_ph = smem + (size_t)PARTS * COUT * UW_LDZ * 2;  // [C0][H0][8][20]

    const int j0 = blockIdx.x * p.spb, j1 = min(p.n, j0 + p.spb);
    if (j0 >= j1) return;  // whole workgroup
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int li = lane & 15, g = lane >> 4;

    // pixels 400 .. UW_LDZ-1 of every plane row stay zero
    for (int e = t; e < PARTS * COUT * (UW_LDZ - UW_P); e += UW_WG) {
        const int row = e / (UW_LDZ - UW_P), q = e - row * (UW_LDZ - UW_P);
        s_dz[row * UW_LDZ + UW_P + q] = (__bf16)0.f;
    }

    // next sample in registers: dz rows wave*RPW .. +RPW-1 (chunks lane, lane + 64),
    // and the 20-byte column blocks of the phase items
    std::conditional_t<DZ16, uint2, f4> vdz[RPW][2];
    uint32_t vb[UW_IPER][5];
    auto load = [&](int j) {
        const size_t dzj = (size_t)j * COUT * UW_P;
#pragma unroll
        for (int q = 0; q < RPW; ++q)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int ch = lane + 64 * h;
                const size_t off = dzj + (wave * RPW + q) * UW_P + 4 * ch;
                if constexpr (DZ16) {
                    if (ch < CPR) vdz[q][h] = *(const uint2*)((const __bf16*)p.dz + off);
                } else {
                    if (ch < CPR) vdz[q][h] = *(const f4*)(p.dz + off);
                }
            }
        const unsigned char* src = sample_ptr(p.in, j);
#pragma unroll
        for (int u = 0; u < UW_IPER; ++u) {
            const int it = t + u * UW_WG;
            if (it < UW_ITEMS) {
                const int row = it / 5, qb = it - row * 5;   // row = c * H0 + r
                const uint32_t* w = (const uint32_t*)(src + row * H0 + 16 * qb);
#pragma unroll
                for (int d = 0; d < 5; ++d) vb[u][d] = w[d];
            }
        }
    };
    // bias sum of row wave * RPW + halving_index<RPW>(lane) (where that is >= 0):
    // the RPW rows' wave sums by halving, in each value's wave_sum order
    float bs = 0.f;
    auto stage = [&]() {
        float parts[RPW];
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int o = wave * RPW + q;
            float& part = parts[q];
            part = 0.f;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int ch = lane + 64 * h;
                if constexpr (DZ16) {
                    if (ch < CPR) *(uint2*)(s_dz + o * UW_LDZ + 4 * ch) = vdz[q][h];
                    continue;
                } else if (ch < CPR) {
                    const f4 v = vdz[q][h];
                    part += (v[0] + v[1]) + (v[2] + v[3]);
                    bf16x4 hv, mv, lv;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        __bf16 hi, mid, lo;
                        split3(v[i], hi, mid, lo);
                        hv[i] = hi;
                        mv[i] = mid;
                        lv[i] = lo;
                    }
                    *(bf16x4*)(s_dz + (0 * COUT + o) * UW_LDZ + 4 * ch) = hv;
                    if constexpr (PARTS == 3) {
                        *(bf16x4*)(s_dz + (1 * COUT + o) * UW_LDZ + 4 * ch) = mv;
                        *(bf16x4*)(s_dz + (2 * COUT + o) * UW_LDZ + 4 * ch) = lv;
                    }
                }
            }
        }
        if constexpr (!DZ16) bs += halving_step<RPW, 32>(parts, lane);
        // phase word (row, kx, block qb) = bytes 16 qb + 4e + kx, e < 4, of the row
#pragma unroll
        for (int u = 0; u < UW_IPER; ++u) {
            const int it = t + u * UW_WG;
            if (it < UW_ITEMS) {
                const int row = it / 5, qb = it - row * 5;
#pragma unroll
                for (int kx = 0; kx < 8; ++kx) {
                    const int m = kx & 3, d = kx >> 2;
                    const uint32_t sel = (uint32_t)m | ((uint32_t)(4 + m) << 8) | 0x0c0c0000u;
                    const uint32_t lo2 = __builtin_amdgcn_perm(vb[u][d + 1], vb[u][d], sel);
                    const uint32_t hi2 = __builtin_amdgcn_perm(vb[u][d + 3], vb[u][d + 2], sel);
                    const uint32_t w = __builtin_amdgcn_perm(hi2, lo2, 0x05040100u);
                    if constexpr (PH16) {   // the four bytes as bfloat16 (exact)
                        bf16x4 h;
#pragma unroll
                        for (int e = 0; e < 4; ++e) h[e] = (__bf16)(float)((w >> (8 * e)) & 0xffu);
                        *(bf16x4*)(s_ph + ((row * 8 + kx) * H1 + 4 * qb) * 2) = h;
                    } else {
                        *(uint32_t*)(s_ph + (row * 8 + kx) * H1 + 4 * qb) = w;
                    }
                }
            }
        }
    };

    // weight column (c, ky, kx) of this lane in each of its two N-tiles (byte offsets)
    int cb[2];
#pragma unroll
    for (int n = 0; n < 2; ++n) {
        const int col = (2 * wave + n) * 16 + li;
        const int c = col / (K1 * K1), ky = (col / K1) % K1, kx = col % K1;
        cb[n] = ((c * H0 + ky) * 8 + kx) * H1 * PHB;
    }
    // phase byte offsets of the lane's pixel groups 32 st + 8 g + 4 h (pixels
    // past 400 read row 0: their dz is zero)
    int po[UW_STEPS][2];
#pragma unroll
    for (int st = 0; st < UW_STEPS; ++st)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int pp = 32 * st + 8 * g + 4 * h;
            const int y = pp < UW_P ? pp / H1 : 0, x = pp < UW_P ? pp - (pp / H1) * H1 : 0;
            po[st][h] = (S1 * y * 8 * H1 + x) * PHB;
        }
    f4 acc[MT][2];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int n = 0; n < 2; ++n) acc[m][n] = f4{0.f, 0.f, 0.f, 0.f};

    // operands of k-step st into buffer slot
    bf16x8 bb[2][2], aa[2][MT][PARTS];
    auto operands = [&](int st, int slot) {
#pragma unroll
        for (int n = 0; n < 2; ++n) {
            if constexpr (PH16) {
                const uint2 w0 = *(const uint2*)(s_ph + cb[n] + po[st][0]);
                const uint2 w1 = *(const uint2*)(s_ph + cb[n] + po[st][1]);
                bb[slot][n] = __builtin_bit_cast(bf16x8, uint4{w0.x, w0.y, w1.x, w1.y});
            } else {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const uint32_t w = *(const uint32_t*)(s_ph + cb[n] + po[st][h]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) bb[slot][n][4 * h + e] = (__bf16)(float)((w >> (8 * e)) & 0xffu);
                }
            }
        }
        const int p0 = 32 * st + 8 * g;
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int part = 0; part < PARTS; ++part)
                aa[slot][m][part] = *(const bf16x8*)(s_dz + (part * COUT + m * 16 + li) * UW_LDZ + p0);
    };

    load(j0);
    for (int j = j0; j < j1; ++j) {
        __syncthreads();  // the previous sample's reads are done
        stage();
        __syncthreads();
        if (j + 1 < j1) load(j + 1);
        operands(0, 0);
#pragma unroll
        for (int st = 0; st < UW_STEPS; ++st) {
            if (st + 1 < UW_STEPS) operands(st + 1, (st + 1) & 1);   // read while step st multiplies
            const int sl = st & 1;
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int part = 0; part < PARTS; ++part)
#pragma unroll
                    for (int n = 0; n < 2; ++n) acc[m][n] = mfma16x16x32bf16(aa[sl][m][part], bb[sl][n], acc[m][n]);
        }
    }
    // D[4g + r][li] of tile (m, n): channel m*16 + 4g + r, column (2 wave + n)*16 + li
    float* wp = p.wpart + (size_t)blockIdx.x * COUT * KW1;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                wp[(size_t)(m * 16 + 4 * g + r) * KW1 + (2 * wave + n) * 16 + li] = acc[m][n][r] * p.in_scale;
    if constexpr (!DZ16) {
        const int bi = halving_index<RPW>(lane);
        if (bi >= 0) p.bpart[(size_t)blockIdx.x * COUT + wave * RPW + bi] = bs;
    }
}

}  // namespace

int conv1_u8_wgrad_slots(int n) {
    const int spb = std::max(1, (n + UW_TARGET_BLOCKS - 1) / UW_TARGET_BLOCKS);
    return (n + spb - 1) / spb;
}

hipError_t launch_conv1_u8_wgrad(ConvId id, const ConvIn& in, const float* dz, int n, float* wpart,
                                 float* bpart, float in_scale, bool bf16, hipStream_t st, bool dz16) {
    if (n <= 0 || !conv_s12_fwd_aligned(in) || in.off != 0 || ((uintptr_t)dz & 15)) return hipErrorInvalidValue;
    if (dz16 && (!bf16 || id != CONV_L1)) return hipErrorInvalidValue;
    const int spb = std::max(1, (n + UW_TARGET_BLOCKS - 1) / UW_TARGET_BLOCKS);
    const int blocks = (n + spb - 1) / spb;
    const U8WgradParams prm{in, dz, n, spb, wpart, bpart, in_scale};
    auto go = [&](auto kern, int cout, int parts) -> hipError_t {
        const size_t lds = uw_lds(cout, parts);
        if (!allow_lds((const void*)kern, lds)) return hipErrorInvalidValue;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(UW_WG), lds, st, prm);
        return hipGetLastError();
    };
    if (id == CONV_L1 && dz16) return go(conv1_u8_wgrad_kernel<32, 1, true>, 32, 1);
    if (id == CONV_L1) return bf16 ? go(conv1_u8_wgrad_kernel<32, 1>, 32, 1) : go(conv1_u8_wgrad_kernel<32, 3>, 32, 3);
    if (id == CONV_S1) return bf16 ? go(conv1_u8_wgrad_kernel<16, 1>, 16, 1) : go(conv1_u8_wgrad_kernel<16, 3>, 16, 3);
    return hipErrorInvalidValue;
}

}  // namespace dqn
