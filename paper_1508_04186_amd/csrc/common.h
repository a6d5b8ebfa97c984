// Internal declarations shared by the translation units of libdqn.so.
// Target: gfx950 (CDNA4), wave64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dqn.h"

namespace dqn {

typedef float f4 __attribute__((ext_vector_type(4)));

// One v_mfma_f32_16x16x4_f32: D[16x16] += A[16x4] * B[4x16] over a wave.
// Lane l supplies A[l%16][l/16] and B[l/16][l%16]; it holds
// D[4*(l/16) + r][l%16] in element r of the accumulator.
__device__ __forceinline__ f4 mfma16x16x4(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// One v_mfma_f32_16x16x32_bf16: D[16x16] += A[16x32] * B[32x16] over a wave.
// Lane l supplies A[l%16][8*(l/16) + e] and B[8*(l/16) + e][l%16] in element
// e of its operands; D as mfma16x16x4.
__device__ __forceinline__ f4 mfma16x16x32bf16(bf16x8 a, bf16x8 b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Exact split of a float32 value into three bfloat16 terms, w = hi + mid +
// lo: each remainder is exactly representable in float32, and after two
// terms at most 8 significand bits remain (values below about 2^-110, whose
// low terms underflow, lose them).
__device__ __forceinline__ void split3(float w, __bf16& hi, __bf16& mid, __bf16& lo) {
    hi = (__bf16)w;
    const float r1 = w - (float)hi;
    mid = (__bf16)r1;
    lo = (__bf16)(r1 - (float)mid);
}

// Operand of the bf16-input contraction step over 32 k-values staged in
// fp32: element e holds the value at k = 4e + g for lane group g (the
// contraction is a sum over k, so any assignment of k to (g, e) that both
// operands share is valid; this one reads, for each e, the addresses the
// fp32 step kk = e reads, so the LDS access pattern is unchanged).  at(k)
// returns the staged fp32 value; the conversion rounds to nearest, ties to
// even.
template <class At>
__device__ __forceinline__ bf16x8 bf16_operand(At at, int g) {
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)at(4 * e + g);
    return v;
}

// Parameter-server update of one parameter theta with gradient g and
// optimizer state st: RULE 0 gradient descent (Sec. III.B), 1 RMSProp (Alg. 2
// RMSPROPUPDATE: r <- decay*r + (1-decay)*g^2, theta <- theta - lr*g/sqrt(r),
// skipped while r == 0), 2 AdaGrad (G <- G + g^2, theta <- theta -
// lr*g/(sqrt(G) + eps)).  Every kernel that updates parameters calls this, so
// fused and standalone updates round identically.
template <int RULE>
__device__ __forceinline__ void ps_update(float& th, float& st, float g, float lr, float decay,
                                          float eps) {
    if constexpr (RULE == 0) {
        th = fmaf(-lr, g, th);
    } else if constexpr (RULE == 1) {
        st = fmaf(decay, st, (1.f - decay) * (g * g));
        if (st > 0.f) th = th - lr * g / sqrtf(st);
    } else {
        st = fmaf(g, g, st);
        th = th - lr * g / (sqrtf(st) + eps);
    }
}

// Output tile (x, y, z) of workgroup (blockIdx) in a grid of gx x gy x gz
// tiles, ordered so that each of the eight XCDs (each with its own L2) runs
// a contiguous range of tiles: workgroups are dealt to the XCDs round-robin
// by linear id, so XCD c runs ids c, c + 8, ...; its r-th one takes tile
// first(c) + r, first(c) being the number of ids dealt to XCDs before c.
// Within a k-slice z, ROWS_SHARE orders the tiles x-major (runs that share
// a row block of the row operand), otherwise y-major (runs that share a
// column block of the column operand).
struct TileXYZ {
    int x, y, z;
};
template <bool ROWS_SHARE>
__device__ __forceinline__ TileXYZ xcd_tile() {
    const int gx = gridDim.x, gy = gridDim.y, gz = gridDim.z;
    const int tiles = gx * gy * gz;
    const int id = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
    const int c = id & 7, q = tiles >> 3, rem = tiles & 7;
    const int t = c * q + min(c, rem) + (id >> 3);
    const int z = t / (gx * gy), u = t - z * (gx * gy);
    if constexpr (ROWS_SHARE) return TileXYZ{u / gy, u % gy, z};
    else return TileXYZ{u % gx, u / gx, z};
}
// The forward contractions (split-K): the XCD-contiguous order when every
// XCD's range spans at least two k-slices.  With fewer, whole XCDs would
// hold one slice each, and a shorter last slice leaves its XCDs idle; the
// launch order then already keeps each row block on one XCD (gx a multiple
// of 8), the weights being fetched once per XCD.
__device__ __forceinline__ TileXYZ fwd_tile_order() {
    if (gridDim.z >= 16) return xcd_tile<true>();   // (gx*gy*gz / 8 >= 2*gx*gy)
    return TileXYZ{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

// Sums over the 64 lanes of a wave of N values per lane, by halving: at
// the step with lane mask M every lane keeps half of its current list (the
// lower half if its bit M is clear, else the upper half, padded with zeros)
// and adds the partner lane's copy of that half.  Each value is summed over
// the lanes in the same butterfly order as wave_sum (xor 32, 16, ..., 1),
// with at most N + 6 shuffles in all instead of 6N.  Lane l ends with the sum of
// value halving_index<N>(l), or of padding where that is -1.
template <int N, int M>
__device__ __forceinline__ float halving_step(const float* v, int lane) {
    if constexpr (M == 0) {
        return v[0];
    } else {
        constexpr int H = (N + 1) / 2;
        const bool up = (lane & M) != 0;
        float w[H];
#pragma unroll
        for (int i = 0; i < H; ++i) {
            const float lo = v[i];
            const float hi = H + i < N ? v[H + i] : 0.f;
            w[i] = (up ? hi : lo) + __shfl_xor(up ? lo : hi, M, 64);
        }
        return halving_step<H, M / 2>(w, lane);
    }
}

template <int N>
__device__ __forceinline__ int halving_index(int lane) {
    int n = N, base = 0, real = N;
    for (int m = 32; m >= 1; m >>= 1) {
        const int h = (n + 1) / 2;
        if (lane & m) {
            base += h;
            real = real > h ? real - h : 0;
        } else {
            real = real < h ? real : h;
        }
        n = h;
    }
    return real > 0 ? base : -1;
}

// The convolution layers the library is built for (valid padding).
enum ConvId { CONV_S1 = 0, CONV_S2 = 1, CONV_L1 = 2, CONV_L2 = 3, CONV_L3 = 4, CONV_COUNT = 5 };

struct ConvDims {
    int cin, ih, iw, cout, k, s, oh, ow;
};

inline ConvDims conv_dims(ConvId id) {
    switch (id) {
        case CONV_S1: return {4, 84, 84, 16, 8, 4, 20, 20};
        case CONV_S2: return {16, 20, 20, 32, 4, 2, 9, 9};
        case CONV_L1: return {4, 84, 84, 32, 8, 4, 20, 20};
        case CONV_L2: return {32, 20, 20, 64, 4, 2, 9, 9};
        default:      return {64, 9, 9, 64, 3, 1, 7, 7};
    }
}

// Where sample j of a layer input lives: base + j*stride (dense), or, for
// replay records addressed by index, base + (idx[j] + off)*stride.
struct ConvIn {
    const void* base;
    const int64_t* idx;
    int64_t stride;  // bytes
    int off;
};

__device__ __forceinline__ const unsigned char* sample_ptr(const ConvIn& in, int j) {
    const int64_t r = in.idx ? in.idx[j] + in.off : (int64_t)j;
    return (const unsigned char*)in.base + r * in.stride;
}

// Side fields of the transitions idx[0..batch) copied (with conversion) from
// the replay's arrays, by block 0 of the first forward launch.
struct SideFields {
    const int64_t* idx;  // NULL: nothing to copy
    const uint8_t* action;
    const int8_t* reward;
    const uint8_t* terminal;
    int32_t* a_out;
    float* r_out;
    uint8_t* t_out;
    int batch;
};

// The copy of SideFields split into stages, so that its two dependent
// global round trips (the index, then the fields it selects) overlap the
// caller's own loads and arithmetic: begin() loads thread t's index, fetch()
// the fields, end() stores them and copies any transitions from nthreads on
// with a plain loop.  on: the copying workgroup.
struct SideCopy {
    int64_t i = 0;
    uint8_t a = 0, term = 0;
    int8_t r = 0;
    __device__ void begin(const SideFields& s, bool on, int t) {
        if (on && t < s.batch) i = s.idx[t];
    }
    __device__ void fetch(const SideFields& s, bool on, int t) {
        if (on && t < s.batch) {
            a = s.action[i];
            r = s.reward[i];
            term = s.terminal[i];
        }
    }
    __device__ void end(const SideFields& s, bool on, int t, int nthreads) {
        if (!on) return;
        if (t < s.batch) {
            s.a_out[t] = a;
            s.r_out[t] = (float)r;
            s.t_out[t] = term;
        }
        for (int j = t + nthreads; j < s.batch; j += nthreads) {
            const int64_t k = s.idx[j];
            s.a_out[j] = s.action[k];
            s.r_out[j] = (float)s.reward[k];
            s.t_out[j] = s.terminal[k];
        }
    }
};

// ---- launchers (host side); every one returns hipGetLastError() ----------

// Measurement hook (dqn_profile.h): the event pair of kernel id `kid` around
// a launch made outside the C ABI file.
void prof_mark_begin(int kid, hipStream_t st);
void prof_mark_end(int kid, hipStream_t st);

// Replay destination of the actor-side kernels (dqn_replay_out in
// dqn_actor.h): game e keeps states in records e*(cap+1) .. e*(cap+1)+cap,
// state t in slot t mod cap, slot cap repeating slot 0.  frames == NULL: no
// replay write.  t: index of the experience being stored (-1: initial
// states).
struct ReplayOut {
    uint8_t* frames;
    int64_t stride;          // bytes between records
    uint8_t* action;
    int8_t* reward;
    uint8_t* terminal;
    int64_t cap;
    int64_t t;
};
// Pointer, stride and capacity checks of a replay destination.
bool replay_ok(const ReplayOut& rp);

// Raise a kernel's dynamic LDS limit to `bytes` if it is below (once per
// kernel and size; thread-safe).  False if the runtime refuses.
bool allow_lds(const void* kern, size_t bytes);

// Forward convolution + bias + ReLU for n samples.  Samples j < n_a read
// sample j of in_a and use (w_a, b_a); samples j >= n_a read sample j - n_a
// of in_b and use (w_b, b_b).  Output float [n][cout][oh][ow].  in_scale
// multiplies the accumulated products before the bias (1/255 for byte
// input).  side (nullable) is copied by block 0.
hipError_t launch_conv_fwd(ConvId id, const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                           const float* w_a, const float* b_a, const float* w_b, const float* b_b,
                           float* out, float in_scale, const SideFields* side, hipStream_t st);

// Both convolution layers of the small network (CONV_S1 then CONV_S2, bias +
// ReLU each) in one launch; sample roles, inputs and weights as
// launch_conv_fwd.  Writes act1 [n][16][20][20] and act2 [n][32][9][9].
// Requires 16-byte aligned weight blocks, input bases and record strides
// (conv_s12_fwd_aligned).
bool conv_s12_fwd_supported(ConvId c1, ConvId c2);
bool conv_s12_fwd_aligned(const ConvIn& in);
hipError_t launch_conv_s12_fwd(const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                               const float* w1_a, const float* b1_a, const float* w2_a,
                               const float* b2_a, const float* w1_b, const float* b1_b,
                               const float* w2_b, const float* b2_b, float* act1, float* act2,
                               const SideFields* side, hipStream_t st);

// The small network's backward below the fc layers in one launch: conv2's
// weight/bias partial sums (as launch_conv_wgrad for CONV_S2: wpart2,
// bpart2 with conv_wgrad_chunks(CONV_S2, batch) slots), and, per sample and
// band of conv1 rows, conv2's input gradient masked by [act1 > 0] and
// conv1's weight/bias partial sums over those rows into
// conv_s12_bwd_slots(batch) slots of wpart1 [slots][16][256], bpart1
// [slots][16].  in: the network input (bytes), 16-byte aligned.
int conv_s12_bwd_slots(int batch);
hipError_t launch_conv_s12_bwd(const ConvIn& in, const float* act1, const float* dz2, const float* w2,
                               int batch, float* wpart2, float* bpart2, float* wpart1, float* bpart1,
                               hipStream_t st);

// The implicit-GEMM launchers below and the fc GEMMs take `bf16`: false
// contracts the fp32 operands on fp32 MFMA; true is the bf16-input variant
// (both operands rounded to bfloat16, nearest-even, fp32 accumulation).

// Forward of the fp32-input large-network layers (CONV_L2, CONV_L3) as one
// implicit GEMM over all n samples (dense input [n][cin][ih][iw]; samples
// below n_a use (w_a, b_a), the rest (w_b, b_b)); bias + ReLU; output
// [n][cout][oh][ow].  Weights 16-byte aligned.  In the bf16-input variant
// from kFwdClMinRows samples, the input (in16) and the output (out16) may be
// held as bfloat16 values: the contraction rounds its input to bfloat16
// anyway, so only the storage changes.
bool conv_igemm_fwd_supported(ConvId id);
hipError_t launch_conv_igemm_fwd(ConvId id, const float* in, int n_a, int n, const float* w_a,
                                 const float* b_a, const float* w_b, const float* b_b, float* out,
                                 bool bf16, bool in16, bool out16, const float* pk_a, const float* pk_b,
                                 hipStream_t st);

// The forward of CONV_L2 / CONV_L3 from kFwdClMinRows samples on, both
// precisions: weights held in registers, each sample staged channels-last in
// LDS (same arguments and result as launch_conv_igemm_fwd, which routes to
// it).
constexpr int kFwdClMinRows = 256;
bool conv_fwd_cl_use(ConvId id, int n, bool bf16);
// pk_a, pk_b (fp32 only; both or neither): the three bf16 planes of w_a,
// w_b written by launch_fwd_x6_pack (NULL: the kernel splits W itself).
hipError_t launch_conv_fwd_cl(ConvId id, const float* in, int n_a, int n, const float* w_a, const float* b_a,
                              const float* w_b, const float* b_b, float* out, bool bf16, bool in16, bool out16,
                              const float* pk_a, const float* pk_b, hipStream_t st);

// Input gradient of CONV_L2 / CONV_L3 for n samples as an implicit GEMM per
// stride phase, masked by [h_in > 0] (as launch_conv_dgrad).
hipError_t launch_conv_igemm_dgrad(ConvId id, const float* dz, const float* w, const float* h_in, float* din,
                                   int n, bool bf16, hipStream_t st);

// Input gradient of CONV_L2 for n samples by stride phase, masked by
// [h_in > 0] (as launch_conv_dgrad), with each phase's weights held in
// registers and dz staged in LDS with a zero border.
// wpk (NULL: read W directly): the weights repacked by launch_weight_repack
// (d2/d3 for fp32, h2/h3 for bf16), which the workgroups load coalesced.
// din16 (bf16 only; then din is unused): the input gradient is written
// rounded to bfloat16 there, and workgroup b's per-channel sums of the
// float32 values (conv1's bias-gradient partials) to bpart[b][32], for
// conv2_dgrad_phase_blocks(n) workgroups, each a run of consecutive samples
// as conv1_u8_wgrad_slots.
int conv2_dgrad_phase_blocks(int n);
hipError_t launch_conv2_dgrad_phase(const float* dz, const float* w, const float* h_in, float* din, int n,
                                    bool bf16, bool h16, const float* wpk, hipStream_t st,
                                    __bf16* din16 = nullptr, float* bpart = nullptr);

// Input gradient of CONV_L3 for n samples, masked by [h_in > 0], in the same
// arrangement (weights in registers, zero-bordered dz in LDS, the sample's
// gradient assembled in LDS).  h_in and din 16-byte aligned.
hipError_t launch_conv3_dgrad(const float* dz, const float* w, const float* h_in, float* din, int n, bool bf16,
                              bool h16, const float* wpk, hipStream_t st);
// conv2's and conv3's weights of set a (theta) in the per-lane order of the
// large network's input-gradient kernels, one launch (at most
// weight_repack_floats(CONV_L2 / CONV_L3) floats each, 16-byte aligned).
// NULL outputs are skipped.
struct WeightRepack {
    const float *w2a, *w3a;
    void *h2, *h3;   // bf16 input-gradient operands (the bf16-input variant)
    void *x2, *x3;   // the three exact bf16 planes of the float32 input gradients
    // The bf16-input variant's forward weights of both sets (a: w2a, w3a;
    // b: w2b, w3b) rounded to bf16 in the per-lane order of its forward
    // kernel: the first plane of the float32 forward's copies (same layout).
    const float *w2b, *w3b;
    void *f2a, *f3a, *f2b, *f3b;
    // The float32 forward's weights of both sets as the three exact bf16
    // planes in the per-lane order of its kernel (X6FwdPack below;
    // fwd_x6_pack_floats(id) floats each), or NULL.
    void *p2a, *p3a, *p2b, *p3b;
};
int64_t weight_repack_floats(ConvId id);
// One launch writes every copy whose output is set (16-byte aligned).
hipError_t launch_weight_repack(const WeightRepack& r, hipStream_t st);
int64_t fwd_x6_pack_floats(ConvId id);

// The float32 forward's conv2/conv3 weights as the three exact bf16 planes,
// in the order that forward's lanes load them: vector
// index(pl, nt, kh, s, lane) of plane pl holds, for lane (li, g) of the wave
// owning output channels 16 nt .. 16 nt + 15 and k-step ks = kh KSH + s
// (tap ks / CH, input channels from 32 (ks % CH)), the values
// W[16 nt + li][32 (ks % CH) + 8 g + q][tap], q = 0..7 (CH = cin / 32,
// KSH = taps * CH / 2).
template <int CIN, int KK>
struct X6FwdPack {
    static constexpr int CH = CIN / 32, KS = KK * CH, KSH = KS / 2;
    static constexpr int VECS = 3 * 4 * KS * 64;   // bf16x8 vectors of the three planes
    __host__ __device__ static constexpr int index(int pl, int nt, int kh, int s, int lane) {
        return (((pl * 4 + nt) * 2 + kh) * KSH + s) * 64 + lane;
    }
};
// Vector e of that layout from W[cout][cin][taps] (nothing when out is NULL).
template <int CIN, int KK>
__device__ __forceinline__ void x6_fwd_pack_job(const float* __restrict__ w, void* out, int e) {
    using X = X6FwdPack<CIN, KK>;
    if (!out || e >= X::VECS) return;
    const int lane = e & 63, r = e >> 6;
    const int s = r % X::KSH, kh = (r / X::KSH) & 1, nt = (r / (2 * X::KSH)) & 3, pl = r / (8 * X::KSH);
    const int li = lane & 15, g = lane >> 4;
    const int ks = kh * X::KSH + s, tap = ks / X::CH, cb = ks % X::CH;
    bf16x8 o;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        __bf16 a, b, d;
        split3(w[(size_t)(16 * nt + li) * CIN * KK + (size_t)(32 * cb + 8 * g + q) * KK + tap], a, b, d);
        o[q] = pl == 0 ? a : pl == 1 ? b : d;
    }
    ((bf16x8*)out)[e] = o;
}

// Weight/bias gradient partial sums of CONV_L2 or CONV_L3 for n samples, one
// workgroup per run of samples holding its outputs in registers (in float32
// from 256 samples, two workgroups per conv2 slot, each over half of the
// input channels): conv_wgrad_reg_slots(id, n, bf16) slots of wpart
// [slots][64][cin*k*k] and bpart [slots][64].  in: the layer input
// [n][cin][ih][iw] (floats, or bfloat16 values when in16).
int conv_wgrad_reg_slots(ConvId id, int n, bool bf16);
hipError_t launch_conv_wgrad_reg(ConvId id, const float* in, const float* dz, int n, float* wpart, float* bpart,
                                 bool bf16, bool in16, hipStream_t st);

// Weight/bias gradient partial sums of a large-network layer for n samples as
// an implicit GEMM over pixel chunks: conv_igemm_wgrad_chunks(id, n) slots of
// wpart [slots][cout][cin*k*k] and bpart [slots][cout].  in: the layer input
// (bytes for CONV_L1, addressed through in.idx when set; floats otherwise).
int conv_igemm_wgrad_chunks(ConvId id, int n);
hipError_t launch_conv_igemm_wgrad(ConvId id, const ConvIn& in, const float* dz, int n, float* wpart,
                                   float* bpart, float in_scale, bool bf16, hipStream_t st);

// conv1 forward on byte input (CONV_L1 or CONV_S1) for many samples, on bf16
// MFMA with an exact three-term split of the fp32 weights (bf16: the weights
// rounded to bfloat16 instead); roles and alignment as launch_conv_s12_fwd;
// output [n][cout][20][20].
bool conv1_u8_fwd_supported(ConvId id);
hipError_t launch_conv1_u8_fwd(ConvId id, const ConvIn& in_a, const ConvIn& in_b, int n_a, int n,
                               const float* w_a, const float* b_a, const float* w_b, const float* b_b,
                               float* out, const SideFields* side, bool bf16, bool out16, hipStream_t st);

// conv1 weight/bias gradient on byte input (CONV_L1 or CONV_S1) for many
// samples: conv1_u8_wgrad_slots(n) partial-sum slots of wpart
// [slots][cout][256] and bpart [slots][cout]; input 16-byte aligned, dz
// [n][cout][20][20].
// dz16 (bf16 only): dz holds bfloat16 values, and the bias partial sums are
// left to the producer of dz (bpart is not written).
int conv1_u8_wgrad_slots(int n);
hipError_t launch_conv1_u8_wgrad(ConvId id, const ConvIn& in, const float* dz, int n, float* wpart,
                                 float* bpart, float in_scale, bool bf16, hipStream_t st, bool dz16 = false);

// Weight and bias gradient partial sums over sample chunks:
// wpart [chunks][cout][cin*k*k], bpart [chunks][cout].
int conv_wgrad_chunks(ConvId id, int batch);
hipError_t launch_conv_wgrad(ConvId id, const ConvIn& in, const float* dz, int batch, float* wpart,
                             float* bpart, float in_scale, hipStream_t st);

// Weight gradient (as launch_conv_wgrad, fp32 input) and input gradient (as
// launch_conv_dgrad) of one layer from the same dz, in a single launch.
hipError_t launch_conv_bwd(ConvId id, const ConvIn& in, const float* dz, int batch, float* wpart,
                           float* bpart, const float* w, const float* h_in, float* din,
                           hipStream_t st);

// Input gradient din = (W^T * dz) masked by [h_in > 0], float [n][cin][ih][iw].
hipError_t launch_conv_dgrad(ConvId id, const float* dz, const float* w, const float* h_in,
                             float* din, int batch, hipStream_t st);

// C = A * B over fp32 MFMA tiles.  A(m,k) = ta ? A[k*lda+m] : A[m*lda+k];
// B(k,n) = tb ? B[n*ldb+k] : B[k*ldb+n].  Split-K: slice z covers
// k in [z*kchunk, min(K,(z+1)*kchunk)) and writes C + z*c_slice.
// GEMM_NN (the fc1 input gradient) requires mask: C = acc * [mask[m*ldc+n] > 0].
// kchunk must be a multiple of 32.
enum GemmKind { GEMM_NT = 0, GEMM_TN = 1, GEMM_NN = 2 };

// k-slicing of the fc1 forward GEMM for `rows` output rows: ks slices of
// kchunk (a multiple of 64, the last one possibly shorter).
void gemm_fwd_split(int rows, int N, int K, int* ks, int* kchunk);
// From a batch of kGemmX6MinRows (M of the forward and of the input
// gradient, K of the weight gradient) the float32 fc1 contractions run on
// bf16 MFMA with the exact three-plane split (launch_gemm_x6: same arguments
// as launch_gemm, kchunk a multiple of 32): the forward on 128x256 tiles,
// the input gradient (B contiguous along n, transposed as it is staged) on
// 64x64 tiles, batch 2,048: 77 -> 68 us; the weight gradient (both operands
// transposed) on 64x64 tiles, or, split into kGemmX6WgradSlices k-slices of
// partial sums, on 128x128 tiles with 64-wide k-stages (each staged operand
// value then serves twice the products; batch 2,048: 77 -> 63 us, the
// finalize adding the slices).  Below that batch the split cost more than
// the six products saved.
constexpr int kGemmX6WgradSlices = 2;
constexpr int kGemmX6MinRows = 1024;
void gemm_fwd_split_x6(int rows, int N, int K, int* ks, int* kchunk);
hipError_t launch_gemm_x6(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B, int ldb,
                          float* C, int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                          hipStream_t st);
hipError_t launch_gemm_x6_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0, const float* A1,
                               const float* B1, float* C1, int lda, int ldb, int ldc, int kslices, int kchunk,
                               int64_t c_slice, hipStream_t st);
// The same for the bf16-input variant's forward GEMM (its own tiles).
void gemm_fwd_split_bf16(int rows, int N, int K, int* ks, int* kchunk);
// The bf16-input contractions of launch_gemm (same arguments; operands
// rounded to bfloat16 as they are staged).
// x16 (bf16 only): the activation operand -- A of GEMM_NT, B of GEMM_TN, the
// mask of GEMM_NN -- holds bfloat16 values.  a16 (bf16 only, GEMM_TN and
// GEMM_NN): so does A, the pre-activation gradient.
hipError_t launch_gemm_bf16(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B, int ldb,
                            float* C, int ldc, int kslices, int kchunk, int64_t c_slice, const float* mask,
                            bool x16, hipStream_t st, bool a16 = false);
hipError_t launch_gemm(GemmKind kind, int M, int N, int K, const float* A, int lda, const float* B,
                       int ldb, float* C, int ldc, int kslices, int kchunk, int64_t c_slice,
                       const float* mask, bool bf16, bool x16, hipStream_t st, bool a16 = false);
// Two fc1 forward contractions of one shape in one launch (GEMM_NT, split-K
// as above): C0 = A0 B0^T and C1 = A1 B1^T, each in its own k-slices.
hipError_t launch_gemm_bf16_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0,
                                 const float* A1, const float* B1, float* C1, int lda, int ldb, int ldc,
                                 int kslices, int kchunk, int64_t c_slice, bool x16, hipStream_t st);
hipError_t launch_gemm_fwd2(int M, int N, int K, const float* A0, const float* B0, float* C0, const float* A1,
                            const float* B1, float* C1, int lda, int ldb, int ldc, int kslices, int kchunk,
                            int64_t c_slice, bool bf16, bool x16, hipStream_t st);

// fc1 backward for batch B: dW [H][F] = dz1^T x (x = first B rows of the last
// conv output) and dx [B][F] = (dz1 W) masked by [x > 0], as one launch where
// possible.
hipError_t launch_gemm_wgrad_dgrad(int H, int F, int B, const float* dz1, const float* x,
                                   float* dW, const float* W, float* dx, bool bf16, hipStream_t st);

struct HeadTdArgs {
    const float* fc1p;   // [ks][2B][H] split-K partials of fc1 (rows < B: s, >= B: s')
    int ks, B;
    const float *b1, *b1t, *W2, *b2, *W2t, *b2t;
    const int32_t* action;
    const float* reward;
    const uint8_t* terminal;
    float gamma;
    float *h1s, *dz1, *delta, *lossj, *q_out, *y_out;
    __bf16* dz1h;        // when set, dz1 rounded to bfloat16 (nearest even) as well
};
hipError_t launch_head_td(int H, int A, const HeadTdArgs& a, hipStream_t st);

struct HeadFwdArgs {
    const float* fc1p;   // [ks][B][H]
    int ks, B;
    const float *b1, *W2, *b2;
    uint64_t thresh;     // explore iff (draw >> 32) < thresh
    const uint64_t* draws;
    float* q_out;
    int32_t* action_out;
};
hipError_t launch_head_fwd(int H, int A, const HeadFwdArgs& a, hipStream_t st);

struct FinalizeArgs {
    int n_conv;
    const float* wpart[3];
    const float* bpart[3];
    int chunks[3];
    int wcount[3];
    int cout[3];
    float* gw[3];
    float* gb[3];
    const float *dz1, *h1s, *delta, *lossj;
    const int32_t* action;
    int B, H, A;
    float *g_b1, *g_W2, *g_b2, *loss_out;
    // Gradient vector the gw/gb/g_* pointers point into, and the range of it
    // (the fc1 weights) that an earlier kernel wrote in full, or, with
    // fc1w_part set, wrote as fc1w_slices partial sums fc1w_part[z][i] (k
    // split into slices) that the finalize adds in slice order.
    const float* grad_base;
    int64_t fc1w_off, fc1w_count;
    const float* fc1w_part;
    int fc1w_slices;
    // Above 128 samples: sample-sum partial slots, one per chunk of 32
    // samples, each A*H + H + A + 1 floats (workspace).
    float* spart;
    int schunks;
};
// Chunk slots of the sums over samples for batch B (0 up to 128 samples).
inline int finalize_sample_chunks(int B) { return B > 128 ? (B + 31) / 32 : 0; }

// A parameter-server update fused into the last kernel of a TD step.
struct PsUpdate {
    int rule;        // 0 SGD, 1 RMSProp, 2 AdaGrad (ps_update)
    float* theta;    // updated in place
    float* state;    // RMSProp r / AdaGrad G; unused for SGD
    float lr, decay, eps;
};

// Reduce the partial sums into the gradient (upd == NULL), or apply the
// update to every parameter instead of storing the reduced gradient; the fc1
// weight range is then read from grad_base.  The loss is stored either way.
hipError_t launch_finalize(const FinalizeArgs& a, const PsUpdate* upd, hipStream_t st);

// Count of idx[0..batch) outside [0, hi] into *bad (one workgroup).
hipError_t launch_validate(const int64_t* idx, int batch, int64_t hi, int32_t* bad, hipStream_t st);
hipError_t launch_gather(const uint8_t* frames, int64_t stride, int64_t rec_bytes,
                         const uint8_t* act, const int8_t* rew, const uint8_t* term,
                         const int64_t* idx, int batch, uint8_t* s, uint8_t* sn, int32_t* a,
                         float* r, uint8_t* t, hipStream_t st);

hipError_t launch_copy(const float* src, float* dst, int64_t n, hipStream_t st);

hipError_t launch_apply(int rule, const float* th_in, float* th_out, float* state, const float* g,
                        int64_t n, float lr, float decay, float eps, hipStream_t st);

// One sequential training step from replay records: the TD gradient of
// dqn_td_gradient_replay with the update `upd` applied by its last kernel
// (theta == upd.theta, updated in place).  grad_ws holds the fc1 weight
// gradient in between.  Host checks as dqn_td_gradient_replay and
// ps_apply_update; returns a dqn_status.
int td_step_replay(const dqn_net* net, const float* theta_target, const dqn_replay* replay,
                   const int64_t* idx, int32_t batch, float gamma, float* grad_ws, float* loss_out,
                   const PsUpdate& upd, void* ws, size_t ws_bytes, hipStream_t st);

}  // namespace dqn
