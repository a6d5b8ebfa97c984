// C ABI of libdqn.so (declared in include/dqn.h): argument checks, the
// workspace layout and the kernel sequence of each entry point.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstddef>
#include <mutex>

#include "common.h"
#include "dqn.h"
#include "dqn_profile.h"

using namespace dqn;

// Scratch of dqn_td_gradient_noalloc: the workspace of the TD step in the
// library's own device memory, one copy per GPU (the loader places it when
// the library's code is loaded on a device; it is held until the process
// ends).  In host code `scratch` is only a stand-in for the symbol: its
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current, and only that address is handed to kernels.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

struct NetInfo {
    int n_conv;
    ConvId conv[3];
    ConvDims d[3];
    int H, A, flat;
    int64_t P;
    int64_t w_off[5], b_off[5];  // conv layers, then fc1, fc2
    bool bf16;                   // DQN_BF16: bf16-input contractions
};

// Only the two network shapes the kernels are built for are accepted.
int identify(const dqn_net* net, NetInfo* ni) {
    if (!net) return DQN_EINVAL;
    if (net->precision != DQN_FP32 && net->precision != DQN_BF16) return DQN_EUNSUPPORTED;
    if (net->in_c != 4 || net->in_h != 84 || net->in_w != 84) return DQN_EUNSUPPORTED;
    if (net->n_conv == 2 && net->conv_out[0] == 16 && net->conv_k[0] == 8 && net->conv_stride[0] == 4 &&
        net->conv_out[1] == 32 && net->conv_k[1] == 4 && net->conv_stride[1] == 2 &&
        net->fc_hidden == 256 && net->n_actions == 6) {
        ni->n_conv = 2;
        ni->conv[0] = CONV_S1;
        ni->conv[1] = CONV_S2;
        ni->H = 256;
        ni->A = 6;
    } else if (net->n_conv == 3 && net->conv_out[0] == 32 && net->conv_k[0] == 8 &&
               net->conv_stride[0] == 4 && net->conv_out[1] == 64 && net->conv_k[1] == 4 &&
               net->conv_stride[1] == 2 && net->conv_out[2] == 64 && net->conv_k[2] == 3 &&
               net->conv_stride[2] == 1 && net->fc_hidden == 512 && net->n_actions == 18) {
        ni->n_conv = 3;
        ni->conv[0] = CONV_L1;
        ni->conv[1] = CONV_L2;
        ni->conv[2] = CONV_L3;
        ni->H = 512;
        ni->A = 18;
    } else {
        return DQN_EUNSUPPORTED;
    }
    // The bf16-input variant is built for the large network.
    ni->bf16 = net->precision == DQN_BF16;
    if (ni->bf16 && ni->n_conv != 3) return DQN_EUNSUPPORTED;
    int64_t off = 0;
    for (int l = 0; l < ni->n_conv; ++l) {
        ni->d[l] = conv_dims(ni->conv[l]);
        const ConvDims& c = ni->d[l];
        ni->w_off[l] = off;
        off += (int64_t)c.cout * c.cin * c.k * c.k;
        ni->b_off[l] = off;
        off += c.cout;
    }
    const ConvDims& last = ni->d[ni->n_conv - 1];
    ni->flat = last.cout * last.oh * last.ow;
    const int L = ni->n_conv;
    ni->w_off[L] = off;
    off += (int64_t)ni->H * ni->flat;
    ni->b_off[L] = off;
    off += ni->H;
    ni->w_off[L + 1] = off;
    off += (int64_t)ni->A * ni->H;
    ni->b_off[L + 1] = off;
    off += ni->A;
    ni->P = off;
    return DQN_OK;
}

inline int64_t act_elems(const ConvDims& c) { return (int64_t)c.cout * c.oh * c.ow; }

// Largest batch whose backward kernels are launched in pairs (above it each
// kernel alone fills the chip and keeps its own occupancy).
constexpr int kPairMaxBatch = 64;
// Samples per forward launch up to which the small network's two conv layers
// run as one fused launch (measured faster at every batch up to 1024
// samples per launch, and by 2x at 64).
constexpr int kFuseMaxRows = 1 << 20;
// dqn_profile_set_fusion (a measurement switch; read once per call)
std::atomic<bool> g_fusion{true};
// Samples per forward launch from which the large network's fp32 conv layers
// run as one implicit GEMM over all samples (2-3x the per-layer kernel from
// 256 samples; slower at 64).
constexpr int kIgemmMinRows = 128;
// Batch from which the conv2/conv3 weight gradients run with the outputs in
// registers across samples.
constexpr int kRegWgradMinRows = 128;

// Backward layers that run as implicit GEMMs at batch B (measured faster
// than the per-layer kernels from 128 samples: the weight gradients of
// conv2/conv3 and the input gradient of conv3 of the large network; its
// conv1 weight gradient uses a dedicated kernel from the same size).  The
// bf16-input variant runs every large-network layer on these kernels (and
// conv1 on the byte-input kernels) at any batch.
bool igemm_wgrad(ConvId id, int B, bool bf16) {
    return (id == CONV_L2 || id == CONV_L3) && (bf16 || B >= kIgemmMinRows);
}
// ... of which the samples-per-workgroup kernel with register-held outputs
// (k_wgrad.hip) takes the batches it is faster for.
bool reg_wgrad(ConvId id, int B, bool bf16) { return igemm_wgrad(id, B, bf16) && B >= kRegWgradMinRows; }
bool igemm_dgrad(ConvId id, int B, bool bf16) { return id == CONV_L3 && (bf16 || B >= kIgemmMinRows); }
// conv2's and conv3's input gradients of the large network with the weights
// in registers (from the same batch size; k_dgrad.hip).
bool phase_dgrad(ConvId id, int B, bool bf16) {
    return (id == CONV_L2 || id == CONV_L3) && (bf16 || B >= kIgemmMinRows);
}
bool igemm_fwd(ConvId id, int rows, bool bf16) {
    return conv_igemm_fwd_supported(id) && (bf16 || rows >= kIgemmMinRows);
}
bool conv1_u8(ConvId id, int rows, bool bf16) { return id == CONV_L1 && (bf16 || rows >= kIgemmMinRows); }

// fc1 forward split-K: enough slices that the launch covers the chip.
struct Carver {
    size_t off = 0;
    template <class T>
    T* take(void* base, int64_t count) {
        T* p = base ? (T*)((char*)base + off) : nullptr;
        off += ((size_t)count * sizeof(T) + 255) / 256 * 256;
        return p;
    }
};

struct TdLayout {
    float* act[3];
    float* fc1p;
    float *h1s, *dz1, *delta, *lossj;
    int32_t* a;     // side fields gathered from a replay (replay source only)
    float* r;
    uint8_t* t;
    float* dconv[3];
    float* wpart[3];
    float* bpart[3];
    int chunks[3];
    int ks, kchunk;
    float* spart;   // sample-sum chunk slots of the finalize (above 128 samples)
    __bf16* dz1h;         // dz1 in bfloat16 (bf16-input variant from 128 samples), else null
    float *wpk2, *wpk3;   // repacked conv2/conv3 weights of the input gradients (large network)
    float *fpk[2][2];     // ... the fp32 forward's bf16 planes: [layer conv2, conv3][set theta, theta^-]
    float* fc1w_part;     // the float32 fc1 weight gradient's k-slices (large batch, wide layer), else null
    size_t bytes;
};

// The float32 fc1 weight gradient of a large batch and a 512-wide hidden
// layer is computed as kGemmX6WgradSlices k-slices of partial sums (larger
// tiles), which the finalize adds.
bool fc1w_split(const NetInfo& ni, int B) { return !ni.bf16 && B >= kGemmX6MinRows && ni.H >= 512; }

TdLayout td_layout(const NetInfo& ni, int B, void* ws) {
    TdLayout t{};
    Carver cv;
    const int n2 = 2 * B;
    for (int l = 0; l < ni.n_conv; ++l) t.act[l] = cv.take<float>(ws, (int64_t)n2 * act_elems(ni.d[l]));
    (ni.bf16 ? gemm_fwd_split_bf16 : gemm_fwd_split)(n2, ni.H, ni.flat, &t.ks, &t.kchunk);
    t.fc1p = cv.take<float>(ws, (int64_t)t.ks * n2 * ni.H);
    t.h1s = cv.take<float>(ws, (int64_t)B * ni.H);
    t.dz1 = cv.take<float>(ws, (int64_t)B * ni.H);
    t.delta = cv.take<float>(ws, B);
    t.lossj = cv.take<float>(ws, B);
    t.a = cv.take<int32_t>(ws, B);
    t.r = cv.take<float>(ws, B);
    t.t = cv.take<uint8_t>(ws, B);
    for (int l = 0; l < ni.n_conv; ++l) t.dconv[l] = cv.take<float>(ws, (int64_t)B * act_elems(ni.d[l]));
    for (int l = 0; l < ni.n_conv; ++l) {
        const ConvDims& c = ni.d[l];
        t.chunks[l] = conv_wgrad_chunks(ni.conv[l], B);
        // The fused small-network backward writes conv1's partial sums per
        // (sample, band) instead: room for whichever count is larger.
        int64_t slots = t.chunks[l];
        if (l == 0 && ni.n_conv == 2 && conv_s12_fwd_supported(ni.conv[0], ni.conv[1]))
            slots = std::max<int64_t>(slots, conv_s12_bwd_slots(B));
        if (igemm_wgrad(ni.conv[l], B, ni.bf16))
            slots = std::max<int64_t>(slots, conv_igemm_wgrad_chunks(ni.conv[l], B));
        if (reg_wgrad(ni.conv[l], B, ni.bf16))
            slots = std::max<int64_t>(slots, conv_wgrad_reg_slots(ni.conv[l], B, ni.bf16));
        if (l == 0 && conv1_u8(ni.conv[0], B, ni.bf16)) slots = std::max<int64_t>(slots, conv1_u8_wgrad_slots(B));
        t.wpart[l] = cv.take<float>(ws, slots * c.cout * c.cin * c.k * c.k);
        t.bpart[l] = cv.take<float>(ws, slots * c.cout);
    }
    t.spart = cv.take<float>(ws, (int64_t)finalize_sample_chunks(B) * ((int64_t)ni.A * ni.H + ni.H + ni.A + 1));
    if (ni.n_conv == 3) {
        t.wpk2 = cv.take<float>(ws, weight_repack_floats(CONV_L2));
        t.wpk3 = cv.take<float>(ws, weight_repack_floats(CONV_L3));
        for (int w = 0; w < 2; ++w) {
            t.fpk[0][w] = cv.take<float>(ws, fwd_x6_pack_floats(CONV_L2));
            t.fpk[1][w] = cv.take<float>(ws, fwd_x6_pack_floats(CONV_L3));
        }
    }
    // (from 128 samples, where the fc1 gradients are separate launches; kept
    // out of smaller workspaces)
    if (ni.bf16 && B >= 128) t.dz1h = cv.take<__bf16>(ws, (int64_t)B * ni.H);
    if (fc1w_split(ni, B)) t.fc1w_part = cv.take<float>(ws, (int64_t)kGemmX6WgradSlices * ni.H * ni.flat);
    t.bytes = cv.off;
    return t;
}

struct FwdLayout {
    float* act[3];
    float* fc1p;
    int ks, kchunk;
    size_t bytes;
};

FwdLayout fwd_layout(const NetInfo& ni, int B, void* ws) {
    FwdLayout f{};
    Carver cv;
    for (int l = 0; l < ni.n_conv; ++l) f.act[l] = cv.take<float>(ws, (int64_t)B * act_elems(ni.d[l]));
    (ni.bf16 ? gemm_fwd_split_bf16 : gemm_fwd_split)(B, ni.H, ni.flat, &f.ks, &f.kchunk);
    f.fc1p = cv.take<float>(ws, (int64_t)f.ks * B * ni.H);
    f.bytes = cv.off;
    return f;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = (const char*)a;
    const char* pb = (const char*)b;
    return pa < pb + nb && pb < pa + na;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }


// Measurement hook (dqn_profile.h): event pairs recorded around one kernel.
struct ProfSlot {
    hipEvent_t* ev = nullptr;
    int n = 0;
    int used = 0;
    int stride = 1;
    int64_t seen = 0;  // launches since the attach
    bool open = false;
};
ProfSlot g_prof[DQN_K_COUNT];
// Number of attached slots.  While it is zero the launches touch no slot, so
// the entry points read and write no process-wide state and concurrent calls
// from several host threads do not interact.
std::atomic<int> g_prof_attached{0};

inline void prof_begin(int k, hipStream_t st) {
    if (g_prof_attached.load(std::memory_order_relaxed) == 0) return;
    ProfSlot& p = g_prof[k];
    if (p.ev && p.used < p.n && p.seen % p.stride == 0) {
        (void)hipEventRecord(p.ev[2 * p.used], st);
        p.open = true;
    }
    ++p.seen;
}
inline void prof_end(int k, hipStream_t st) {
    if (g_prof_attached.load(std::memory_order_relaxed) == 0) return;
    ProfSlot& p = g_prof[k];
    if (p.open) {
        (void)hipEventRecord(p.ev[2 * p.used + 1], st);
        ++p.used;
        p.open = false;
    }
}

}  // namespace

namespace dqn {
void prof_mark_begin(int kid, hipStream_t st) { prof_begin(kid, st); }
void prof_mark_end(int kid, hipStream_t st) { prof_end(kid, st); }
}  // namespace dqn

namespace {

// Launch one kernel of the hot path, bracketed by the profiling events of
// kernel id `kid` when attached.
#define RUN(kid, expr)                                  \
    do {                                                \
        prof_begin((kid), st);                          \
        if ((expr) != hipSuccess) return DQN_EHIP;      \
        prof_end((kid), st);                            \
    } while (0)


// Where a TD step's transitions come from: dense device buffers, or replay
// records and side arrays addressed by an index array.
struct TdSource {
    const uint8_t *s, *s_next;
    const int32_t* action;
    const float* reward;
    const uint8_t* terminal;
    const dqn_replay* replay;
    const int64_t* idx;
};

int td_gradient_impl(const dqn_net* net, const NetInfo& ni, const float* theta,
                            const float* theta_target, const TdSource& src, int32_t batch,
                            float gamma, float* grad_out, float* loss_out, float* q_out,
                            float* y_out, void* ws, size_t ws_bytes, hipStream_t st,
                            const PsUpdate* upd = nullptr) {
    if (!theta || !grad_out || !loss_out || !ws) return DQN_EINVAL;
    if (batch <= 0 || !std::isfinite(gamma)) return DQN_EINVAL;
    const float* tt = theta_target ? theta_target : theta;
    const size_t pbytes = (size_t)ni.P * sizeof(float);
    if (overlaps(grad_out, pbytes, theta, pbytes) || overlaps(grad_out, pbytes, tt, pbytes))
        return DQN_EINVAL;
    if (!aligned(ws, 256) || !aligned(theta, 16) || !aligned(tt, 16) || !aligned(grad_out, 16))
        return DQN_EINVAL;
    TdLayout t = td_layout(ni, batch, nullptr);
    if (ws_bytes < t.bytes) return DQN_EWORKSPACE;
    t = td_layout(ni, batch, ws);
    const int B = batch, L = ni.n_conv;
    const float* th = theta;
    const int64_t rec = (int64_t)net->in_c * net->in_h * net->in_w;

    // Layer-0 inputs and the side fields.
    ConvIn s0, sn0;
    SideFields side{};
    const int32_t* action = src.action;
    const float* reward = src.reward;
    const uint8_t* terminal = src.terminal;
    if (src.replay) {
        s0 = ConvIn{src.replay->frames, src.idx, src.replay->record_stride, 0};
        sn0 = ConvIn{src.replay->frames, src.idx, src.replay->record_stride, 1};
        side = SideFields{src.idx, src.replay->action, src.replay->reward, src.replay->terminal,
                          t.a, t.r, t.t, B};
        action = t.a;
        reward = t.r;
        terminal = t.t;
    } else {
        s0 = ConvIn{src.s, nullptr, rec, 0};
        sn0 = ConvIn{src.s_next, nullptr, rec, 0};
    }
    // The bf16-input variant reads the network input with the byte-input
    // conv1 kernels, which need 16-byte aligned samples.
    if (ni.bf16 && (!conv_s12_fwd_aligned(s0) || !conv_s12_fwd_aligned(sn0))) return DQN_EINVAL;
    // bf16-input variant of the large network from 128 samples: the conv
    // layers' outputs are stored as bfloat16 values.  Every reader rounds them
    // to bfloat16 anyway (the next layer's forward and weight gradient, the fc1
    // contractions) or takes only their sign (the ReLU masks of the input
    // gradients), and all of those readers are the kernels that accept
    // bfloat16 storage.
    const bool a16 = ni.bf16 && L == 3 && B >= kRegWgradMinRows && 2 * B >= kFwdClMinRows;

    // The large network's conv2 and conv3 kernels that hold their weights in
    // registers load them from copies in per-lane order, written at the start
    // of the step: the fp32 forward's three bf16 planes of both weight sets,
    // and the input gradients' weights of both precisions (instead of
    // gathering 64 to 144 scattered words per lane; the gather dominated a
    // workgroup's first sample: batch 256, conv2's fp32 input gradient 33 ->
    // 21 us, bf16 23 -> 9 us).
    // (the bf16-input variant's forward copies, for its bf16 activations,
    // are jobs of the input gradients' repack launch: batch 2,048, conv2 and
    // conv3 forward 44.6 -> 42.4 and 37.2 -> 31.7 us)
    const bool repack_fwd = !ni.bf16 && L == 3 && conv_fwd_cl_use(CONV_L2, 2 * B, false);
    const bool fwd16 = a16 && conv_fwd_cl_use(CONV_L2, 2 * B, true) && conv_fwd_cl_use(CONV_L3, 2 * B, true);
    const bool repack = L == 3 && phase_dgrad(CONV_L2, B, ni.bf16);
    if (repack_fwd || repack || fwd16) {
        WeightRepack r{th + ni.w_off[1], th + ni.w_off[2], nullptr, nullptr, nullptr, nullptr,
                       tt + ni.w_off[1], tt + ni.w_off[2], nullptr, nullptr, nullptr, nullptr,
                       nullptr, nullptr, nullptr, nullptr};
        if (repack && ni.bf16) {
            r.h2 = t.wpk2;
            r.h3 = t.wpk3;
        } else if (repack) {
            r.x2 = t.wpk2;
            r.x3 = t.wpk3;
        }
        if (fwd16) {
            r.f2a = t.fpk[0][0];
            r.f3a = t.fpk[1][0];
            r.f2b = t.fpk[0][1];
            r.f3b = t.fpk[1][1];
        }
        if (repack_fwd) {
            r.p2a = t.fpk[0][0];
            r.p3a = t.fpk[1][0];
            r.p2b = t.fpk[0][1];
            r.p3b = t.fpk[1][1];
        }
        RUN(DQN_K_WEIGHT_REPACK, launch_weight_repack(r, st));   // (every copy in one launch)
    }

    // Forward of s under theta (samples 0..B-1) and of s' under theta^-
    // (samples B..2B-1): one launch per layer, or both conv layers of the
    // small network in one launch at small batch.
    const bool fusion = g_fusion.load(std::memory_order_relaxed);
    const bool fused_fwd = fusion && L == 2 && conv_s12_fwd_supported(ni.conv[0], ni.conv[1]) &&
                           2 * B <= kFuseMaxRows && conv_s12_fwd_aligned(s0) && conv_s12_fwd_aligned(sn0);
    if (fused_fwd)
        RUN(DQN_K_CONV12_FWD,
            launch_conv_s12_fwd(s0, sn0, B, 2 * B, th + ni.w_off[0], th + ni.b_off[0], th + ni.w_off[1],
                                th + ni.b_off[1], tt + ni.w_off[0], tt + ni.b_off[0], tt + ni.w_off[1],
                                tt + ni.b_off[1], t.act[0], t.act[1], src.replay ? &side : nullptr, st));
    for (int l = 0; l < L && !fused_fwd; ++l) {
        const int64_t ae = l > 0 ? act_elems(ni.d[l - 1]) : 0;
        if (l == 0 && conv1_u8(ni.conv[0], 2 * B, ni.bf16) && conv_s12_fwd_aligned(s0) &&
            conv_s12_fwd_aligned(sn0)) {
            RUN(DQN_K_CONV1_FWD,
                launch_conv1_u8_fwd(CONV_L1, s0, sn0, B, 2 * B, th + ni.w_off[0], th + ni.b_off[0],
                                    tt + ni.w_off[0], tt + ni.b_off[0], t.act[0],
                                    src.replay ? &side : nullptr, ni.bf16, a16, st));
            continue;
        }
        if (l > 0 && igemm_fwd(ni.conv[l], 2 * B, ni.bf16)) {
            RUN(DQN_K_CONV1_FWD + l,
                launch_conv_igemm_fwd(ni.conv[l], t.act[l - 1], B, 2 * B, th + ni.w_off[l], th + ni.b_off[l],
                                      tt + ni.w_off[l], tt + ni.b_off[l], t.act[l], ni.bf16, a16, a16,
                                      repack_fwd || fwd16 ? t.fpk[l - 1][0] : nullptr,
                                      repack_fwd || fwd16 ? t.fpk[l - 1][1] : nullptr,
                                      st));
            continue;
        }
        if (ni.bf16) return DQN_EUNSUPPORTED;  // the per-layer kernels are fp32 only
        const ConvIn in_a = l == 0 ? s0 : ConvIn{t.act[l - 1], nullptr, ae * 4, 0};
        const ConvIn in_b = l == 0 ? sn0 : ConvIn{t.act[l - 1] + (int64_t)B * ae, nullptr, ae * 4, 0};
        const float scale = l == 0 ? (float)(1.0 / 255.0) : 1.f;
        RUN(DQN_K_CONV1_FWD + l,
            launch_conv_fwd(ni.conv[l], in_a, in_b, B, 2 * B, th + ni.w_off[l], th + ni.b_off[l],
                            tt + ni.w_off[l], tt + ni.b_off[l], t.act[l], scale,
                            l == 0 && src.replay ? &side : nullptr, st));
    }
    const float* xlast = t.act[L - 1];
    // s' rows of the last conv output (bfloat16 elements when a16)
    const float* xlast_b = a16 ? (const float*)((const __bf16*)xlast + (int64_t)B * ni.flat)
                               : xlast + (int64_t)B * ni.flat;
    const int64_t slice = (int64_t)2 * B * ni.H;
    if (tt == th) {
        RUN(DQN_K_FC1_FWD,
            launch_gemm(GEMM_NT, 2 * B, ni.H, ni.flat, xlast, ni.flat, th + ni.w_off[L], ni.flat,
                        t.fc1p, ni.H, t.ks, t.kchunk, slice, nullptr, ni.bf16, a16, st));
    } else {
        RUN(DQN_K_FC1_FWD,
            launch_gemm_fwd2(B, ni.H, ni.flat, xlast, th + ni.w_off[L], t.fc1p, xlast_b,
                             tt + ni.w_off[L], t.fc1p + (int64_t)B * ni.H, ni.flat, ni.flat, ni.H, t.ks,
                             t.kchunk, slice, ni.bf16, a16, st));
    }
    HeadTdArgs h{};
    h.fc1p = t.fc1p;
    h.ks = t.ks;
    h.B = B;
    h.b1 = th + ni.b_off[L];
    h.b1t = tt + ni.b_off[L];
    h.W2 = th + ni.w_off[L + 1];
    h.b2 = th + ni.b_off[L + 1];
    h.W2t = tt + ni.w_off[L + 1];
    h.b2t = tt + ni.b_off[L + 1];
    h.action = action;
    h.reward = reward;
    h.terminal = terminal;
    h.gamma = gamma;
    h.h1s = t.h1s;
    h.dz1 = t.dz1;
    h.delta = t.delta;
    h.lossj = t.lossj;
    h.q_out = q_out;
    h.y_out = y_out;
    h.dz1h = t.dz1h;
    RUN(DQN_K_HEAD, launch_head_td(ni.H, ni.A, h, st));

    // fc1: weight gradient and the masked gradient of the last conv output;
    // then the conv layers, last to first.  At small batch each layer's two
    // independent backward kernels share one launch.
    // Up to 512 samples (one or two per input-gradient workgroup) the fp32
    // input-gradient kernels load their weights from a copy in per-lane order
    // instead of gathering 64 / 144 scattered words per lane.
    const bool paired = B <= kPairMaxBatch;
    if (paired) {
        RUN(DQN_K_FC1_BWD,
            launch_gemm_wgrad_dgrad(ni.H, ni.flat, B, t.dz1, xlast, grad_out + ni.w_off[L],
                                    th + ni.w_off[L], t.dconv[L - 1], ni.bf16, st));
    } else {
        // the bf16-input variant reads the head's bfloat16 copy of dz1 (the
        // same rounding the staging would apply)
        const float* dzA = t.dz1h ? (const float*)t.dz1h : t.dz1;
        if (t.fc1w_part) {   // k-slices of ceil(B / 128) * 64 samples (the last one at most that)
            constexpr int S = kGemmX6WgradSlices;
            RUN(DQN_K_FC1_WGRAD,
                launch_gemm(GEMM_TN, ni.H, ni.flat, B, t.dz1, ni.H, xlast, ni.flat, t.fc1w_part, ni.flat, S,
                            (B + 64 * S - 1) / (64 * S) * 64, (int64_t)ni.H * ni.flat, nullptr, false, false, st));
        } else {
            RUN(DQN_K_FC1_WGRAD,
                launch_gemm(GEMM_TN, ni.H, ni.flat, B, dzA, ni.H, xlast, ni.flat, grad_out + ni.w_off[L], ni.flat, 1,
                            (B + 31) / 32 * 32, 0, nullptr, ni.bf16, a16, st, t.dz1h != nullptr));
        }
        RUN(DQN_K_FC1_DGRAD,
            launch_gemm(GEMM_NN, B, ni.flat, ni.H, dzA, ni.H, th + ni.w_off[L], ni.flat, t.dconv[L - 1], ni.flat, 1,
                        (ni.H + 31) / 32 * 32, 0, xlast, ni.bf16, a16, st, t.dz1h != nullptr));
    }
    // The small network's conv layers in one launch: conv2's weight gradient,
    // and conv2's input gradient with conv1's weight gradient per (sample,
    // band of conv1 rows).
    const bool fused_bwd = fusion && L == 2 && conv_s12_fwd_supported(ni.conv[0], ni.conv[1]) &&
                           B <= kFuseMaxRows && conv_s12_fwd_aligned(s0);
    int chunks_used[3] = {t.chunks[0], t.chunks[1], t.chunks[2]};
    int& chunks0 = chunks_used[0];
    if (fused_bwd) {
        RUN(DQN_K_CONV12_BWD,
            launch_conv_s12_bwd(s0, t.act[0], t.dconv[1], th + ni.w_off[1], B, t.wpart[1], t.bpart[1],
                                t.wpart[0], t.bpart[0], st));
        chunks0 = conv_s12_bwd_slots(B);
    }
    // The bf16-input variant of the large network carries conv1's output
    // gradient in bfloat16 (the rounding its weight gradient applies anyway);
    // conv2's input-gradient kernel then also sums conv1's bias gradient
    // from the float32 values, in the same per-workgroup slots.
    const bool dz16_0 = !fused_bwd && ni.bf16 && a16 && L == 3 && conv1_u8(ni.conv[0], B, true) &&
                        conv_s12_fwd_aligned(s0) && phase_dgrad(ni.conv[1], B, true) &&
                        conv2_dgrad_phase_blocks(B) == conv1_u8_wgrad_slots(B);
    for (int l = L - 1; l >= 0 && !fused_bwd; --l) {
        const ConvIn in = l == 0 ? s0 : ConvIn{t.act[l - 1], nullptr, act_elems(ni.d[l - 1]) * 4, 0};
        const float scale = l == 0 ? (float)(1.0 / 255.0) : 1.f;
        if (l > 0 && paired && !ni.bf16) {
            RUN(DQN_K_CONV2_BWD + (l - 1),
                launch_conv_bwd(ni.conv[l], in, t.dconv[l], B, t.wpart[l], t.bpart[l],
                                th + ni.w_off[l], t.act[l - 1], t.dconv[l - 1], st));
            continue;
        }
        if (l == 0 && conv1_u8(ni.conv[0], B, ni.bf16) && conv_s12_fwd_aligned(s0)) {
            RUN(DQN_K_CONV1_WGRAD,
                launch_conv1_u8_wgrad(CONV_L1, s0, t.dconv[0], B, t.wpart[0], t.bpart[0], scale, ni.bf16, st,
                                      dz16_0));
            chunks_used[0] = conv1_u8_wgrad_slots(B);
        } else if (reg_wgrad(ni.conv[l], B, ni.bf16)) {
            RUN(DQN_K_CONV1_WGRAD + l,
                launch_conv_wgrad_reg(ni.conv[l], t.act[l - 1], t.dconv[l], B, t.wpart[l], t.bpart[l], ni.bf16,
                                      a16, st));
            chunks_used[l] = conv_wgrad_reg_slots(ni.conv[l], B, ni.bf16);
        } else if (igemm_wgrad(ni.conv[l], B, ni.bf16)) {
            RUN(DQN_K_CONV1_WGRAD + l,
                launch_conv_igemm_wgrad(ni.conv[l], in, t.dconv[l], B, t.wpart[l], t.bpart[l], scale,
                                        ni.bf16, st));
            chunks_used[l] = conv_igemm_wgrad_chunks(ni.conv[l], B);
        } else {
            if (ni.bf16) return DQN_EUNSUPPORTED;  // the per-layer kernels are fp32 only
            RUN(DQN_K_CONV1_WGRAD + l,
                launch_conv_wgrad(ni.conv[l], in, t.dconv[l], B, t.wpart[l], t.bpart[l], scale, st));
        }
        if (l > 0 && phase_dgrad(ni.conv[l], B, ni.bf16))
            RUN(DQN_K_CONV2_DGRAD + (l - 1),
                ni.conv[l] == CONV_L2
                    ? launch_conv2_dgrad_phase(t.dconv[l], th + ni.w_off[l], t.act[l - 1], t.dconv[l - 1], B,
                                               ni.bf16, a16, repack ? t.wpk2 : nullptr, st,
                                               dz16_0 ? (__bf16*)t.dconv[0] : nullptr,
                                               dz16_0 ? t.bpart[0] : nullptr)
                    : launch_conv3_dgrad(t.dconv[l], th + ni.w_off[l], t.act[l - 1], t.dconv[l - 1], B,
                                         ni.bf16, a16, repack ? t.wpk3 : nullptr, st));
        else if (l > 0 && igemm_dgrad(ni.conv[l], B, ni.bf16))
            RUN(DQN_K_CONV2_DGRAD + (l - 1),
                launch_conv_igemm_dgrad(ni.conv[l], t.dconv[l], th + ni.w_off[l], t.act[l - 1],
                                        t.dconv[l - 1], B, ni.bf16, st));
        else if (l > 0)
            RUN(DQN_K_CONV2_DGRAD + (l - 1),
                launch_conv_dgrad(ni.conv[l], t.dconv[l], th + ni.w_off[l], t.act[l - 1],
                                  t.dconv[l - 1], B, st));
    }
    FinalizeArgs fa{};
    fa.n_conv = L;
    for (int l = 0; l < L; ++l) {
        const ConvDims& c = ni.d[l];
        fa.wpart[l] = t.wpart[l];
        fa.bpart[l] = t.bpart[l];
        fa.chunks[l] = chunks_used[l];
        fa.wcount[l] = c.cout * c.cin * c.k * c.k;
        fa.cout[l] = c.cout;
        fa.gw[l] = grad_out + ni.w_off[l];
        fa.gb[l] = grad_out + ni.b_off[l];
    }
    fa.dz1 = t.dz1;
    fa.h1s = t.h1s;
    fa.delta = t.delta;
    fa.lossj = t.lossj;
    fa.action = action;
    fa.B = B;
    fa.H = ni.H;
    fa.A = ni.A;
    fa.g_b1 = grad_out + ni.b_off[L];
    fa.g_W2 = grad_out + ni.w_off[L + 1];
    fa.g_b2 = grad_out + ni.b_off[L + 1];
    fa.loss_out = loss_out;
    fa.grad_base = grad_out;
    fa.fc1w_off = ni.w_off[L];
    fa.fc1w_count = (int64_t)ni.H * ni.flat;
    fa.fc1w_part = t.fc1w_part;
    fa.fc1w_slices = t.fc1w_part ? kGemmX6WgradSlices : 0;
    fa.spart = t.spart;
    fa.schunks = finalize_sample_chunks(B);
    if (upd)
        RUN(DQN_K_FINALIZE_APPLY, launch_finalize(fa, upd, st));
    else
        RUN(DQN_K_FINALIZE, launch_finalize(fa, nullptr, st));
    return DQN_OK;
}

// Host checks of a replay descriptor shared by the gather and the fused TD step.
int check_replay(const dqn_replay* rp, bool with_next) {
    if (!rp || !rp->frames || rp->c <= 0 || rp->h <= 0 || rp->w <= 0) return DQN_EINVAL;
    const int64_t rec = (int64_t)rp->c * rp->h * rp->w;
    if (rec % 16 != 0 || rp->record_stride < rec || rp->record_stride % 16 != 0) return DQN_EINVAL;
    if (!aligned(rp->frames, 16)) return DQN_EINVAL;
    if (rp->size < (with_next ? 2 : 1)) return DQN_EINVAL;
    return DQN_OK;
}

}  // namespace


namespace dqn {

int td_step_replay(const dqn_net* net, const float* theta_target, const dqn_replay* replay,
                   const int64_t* idx, int32_t batch, float gamma, float* grad_ws, float* loss_out,
                   const PsUpdate& upd, void* ws, size_t ws_bytes, hipStream_t st) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    rc = check_replay(replay, true);
    if (rc != DQN_OK) return rc;
    if (!idx || !replay->action || !replay->reward || !replay->terminal) return DQN_EINVAL;
    if (replay->c != net->in_c || replay->h != net->in_h || replay->w != net->in_w) return DQN_EINVAL;
    if (upd.rule != PS_SGD && upd.rule != PS_RMSPROP && upd.rule != PS_ADAGRAD) return DQN_EINVAL;
    if (!upd.theta || (upd.rule != PS_SGD && !upd.state)) return DQN_EINVAL;
    if (upd.state && !aligned(upd.state, 16)) return DQN_EINVAL;
    if (!std::isfinite(upd.lr) || !std::isfinite(upd.decay) || !std::isfinite(upd.eps)) return DQN_EINVAL;
    const size_t pb = (size_t)ni.P * sizeof(float);
    if (upd.state && (overlaps(upd.state, pb, upd.theta, pb) || (grad_ws && overlaps(upd.state, pb, grad_ws, pb))))
        return DQN_EINVAL;
    TdSource src{nullptr, nullptr, nullptr, nullptr, nullptr, replay, idx};
    return td_gradient_impl(net, ni, upd.theta, theta_target, src, batch, gamma, grad_ws, loss_out,
                            nullptr, nullptr, ws, ws_bytes, st, &upd);
}

}  // namespace dqn

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_dev[kMaxDevices];
std::mutex g_scratch_mu;

// The scratch address on the current device (looked up on the first call on
// that device).  The stream must belong to the current device.
int scratch_on_current_device(hipStream_t st, void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return DQN_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return DQN_EUNSUPPORTED;
    if (st) {
        hipDevice_t sdev = -1;
        if (hipStreamGetDevice(st, &sdev) != hipSuccess) return DQN_EHIP;
        if (sdev != dev) return DQN_EINVAL;
    }
    void* p = g_scratch_dev[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_dev[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DQN_EHIP;
            if ((uintptr_t)p % 256 != 0) return DQN_EHIP;
            g_scratch_dev[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return DQN_OK;
}

}  // namespace

extern "C" {

const char* dqn_status_string(int status) {
    switch (status) {
        case DQN_OK: return "ok";
        case DQN_EINVAL: return "invalid argument";
        case DQN_EWORKSPACE: return "workspace too small";
        case DQN_EHIP: return "HIP launch failed";
        case DQN_EUNSUPPORTED: return "unsupported network";
        default: return "unknown status";
    }
}

int64_t dqn_param_count(const dqn_net* net) {
    NetInfo ni;
    int rc = identify(net, &ni);
    return rc != DQN_OK ? rc : ni.P;
}

int64_t dqn_param_offset(const dqn_net* net, int32_t layer, int32_t is_bias) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    if (layer < 0 || layer > ni.n_conv + 1) return DQN_EINVAL;
    return is_bias ? ni.b_off[layer] : ni.w_off[layer];
}

int64_t dqn_workspace_bytes(const dqn_net* net, int32_t batch, int32_t op) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    if (batch <= 0) return DQN_EINVAL;
    if (op == DQN_OP_FORWARD) return (int64_t)fwd_layout(ni, batch, nullptr).bytes;
    if (op == DQN_OP_TD_GRADIENT) return (int64_t)td_layout(ni, batch, nullptr).bytes;
    return DQN_EINVAL;
}

int replay_gather(const dqn_replay* rp, const int64_t* idx, int32_t batch, uint8_t* s_out,
                  uint8_t* s_next_out, int32_t* a_out, float* r_out, uint8_t* term_out,
                  void* stream) {
    if (!idx || !s_out || batch <= 0) return DQN_EINVAL;
    const int vr = check_replay(rp, s_next_out != nullptr);
    if (vr != DQN_OK) return vr;
    const int64_t rec = (int64_t)rp->c * rp->h * rp->w;
    if (!aligned(s_out, 16) || (s_next_out && !aligned(s_next_out, 16))) return DQN_EINVAL;
    if ((a_out && !rp->action) || (r_out && !rp->reward) || (term_out && !rp->terminal))
        return DQN_EINVAL;
    if (batch > 65535) return DQN_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    RUN(DQN_K_GATHER, launch_gather(rp->frames, rp->record_stride, rec, rp->action, rp->reward,
                                    rp->terminal, idx, batch, s_out, s_next_out, a_out, r_out,
                                    term_out, st));
    return DQN_OK;
}

int replay_gather_validate(const dqn_replay* rp, const int64_t* idx, int32_t batch, int32_t with_next,
                           int32_t* bad_count, void* stream) {
    if (!rp || !idx || !bad_count || batch <= 0) return DQN_EINVAL;
    if (rp->size < (with_next ? 2 : 1)) return DQN_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    if (launch_validate(idx, batch, rp->size - (with_next ? 2 : 1), bad_count, st) != hipSuccess) return DQN_EHIP;
    return DQN_OK;
}

}  // extern "C"

namespace {

// The forward pass of dqn_forward / dqn_forward_replay on layer-0 input in0.
int forward_impl(const dqn_net* net, const NetInfo& ni, const float* theta, const ConvIn& in0, int32_t batch,
                 float epsilon, const uint64_t* draws, float* q_out, int32_t* action_out, void* ws,
                 size_t ws_bytes, hipStream_t st) {
    if (!theta || batch <= 0 || !ws) return DQN_EINVAL;
    if (!(epsilon >= 0.f && epsilon <= 1.f)) return DQN_EINVAL;
    const double te = std::floor((double)epsilon * 4294967296.0);
    const uint64_t thresh = te >= 4294967296.0 ? 4294967296ull : (uint64_t)te;
    if (thresh > 0 && !draws) return DQN_EINVAL;
    if (!aligned(ws, 256) || !aligned(theta, 16)) return DQN_EINVAL;
    FwdLayout f = fwd_layout(ni, batch, nullptr);
    if (ws_bytes < f.bytes) return DQN_EWORKSPACE;
    f = fwd_layout(ni, batch, ws);
    const float* th = theta;
    const bool fused_fwd = g_fusion.load(std::memory_order_relaxed) && ni.n_conv == 2 && conv_s12_fwd_supported(ni.conv[0], ni.conv[1]) &&
                           batch <= kFuseMaxRows && conv_s12_fwd_aligned(in0);
    if (fused_fwd)
        RUN(DQN_K_CONV12_FWD,
            launch_conv_s12_fwd(in0, in0, batch, batch, th + ni.w_off[0], th + ni.b_off[0],
                                th + ni.w_off[1], th + ni.b_off[1], th + ni.w_off[0], th + ni.b_off[0],
                                th + ni.w_off[1], th + ni.b_off[1], f.act[0], f.act[1], nullptr, st));
    // bfloat16 storage of the conv layers' outputs, as in the TD step
    const bool a16 = ni.bf16 && ni.n_conv == 3 && batch >= kFwdClMinRows;
    for (int l = 0; l < ni.n_conv && !fused_fwd; ++l) {
        if (l == 0 && conv1_u8(ni.conv[0], batch, ni.bf16) && conv_s12_fwd_aligned(in0)) {
            RUN(DQN_K_CONV1_FWD,
                launch_conv1_u8_fwd(CONV_L1, in0, in0, batch, batch, th + ni.w_off[0], th + ni.b_off[0],
                                    th + ni.w_off[0], th + ni.b_off[0], f.act[0], nullptr, ni.bf16, a16, st));
            continue;
        }
        if (l > 0 && igemm_fwd(ni.conv[l], batch, ni.bf16)) {
            RUN(DQN_K_CONV1_FWD + l,
                launch_conv_igemm_fwd(ni.conv[l], f.act[l - 1], batch, batch, th + ni.w_off[l], th + ni.b_off[l],
                                      th + ni.w_off[l], th + ni.b_off[l], f.act[l], ni.bf16, a16, a16, nullptr,
                                      nullptr, st));
            continue;
        }
        if (ni.bf16) return DQN_EUNSUPPORTED;  // the per-layer kernels are fp32 only
        const ConvIn in = l == 0 ? in0
                                 : ConvIn{f.act[l - 1], nullptr, act_elems(ni.d[l - 1]) * 4, 0};
        const float scale = l == 0 ? (float)(1.0 / 255.0) : 1.f;
        RUN(DQN_K_CONV1_FWD + l,
            launch_conv_fwd(ni.conv[l], in, in, batch, batch, th + ni.w_off[l], th + ni.b_off[l],
                            th + ni.w_off[l], th + ni.b_off[l], f.act[l], scale, nullptr, st));
    }
    const int L = ni.n_conv;
    RUN(DQN_K_FC1_FWD,
        launch_gemm(GEMM_NT, batch, ni.H, ni.flat, f.act[L - 1], ni.flat, th + ni.w_off[L], ni.flat,
                    f.fc1p, ni.H, f.ks, f.kchunk, (int64_t)batch * ni.H, nullptr, ni.bf16, a16, st));
    HeadFwdArgs h{};
    h.fc1p = f.fc1p;
    h.ks = f.ks;
    h.B = batch;
    h.b1 = th + ni.b_off[L];
    h.W2 = th + ni.w_off[L + 1];
    h.b2 = th + ni.b_off[L + 1];
    h.thresh = thresh;
    h.draws = draws;
    h.q_out = q_out;
    h.action_out = action_out;
    RUN(DQN_K_HEAD, launch_head_fwd(ni.H, ni.A, h, st));
    return DQN_OK;
}

}  // namespace

extern "C" {

int dqn_forward(const dqn_net* net, const float* theta, const uint8_t* states, int32_t batch,
                float epsilon, const uint64_t* draws, float* q_out, int32_t* action_out, void* ws,
                size_t ws_bytes, void* stream) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    if (!states || !aligned(states, 16)) return DQN_EINVAL;
    const ConvIn in0{states, nullptr, (int64_t)net->in_c * net->in_h * net->in_w, 0};
    return forward_impl(net, ni, theta, in0, batch, epsilon, draws, q_out, action_out, ws, ws_bytes,
                        (hipStream_t)stream);
}

int dqn_forward_replay(const dqn_net* net, const float* theta, const dqn_replay* replay, const int64_t* idx,
                       int32_t batch, float epsilon, const uint64_t* draws, float* q_out, int32_t* action_out,
                       void* ws, size_t ws_bytes, void* stream) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    rc = check_replay(replay, false);
    if (rc != DQN_OK) return rc;
    if (!idx) return DQN_EINVAL;
    if (replay->c != net->in_c || replay->h != net->in_h || replay->w != net->in_w) return DQN_EINVAL;
    const ConvIn in0{replay->frames, idx, replay->record_stride, 0};
    return forward_impl(net, ni, theta, in0, batch, epsilon, draws, q_out, action_out, ws, ws_bytes,
                        (hipStream_t)stream);
}

int dqn_td_gradient(const dqn_net* net, const float* theta, const float* theta_target,
                    const uint8_t* s, const uint8_t* s_next, const int32_t* action,
                    const float* reward, const uint8_t* terminal, int32_t batch, float gamma,
                    float* grad_out, float* loss_out, float* q_out, float* y_out, void* ws,
                    size_t ws_bytes, void* stream) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    if (!s || !s_next || !action || !reward || !terminal) return DQN_EINVAL;
    if (!aligned(s, 16) || !aligned(s_next, 16)) return DQN_EINVAL;
    TdSource src{s, s_next, action, reward, terminal, nullptr, nullptr};
    return td_gradient_impl(net, ni, theta, theta_target, src, batch, gamma, grad_out, loss_out,
                            q_out, y_out, ws, ws_bytes, (hipStream_t)stream);
}

int dqn_td_gradient_noalloc(const dqn_net* net, const float* theta, const float* theta_target,
                            const uint8_t* s, const uint8_t* s_next, const int32_t* action,
                            const float* reward, const uint8_t* terminal, int32_t batch, float gamma,
                            float* grad_out, float* loss_out, float* q_out, float* y_out, void* stream) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    if (!s || !s_next || !action || !reward || !terminal) return DQN_EINVAL;
    if (!aligned(s, 16) || !aligned(s_next, 16)) return DQN_EINVAL;
    if (batch <= 0) return DQN_EINVAL;
    // Reject a batch whose workspace exceeds the scratch before touching it.
    if (td_layout(ni, batch, nullptr).bytes > kNoAllocScratchBytes) return DQN_EWORKSPACE;
    const hipStream_t st = (hipStream_t)stream;
    void* ws = nullptr;
    rc = scratch_on_current_device(st, &ws);
    if (rc != DQN_OK) return rc;
    TdSource src{s, s_next, action, reward, terminal, nullptr, nullptr};
    return td_gradient_impl(net, ni, theta, theta_target, src, batch, gamma, grad_out, loss_out,
                            q_out, y_out, ws, kNoAllocScratchBytes, st);
}

int dqn_td_gradient_replay(const dqn_net* net, const float* theta, const float* theta_target,
                           const dqn_replay* replay, const int64_t* idx, int32_t batch, float gamma,
                           float* grad_out, float* loss_out, float* q_out, float* y_out, void* ws,
                           size_t ws_bytes, void* stream) {
    NetInfo ni;
    int rc = identify(net, &ni);
    if (rc != DQN_OK) return rc;
    rc = check_replay(replay, true);
    if (rc != DQN_OK) return rc;
    if (!idx || !replay->action || !replay->reward || !replay->terminal) return DQN_EINVAL;
    if (replay->c != net->in_c || replay->h != net->in_h || replay->w != net->in_w) return DQN_EINVAL;
    TdSource src{nullptr, nullptr, nullptr, nullptr, nullptr, replay, idx};
    return td_gradient_impl(net, ni, theta, theta_target, src, batch, gamma, grad_out, loss_out,
                            q_out, y_out, ws, ws_bytes, (hipStream_t)stream);
}

int ps_apply_update(int32_t rule, const float* theta_in, float* theta_out, float* state,
                    const float* grad, int64_t n, float lr, float decay, float eps, void* stream) {
    if (rule != PS_SGD && rule != PS_RMSPROP && rule != PS_ADAGRAD) return DQN_EINVAL;
    if (!theta_in || !theta_out || !grad || n <= 0) return DQN_EINVAL;
    if (rule != PS_SGD && !state) return DQN_EINVAL;
    if (!aligned(theta_in, 16) || !aligned(theta_out, 16) || !aligned(grad, 16) ||
        (state && !aligned(state, 16)))
        return DQN_EINVAL;
    const size_t nb = (size_t)n * sizeof(float);
    if (theta_out != theta_in && overlaps(theta_out, nb, theta_in, nb)) return DQN_EINVAL;
    if (overlaps(grad, nb, theta_out, nb) || (state && overlaps(grad, nb, state, nb)) ||
        (state && overlaps(state, nb, theta_out, nb)))
        return DQN_EINVAL;
    if (!std::isfinite(lr) || !std::isfinite(decay) || !std::isfinite(eps)) return DQN_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    RUN(DQN_K_APPLY, launch_apply(rule, theta_in, theta_out, state, grad, n, lr, decay, eps, st));
    return DQN_OK;
}

int dqn_profile_attach(int32_t kernel, void** events, int32_t n_pairs, int32_t stride) {
    if (kernel < 0 || kernel >= DQN_K_COUNT || n_pairs < 0 || stride < 1) return DQN_EINVAL;
    ProfSlot& p = g_prof[kernel];
    const bool was = p.ev != nullptr;
    p.ev = (events && n_pairs > 0) ? (hipEvent_t*)events : nullptr;
    p.n = p.ev ? n_pairs : 0;
    p.used = 0;
    p.stride = stride;
    p.seen = 0;
    p.open = false;
    if (p.ev && !was) g_prof_attached.fetch_add(1, std::memory_order_relaxed);
    if (!p.ev && was) g_prof_attached.fetch_sub(1, std::memory_order_relaxed);
    return DQN_OK;
}

int dqn_profile_set_fusion(int32_t enabled) {
    g_fusion.store(enabled != 0, std::memory_order_relaxed);
    return DQN_OK;
}

int32_t dqn_profile_used(int32_t kernel) {
    if (kernel < 0 || kernel >= DQN_K_COUNT) return DQN_EINVAL;
    return g_prof[kernel].used;
}

}  // extern "C"
