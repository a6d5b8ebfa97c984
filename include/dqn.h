/*
 * dqn.h -- C ABI of the MI355X (gfx950) DQN hot-path library, libdqn.so.
 *
 * The hot path of distributed deep Q-learning (Ong, Chavez and Hong,
 * arXiv 1508.04186): a worker samples a minibatch of transitions from its
 * replay memory, computes the gradient of the TD loss of its Q-network, and
 * the parameter server applies that gradient (Alg. 1 and Alg. 2).
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless the parameter is a struct passed by
 *    host pointer (dqn_net, dqn_replay), which is read on the host during the
 *    call and not retained.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t passed as
 *    void*; NULL is the default stream).  No entry point allocates, frees or
 *    synchronizes; device memory is owned by the caller.
 *  - Return value: DQN_OK (0) or a negative dqn_status.  Argument checks run
 *    on the host before anything is enqueued; when one fails nothing is
 *    enqueued.  DQN_EHIP reports a failed kernel launch.  Faults inside a
 *    kernel surface at the caller's next synchronization.
 *  - Calls on different streams that write different buffers may overlap.
 *  - Thread safety: the entry points keep no mutable process-wide state, so
 *    they may be called concurrently from several host threads (on their
 *    own streams and buffers).  The only process-wide state is the
 *    measurement hook of dqn_profile.h: while a kernel is attached there,
 *    calls must not race with attach/detach or with each other.
 *
 * Networks (Sec. III.A; Appendix A's figure is not available, so the two
 * supported shapes are fixed here): input 4x84x84 bytes scaled by 1/255,
 * valid-padding convolutions with ReLU, a hidden fully connected layer with
 * ReLU, and a linear output layer with one unit per action.
 *   small: conv 16@8x8/4, conv 32@4x4/2, fc 256, fc 6   (677,686 parameters)
 *   large: conv 32@8x8/4, conv 64@4x4/2, conv 64@3x3/1, fc 512, fc 18
 *          (1,693,362 parameters)
 * Other shapes return DQN_EUNSUPPORTED.
 *
 * Flat parameter layout (float32): for each conv layer W[out][in][k][k] then
 * b[out]; then fc1 W[hidden][flat] and b[hidden]; then fc2 W[actions][hidden]
 * and b[actions].  fc1 reads the last conv output flattened channel-major,
 * flat index = c*H*W + y*W + x.  Gradients use the same layout.
 */
#ifndef DQN_H
#define DQN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DQN_OK = 0,
    DQN_EINVAL = -1,        /* null pointer, bad size, aliasing, misalignment */
    DQN_EWORKSPACE = -2,    /* workspace smaller than dqn_workspace_bytes() */
    DQN_EHIP = -3,          /* a HIP launch failed */
    DQN_EUNSUPPORTED = -4   /* network shape or precision not supported */
} dqn_status;

/* Arithmetic of the layer contractions (dqn_net.precision):
 *   DQN_FP32  float32 operands and accumulation (the first conv layer runs
 *             its byte inputs against an exact three-term bfloat16 split of
 *             each float32 weight, which reproduces float32 products);
 *   DQN_BF16  the bf16-input variant, large network only: every operand of
 *             the conv and fc1 contractions (weights, input activations,
 *             back-propagated gradients) is rounded to bfloat16 (round to
 *             nearest, ties to even) and the products are accumulated in
 *             float32.  Input bytes are exact in bfloat16 and the 1/255 scale
 *             is applied to the float32 sum.  The output layer, the TD target
 *             and loss, bias gradients, ReLU decisions and the update stay
 *             float32.  The small network returns DQN_EUNSUPPORTED. */
enum { DQN_FP32 = 0, DQN_BF16 = 1 };

typedef struct {
    int32_t in_c, in_h, in_w;      /* 4, 84, 84 */
    int32_t n_conv;                /* 2 or 3 */
    int32_t conv_out[3];           /* output channels per conv layer */
    int32_t conv_k[3];             /* square kernel size */
    int32_t conv_stride[3];
    int32_t fc_hidden;             /* 256 or 512 */
    int32_t n_actions;             /* 6 or 18 */
    int32_t precision;             /* DQN_FP32 or DQN_BF16 */
} dqn_net;

/* Replay memory (Sec. III.C): the last N experiences.  Record i holds the
 * stacked preprocessed frames phi_i (c*h*w bytes) at frames + i*record_stride;
 * transition i is (phi_i, action[i], reward[i], terminal[i], phi_{i+1}), so
 * indices 0 .. size-2 are valid; terminal[i] = 1 marks phi_{i+1} terminal. */
typedef struct {
    const uint8_t* frames;     /* device; 16-byte aligned */
    const uint8_t* action;     /* device [size] */
    const int8_t* reward;      /* device [size], clipped game reward */
    const uint8_t* terminal;   /* device [size], 0 or 1 */
    int64_t record_stride;     /* bytes between records; multiple of 16, >= c*h*w */
    int64_t size;              /* number of valid records, >= 2 */
    int32_t c, h, w;           /* record shape; c*h*w must be a multiple of 16 */
} dqn_replay;

/* Parameter-server update rules (ps_apply_update). */
enum {
    PS_SGD = 0,       /* theta <- theta - lr*g */
    PS_RMSPROP = 1,   /* Alg. 2: r <- decay*r + (1-decay)*g^2; theta <- theta - lr*g/sqrt(r) */
    PS_ADAGRAD = 2    /* Sec. IV.D.2: G <- G + g^2; theta <- theta - lr*g/(sqrt(G)+eps) */
};

enum { DQN_OP_FORWARD = 0, DQN_OP_TD_GRADIENT = 1 };

/* Number of float32 parameters of `net`, or a negative dqn_status. */
int64_t dqn_param_count(const dqn_net* net);

/* Element offset of a layer's weight (is_bias = 0) or bias (is_bias = 1) in
 * the flat layout.  Layers: 0 .. n_conv-1 are the convs, n_conv is fc1,
 * n_conv+1 is fc2.  Negative dqn_status on a bad argument. */
int64_t dqn_param_offset(const dqn_net* net, int32_t layer, int32_t is_bias);

/* Bytes of device workspace that dqn_forward (op = DQN_OP_FORWARD) or
 * dqn_td_gradient (op = DQN_OP_TD_GRADIENT) needs for `batch` samples, or a
 * negative dqn_status. */
int64_t dqn_workspace_bytes(const dqn_net* net, int32_t batch, int32_t op);

/* Uniform minibatch draw from the replay memory (Sec. III.C; Alg. 1 "uniformly
 * sample minibatch X from D_k"): for j < batch, with i = idx[j],
 *   s_out[j] = phi_i, s_next_out[j] = phi_{i+1}   (c*h*w bytes each),
 *   a_out[j] = action[i], r_out[j] = reward[i] as float, term_out[j] = terminal[i].
 * idx: device int64 [batch], drawn by the caller; values must lie in
 * [0, size-2] (or [0, size-1] when s_next_out is NULL); they are not checked
 * on the device and an out-of-range value reads out of bounds.
 * s_next_out, a_out, r_out and term_out may each be NULL (not written).
 * Outputs are densely packed [batch][c][h][w]; s_out must be 16-byte aligned. */
int replay_gather(const dqn_replay* replay, const int64_t* idx, int32_t batch,
                  uint8_t* s_out, uint8_t* s_next_out, int32_t* a_out, float* r_out,
                  uint8_t* term_out, void* stream);

/* Check of an index stream before replay_gather, which does not check on
 * the device (Sec. III.C: transition i needs record i+1 when with_next is
 * nonzero): writes to *bad_count (device int32) the number of idx[0..batch)
 * outside [0, size-2] (with_next != 0) or [0, size-1] (with_next == 0).
 * Only replay->size is read.  DQN_EINVAL for null pointers, batch <= 0 or a
 * replay too small for any valid index. */
int replay_gather_validate(const dqn_replay* replay, const int64_t* idx, int32_t batch, int32_t with_next,
                           int32_t* bad_count, void* stream);

/* Setup, not part of the method: fills the replay memory that `replay`
 * describes (records 0 .. size-1 and the side arrays; the call writes through
 * its pointers) with a seeded synthetic stream standing in for preprocessed
 * game frames (Sec. III.A).  Record i stacks stream frames i .. i+c-1; a frame
 * is 84 x 84 bytes: noise uniform on 0..8 under one to four bright moving
 * rectangles (a fresh set every 100 frames).  Every byte and side field is a
 * pure function of (seed, frame, pixel) or (seed, record) through
 * SplitMix64's output mix of seed + 0x9E3779B97F4A7C15 * ((stream << 40) |
 * counter); side fields: action = bounded(H(3, i), n_actions), reward =
 * bounded(H(4, i), 3) - 1, terminal iff (H(5, i) >> 32) < floor(0.01 * 2^32),
 * with bounded(h, n) = ((h >> 32) * n) >> 32.  Requires h = w = 84, c >= 1,
 * n_actions in 1..256, the frames pointer 16-byte aligned and record_stride a
 * multiple of 16 of at least c*84*84. */
int replay_fill_synthetic(const dqn_replay* replay, int32_t n_actions, uint64_t seed, void* stream);

/* Q-network forward pass and epsilon-greedy action choice (Sec. II.A,
 * Sec. III.A-B; Alg. 1 "select action").
 * states: uint8 [batch][4][84][84]; theta: flat parameters.
 * q_out: float [batch][A], may be NULL.  action_out: int32 [batch], may be
 * NULL.  The greedy action is the lowest index attaining the maximum of the
 * float32 Q values written to q_out.  With epsilon > 0, draws (uint64
 * [batch], uniform bits supplied by the caller) decide exploration: state j
 * explores iff (draws[j] >> 32) < floor(epsilon * 2^32) (computed on the host
 * in double from the float epsilon) and then takes action
 * ((draws[j] & 0xffffffff) * A) >> 32.  epsilon must lie in [0, 1]; draws may
 * be NULL only when epsilon == 0.
 * ws: device workspace of at least dqn_workspace_bytes(net, batch, DQN_OP_FORWARD)
 * bytes, 256-byte aligned; its contents are scratch. */
int dqn_forward(const dqn_net* net, const float* theta, const uint8_t* states, int32_t batch,
                float epsilon, const uint64_t* draws, float* q_out, int32_t* action_out,
                void* ws, size_t ws_bytes, void* stream);

/* The same forward pass and action choice on states read in place from the
 * replay memory: state j is phi_i of record i = idx[j], the bytes
 * replay_gather would copy to s_out[j], read by the first convolution
 * instead of being copied first.  idx: device int64 [batch] with values in
 * [0, size-1] (not checked on the device; an out-of-range value reads out of
 * bounds; replay_gather_validate checks them).  The replay record shape must
 * equal the network input.  Outputs, epsilon, draws, workspace
 * (DQN_OP_FORWARD) and errors as dqn_forward. */
int dqn_forward_replay(const dqn_net* net, const float* theta, const dqn_replay* replay,
                       const int64_t* idx, int32_t batch, float epsilon, const uint64_t* draws,
                       float* q_out, int32_t* action_out, void* ws, size_t ws_bytes, void* stream);

/* Worker minibatch gradient (Alg. 1; Eq. (1)):
 *   y_j = r_j                                          if terminal_j,
 *   y_j = r_j + gamma * max_a' Q(s_next_j, a'; theta_target)   otherwise;
 *   loss = (1/B) sum_j 1/2 (Q(s_j, a_j; theta) - y_j)^2;
 *   grad_out = d loss / d theta, with y held constant (no gradient flows
 *   through the target network, even when theta_target == theta).
 * theta_target may equal theta or be NULL (then theta is used).
 * s, s_next: uint8 [batch][4][84][84]; action int32 [batch] in [0, A);
 * reward float [batch]; terminal uint8 [batch].  An action outside [0, A)
 * is clamped into that range.
 * Outputs: grad_out float [p] (overwritten, never accumulated), loss_out
 * float [1]; optional q_out float [batch][A] = Q(s_j, .; theta) and y_out
 * float [batch] (NULL to skip).  grad_out must not overlap theta or
 * theta_target.  Deterministic: the same inputs give bitwise-identical
 * outputs.
 * ws: at least dqn_workspace_bytes(net, batch, DQN_OP_TD_GRADIENT) bytes,
 * 256-byte aligned; scratch. */
int dqn_td_gradient(const dqn_net* net, const float* theta, const float* theta_target,
                    const uint8_t* s, const uint8_t* s_next, const int32_t* action,
                    const float* reward, const uint8_t* terminal, int32_t batch, float gamma,
                    float* grad_out, float* loss_out, float* q_out, float* y_out,
                    void* ws, size_t ws_bytes, void* stream);

/* dqn_td_gradient for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving or training loops, harnesses that forbid
 * hipMalloc): the same arguments without a workspace, the same kernels and
 * bitwise the same outputs.  The workspace is the library's own static
 * device array of 64 MiB, one per GPU, held from the library's load on that
 * GPU until the process ends; the call allocates and frees nothing.
 * The batch is limited by that size: when dqn_workspace_bytes(net, batch,
 * DQN_OP_TD_GRADIENT) exceeds 64 MiB the call returns DQN_EWORKSPACE and
 * enqueues nothing.  Every batch up to 289 samples fits for the small
 * network, up to 100 for the large one and up to 93 for its bf16-input
 * variant.  The array needs no clearing between calls (every call writes
 * what it reads).  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (concurrent streams or host threads) race, so serialize
 * them.  The stream must belong to the current device (else DQN_EINVAL).
 * The first call on a device looks up the array's address there
 * (hipGetSymbolAddress); make that first call outside graph capture. */
int dqn_td_gradient_noalloc(const dqn_net* net, const float* theta, const float* theta_target,
                            const uint8_t* s, const uint8_t* s_next, const int32_t* action,
                            const float* reward, const uint8_t* terminal, int32_t batch, float gamma,
                            float* grad_out, float* loss_out, float* q_out, float* y_out,
                            void* stream);

/* The same gradient with the minibatch drawn from the replay memory in the
 * same call (Alg. 1: "uniformly sample minibatch X from D_k", then the
 * gradient): transition j is idx[j] of `replay`, exactly as replay_gather
 * would deliver it (s_j = phi_i, s_next_j = phi_{i+1}, a, r, terminal of
 * record i = idx[j]), but the records are read in place by the first
 * convolution instead of being copied first.  idx: device int64 [batch] with
 * values in [0, size-2] (not checked on the device; an out-of-range value
 * reads out of bounds).  The replay record shape must equal the network
 * input (4x84x84).  Outputs, workspace (dqn_workspace_bytes with
 * DQN_OP_TD_GRADIENT) and errors as dqn_td_gradient. */
int dqn_td_gradient_replay(const dqn_net* net, const float* theta, const float* theta_target,
                           const dqn_replay* replay, const int64_t* idx, int32_t batch, float gamma,
                           float* grad_out, float* loss_out, float* q_out, float* y_out, void* ws,
                           size_t ws_bytes, void* stream);

/* Parameter-server update applied to one received gradient (Alg. 2
 * RMSPROPUPDATE; plain gradient descent of Sec. III.B; AdaGrad of
 * Sec. IV.D.2), elementwise over n float32 parameters:
 *   PS_SGD:     theta_out = theta_in - lr*g                       (state unused, may be NULL)
 *   PS_RMSPROP: r = decay*r + (1-decay)*g^2 (new r stored in state);
 *               theta_out = theta_in - lr*g/sqrt(r), or theta_in where r == 0
 *               (Alg. 2 has no epsilon; eps is ignored)
 *   PS_ADAGRAD: G = G + g^2 (stored in state);
 *               theta_out = theta_in - lr*g/(sqrt(G) + eps)
 * theta_out may equal theta_in (in place) or be a separate buffer (an
 * out-of-place new parameter version); grad must not overlap theta_out or
 * state.  All pointers 16-byte aligned. */
int ps_apply_update(int32_t rule, const float* theta_in, float* theta_out, float* state,
                    const float* grad, int64_t n, float lr, float decay, float eps,
                    void* stream);

/* Human-readable name of a dqn_status value (static string). */
const char* dqn_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* DQN_H */
