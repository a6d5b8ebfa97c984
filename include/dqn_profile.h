/*
 * dqn_profile.h -- measurement hook of libdqn.so.
 *
 * Lets a benchmark time one internal kernel of the hot path with HIP events
 * recorded on the stream that kernel runs on.  Not needed for normal use.
 *
 * dqn_profile_attach(kernel, events, n_pairs, stride): from now on, every
 * stride-th launch of `kernel` (launches 0, stride, 2*stride, ... counted
 * from the attach) is bracketed by hipEventRecord(events[2*i]) before and
 * hipEventRecord(events[2*i+1]) after, for i = 0, 1, ... up to n_pairs - 1;
 * later launches are not bracketed.  `events` is a host array of hipEvent_t
 * created by the caller; it must stay valid while attached.  Pass
 * events = NULL (or n_pairs = 0) to detach.  stride >= 1.  Returns DQN_OK or
 * DQN_EINVAL.
 * dqn_profile_used(kernel): number of pairs recorded since the last attach.
 * dqn_profile_set_fusion(enabled): with 0, the small network's conv layers
 * run as one launch per layer and pass instead of the fused two-layer
 * launches (DQN_K_CONV12_FWD / DQN_K_CONV12_BWD), so that the two can be
 * compared; 1 (the default) restores them.  Returns DQN_OK.
 *
 * The hook is process-wide state: attach/detach must not race with calls of
 * the hot-path entry points on other host threads.
 */
#ifndef DQN_PROFILE_H
#define DQN_PROFILE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DQN_K_GATHER = 0,
    DQN_K_CONV1_FWD = 1,
    DQN_K_CONV2_FWD = 2,
    DQN_K_CONV3_FWD = 3,
    DQN_K_FC1_FWD = 4,
    DQN_K_HEAD = 5,
    DQN_K_FC1_WGRAD = 6,
    DQN_K_FC1_DGRAD = 7,
    DQN_K_CONV1_WGRAD = 8,
    DQN_K_CONV2_WGRAD = 9,
    DQN_K_CONV3_WGRAD = 10,
    DQN_K_CONV2_DGRAD = 11,
    DQN_K_CONV3_DGRAD = 12,
    DQN_K_FINALIZE = 13,
    DQN_K_APPLY = 14,
    DQN_K_FC1_BWD = 15,     /* fc1 weight + input gradient in one launch (small batch) */
    DQN_K_CONV2_BWD = 16,   /* conv2 weight + input gradient in one launch (small batch) */
    DQN_K_CONV3_BWD = 17,   /* conv3 weight + input gradient in one launch (small batch) */
    DQN_K_FINALIZE_APPLY = 18, /* finalize with the update applied (dqn_train_steps) */
    DQN_K_CONV12_FWD = 19,  /* both conv layers of the small network */
    DQN_K_CONV12_BWD = 20,  /* conv2 weight + input gradient and conv1 weight gradient, small network */
    DQN_K_SNAKE_STEP = 21,  /* one move of every game with its replay write (dqn_actor.h) */
    DQN_K_OBSERVE = 22,     /* preprocessing of raw screens (dqn_preprocess, dqn_observe) */
    DQN_K_WEIGHT_REPACK = 23, /* conv2/conv3 weights in the per-lane order of the fp32 kernels */
    DQN_K_COUNT = 24
} dqn_kernel;

int dqn_profile_attach(int32_t kernel, void** events, int32_t n_pairs, int32_t stride);
int32_t dqn_profile_used(int32_t kernel);
int dqn_profile_set_fusion(int32_t enabled);

/* Checks of the roofline denominators on the running device (the spec-sheet
 * peaks are what the figures are divided by; these show what the chip
 * reaches with the instruction forms the hot path uses).
 *
 * dqn_profile_mfma_peak(dtype, workgroups, iters, out, stream): enqueues one
 * launch of `workgroups` workgroups of four waves; every wave issues iters x 4
 * independent matrix-core instructions on register operands (DQN_PEAK_FP32:
 * v_mfma_f32_16x16x4_f32, 2,048 FLOP each; DQN_PEAK_BF16:
 * v_mfma_f32_16x16x32_bf16, 16,384 FLOP each) and stores one float per
 * workgroup to out (device float [workgroups]).  Returns the FLOP count of the
 * launch (> 0), or DQN_EINVAL / DQN_EHIP.  The caller times the launch with
 * events on `stream`.
 *
 * dqn_profile_stream_copy(src, dst, bytes, workgroups, stream): enqueues a
 * copy of `bytes` (a multiple of 16; src and dst device pointers, 16-byte
 * aligned, not overlapping) with 16-byte loads and stores, grid-stride over
 * `workgroups` workgroups of 256 threads; it moves 2 x bytes through HBM when
 * the buffers exceed the caches.  Returns DQN_OK, DQN_EINVAL or DQN_EHIP. */
enum { DQN_PEAK_FP32 = 0, DQN_PEAK_BF16 = 1 };
int64_t dqn_profile_mfma_peak(int32_t dtype, int32_t workgroups, int32_t iters, float* out, void* stream);
int dqn_profile_stream_copy(const void* src, void* dst, int64_t bytes, int32_t workgroups, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DQN_PROFILE_H */
