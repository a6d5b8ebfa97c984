/*
 * dqn_train.h -- worker and parameter-server loops of libdqn.so.
 *
 * Distributed deep Q-learning (arXiv 1508.04186) repeats, per worker, "fetch
 * the model, sample a minibatch from the local replay memory, compute the
 * gradient, send it" (Alg. 1), while the parameter server applies each
 * gradient it receives, in arrival order, and counts updates (Alg. 2).  These
 * two entry points run those loops on one GPU from the calls in dqn.h:
 *
 *  dqn_train_steps      one worker and the server in lockstep on one stream,
 *                       with the held target network refreshed every C steps
 *                       (Alg. 1's test n >= l*C, generation l starting at 0:
 *                       theta^- <- theta_n at n = 0, C, 2C, ... before step
 *                       n's gradient).
 *  dqn_train_replicas   R workers on R streams and the server on its own
 *                       stream (Sec. IV.A's asynchronous Downpour variant),
 *                       with a deterministic bounded-staleness schedule:
 *                       update u is computed by replica u mod R from the
 *                       parameter version v(u) = max(0, u - S), which is also
 *                       its target network, and the server applies updates
 *                       in order u = 0, 1, ..., producing version u + 1.  The
 *                       paper's write-lock becomes stream order plus
 *                       out-of-place versions in a ring of S + 1 slots.
 *
 * Conventions as in dqn.h: device pointers, caller-owned memory, asynchronous
 * on the given streams, DQN_OK or a negative dqn_status, argument checks on
 * the host before anything is enqueued.
 */
#ifndef DQN_TRAIN_H
#define DQN_TRAIN_H

#include <stddef.h>
#include <stdint.h>

#include "dqn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Device workspace bytes for dqn_train_steps (replicas = 1) or
 * dqn_train_replicas (replicas = R), or a negative dqn_status. */
int64_t dqn_train_workspace_bytes(const dqn_net* net, int32_t batch, int32_t replicas);

/* n_steps sequential steps n = 0 .. n_steps-1 (global step g = step0 + n):
 *   if target_period > 0 and g % target_period == 0: theta_target <- theta;
 *   dqn_td_gradient_replay(theta, theta_target or, when target_period == 0,
 *   theta itself, minibatch idx + n*batch); ps_apply_update(rule, theta in
 *   place).
 * The update is applied by the last kernel of each step rather than by a
 * separate pass; theta, opt_state and the losses are bit-identical to those
 * of the two calls above.
 * idx: device int64 [n_steps][batch] (transition indices, as replay_gather).
 * theta_target: device float [p]; may be NULL when target_period == 0.
 * opt_state: device float [p] (RMSProp r or AdaGrad G); NULL for PS_SGD.
 * losses_out: device float [n_steps], the loss of each step; may be NULL.
 * ws: at least dqn_train_workspace_bytes(net, batch, 1) bytes, 256-aligned. */
int dqn_train_steps(const dqn_net* net, float* theta, float* theta_target, float* opt_state,
                    int32_t rule, float lr, float decay, float eps, float gamma,
                    const dqn_replay* replay, const int64_t* idx, int32_t batch,
                    int64_t n_steps, int64_t step0, int64_t target_period, float* losses_out,
                    void* ws, size_t ws_bytes, void* stream);

/* Floats between consecutive slots of dqn_train_replicas' parameter ring:
 * the parameter count rounded up to a multiple of 64 (so every slot is
 * 256-byte aligned when the ring is), or a negative dqn_status. */
int64_t dqn_train_ring_stride(const dqn_net* net);

/* n_updates asynchronous-style updates with bounded staleness (see above).
 * theta_ring: device float [staleness + 1][dqn_train_ring_stride(net)],
 * 16-byte aligned; slot 0 holds the initial parameters on entry; after the
 * call (once the server stream is done), version n_updates is in slot
 * n_updates % (staleness + 1).
 * opt_state: server's optimizer state, device float [p] (NULL for PS_SGD).
 * streams: host array of replicas + 1 hipStream_t (as void*): the replica
 * streams, then the server stream.  All must be distinct.  On return every
 * update is enqueued; the caller synchronizes the server stream.  The call
 * creates replicas + staleness + 2 HIP events for the cross-stream
 * dependencies and releases them before returning (no device memory is
 * allocated).  Inputs written on other streams must be complete before the
 * call (the replica streams do not wait for the caller's stream).
 * replicas must exceed staleness (a replica's gradient buffer is reused only
 * after the server consumed it).  idx: device int64 [n_updates][batch];
 * losses_out: device float [n_updates] or NULL.
 * ws: at least dqn_train_workspace_bytes(net, batch, replicas) bytes. */
int dqn_train_replicas(const dqn_net* net, float* theta_ring, float* opt_state, int32_t rule,
                       float lr, float decay, float eps, float gamma, const dqn_replay* replay,
                       const int64_t* idx, int32_t batch, int64_t n_updates, int32_t replicas,
                       int32_t staleness, float* losses_out, void* ws, size_t ws_bytes,
                       void* const* streams);

#ifdef __cplusplus
}
#endif

#endif /* DQN_TRAIN_H */
