// Worker and parameter-server loops (include/dqn_train.h): sequences of the
// dqn.h calls on one stream (one worker in lockstep with the server) or on
// replica streams plus a server stream with a bounded-staleness schedule.
#include <vector>

#include "common.h"
#include "dqn.h"
#include "dqn_train.h"

using namespace dqn;

namespace {

// Per-replica slice of the workspace: gradient, loss and the TD workspace.
// The minibatch is read from the replay in place (dqn_td_gradient_replay).
struct ReplicaWs {
    float* grad;
    float* loss;
    void* td_ws;
    size_t td_bytes;
};

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

// Bytes of one replica slice; negative dqn_status on a bad network.
int64_t replica_bytes(const dqn_net* net, int32_t batch) {
    const int64_t p = dqn_param_count(net);
    if (p < 0) return p;
    const int64_t td = dqn_workspace_bytes(net, batch, DQN_OP_TD_GRADIENT);
    if (td < 0) return td;
    return (int64_t)(round256(4 * (size_t)p) + 256 + (size_t)td);
}

ReplicaWs carve(const dqn_net* net, int32_t batch, char* base) {
    ReplicaWs w;
    const size_t p = (size_t)dqn_param_count(net);
    w.grad = (float*)base;
    w.loss = (float*)(base + round256(4 * p));
    w.td_ws = base + round256(4 * p) + 256;
    w.td_bytes = (size_t)dqn_workspace_bytes(net, batch, DQN_OP_TD_GRADIENT);
    return w;
}

bool valid_rule(int32_t rule, const float* state) {
    if (rule != PS_SGD && rule != PS_RMSPROP && rule != PS_ADAGRAD) return false;
    return rule == PS_SGD || state != nullptr;
}

#define TRY(expr)                       \
    do {                                \
        const int rc_ = (expr);         \
        if (rc_ != DQN_OK) return rc_;  \
    } while (0)

}  // namespace

extern "C" {

int64_t dqn_train_ring_stride(const dqn_net* net) {
    const int64_t p = dqn_param_count(net);
    return p < 0 ? p : (p + 63) / 64 * 64;
}

int64_t dqn_train_workspace_bytes(const dqn_net* net, int32_t batch, int32_t replicas) {
    if (batch <= 0 || replicas <= 0) return DQN_EINVAL;
    const int64_t one = replica_bytes(net, batch);
    if (one < 0) return one;
    return one * replicas;
}

int dqn_train_steps(const dqn_net* net, float* theta, float* theta_target, float* opt_state,
                    int32_t rule, float lr, float decay, float eps, float gamma,
                    const dqn_replay* replay, const int64_t* idx, int32_t batch,
                    int64_t n_steps, int64_t step0, int64_t target_period, float* losses_out,
                    void* ws, size_t ws_bytes, void* stream) {
    const int64_t need = dqn_train_workspace_bytes(net, batch, 1);
    if (need < 0) return (int)need;
    if (!theta || !replay || !idx || !ws || n_steps < 0 || step0 < 0 || target_period < 0)
        return DQN_EINVAL;
    if (target_period > 0 && !theta_target) return DQN_EINVAL;
    if (((uintptr_t)theta | (uintptr_t)theta_target) % 16 != 0) return DQN_EINVAL;
    if (!valid_rule(rule, opt_state)) return DQN_EINVAL;
    if ((uintptr_t)ws % 256 != 0) return DQN_EINVAL;
    if (ws_bytes < (size_t)need) return DQN_EWORKSPACE;
    const int64_t p = dqn_param_count(net);
    if (theta_target) {
        const char* a = (const char*)theta;
        const char* b = (const char*)theta_target;
        if (a < b + 4 * p && b < a + 4 * p) return DQN_EINVAL;
    }
    const ReplicaWs w = carve(net, batch, (char*)ws);
    hipStream_t st = (hipStream_t)stream;
    // The update is applied by the step's last kernel (same arithmetic as
    // ps_apply_update on the stored gradient).
    const PsUpdate upd{rule, theta, opt_state, lr, decay, eps};
    for (int64_t n = 0; n < n_steps; ++n) {
        const int64_t g = step0 + n;
        if (target_period > 0 && g % target_period == 0)
            if (launch_copy(theta, theta_target, p, st) != hipSuccess) return DQN_EHIP;
        TRY(td_step_replay(net, target_period > 0 ? theta_target : theta, replay, idx + n * batch,
                           batch, gamma, w.grad, losses_out ? losses_out + n : w.loss, upd, w.td_ws,
                           w.td_bytes, st));
    }
    return DQN_OK;
}

int dqn_train_replicas(const dqn_net* net, float* theta_ring, float* opt_state, int32_t rule,
                       float lr, float decay, float eps, float gamma, const dqn_replay* replay,
                       const int64_t* idx, int32_t batch, int64_t n_updates, int32_t replicas,
                       int32_t staleness, float* losses_out, void* ws, size_t ws_bytes,
                       void* const* streams) {
    if (replicas <= 0 || staleness < 0 || replicas <= staleness) return DQN_EINVAL;
    const int64_t need = dqn_train_workspace_bytes(net, batch, replicas);
    if (need < 0) return (int)need;
    if (!theta_ring || !replay || !idx || !ws || !streams || n_updates < 0) return DQN_EINVAL;
    if (!valid_rule(rule, opt_state)) return DQN_EINVAL;
    if ((uintptr_t)ws % 256 != 0) return DQN_EINVAL;
    if (ws_bytes < (size_t)need) return DQN_EWORKSPACE;
    for (int i = 0; i <= replicas; ++i) {
        if (!streams[i]) return DQN_EINVAL;
        for (int j = 0; j < i; ++j)
            if (streams[i] == streams[j]) return DQN_EINVAL;
    }
    if ((uintptr_t)theta_ring % 16 != 0) return DQN_EINVAL;
    const int64_t p = dqn_param_count(net);
    const int64_t rs = dqn_train_ring_stride(net);
    const int64_t one = replica_bytes(net, batch);
    std::vector<ReplicaWs> w(replicas);
    for (int k = 0; k < replicas; ++k) w[k] = carve(net, batch, (char*)ws + k * one);
    const int slots = staleness + 1;
    const int nv = staleness + 2;  // version events: V[v] lives in ev_v[v % nv]
    std::vector<hipEvent_t> ev_v(nv, nullptr), ev_g(replicas, nullptr);
    int rc = DQN_OK;
    for (auto& e : ev_v)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) rc = DQN_EHIP;
    for (auto& e : ev_g)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) rc = DQN_EHIP;
    hipStream_t server = (hipStream_t)streams[replicas];
    for (int64_t u = 0; u < n_updates && rc == DQN_OK; ++u) {
        const int k = (int)(u % replicas);
        hipStream_t st = (hipStream_t)streams[k];
        const int64_t v = u > staleness ? u - staleness : 0;
        // fetch (theta_v, v): wait until the server has produced version v
        if (v > 0 && hipStreamWaitEvent(st, ev_v[v % nv], 0) != hipSuccess) { rc = DQN_EHIP; break; }
        float* th_v = theta_ring + (v % slots) * rs;
        const ReplicaWs& r = w[k];
        rc = dqn_td_gradient_replay(net, th_v, th_v, replay, idx + u * batch, batch, gamma, r.grad,
                                    losses_out ? losses_out + u : r.loss, nullptr, nullptr, r.td_ws,
                                    r.td_bytes, st);
        if (rc != DQN_OK) break;
        // send the gradient; the server applies update u to version u
        if (hipEventRecord(ev_g[k], st) != hipSuccess || hipStreamWaitEvent(server, ev_g[k], 0) != hipSuccess) {
            rc = DQN_EHIP;
            break;
        }
        rc = ps_apply_update(rule, theta_ring + (u % slots) * rs, theta_ring + ((u + 1) % slots) * rs,
                             opt_state, r.grad, p, lr, decay, eps, server);
        if (rc != DQN_OK) break;
        if (hipEventRecord(ev_v[(u + 1) % nv], server) != hipSuccess) rc = DQN_EHIP;
    }
    for (auto& e : ev_v)
        if (e) (void)hipEventDestroy(e);
    for (auto& e : ev_g)
        if (e) (void)hipEventDestroy(e);
    return rc;
}

}  // extern "C"
