"""MI355X (gfx950) hot path of distributed deep Q-learning (arXiv 1508.04186).

Thin Python binding over libdqn.so: the same entry points as the C ABI in
include/dqn.h (replay_gather, dqn_forward, dqn_forward_replay, dqn_td_gradient, ps_apply_update
and the layout/workspace queries) and include/dqn_train.h (the worker and
parameter-server loops dqn_train_steps and dqn_train_replicas), with torch
tensors for device memory and streams.  All arithmetic runs in the library's HIP kernels; there is no CPU
or PyTorch fallback, and loading fails loudly when the library is missing.
"""
from .native import (  # noqa: F401
    DQN_OK, DQN_EINVAL, DQN_EWORKSPACE, DQN_EHIP, DQN_EUNSUPPORTED,
    PS_SGD, PS_RMSPROP, PS_ADAGRAD, DQN_OP_FORWARD, DQN_OP_TD_GRADIENT,
    DqnError, Net, NET_SMALL, NET_LARGE, NET_LARGE_BF16, DQN_FP32, DQN_BF16, Replay,
    lib, lib_path, dqn_param_count, dqn_param_offset, dqn_workspace_bytes,
    replay_gather, dqn_forward, dqn_forward_replay, dqn_td_gradient, dqn_td_gradient_replay, dqn_td_gradient_noalloc,
    ps_apply_update,
    dqn_status_string,
    workspace, profile_attach, profile_used, profile_set_fusion, KERNEL_NAMES,
    dqn_train_workspace_bytes, dqn_train_ring_stride, dqn_train_steps, dqn_train_replicas,
    HipStreams, DQN_PEAK_FP32, DQN_PEAK_BF16, profile_mfma_peak, profile_stream_copy,
    ActorReplay, snake_games, snake_reset, snake_step, dqn_anneal_epsilon, dqn_act, SNAKE_STATE_BYTES,
    dqn_preprocess, dqn_observe, replay_fill_synthetic, replay_gather_validate,
)
