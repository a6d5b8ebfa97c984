"""Helpers shared by the GPU parity tests: device copies, per-tensor error
norms against the oracle, and the action-choice comparison rule."""
import sys

import numpy as np

FP32_TOL = 1e-4      # relative L2 error per tensor (each W and b separately)


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def dev_tensor(a, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def host(t):
    return t.detach().cpu().numpy()


def rel_l2(x, ref):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.linalg.norm((x - ref).ravel())
    den = np.linalg.norm(ref.ravel())
    if den == 0.0:
        return 0.0 if num == 0.0 else np.inf
    return num / den


def grad_errors(net_shape, g, ref):
    """{tensor name: relative L2 error} over the flat parameter layout."""
    out = {}
    for name, (off, shape) in net_shape.slices().items():
        n = int(np.prod(shape))
        out[name] = rel_l2(g[off:off + n], ref[off:off + n])
    return out


def assert_grad_close(net_shape, g, ref, tol=FP32_TOL, what="grad"):
    errs = grad_errors(net_shape, g, ref)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{what}: per-tensor relative L2 errors above {tol}: {bad} (all: {errs})"
    return errs


def check_actions(act_gpu, q_gpu, q_ref, act_ref, explore_mask, tol=FP32_TOL):
    """Action parity rule.  (i) Every greedy action is the lowest index of the
    maximum of the GPU's own Q row (bit-exact).  (ii) It equals the oracle's
    choice wherever the oracle's top-two gap exceeds 2*tol*max|Q| (the Q
    tolerance); inside that band any action whose oracle value is within the
    band of the maximum is valid.  (iii) Exploring states take exactly the
    oracle's random action.  Returns the number of near-tie states."""
    act_gpu = np.asarray(act_gpu)
    greedy = ~explore_mask
    own = np.argmax(q_gpu, axis=1)  # numpy argmax returns the first maximum
    assert np.array_equal(act_gpu[greedy], own[greedy]), "action is not the argmax of q_out"
    assert np.array_equal(act_gpu[explore_mask], act_ref[explore_mask]), "exploration differs"
    scale = np.abs(q_ref).max(axis=1)
    band = 2 * tol * np.maximum(scale, 1e-30)
    srt = np.sort(q_ref, axis=1)
    gap = srt[:, -1] - srt[:, -2] if q_ref.shape[1] > 1 else np.full(len(q_ref), np.inf)
    clear = greedy & (gap > band)
    assert np.array_equal(act_gpu[clear], act_ref[clear]), "greedy action differs from oracle"
    near = greedy & ~clear
    if near.any():
        rows = np.nonzero(near)[0]
        chosen = q_ref[rows, act_gpu[rows]]
        assert np.all(chosen >= q_ref[rows].max(axis=1) - band[rows]), "near-tie action not near max"
    return int(near.sum())


# Normalized ReLU margin below which float32 rounding may decide a ReLU
# derivative differently from the float64 oracle (the derivative at a
# pre-activation within rounding of zero is not fixed by the arithmetic).
# float32 errors in a pre-activation are ~1e-7 of the magnitude of its
# terms; 1e-6 leaves a factor of ten.
MARGIN_MIN = 1e-6


def split_by_margin(net_shape, theta, states):
    """Boolean mask: True where the oracle's smallest normalized ReLU margin of
    Q(state; theta) is at least MARGIN_MIN (the gradient is then unique)."""
    import oracle
    return oracle.relu_margins(net_shape, theta, states) >= MARGIN_MIN
