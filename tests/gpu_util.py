"""Helpers shared by the GPU parity tests: device copies, per-tensor error
bounds against the oracle (normwise and element by element), and the
action-choice comparison rule."""
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


def max_elem_err(x, ref, slack=None):
    """Largest elementwise error relative to the tensor's largest magnitude:
    max (|x - ref| - slack) / max |ref| (0 when both are zero).  slack: an
    elementwise allowance (e.g. one float32 ulp of a stored result)."""
    x = np.asarray(x, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    if x.size == 0:
        return 0.0
    d = np.abs(x - ref)
    if slack is not None:
        d = np.maximum(d - np.asarray(slack, np.float64).ravel(), 0.0)
    num = d.max()
    den = np.abs(ref).max()
    if den == 0.0:
        return 0.0 if num == 0.0 else np.inf
    return num / den


def assert_close(x, ref, tol=FP32_TOL, what="value"):
    """Per tensor: the relative L2 error is at most tol, and so is every
    element's error relative to the tensor's largest magnitude
    (|x_i - ref_i| <= tol * max |ref|).  Returns (normwise, elementwise)."""
    n, e = rel_l2(x, ref), max_elem_err(x, ref)
    assert n <= tol and e <= tol, f"{what}: relative L2 {n:.3e}, max elementwise {e:.3e} (bound {tol})"
    return n, e


def grad_errors(net_shape, g, ref):
    """{tensor name: relative L2 error} over the flat parameter layout."""
    out = {}
    for name, (off, shape) in net_shape.slices().items():
        n = int(np.prod(shape))
        out[name] = rel_l2(g[off:off + n], ref[off:off + n])
    return out


def grad_elem_errors(net_shape, g, ref, slack=None):
    """{tensor name: max elementwise error / max |ref|} over the flat layout."""
    out = {}
    for name, (off, shape) in net_shape.slices().items():
        n = int(np.prod(shape))
        out[name] = max_elem_err(g[off:off + n], ref[off:off + n],
                                 None if slack is None else slack[off:off + n])
    return out


def assert_grad_close(net_shape, g, ref, tol=FP32_TOL, what="grad", slack=None):
    """Every tensor of the flat layout (each W and b separately) within tol,
    normwise and element by element (assert_close's bounds).  slack: an
    elementwise allowance added to the elementwise bound, for differences of
    float32-stored values (a parameter change theta_new - theta carries one
    ulp of the stored theta_new, whatever computed it).  The largest
    elementwise error is printed as a diagnostic.  Returns the normwise
    errors."""
    errs = grad_errors(net_shape, g, ref)
    elem = grad_elem_errors(net_shape, g, ref, slack)
    worst = max(elem, key=elem.get)
    say(f"{what}: max elementwise error {elem[worst]:.2e} ({worst}), max relative L2 "
        f"{max(errs.values()):.2e}")
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{what}: per-tensor relative L2 errors above {tol}: {bad} (all: {errs})"
    bad = {k: v for k, v in elem.items() if not v <= tol}
    assert not bad, f"{what}: per-tensor max elementwise errors above {tol} x max|ref|: {bad} (all: {elem})"
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
