"""Pins of the oracle's bf16-input variant (every operand of the conv and fc1
contractions rounded to bfloat16 before the products, fp32-style
accumulation replaced by exact double sums).

The rounding itself is checked against torch's float32 -> bfloat16
conversion (round to nearest, ties to even), a library routine.  Where the
rounding is applied is checked against an independent batched numpy
formulation of the forward pass and of the TD gradient (im2col, matrix
products, col2im), whose operands are rounded with torch; with rounding
switched off that formulation reproduces the float64 oracle, which the
finite-difference pins fix.  A rounding placed on the wrong tensor (a bias
gradient taken from the rounded dz, an unrounded weight, the 1/255 applied
before rounding) fails one of these.
"""
import numpy as np
import pytest
import torch

import dqn_inputs as di
import oracle


def torch_bf16(x):
    t = torch.from_numpy(np.asarray(x, np.float64).astype(np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.normal(0, 1, 20000),
        rng.normal(0, 1e-30, 1000),              # float32 subnormal range
        rng.uniform(-1e30, 1e30, 1000),
        np.array([0.0, -0.0, 1.0, -1.0, 255.0, 1 / 255, 65504.0]),
    ])
    # exact ties: float32 values whose discarded 16 bits are 0x8000, with odd
    # and even kept parts
    u = (rng.integers(0x3f000000, 0x40000000, 4000, dtype=np.uint32) & np.uint32(0xffff0000)) | np.uint32(0x8000)
    x = np.concatenate([x, u.view(np.float32).astype(np.float64)])
    assert np.array_equal(oracle.bf16_round(x), torch_bf16(x))
    # bytes are exact in bfloat16
    b = np.arange(256, dtype=np.float64)
    assert np.array_equal(oracle.bf16_round(b), b)


# ---------------------------------------------------------------------------
# The independent batched formulation.

def _params(net, th):
    sl = net.slices()
    get = lambda k: th[sl[k][0]:sl[k][0] + int(np.prod(sl[k][1]))].reshape(sl[k][1])
    convs = [(get(f"conv{i+1}.W"), get(f"conv{i+1}.b")) for i in range(len(net.conv))]
    return convs, (get("fc1.W"), get("fc1.b")), (get("fc2.W"), get("fc2.b"))


def _im2col(x, k, s, oh, ow):
    win = np.lib.stride_tricks.sliding_window_view(x, (k, k), axis=(2, 3))[:, :, ::s, ::s][:, :, :oh, :ow]
    return win.transpose(0, 2, 3, 1, 4, 5).reshape(x.shape[0], oh * ow, -1)      # B P (C k k)


def _col2im(cols, shape, k, s, oh, ow):
    B, C, H, W = shape
    out = np.zeros(shape)
    c6 = cols.reshape(B, oh, ow, C, k, k)
    for ky in range(k):
        for kx in range(k):
            out[:, :, ky:ky + s * oh:s, kx:kx + s * ow:s] += c6[:, :, :, :, ky, kx].transpose(0, 3, 1, 2)
    return out


def np_forward(net, th, states, rnd):
    """Batched forward; returns Q and the per-layer values backprop needs."""
    convs, (W1, b1), (W2, b2) = _params(net, th)
    x = states.astype(np.float64) / 255.0
    cache = []
    for i, ((W, b), (cin, ih, iw, cout, k, s, oh, ow)) in enumerate(zip(convs, net.conv_dims())):
        xo = x if i == 0 else rnd(x)                     # input bytes are exact
        cols = _im2col(xo, k, s, oh, ow)
        z = cols @ rnd(W).reshape(cout, -1).T + b        # B P O
        cache.append((x.shape, cols, z, W, k, s, oh, ow))
        x = np.maximum(z, 0).transpose(0, 2, 1).reshape(x.shape[0], cout, oh, ow)
    flat = x.reshape(x.shape[0], -1)
    z1 = rnd(flat) @ rnd(W1).T + b1
    h1 = np.maximum(z1, 0)
    return h1 @ W2.T + b2, (cache, flat, z1, h1, W1, W2)


def np_td_gradient(net, th, tt, s, sn, a, r, t, gamma, rnd):
    B = s.shape[0]
    qn, _ = np_forward(net, tt, sn, rnd)
    y = np.where(t > 0, r.astype(np.float64), r.astype(np.float64) + gamma * qn.max(axis=1))
    q, (cache, flat, z1, h1, W1, W2) = np_forward(net, th, s, rnd)
    diff = q[np.arange(B), a] - y
    loss = np.sum(0.5 * diff ** 2) / B
    dq = np.zeros_like(q)
    dq[np.arange(B), a] = diff / B
    grads = {}
    grads["fc2.W"] = dq.T @ h1
    grads["fc2.b"] = dq.sum(0)
    dz1 = (dq @ W2) * (z1 > 0)
    grads["fc1.W"] = rnd(dz1).T @ rnd(flat)
    grads["fc1.b"] = dz1.sum(0)
    dx = (rnd(dz1) @ rnd(W1)).reshape(B, -1)
    for i in range(len(cache) - 1, -1, -1):
        shape, cols, z, W, k, s_, oh, ow = cache[i]
        cout = W.shape[0]
        dz = dx.reshape(B, cout, oh * ow).transpose(0, 2, 1) * (z > 0)          # B P O
        grads[f"conv{i+1}.W"] = np.einsum("bpo,bpk->ok", rnd(dz), cols).reshape(W.shape)
        grads[f"conv{i+1}.b"] = dz.sum((0, 1))
        if i > 0:
            dcols = rnd(dz) @ rnd(W).reshape(cout, -1)                          # B P (C k k)
            dx = _col2im(dcols, shape, k, s_, oh, ow)
    g = np.empty(net.param_count())
    for name, (off, shp) in net.slices().items():
        g[off:off + int(np.prod(shp))] = grads[name].ravel()
    return g, loss, q, y


NETS = [
    di.tiny_net(2, 12, 12, ((3, 4, 2),), 5, 3),
    di.tiny_net(3, 14, 14, ((4, 4, 2), (3, 3, 1)), 6, 4),
    di.tiny_net(2, 20, 20, ((3, 8, 4), (4, 2, 1), (2, 2, 1)), 4, 5),
]
IDENT = lambda v: v  # noqa: E731


def _case(net, B=4, seed=31):
    th = di.xavier_theta(net, seed, bias_scale=0.1).astype(np.float64)
    tt = th + np.random.default_rng(seed).normal(0, 0.03, th.shape)
    s = di.random_states(B, seed + 1, net.in_c, net.in_h, net.in_w)
    sn = di.random_states(B, seed + 2, net.in_c, net.in_h, net.in_w)
    a = (np.arange(B) % net.n_actions).astype(np.int32)
    r = np.array([1.0, -1.0, 0.0, 1.0] * B, np.float32)[:B]
    t = np.array([0, 1, 0, 0] * B, np.uint8)[:B]
    return th, tt, s, sn, a, r, t


@pytest.mark.parametrize("net", NETS + [di.NET_S], ids=lambda n: str(n.conv))
def test_batched_formulation_reproduces_fp64_oracle(net):
    th, tt, s, sn, a, r, t = _case(net)
    g, loss, q, y = np_td_gradient(net, th, tt, s, sn, a, r, t, 0.9, IDENT)
    ref = oracle.td_gradient(net, th, tt, s, sn, a, r, t, 0.9)
    assert np.allclose(g, ref["grad"], rtol=1e-10, atol=1e-14)
    assert abs(loss - ref["loss"]) <= 1e-12 * abs(ref["loss"])


@pytest.mark.parametrize("net", NETS + [di.NET_S, di.NET_L], ids=lambda n: str(n.conv))
def test_bf16_forward_matches_batched_formulation(net):
    th = di.xavier_theta(net, 7, bias_scale=0.1)
    st = di.random_states(3, 8, net.in_c, net.in_h, net.in_w)
    q = oracle.forward_q(net, th, st, bf16=True)
    ref, _ = np_forward(net, th.astype(np.float64), st, torch_bf16)
    assert np.allclose(q, ref, rtol=1e-11, atol=1e-13)
    # and it differs from the unrounded forward by a bf16-sized amount
    q64 = oracle.forward_q(net, th, st)
    rel = np.linalg.norm(q - q64) / np.linalg.norm(q64)
    assert 1e-5 < rel < 3e-2, rel


@pytest.mark.parametrize("net", NETS + [di.NET_S], ids=lambda n: str(n.conv))
def test_bf16_td_gradient_matches_batched_formulation(net):
    th, tt, s, sn, a, r, t = _case(net)
    out = oracle.td_gradient(net, th, tt, s, sn, a, r, t, 0.9, bf16=True)
    g, loss, q, y = np_td_gradient(net, th, tt, s, sn, a, r, t, 0.9, torch_bf16)
    assert np.allclose(out["q"], q, rtol=1e-11, atol=1e-13)
    assert np.allclose(out["y"], y, rtol=1e-11, atol=1e-13)
    assert abs(out["loss"] - loss) <= 1e-10 * abs(loss)
    for name, (off, shp) in net.slices().items():
        n = int(np.prod(shp))
        assert np.allclose(out["grad"][off:off + n], g[off:off + n], rtol=1e-9, atol=1e-13), name
