"""Free-running trajectories of the GPU path beside the float64 oracle, and
the float32 pre-activation error that the margin rule of the full-size
parity tests has to cover.  A report, not a test: it asserts nothing about
the gaps it prints.

Run on a GPU machine from the repository root:  python -u tests/drift_report.py

Part 1 (config 1: small network, batch 32, SGD lr 2.5e-4, the seeded
100,000-transition replay) and part 2 (config 2: 16 replicas, staleness 4,
AdaGrad lr 0.01 eps 1e-8 from a zero state) run the GPU and the oracle
side by side, each on its own trajectory from the same initial parameters
(Alg. 1 and Alg. 2).  At logged steps they print, per tensor, the gap
|theta_gpu - theta_oracle| relative to how far the oracle's parameters have
moved, |theta_oracle - theta_0|, and two counts at the GPU's own state: the
gradient elements whose sign differs between the GPU and the oracle
(computed from the same parameters; an element that is exactly zero on one
side only counts too), and the elements whose float64 gradient is nonzero
but below 1e-6 of the tensor's largest (sign-ambiguous at float32
precision; exact zeros, from ReLUs that are off, are not).  Under AdaGrad from a zero state each element's first step is
about lr * sign(g), so a sign decided by rounding moves that parameter by up
to 2 lr (the reading of Sec. IV.D.2's AdaGrad that the tests follow).

Part 3: for the large network in float32 at 64 and 256 states (the
per-layer and the large-batch conv kernels), the GPU's conv outputs and fc1
sums are read back from dqn_forward's workspace and compared with float64
pre-activations z of the same layer computed from the float64 activations
below (an independent numpy formulation): the normalized error
|z_gpu - z| / (|b| + sum |w x|) at units with z > 0, per layer, and the
number of units whose ReLU decision differs.  This is what the margin rule
MARGIN_MIN (minimum normalized margin of a transition's pre-activations)
must exceed for the float32 and float64 ReLU decisions to agree."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
for p in (ROOT, os.path.join(ROOT, "tests")):
    if p not in sys.path:
        sys.path.insert(0, p)

import dqn_inputs as di  # noqa: E402
import oracle  # noqa: E402
import paper_1508_04186_amd as dq  # noqa: E402

F32 = np.float32
LOG_STEPS = (1, 10, 50, 100, 200)


def say(msg):
    print(msg, flush=True)


def host(t):
    return t.detach().cpu().numpy()


def tensor_table(shape, th_g, th_o, th0, g_g, g_o):
    rows = []
    for name, (off, shp) in shape.slices().items():
        n = int(np.prod(shp))
        sl = slice(off, off + n)
        moved = np.linalg.norm(th_o[sl].astype(np.float64) - th0[sl])
        gap = np.linalg.norm(th_g[sl].astype(np.float64) - th_o[sl])
        flips = int(np.sum(np.sign(g_g[sl]) != np.sign(g_o[sl])))
        ao = np.abs(g_o[sl])
        amb = int(np.sum((ao > 0) & (ao < 1e-6 * max(ao.max(), 1e-300))))
        rows.append((name, gap / moved if moved > 0 else float("nan"), flips, amb, n))
    return rows


def print_rows(step, rows):
    for name, rel, flips, amb, n in rows:
        say(f"| {step} | {name} | {rel:.3e} | {flips} | {amb} | {n} |")


def part1():
    import torch
    dev = torch.device("cuda:0")
    net, shape = dq.NET_SMALL, di.NET_S
    B, SIZE, SEED, LR, GAMMA = 32, 100_000, 1001, 2.5e-4, 0.99
    steps = max(LOG_STEPS)
    say(f"## config 1 free-running: small network, batch {B}, SGD lr {LR}, {steps} steps")
    hr = di.host_replay(SIZE, shape.n_actions, SEED)
    rec, a, r, t = di.device_replay(SIZE, shape.n_actions, SEED, host=hr)
    rp = dq.Replay(rec, a, r, t, SIZE)
    th0 = di.xavier_theta(shape, SEED)
    idx_h = di.index_stream(steps, B, SIZE, SEED)
    idx = torch.from_numpy(idx_h).to(dev)
    theta = torch.from_numpy(th0).to(dev)
    ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, 1), dtype=torch.uint8, device=dev)
    g = torch.empty_like(theta)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    th_o = th0.copy()
    say("| step | tensor | gap / moved | sign flips | sign-ambiguous | elements |")
    say("|---:|---|---:|---:|---:|---:|")
    done = 0
    for n in range(steps):
        s, sn, aa, rr, tt = oracle.gather_from_host_replay(hr, idx_h[n])
        out = oracle.td_gradient(shape, th_o, th_o, s, sn, aa, rr, tt, float(F32(GAMMA)))
        th_o, _ = oracle.apply_update("sgd", th_o, None, out["grad"], float(F32(LR)))
        if n + 1 in LOG_STEPS:
            dq.dqn_train_steps(net, theta, None, None, dq.PS_SGD, LR, 0.9, 0.0, GAMMA, rp, idx[done:n + 1],
                               step0=done, ws=ws)
            done = n + 1
            th_g = host(theta)
            # gradients at the GPU's state, on the next minibatch
            nxt = min(n + 1, steps - 1)
            dq.dqn_td_gradient_replay(net, theta, theta, rp, idx[nxt], GAMMA, g, loss)
            torch.cuda.synchronize()
            s, sn, aa, rr, tt = oracle.gather_from_host_replay(hr, idx_h[nxt])
            ref = oracle.td_gradient(shape, th_g, th_g, s, sn, aa, rr, tt, float(F32(GAMMA)))
            print_rows(n + 1, tensor_table(shape, th_g, th_o, th0, host(g), ref["grad"]))


def part2():
    import torch
    dev = torch.device("cuda:0")
    net, shape = dq.NET_SMALL, di.NET_S
    B, SIZE, SEED, LR, EPS, GAMMA, R, S = 32, 100_000, 1002, 0.01, 1e-8, 0.99, 16, 4
    U = max(LOG_STEPS)
    say(f"## config 2 free-running: {R} replicas, staleness {S}, AdaGrad lr {LR} eps {EPS} from a zero "
        f"state, {U} updates")
    hr = di.host_replay(SIZE, shape.n_actions, SEED)
    rec, a, r, t = di.device_replay(SIZE, shape.n_actions, SEED, host=hr)
    rp = dq.Replay(rec, a, r, t, SIZE)
    th0 = di.xavier_theta(shape, SEED)
    idx_h = di.index_stream(U, B, SIZE, SEED)
    idx = torch.from_numpy(idx_h).to(dev)
    P = dq.dqn_param_count(net)
    RS = dq.dqn_train_ring_stride(net)
    ring = torch.empty((S + 1) * RS, dtype=torch.float32, device=dev)
    G = torch.zeros(P, dtype=torch.float32, device=dev)
    ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, R), dtype=torch.uint8, device=dev)
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    say("| update | tensor | gap / moved | sign flips | sign-ambiguous | elements |")
    say("|---:|---|---:|---:|---:|---:|")
    logged = {}

    def cb(u, theta, state, out):
        if u + 1 in LOG_STEPS:
            logged[u + 1] = theta.copy()
    oracle.stale_replica_training(shape, th0, hr, idx_h, float(F32(GAMMA)), float(F32(LR)), S,
                                  rule="adagrad", eps=float(F32(EPS)), callback=cb)
    with dq.HipStreams(R + 1) as hs:
        for n in LOG_STEPS:
            ring[:P].copy_(torch.from_numpy(th0).to(dev))
            G.zero_()
            torch.cuda.synchronize()
            dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA, rp, idx[:n], R, S,
                                  hs.handles, ws=ws)
            torch.cuda.synchronize()
            slot = n % (S + 1)
            th_g = host(ring[slot * RS:slot * RS + P])
            nxt = min(n, U - 1)
            th_d = torch.from_numpy(th_g).to(dev)
            dq.dqn_td_gradient_replay(net, th_d, th_d, rp, idx[nxt], GAMMA, g, loss)
            torch.cuda.synchronize()
            s, sn, aa, rr, tt = oracle.gather_from_host_replay(hr, idx_h[nxt])
            ref = oracle.td_gradient(shape, th_g, th_g, s, sn, aa, rr, tt, float(F32(GAMMA)))
            print_rows(n, tensor_table(shape, th_g, logged[n], th0, host(g), ref["grad"]))


def _windows(x, k, s):
    """im2col: [B][C][H][W] -> [B][OH][OW][C*k*k] (channel-major taps)."""
    B, C, H, W = x.shape
    oh, ow = (H - k) // s + 1, (W - k) // s + 1
    v = np.lib.stride_tricks.sliding_window_view(x, (k, k), axis=(2, 3))[:, :, ::s, ::s]
    return v[:, :, :oh, :ow].transpose(0, 2, 3, 1, 4, 5).reshape(B, oh, ow, C * k * k)


def part3():
    import torch
    dev = torch.device("cuda:0")
    net, shape = dq.NET_LARGE, di.NET_L
    say("## float32 pre-activation error of the large network's forward (normalized by |b| + sum |w x|)")
    say("| states | layer | units with z > 0 | median | 99.9th percentile | max | ReLU decisions differing |")
    say("|---:|---|---:|---:|---:|---:|---:|")
    sl = shape.slices()
    for B in (64, 256):
        th = di.xavier_theta(shape, 4000 + B, bias_scale=0.02)
        hr = di.host_replay(B + 10, shape.n_actions, seed=4100 + B)
        idx = np.arange(B)
        st, _, _, _, _ = oracle.gather_from_host_replay(hr, idx, with_next=False)
        st = st.reshape(B, 4, 84, 84)
        ws = dq.workspace(net, B, dq.DQN_OP_FORWARD, dev)
        q = torch.empty((B, net.n_actions), dtype=torch.float32, device=dev)
        dq.dqn_forward(net, torch.from_numpy(th).to(dev), torch.from_numpy(st).to(dev), 0.0, None, q, None,
                       ws=ws)
        torch.cuda.synchronize()
        wsh = host(ws)
        # the workspace holds each conv layer's float32 output [B][C][H][W] in order, each
        # buffer starting on a 256-byte boundary, then the fc1 split-K partial sums
        # [slices][B][hidden] (the head adds the slices and the bias)
        off = 0
        x = st.astype(np.float64) / 255.0
        dims = shape.conv_dims()
        for l, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(dims):
            n = B * cout * oh * ow
            h_gpu = wsh[off:off + 4 * n].view(np.float32).reshape(B, cout, oh, ow).astype(np.float64)
            off += (4 * n + 255) // 256 * 256
            W = th[sl[f"conv{l + 1}.W"][0]:][:cout * cin * k * k].astype(np.float64).reshape(cout, -1)
            b = th[sl[f"conv{l + 1}.b"][0]:][:cout].astype(np.float64)
            cols = _windows(x, k, s)
            z = (cols @ W.T + b).transpose(0, 3, 1, 2)
            nz = (np.abs(cols) @ np.abs(W).T + np.abs(b)).transpose(0, 3, 1, 2)
            report(B, f"conv{l + 1}", h_gpu, z, nz)
            x = np.maximum(z, 0.0)
        flat = x.reshape(B, -1)
        W1 = th[sl["fc1.W"][0]:][:shape.fc_hidden * flat.shape[1]].astype(np.float64).reshape(shape.fc_hidden, -1)
        b1 = th[sl["fc1.b"][0]:][:shape.fc_hidden].astype(np.float64)
        rest = wsh[off:].view(np.float32)
        ks = rest.size // (B * shape.fc_hidden)
        parts = rest[:ks * B * shape.fc_hidden].reshape(ks, B, shape.fc_hidden).astype(np.float64)
        z1_gpu = parts.sum(axis=0) + b1
        z1 = flat @ W1.T + b1
        n1 = np.abs(flat) @ np.abs(W1).T + np.abs(b1)
        report(B, "fc1", np.maximum(z1_gpu, 0.0), z1, n1)


def report(B, name, h_gpu, z, nz):
    pos = z > 0
    e = np.abs(h_gpu[pos] - z[pos]) / np.maximum(nz[pos], 1e-300)
    differ = int(np.sum((h_gpu > 0) != pos))
    say(f"| {B} | {name} | {int(pos.sum())} | {np.median(e):.2e} | {np.quantile(e, 0.999):.2e} | "
        f"{e.max():.2e} | {differ} |")


if __name__ == "__main__":
    import torch
    assert torch.cuda.is_available(), "the drift report needs a GPU"
    part3()
    part1()
    part2()
