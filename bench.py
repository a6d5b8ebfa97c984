#!/usr/bin/env python3
"""Throughput of the DQN TD-gradient + parameter-server update hot path on one
MI355X (arXiv 1508.04186, Alg. 1 and Alg. 2 with one worker).

Workload (one "step" = one pass of the whole hot path over one minibatch):
  replay_gather   32 transitions drawn uniformly (seeded index stream) from a
                  replay memory of 100,000 synthetic uint8 4x84x84 transitions
                  held in device memory;
  dqn_td_gradient targets from theta^- = theta, loss and full gradient of the
                  small Q-network (conv 16@8x8/4, conv 32@4x4/2, fc 256, fc 6);
  ps_apply_update plain gradient-descent step, lr 2.5e-4.
2,000 sequential steps are timed (after warmup) between HIP events on the
stream the work runs on.  Inputs are resident in device memory before timing.

The JSON line adds:
  roofline      the dominant kernel (largest time per step, chosen by a short
                event-bracketed breakdown pass before timing): algorithmic
                FLOP per launch / its average launch time, measured with HIP
                event pairs around every launch inside the timed region;
  cpu_baseline  the CPU oracle (fp64, direct loops) timed on this host on the
                first steps of the same run;
  breakdown     per-kernel average times (us) from the breakdown pass, and the
                paper's T (gradient) and tau (server update) times.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DQN TD-gradient+update steps/sec (transitions/sec); % MFMA peak and HBM GB/s"
PEAK_FP32_MFMA = 157.3e12   # MI355X dense fp32 matrix FLOP/s
PEAK_HBM = 8.0e12           # MI355X HBM3E bytes/s


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (one runtime per process)."""

    def __init__(self):
        import torch
        path = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
        if not os.path.exists(path):
            path = "libamdhip64.so"
        L = ctypes.CDLL(path)
        L.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        L.hipEventCreate.restype = ctypes.c_int
        L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                          ctypes.c_void_p]
        L.hipEventElapsedTime.restype = ctypes.c_int
        L.hipEventDestroy.argtypes = [ctypes.c_void_p]
        L.hipEventDestroy.restype = ctypes.c_int
        self.L = L

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self.L.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            out.append(e.value)
        return out

    def ms(self, a, b):
        v = ctypes.c_float()
        if self.L.hipEventElapsedTime(ctypes.byref(v), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return v.value

    def destroy(self, evs):
        for e in evs:
            self.L.hipEventDestroy(e)


def kernel_work(shape, B):
    """Algorithmic work per launch of each kernel for one TD step at batch B
    (theta^- = theta, so s and s' share one forward launch of 2B samples).
    Returns {name: (flop, bytes)}: MACs x 2 of the dense contractions; bytes
    for the memory-bound kernels."""
    dims = shape.conv_dims()
    H, A, F = shape.fc_hidden, shape.n_actions, shape.flat()
    P = shape.param_count()
    rec = shape.in_c * shape.in_h * shape.in_w
    w = {}
    for l, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(dims):
        macs = oh * ow * cout * cin * k * k
        w[f"conv{l+1}_fwd"] = (2 * (2 * B) * macs, 0)
        w[f"conv{l+1}_wgrad"] = (2 * B * macs, 0)
        if l > 0:
            w[f"conv{l+1}_dgrad"] = (2 * B * macs, 0)
    w["fc1_fwd"] = (2 * (2 * B) * H * F, 0)
    w["fc1_wgrad"] = (2 * B * H * F, 0)
    w["fc1_dgrad"] = (2 * B * H * F, 0)
    w["head"] = (2 * (2 * B) * A * H + 2 * B * H, 0)
    w["gather"] = (0, 4 * B * rec)             # read s and s', write both
    w["apply"] = (0, 12 * P)                   # SGD: read theta and g, write theta
    w["finalize"] = (0, 0)
    return w


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--breakdown-steps", type=int, default=100)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall time budget of the CPU-oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(reference kernel for scaling HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(one worker and its parameter server on one device); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import dqn_inputs as di
    import paper_1508_04186_amd as dq

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.init()
    hip = HipEvents()

    net, shape = dq.NET_SMALL, di.NET_S
    B, SIZE, SEED, LR, GAMMA = 32, 100_000, 1001, 2.5e-4, 0.99
    K, W = args.steps, args.warmup
    total = K + W

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    t0 = time.time()
    log(f"replay: generating {SIZE} transitions (seed {SEED})")
    hr = di.host_replay(SIZE, shape.n_actions, SEED)
    rec, ra, rr, rt = di.device_replay(SIZE, shape.n_actions, SEED, device=dev, host=hr)
    rp = dq.Replay(rec, ra, rr, rt, SIZE)
    log(f"replay ready in {time.time() - t0:.1f}s ({rec.numel() / 2**30:.2f} GiB on device)")

    theta0 = di.xavier_theta(shape, SEED)
    idx_host = di.index_stream(max(total, 1), B, SIZE, SEED)
    idx = torch.from_numpy(idx_host).to(dev)
    theta = torch.from_numpy(theta0).to(dev)
    P = dq.dqn_param_count(net)
    s = torch.empty((B, 4, 84, 84), dtype=torch.uint8, device=dev)
    sn = torch.empty_like(s)
    a = torch.empty(B, dtype=torch.int32, device=dev)
    r = torch.empty(B, dtype=torch.float32, device=dev)
    t = torch.empty(B, dtype=torch.uint8, device=dev)
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    ws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)
    stream = torch.cuda.current_stream()

    def step(i):
        dq.replay_gather(rp, idx[i], s, sn, a, r, t, stream=stream)
        dq.dqn_td_gradient(net, theta, theta, s, sn, a, r, t, GAMMA, g, loss, ws=ws, stream=stream)
        dq.ps_apply_update(dq.PS_SGD, theta, theta, None, g, LR, stream=stream)

    # ---- warmup (also the first W steps of the run)
    for i in range(W):
        step(i)
    torch.cuda.synchronize()

    # ---- breakdown pass on a copy of the state: per-kernel event pairs
    work = kernel_work(shape, B)
    names = dq.KERNEL_NAMES
    nb = args.breakdown_steps
    theta_save = theta.clone()
    ev_all = {}
    for kid, name in enumerate(names):
        if name in work:
            ev_all[kid] = hip.create(2 * nb)
            dq.profile_attach(kid, ev_all[kid])
    for i in range(nb):
        step(W + (i % max(K, 1)))
    torch.cuda.synchronize()
    per_kernel = {}
    for kid, evs in ev_all.items():
        used = dq.profile_used(kid)
        dq.profile_attach(kid, None)
        if used:
            per_kernel[names[kid]] = 1e3 * sum(hip.ms(evs[2 * j], evs[2 * j + 1]) for j in range(used)) / used
        hip.destroy(evs)
    theta.copy_(theta_save)
    torch.cuda.synchronize()
    dominant = max((k for k in per_kernel if work[k][0] > 0), key=lambda k: per_kernel[k])
    dom_id = names.index(dominant)
    log("breakdown (us/launch): " + ", ".join(f"{k} {v:.1f}" for k, v in per_kernel.items()))

    # ---- timed region: K steps, events around every launch of the dominant kernel
    dom_ev = hip.create(2 * K)
    dq.profile_attach(dom_id, dom_ev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(K):
        step(W + i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    used = dq.profile_used(dom_id)
    dq.profile_attach(dom_id, None)
    dom_us = 1e3 * sum(hip.ms(dom_ev[2 * j], dom_ev[2 * j + 1]) for j in range(used)) / max(used, 1)
    hip.destroy(dom_ev)
    final_loss = float(loss.item())
    log(f"timed {K} steps in {ms:.1f} ms; dominant kernel {dominant} {dom_us:.2f} us/launch")

    # ---- the paper's T (worker gradient) and tau (server update), separately
    def time_calls(fn, n):
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a0.record(stream)
        for _ in range(n):
            fn()
        a1.record(stream)
        torch.cuda.synchronize()
        return 1e3 * a0.elapsed_time(a1) / n
    th_copy = theta.clone()
    T_us = time_calls(lambda: (dq.replay_gather(rp, idx[0], s, sn, a, r, t, stream=stream),
                               dq.dqn_td_gradient(net, theta, theta, s, sn, a, r, t, GAMMA, g, loss,
                                                  ws=ws, stream=stream)), 200)
    tau_us = time_calls(lambda: dq.ps_apply_update(dq.PS_SGD, th_copy, th_copy, None, g, LR,
                                                   stream=stream), 200)

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * 2**20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mib} MiB done")

    steps_per_s = K / (ms / 1e3)
    flop, byts = work[dominant]
    roof = {
        "kernel": dominant,
        "bound": "mfma" if flop > 0 else "hbm",
        "achieved": (flop / (dom_us * 1e-6) / 1e12) if flop > 0 else (byts / (dom_us * 1e-6) / 1e9),
        "peak": PEAK_FP32_MFMA / 1e12 if flop > 0 else PEAK_HBM / 1e9,
        "unit": "TFLOP/s" if flop > 0 else "GB/s",
        "traffic": None,
        "per_launch": {"flop": flop, "bytes": byts, "avg_us": round(dom_us, 3), "launches": used},
    }
    roof["frac"] = roof["achieved"] / roof["peak"]

    out = {
        "metric": METRIC,
        "value": round(steps_per_s, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms / K, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "small Q-network, batch 32, 100,000-transition device replay, "
                        "2,000 sequential TD-gradient + SGD steps",
            "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "batch": B,
            "replay_transitions": SIZE, "update": "sgd", "lr": LR, "gamma": GAMMA,
            "target": "theta", "parallelism": "single worker + server on one GPU",
        },
        "transitions_per_s": round(steps_per_s * B, 1),
        "step_tflops": round(sum(v[0] for v in work.values()) * steps_per_s / 1e12, 4),
        "final_loss": final_loss,
        "roofline": roof,
        "breakdown": {"us_per_launch": {k: round(v, 2) for k, v in per_kernel.items()},
                      "T_us": round(T_us, 2), "tau_us": round(tau_us, 2),
                      "T_over_tau": round(T_us / tau_us, 2)},
    }

    if not args.no_cpu_baseline:
        import oracle
        log(f"cpu baseline: oracle steps for about {args.cpu_seconds:.0f}s")
        th = theta0.copy()
        n_done = 0
        c0 = time.perf_counter()
        while True:
            si, sni, ai, ri, ti = oracle.gather_from_host_replay(hr, idx_host[n_done])
            res = oracle.td_gradient(shape, th, None, si, sni, ai, ri, ti, float(np.float32(GAMMA)))
            th, _ = oracle.apply_update("sgd", th, None, res["grad"], float(np.float32(LR)))
            n_done += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds or n_done >= total:
                break
        out["cpu_baseline"] = {
            "value": round(n_done / el, 3), "unit": "steps/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"first {n_done} steps of the same run (batch 32, same replay and index "
                      f"stream), gather + fp64 TD gradient + SGD, {el:.1f}s wall",
        }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
