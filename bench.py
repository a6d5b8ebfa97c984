#!/usr/bin/env python3
"""Throughput of the DQN TD-gradient + parameter-server update hot path on one
MI355X (arXiv 1508.04186, Alg. 1 and Alg. 2), on seeded synthetic inputs.

Configurations (--config; the default line is config 4b, the largest
single-GPU workload):
  0   small Q-network (conv 16@8x8/4, conv 32@4x4/2, fc 256, fc 6), one
      batch of 32 uniform random states: TD gradient + SGD step, repeated.
  1   small Q-network, 100,000-transition replay in device memory,
      sequential steps of gather (batch 32) -> TD gradient -> SGD.
  2   small Q-network, 16 worker replicas on 16 streams + a server stream
      applying AdaGrad (lr 0.01, eps 1e-8) in order, gradients at most 4
      versions stale, 5,000 updates, 100,000-transition replay.
  3   large Q-network (conv 32@8x8/4, 64@4x4/2, 64@3x3/1, fc 512, fc 18),
      batch 256, 1,000,000-transition replay (28 GB), target network
      refreshed every 1,000 steps, SGD.
  4a  large Q-network, epsilon-greedy forward pass (eps 0.05) over 8,192
      states drawn from the 1,000,000-transition replay (read in place by
      the first convolution, dqn_forward_replay).
  4b  large Q-network, TD gradient + SGD at batch 2,048 from that replay.
  actor  Alg. 1 closed: 32 Snake games act with the small network
      (epsilon-greedy, annealed epsilon), store into a replay pooled over
      the games, and one TD gradient + SGD step follows on a minibatch of 32
      drawn from it (a step = one such iteration).
  observe  preprocessing phi on the device: 1,024 games each hand over a
      raw 176 x 176 RGB screen per step; phi (gray, crop, 2 x 2 mean) goes
      into each game's 4-frame state and the state into a replay keeping
      64 states per game, 10% of the games restarting per step (a step = one
      observe launch over all games).

--precision bf16 runs configs 3, 4a and 4b with the bf16-input variant;
--config 2 --sweep runs the server-bottleneck study over replicas and batch.

A step is one pass of the whole hot path over one batch (config 2: one
update; config 4a: one forward pass over 8,192 states).  Inputs are resident
in device memory before the timed region.  After warm-up, --repeats timed
runs of --steps consecutive steps each are bracketed by device
synchronizations and events, with nothing attached to the library's
measurement hook; `value` is their median and `timed_runs_ms` lists them.

The JSON line adds:
  step_tflops   the step's algorithmic FLOP (Alg. 1: forward of s and s',
                every weight and input gradient) times steps/s;
  roofline      the dominant kernel (largest time per step, from an
                event-bracketed breakdown pass before timing): its
                algorithmic FLOP (or bytes) per launch divided by its average
                launch time, measured in a separate pass over the steps that
                follow the timed runs, with a HIP event pair on the kernel's
                stream around every launch, less what a pair adds around a
                one-element fill kernel compared with that kernel's
                per-launch time in a chain (so the figure includes the
                kernel's dispatch and drain, as a rocprofv3 kernel duration
                does);
                `traffic` is the HBM bytes per launch from the committed
                rocprofv3 PMC summary (profiles/) while the kernel's source
                is unchanged;
  cpu_baseline  the CPU oracle (fp64, direct loops) timed on this host on a
                bounded sample of the same workload, on all its threads and
                (`single_thread`) on one;
  breakdown     per-kernel average times (us) and the paper's T (worker
                gradient time) and tau (server update time) on the GPU clock.
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
PEAK_BF16_MFMA = 2.5e15     # MI355X dense bf16 matrix FLOP/s
# Timed runs per configuration; `value` is their median.
REPEATS = 5
# Steps of the separate pass, after the timed runs, that times the dominant
# kernel with an event pair around each of its launches (the first launches
# of a short run read a few per cent slow).
KERNEL_PASS_STEPS = 200
F32 = np.float32


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch loaded (one runtime per process)."""

    def __init__(self):
        import torch
        path = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
        L = ctypes.CDLL(path if os.path.exists(path) else "libamdhip64.so")
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


def kernel_work(shape, B, forward_only=False, rule="sgd"):
    """Algorithmic work per launch of each kernel: {name: (flop, bytes)}.
    FLOP = 2 x multiply-adds of the dense contractions; bytes for the
    memory-bound kernels.  A TD step runs the forward on 2B samples (s under
    theta, s' under theta^-) in one launch per layer; dgrad and wgrad run on
    B samples."""
    dims = shape.conv_dims()
    H, A, F = shape.fc_hidden, shape.n_actions, shape.flat()
    P = shape.param_count()
    rec = shape.in_c * shape.in_h * shape.in_w
    nf = B if forward_only else 2 * B
    w = {}
    for l, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(dims):
        macs = oh * ow * cout * cin * k * k
        w[f"conv{l+1}_fwd"] = (2 * nf * macs, 0)
        if not forward_only:
            w[f"conv{l+1}_wgrad"] = (2 * B * macs, 0)
            if l > 0:
                w[f"conv{l+1}_dgrad"] = (2 * B * macs, 0)
    if len(dims) == 2:   # fused conv1 + conv2 launches of the small network
        w["conv12_fwd"] = (w["conv1_fwd"][0] + w["conv2_fwd"][0], 0)
        if not forward_only:
            w["conv12_bwd"] = (w["conv1_wgrad"][0] + w["conv2_wgrad"][0] + w["conv2_dgrad"][0], 0)
    w["fc1_fwd"] = (2 * nf * H * F, 0)
    w["head"] = (2 * nf * A * H, 0)
    if forward_only:
        w["gather"] = (0, 2 * B * rec)          # read s, write s
    else:
        w["fc1_wgrad"] = (2 * B * H * F, 0)
        w["fc1_dgrad"] = (2 * B * H * F, 0)
        # paired launches (weight + input gradient of one layer)
        w["fc1_bwd"] = (4 * B * H * F, 0)
        for l in range(1, len(dims)):
            w[f"conv{l+1}_bwd"] = (w[f"conv{l+1}_wgrad"][0] + w[f"conv{l+1}_dgrad"][0], 0)
        w["gather"] = (0, 4 * B * rec)          # read s and s', write both
        if len(dims) == 3:                      # conv2/conv3 weights into the fp32 kernels' lane order
            w["weight_repack"] = (0, 2 * 4 * 2 * (4 * 128 * 64 + 4 * 144 * 64) + 2 * 4 * (8 * 64 * 64 + 4 * 144 * 64))
        # SGD reads theta and g and writes theta; RMSProp and AdaGrad also
        # read and write their state
        ub = 12 * P if rule == "sgd" else 20 * P
        w["apply"] = (0, ub)
        w["finalize"] = (0, 0)
        w["finalize_apply"] = (0, ub)           # as apply, with the reductions fused
    return w


def step_flop(shape, B, forward_only=False):
    """Algorithmic FLOP of one step: 2 x multiply-adds of the forward pass of
    s through every layer (and of s' under theta^-, whose activations are
    not kept), and of every layer's weight gradient and every input gradient
    below the output layer except the first conv layer's (the input is
    data), plus the output layer's backward, which is sparse in the taken
    action (one row of B x hidden per gradient).  Forward only: the forward
    pass of B states."""
    dims = shape.conv_dims()
    H, A, F = shape.fc_hidden, shape.n_actions, shape.flat()
    nf = B if forward_only else 2 * B
    f = 0
    for l, (cin, ih, iw, cout, k, s, oh, ow) in enumerate(dims):
        macs = oh * ow * cout * cin * k * k
        f += 2 * nf * macs
        if not forward_only:
            f += 2 * B * macs * (2 if l > 0 else 1)
    f += 2 * nf * (H * F + A * H)
    if not forward_only:
        f += 4 * B * H * F + 4 * B * H
    return f


# Kernels whose roofline is reported (dense contractions and the
# memory-bound gather); the head and finalize are latency-bound reductions.
ROOFLINE_KERNELS = ("conv1_fwd", "conv2_fwd", "conv3_fwd", "conv12_fwd", "conv12_bwd", "fc1_fwd", "fc1_wgrad", "fc1_dgrad",
                    "conv1_wgrad", "conv2_wgrad", "conv3_wgrad", "conv2_dgrad", "conv3_dgrad",
                    "fc1_bwd", "conv2_bwd", "conv3_bwd", "gather", "apply", "finalize_apply")


class Profiler:
    """Event-bracketed timing of the library's kernels via dqn_profile.h.

    Nothing is attached while a run that sets `value` is timed.  Kernel times
    come from separate passes in which an event pair brackets every launch of
    the kernel; a pair adds a fixed time to what it brackets, measured here
    and subtracted (`overhead`)."""

    def __init__(self, hip):
        import torch
        import paper_1508_04186_amd as dq
        self.dq, self.hip = dq, hip
        self._overhead = None
        self._busy_out = torch.empty(2048, device="cuda")
        rec = hip.L.hipEventRecord
        rec.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        rec.restype = ctypes.c_int
        self.rec = rec

    def busy(self, ms=15.0):
        """Enqueue a matrix-core loop of about `ms` milliseconds on the current
        stream, so that the host enqueues what follows before the GPU reaches
        it (the spans measured after it hold no host time)."""
        iters = max(1, int(ms * 1e-3 * 1.2e14 / (2048 * 4 * 4 * 2048)))
        self.dq.profile_mfma_peak(self.dq.DQN_PEAK_FP32, 2048, iters, self._busy_out)

    def overhead(self):
        """Event-pair overhead in microseconds (measured once)."""
        if self._overhead is None:
            self._overhead = self.empty_pair_us()
        return self._overhead

    def breakdown(self, run, n, kernels):
        """{kernel: (us per launch, launches)} over `run()`, every launch of
        every listed kernel bracketed (an untimed pass)."""
        dq = self.dq
        evs = {}
        for name in kernels:
            kid = dq.KERNEL_NAMES.index(name)
            evs[kid] = self.hip.create(2 * n * 2)
            dq.profile_attach(kid, evs[kid])
        run()
        import torch
        torch.cuda.synchronize()
        out = {}
        for kid, ev in evs.items():
            used = dq.profile_used(kid)
            dq.profile_attach(kid, None)
            if used:
                raw = 1e3 * sum(self.hip.ms(ev[2 * j], ev[2 * j + 1]) for j in range(used)) / used
                out[dq.KERNEL_NAMES[kid]] = (raw - self.overhead(), used)
            self.hip.destroy(ev)
        return out

    def kernel_pass(self, name, run, launches):
        """Average launch time (us) of kernel `name` over a pass `run()` (the
        same steps as a timed run) with an event pair around every launch:
        (time less the pair overhead, raw pair time, launches bracketed)."""
        import torch
        dq = self.dq
        kid = dq.KERNEL_NAMES.index(name)
        ev = self.hip.create(2 * launches)
        dq.profile_attach(kid, ev, 1)
        torch.cuda.synchronize()
        run()
        torch.cuda.synchronize()
        used = dq.profile_used(kid)
        dq.profile_attach(kid, None)
        raw = 1e3 * sum(self.hip.ms(ev[2 * j], ev[2 * j + 1]) for j in range(used)) / max(used, 1)
        self.hip.destroy(ev)
        return raw - self.overhead(), raw, used

    def chain_us(self, fn, n):
        """GPU time (us) per call of n back-to-back calls fn(0..n-1) on the
        current stream, between one event before the first and one after the
        last, queued behind `busy` (so no host time is in it)."""
        import torch
        stream = torch.cuda.current_stream().cuda_stream
        ev = self.hip.create(2)
        torch.cuda.synchronize()
        self.busy()
        self.rec(ev[0], stream)
        for i in range(n):
            fn(i)
        self.rec(ev[1], stream)
        torch.cuda.synchronize()
        us = 1e3 * self.hip.ms(ev[0], ev[1]) / n
        self.hip.destroy(ev)
        return us

    def empty_pair_us(self, n=100):
        """What an event pair adds to the time of the launch it brackets: the
        mean bracketed time of a 16 MiB fill kernel, less that kernel's
        per-launch time in a chain of n launches (which, like a rocprofv3
        kernel duration, includes its dispatch and drain; a kernel this size
        leaves the chain no launch latency to hide).  Both are queued behind
        `busy` on the current stream, so neither holds host time."""
        import torch
        stream = torch.cuda.current_stream().cuda_stream
        x = torch.zeros(1 << 22, device="cuda")
        for _ in range(20):
            x.fill_(1.0)
        ev = self.hip.create(2 * n + 2)
        torch.cuda.synchronize()
        self.busy()
        self.rec(ev[2 * n], stream)
        for _ in range(n):
            x.fill_(1.0)
        self.rec(ev[2 * n + 1], stream)
        for j in range(n):
            self.rec(ev[2 * j], stream)
            x.fill_(1.0)
            self.rec(ev[2 * j + 1], stream)
        torch.cuda.synchronize()
        chain_us = 1e3 * self.hip.ms(ev[2 * n], ev[2 * n + 1]) / n
        us = 1e3 * sum(self.hip.ms(ev[2 * j], ev[2 * j + 1]) for j in range(n)) / n
        self.hip.destroy(ev)
        return us - chain_us


def timed_runs(run, lo, K, R):
    """R timed runs of the K consecutive steps run(lo, lo + K), then the next
    K, ...; nothing is attached to the measurement hook.  Returns (median ms,
    every run's ms, the first step after them)."""
    import torch
    ms = []
    for _ in range(R):
        ms.append(time_region(torch.cuda.synchronize, lambda a=lo: run(a, a + K)))
        lo += K
    return float(np.median(ms)), ms, lo


def worker_server_times(prof, grad_one, update_one, n=50):
    """The paper's T (one worker gradient: the minibatch read from the replay
    and the TD gradient) and tau (one server update: the apply kernel) on the
    GPU clock (Sec. IV.D.1): the time per call of n back-to-back calls, so
    1/tau is the update rate the server sustains and T the time a worker
    takes per gradient."""
    grad_one(0)
    update_one(0)
    T = prof.chain_us(grad_one, n)
    tau = prof.chain_us(update_one, n)
    return {"T_us": round(T, 2), "tau_us": round(tau, 2), "T_over_tau": round(T / tau, 2),
            "server_bound_updates_per_s": round(1e6 / tau, 1),
            "method": f"GPU time per call over {n} back-to-back calls on one stream, between events queued "
                      f"behind a matrix-core loop so that no host time is in them"}


def single_thread_baseline(grad_fn, update_fn, B, b, budget_s=3.0):
    """The oracle on one thread: grad_fn(b) computes the gradient (or the
    forward pass) of b of a step's B transitions and update_fn() the step's
    update (None: no update); the gradient is repeated for about budget_s and
    scaled by B / b, the update is timed once."""
    import oracle
    n0 = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        n, c0 = 0, time.perf_counter()
        while True:
            grad_fn(b)
            n += 1
            el = time.perf_counter() - c0
            if el >= budget_s:
                break
        c1 = time.perf_counter()
        if update_fn is not None:
            update_fn()
        upd = time.perf_counter() - c1
    finally:
        oracle.set_num_threads(n0)
    step_s = el / n * B / b + upd
    return {"value": round(1.0 / step_s, 5), "unit": "steps/s", "cores": 1,
            "sample": f"{n} x {b} of the {B} transitions of the first step ({el:.1f}s wall), scaled by "
                      f"{B}/{b}" + (f", plus one update ({upd * 1e3:.1f} ms)" if update_fn is not None else "")}


def measured_traffic(config, name):
    """HBM bytes per launch of kernel role `name` under `config`, from the
    committed rocprofv3 PMC summaries (profiles/*_traffic.md lines
    'traffic|config|role|read|write|source|sha256-16'), or None when no
    summary exists or the kernel's source changed since it was measured."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*_traffic.md"))):
        for line in open(path):
            f = line.strip().split("|")
            if len(f) == 7 and f[0] == "traffic" and f[1] == f"config {config}" and f[2] == name:
                h = hashlib.sha256()
                for part in f[5].split("+"):
                    src = os.path.join(ROOT, "paper_1508_04186_amd", "csrc", part)
                    if not os.path.exists(src):
                        return None
                    h.update(open(src, "rb").read())
                return int(f[3]) + int(f[4]) if h.hexdigest()[:16] == f[6] else None
    return None


# Large-network float32 kernels that run their contraction on bf16 MFMA with
# exact three-term bf16 splits of float32 operands: the number of bf16
# products per float32 product (both operands split: 6 of the 9 pairs; one
# operand exact in bf16, the input bytes: 3).  Their matrix ceiling is the
# bf16 dense peak divided by that count.
SPLIT_PRODUCTS = {"conv1_fwd": 3, "conv1_wgrad": 3, "conv2_fwd": 6, "conv3_fwd": 6}


def roofline(work, name, avg_us, launches, per_step_launches, raw_us=None, config=None,
             peak_flops=PEAK_FP32_MFMA, products=1):
    flop, byts = work[name]           # per step: per launch when a step launches the kernel several times
    if per_step_launches > 1:
        flop, byts = flop // per_step_launches, byts // per_step_launches
    if flop > 0:
        achieved, peak, unit, bound = flop / (avg_us * 1e-6) / 1e12, peak_flops / 1e12 / products, "TFLOP/s", "mfma"
    else:
        achieved, peak, unit, bound = byts / (avg_us * 1e-6) / 1e9, PEAK_HBM / 1e9, "GB/s", "hbm"
    out = {"kernel": name, "bound": bound, "achieved": round(achieved, 4), "peak": round(peak, 4),
           "unit": unit, "frac": round(achieved / peak, 6),
           "traffic": measured_traffic(config, name) if config is not None else None,
           "per_launch": {"flop": flop, "bytes": byts, "avg_us": round(avg_us, 3),
                          "launches": launches, "launches_per_step": per_step_launches}}
    if raw_us is not None:
        out["per_launch"]["event_pair_us"] = round(raw_us, 3)
        out["per_launch"]["event_overhead_us"] = round(raw_us - avg_us, 3)
    if products > 1:
        out["peak_basis"] = (f"float32 contraction on bf16 MFMA, {products} bf16 products per float32 product "
                             f"(exact three-term splits): bf16 dense {PEAK_BF16_MFMA / 1e12:.0f} TFLOP/s / {products}")
        out["frac_of_fp32_matrix_peak"] = round(achieved / (PEAK_FP32_MFMA / 1e12), 6)
    return out


def time_region(stream_sync, fn):
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    fn()
    stream_sync()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", default="4b", choices=["0", "1", "2", "3", "4a", "4b", "actor", "observe"])
    ap.add_argument("--steps", type=int, default=None, help="timed steps per run (default per config)")
    ap.add_argument("--repeats", type=int, default=REPEATS,
                    help="timed runs of --steps steps each; value is their median")
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--breakdown-steps", type=int, default=50)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall time budget of the CPU-oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--precision", default="fp32", choices=["fp32", "bf16"],
                    help="configs 3, 4a, 4b: fp32, or the bf16-input MFMA variant (fp32 accumulation)")
    ap.add_argument("--sweep", action="store_true",
                    help="config 2: the server-bottleneck sweep over replicas and batch instead of the fixed run")
    ap.add_argument("--no-denominators", action="store_true",
                    help="skip the measured matrix-core and HBM copy peaks")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB "
                         "(reference kernel for scaling HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this implementation has no multi-GPU path (workers and "
              "their parameter server run on one device); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.init()
    if args.precision == "bf16" and args.config not in ("3", "4a", "4b"):
        print("--precision bf16 applies to the large network (configs 3, 4a, 4b)", file=sys.stderr)
        sys.exit(2)
    if args.sweep and args.config != "2":
        print("--sweep applies to config 2", file=sys.stderr)
        sys.exit(2)
    out = {"0": bench_single, "1": bench_sequential, "2": bench_replica_sweep if args.sweep else bench_replicas,
           "3": bench_large, "4a": bench_forward, "4b": bench_large, "actor": bench_actor,
           "observe": bench_observe}[args.config](args)
    if not args.no_denominators:
        out["denominators"] = measure_denominators()
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * 2**20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mib} MiB done")
    print(json.dumps(out), flush=True)


def measure_denominators():
    """The roofline denominators as this GPU reaches them (dqn_profile.h): a
    pure matrix-core loop for fp32 and bf16 MFMA and a streaming copy of
    1 GiB, each the best of five launches timed with events; reported beside
    the spec-sheet peaks that the roofline fractions use."""
    import torch
    import paper_1508_04186_amd as dq
    workgroups = 256 * 8
    out = torch.empty(workgroups, device="cuda")

    def best_ms(fn, reps=5):
        fn()
        t = []
        for _ in range(reps):
            t.append(time_region(torch.cuda.synchronize, fn))
        return min(t)

    res = {}
    for name, dt, iters, spec in (("mfma_fp32_tflops", dq.DQN_PEAK_FP32, 4096, PEAK_FP32_MFMA / 1e12),
                                  ("mfma_bf16_tflops", dq.DQN_PEAK_BF16, 8192, PEAK_BF16_MFMA / 1e12)):
        flop = [0]

        def run():
            flop[0] = dq.profile_mfma_peak(dt, workgroups, iters, out)
        ms = best_ms(run)
        res[name] = {"spec": spec, "measured": round(flop[0] / (ms * 1e-3) / 1e12, 1)}
    n = 1 << 30
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ms = best_ms(lambda: dq.profile_stream_copy(src, dst, 256 * 16))
    res["hbm_copy_gbs"] = {"spec": PEAK_HBM / 1e9, "measured": round(2 * n / (ms * 1e-3) / 1e9, 1)}
    del src, dst
    log(f"denominators: {res}")
    return res


def base_record(K, W, ms, unit="steps/s"):
    return {"metric": METRIC, "value": round(K / (ms / 1e3), 2), "unit": unit, "n_gpus": 1,
            "steps": K, "warmup": W, "ms_per_step": round(ms / K, 5), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic"}


# ---------------------------------------------------------------------------
# configs 0 and 1

def _small_setup(dev):
    import dqn_inputs as di
    import paper_1508_04186_amd as dq
    return dq.NET_SMALL, di.NET_S


def bench_single(args):
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    hip = HipEvents()
    prof = Profiler(hip)
    net, shape = _small_setup(dev)
    B, SEED, LR, GAMMA = 32, 1000, 2.5e-4, 0.99
    K = args.steps or 2000
    W = args.warmup if args.warmup is not None else 50
    s_h = di.random_states(B, SEED)
    sn_h = di.random_states(B, SEED + 1)
    a_h, r_h, t_h = di.random_transitions(B, shape.n_actions, SEED + 2)
    th0 = di.xavier_theta(shape, SEED)
    d = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    s, sn, a, r, t = d(s_h), d(sn_h), d(a_h), d(r_h), d(t_h)
    theta = d(th0)
    P = dq.dqn_param_count(net)
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    ws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)

    def steps(n):
        for _ in range(n):
            dq.dqn_td_gradient(net, theta, theta, s, sn, a, r, t, GAMMA, g, loss, ws=ws)
            dq.ps_apply_update(dq.PS_SGD, theta, theta, None, g, LR)

    steps(W)
    work = kernel_work(shape, B)
    work.pop("gather")
    nb = min(args.breakdown_steps, K)
    bd = prof.breakdown(lambda: steps(nb), nb, list(work))
    dom = max((k for k in bd if k in ROOFLINE_KERNELS), key=lambda k: bd[k][0] * bd[k][1])
    R = args.repeats
    ms, runs, _ = timed_runs(lambda lo, hi: steps(hi - lo), 0, K, R)
    kp = KERNEL_PASS_STEPS
    dom_us, raw_us, used = prof.kernel_pass(dom, lambda: steps(kp), kp)
    rec = base_record(K, W, ms)
    rec["timed_runs_ms"] = [round(x, 3) for x in runs]
    rec["config"] = {"workload": f"config 0: small Q-network, one batch of 32 uniform random "
                                 f"states, TD gradient + SGD step (lr 2.5e-4) repeated {K} times "
                                 f"(median of {R} timed runs)",
                     "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "batch": B, "update": "sgd",
                     "gamma": GAMMA, "target": "theta"}
    rec["transitions_per_s"] = round(rec["value"] * B, 1)
    rec["step_tflops"] = round(step_flop(shape, B) * rec["value"] / 1e12, 4)
    rec["roofline"] = roofline(work, dom, dom_us, used, 1, raw_us, "0")
    rec["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()}}
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle steps for about {args.cpu_seconds:.0f}s")
        th = th0.copy()
        n, c0 = 0, time.perf_counter()
        while True:
            res = oracle.td_gradient(shape, th, None, s_h, sn_h, a_h, r_h, t_h, float(F32(GAMMA)))
            th, _ = oracle.apply_update("sgd", th, None, res["grad"], float(F32(LR)))
            n += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds:
                break
        rec["cpu_baseline"] = {"value": round(n / el, 3), "unit": "steps/s",
                               "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"{n} repetitions of the same step (fp64 TD gradient + "
                                         f"SGD), {el:.1f}s wall"}
        rec["cpu_baseline"]["single_thread"] = single_thread_baseline(
            lambda b: oracle.td_gradient(shape, th0, None, s_h[:b], sn_h[:b], a_h[:b], r_h[:b], t_h[:b],
                                         float(F32(GAMMA))),
            lambda: oracle.apply_update("sgd", th0, None, res["grad"], float(F32(LR))), B, B)
    return rec


def bench_sequential(args):
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    hip = HipEvents()
    prof = Profiler(hip)
    net, shape = _small_setup(dev)
    B, SIZE, SEED, LR, GAMMA = 32, 100_000, 1001, 2.5e-4, 0.99
    K = args.steps or 2000
    W = args.warmup if args.warmup is not None else 50
    t0 = time.time()
    log(f"replay: generating {SIZE} transitions (seed {SEED})")
    hr = di.host_replay(SIZE, shape.n_actions, SEED)
    rp = _filled_replay(dev, SIZE, shape.n_actions, SEED)
    rec = rp.frames
    log(f"replay ready in {time.time() - t0:.1f}s ({rec.numel() / 2**30:.2f} GiB on device)")
    th0 = di.xavier_theta(shape, SEED)
    R = args.repeats
    nb = min(args.breakdown_steps, K)
    kp = KERNEL_PASS_STEPS
    total = W + nb + R * K + kp
    idx_host = di.index_stream(total, B, SIZE, SEED)
    idx = torch.from_numpy(idx_host).to(dev)
    theta = torch.from_numpy(th0).to(dev)
    losses = torch.empty(total, dtype=torch.float32, device=dev)
    ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, 1), dtype=torch.uint8, device=dev)

    def run(lo, hi):
        dq.dqn_train_steps(net, theta, None, None, dq.PS_SGD, LR, 0.9, 0.0, GAMMA, rp, idx[lo:hi],
                           step0=lo, losses_out=losses[lo:hi], ws=ws)

    run(0, W)
    torch.cuda.synchronize()
    work = kernel_work(shape, B)
    bd = prof.breakdown(lambda: run(W, W + nb), nb, list(work))
    dom = max((k for k in bd if k in ROOFLINE_KERNELS), key=lambda k: bd[k][0] * bd[k][1])
    ms, runs, lo = timed_runs(run, W + nb, K, R)
    final_loss = float(losses[lo - 1].item())
    dom_us, raw_us, used = prof.kernel_pass(dom, lambda: run(lo, lo + kp), kp)
    log(f"timed {R} x {K} steps, median {ms:.1f} ms; dominant kernel {dom} {dom_us:.2f} us/launch")

    # the paper's T (worker gradient) and tau (server update) on the GPU clock
    g = torch.empty(dq.dqn_param_count(net), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    tws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)
    th_copy = theta.clone()
    Tt = worker_server_times(
        prof, lambda i: dq.dqn_td_gradient_replay(net, th_copy, th_copy, rp, idx[i], GAMMA, g, loss, ws=tws),
        lambda i: dq.ps_apply_update(dq.PS_SGD, th_copy, th_copy, None, g, LR))

    rec_ = base_record(K, W, ms)
    rec_["timed_runs_ms"] = [round(x, 3) for x in runs]
    rec_["config"] = {
        "workload": f"config 1: small Q-network, batch 32, 100,000-transition device replay, "
                    f"{K} sequential gather + TD-gradient + SGD steps (median of {R} timed runs)",
        "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "batch": B, "replay_transitions": SIZE,
        "update": "sgd", "lr": LR, "gamma": GAMMA, "target": "theta",
        "parallelism": "one worker + server on one GPU"}
    rec_["transitions_per_s"] = round(rec_["value"] * B, 1)
    rec_["step_tflops"] = round(step_flop(shape, B) * rec_["value"] / 1e12, 4)
    rec_["final_loss"] = final_loss
    rec_["roofline"] = roofline(work, dom, dom_us, used, 1, raw_us, "1")
    rec_["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()}, **Tt}
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle steps for about {args.cpu_seconds:.0f}s")
        th = th0.copy()
        n, c0 = 0, time.perf_counter()
        while True:
            si, sni, ai, ri, ti = oracle.gather_from_host_replay(hr, idx_host[n])
            res = oracle.td_gradient(shape, th, None, si, sni, ai, ri, ti, float(F32(GAMMA)))
            th, _ = oracle.apply_update("sgd", th, None, res["grad"], float(F32(LR)))
            n += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds or n >= total:
                break
        rec_["cpu_baseline"] = {
            "value": round(n / el, 3), "unit": "steps/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"first {n} steps of the same run (batch 32, same replay and index stream), "
                      f"gather + fp64 TD gradient + SGD, {el:.1f}s wall"}
        si, sni, ai, ri, ti = oracle.gather_from_host_replay(hr, idx_host[0])
        rec_["cpu_baseline"]["single_thread"] = single_thread_baseline(
            lambda b: oracle.td_gradient(shape, th0, None, si[:b], sni[:b], ai[:b], ri[:b], ti[:b],
                                         float(F32(GAMMA))),
            lambda: oracle.apply_update("sgd", th0, None, res["grad"], float(F32(LR))), B, B)
    return rec_


# ---------------------------------------------------------------------------
# config 2

def bench_actor(args):
    """Alg. 1 closed on one GPU: 32 Snake games act (epsilon-greedy forward
    with the annealed epsilon, one move each, the experiences stored in a
    replay pooled over the games that keeps the last 3,125 states per game,
    100,000 in all), then one TD gradient + SGD step on a minibatch of 32
    drawn uniformly from that replay, target network refreshed every 1,000
    iterations.  A step is one such iteration."""
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    net, shape = _small_setup(dev)
    E, N, B, SEED, LR, GAMMA, C = 32, 3125, 32, 1005, 2.5e-4, 0.99, 1000
    NMAX, EMIN, EMAX = 1000, 0.1, 1.0
    FILL = 64
    K = args.steps or 2000
    W = args.warmup if args.warmup is not None else 50
    R = args.repeats
    nb = min(args.breakdown_steps, K, 50)
    kp = KERNEL_PASS_STEPS
    total = FILL + W + nb + R * K + kp
    th0 = di.xavier_theta(shape, SEED)
    theta = torch.from_numpy(th0).to(dev)
    tgt = torch.empty_like(theta)
    games = dq.snake_games(E, dev)
    states = torch.empty((E, 4, 84, 84), dtype=torch.uint8, device=dev)
    rp = dq.ActorReplay(E, N, dev)
    gd_host = np.stack([di.game_draws(E, SEED, t) for t in range(-1, total)])
    gd = torch.from_numpy(gd_host).to(dev)
    ed = torch.from_numpy(np.stack([di.egreedy_draws(E, SEED * 100003 + t) for t in range(total)])).to(dev)
    eps = [float(F32(dq.dqn_anneal_epsilon(t, NMAX, EMIN, EMAX))) for t in range(total)]
    # minibatch of iteration t is drawn after its move: t + 1 moves made
    idx_host = np.stack([di.actor_minibatch(B, SEED, t, E, N, t + 1) for t in range(total)])
    idx = torch.from_numpy(idx_host).to(dev)
    acts = torch.empty(E, dtype=torch.int32, device=dev)
    rew = torch.empty(E, dtype=torch.float32, device=dev)
    term = torch.empty(E, dtype=torch.uint8, device=dev)
    fws = dq.workspace(net, E, dq.DQN_OP_FORWARD, dev)
    tws = torch.empty(dq.dqn_train_workspace_bytes(net, B, 1), dtype=torch.uint8, device=dev)
    losses = torch.empty(total, dtype=torch.float32, device=dev)

    def act(t):
        dq.dqn_act(net, theta, games, states, eps[t], ed[t], gd[t + 1], acts, rew, term, rp, t, ws=fws)

    def run(lo, hi):
        for t in range(lo, hi):
            act(t)
            if t >= FILL:
                dq.dqn_train_steps(net, theta, tgt, None, dq.PS_SGD, LR, 0.9, 0.0, GAMMA, rp.view, idx[t:t + 1],
                                   step0=t - FILL, target_period=C, losses_out=losses[t:t + 1], ws=tws)

    dq.snake_reset(games, gd[0], states, rp)
    run(0, FILL + W)
    torch.cuda.synchronize()
    hip = HipEvents()
    prof = Profiler(hip)
    work = kernel_work(shape, B)
    ebytes = E * 11 * 84 * 84          # read 3 frames, write the 4-frame state and its replay record
    work["snake_step"] = (0, ebytes)
    # the acting forward shares conv12_fwd, fc1_fwd and head with the TD step, so the roofline is
    # taken over kernels that only one of them launches
    cands = ("conv12_bwd", "fc1_bwd", "finalize_apply", "snake_step")
    bd = prof.breakdown(lambda: run(FILL + W, FILL + W + nb), nb, [k for k in work if k in cands] +
                        ["conv12_fwd", "fc1_fwd", "head"])
    # the games and the learner go on from where the breakdown left them
    dom = max((k for k in bd if k in cands), key=lambda k: bd[k][0] * bd[k][1])
    ms, runs, lo = timed_runs(run, FILL + W + nb, K, R)
    final_loss = float(losses[lo - 1].item())
    dom_us, raw_us, used = prof.kernel_pass(dom, lambda: run(lo, lo + kp), kp)
    out = base_record(K, W, ms)
    out["timed_runs_ms"] = [round(x, 3) for x in runs]
    out["config"] = {
        "workload": f"Alg. 1 closed: {E} Snake games (12x12 board, 84x84 frames) act epsilon-greedily with "
                    f"annealed epsilon and store into a {E * N:,}-experience replay pooled over the games, then "
                    f"one TD gradient + SGD step on a minibatch of {B}; target refreshed every {C}; "
                    f"{K} iterations (median of {R} timed runs)",
        "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "games": E, "batch": B, "replay_states": E * N,
        "update": "sgd", "lr": LR, "gamma": GAMMA, "epsilon": f"{EMAX} -> {EMIN} over {NMAX} iterations"}
    out["env_steps_per_s"] = round(out["value"] * E, 1)
    out["transitions_per_s"] = round(out["value"] * B, 1)
    out["final_loss"] = final_loss
    out["roofline"] = roofline(work, dom, dom_us, used, 1, raw_us, None)
    out["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()},
                        "launches_per_step": {k: v[1] / nb for k, v in bd.items()}}
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle loop for about {args.cpu_seconds:.0f}s")
        og = oracle.SnakeGames(E, gd_host[0])
        orp = oracle.SegmentedReplay(E, N)
        orp.append(-1, og.states)
        th = th0.copy()
        n, c0 = 0, time.perf_counter()
        while True:
            q = oracle.forward_q(shape, th, og.states)
            a = oracle.select_actions(q, eps[n], host_u64(ed, n))
            r, tt = og.step(a, gd_host[n + 1])
            orp.append(n, og.states, a, r, tt)
            s, sn, aa, rr, ttt = oracle.replay_gather(orp.frames, orp.rec, orp.rec, len(orp.frames), orp.action,
                                                      orp.reward, orp.terminal, idx_host[n])
            res = oracle.td_gradient(shape, th, None, s.reshape(B, 4, 84, 84), sn.reshape(B, 4, 84, 84), aa, rr,
                                     ttt, float(F32(GAMMA)))
            th, _ = oracle.apply_update("sgd", th, None, res["grad"], float(F32(LR)))
            n += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds or n >= total:
                break
        out["cpu_baseline"] = {"value": round(n / el, 3), "unit": "steps/s", "cores": oracle.num_threads(),
                               "kind": "oracle",
                               "sample": f"first {n} iterations of the same loop (act {E} games, store, "
                                         f"minibatch {B} TD gradient + SGD), {el:.1f}s wall"}
    return out


def bench_observe(args):
    """Preprocessing phi on the device (Sec. III.A, Fig. 2): every step, E
    games hand over one raw RGB screen each (resident in device memory, a
    pool of 8 screen sets cycled so that no step finds its screens in a
    cache); dqn_observe turns them into 84 x 84 gray frames, shifts them
    into the games' 4-frame states (restarting the games flagged terminal)
    and stores the states with the step's action, reward and flag in a
    replay that keeps the last N states per game."""
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    E, N, H, Wd, TOP, LEFT, F, POOL, SEED = 1024, 64, 176, 176, 4, 4, 2, 8, 1006
    K = args.steps or 2000
    W = args.warmup if args.warmup is not None else 50
    R = args.repeats
    kp = KERNEL_PASS_STEPS
    total = W + R * K + kp
    log(f"observe: generating {POOL} sets of {E} screens {H}x{Wd}")
    screens_host = [di.rgb_screens(E, SEED * 100 + i, H, Wd) for i in range(POOL)]
    screens = [torch.from_numpy(x).to(dev) for x in screens_host]
    rng = np.random.default_rng(SEED)
    acts_h = rng.integers(0, 18, size=(total, E)).astype(np.int32)
    rew_h = rng.integers(-1, 2, size=(total, E)).astype(np.int8)
    term_h = (rng.random((total, E)) < 0.1).astype(np.uint8)
    acts, rew, term = (torch.from_numpy(x).to(dev) for x in (acts_h, rew_h, term_h))
    states = torch.empty((E, 4, 84, 84), dtype=torch.uint8, device=dev)
    rp = dq.ActorReplay(E, N, dev)

    def run(lo, hi):
        for t in range(lo, hi):
            dq.dqn_observe(screens[(t + 1) % POOL], TOP, LEFT, F, states, acts[t], rew[t], term[t], rp, t)

    dq.dqn_observe(screens[0], TOP, LEFT, F, states, replay=rp, t=-1)
    run(0, W)
    torch.cuda.synchronize()
    hip = HipEvents()
    prof = Profiler(hip)
    ms, runs, lo = timed_runs(run, W, K, R)
    dom_us, raw_us, used = prof.kernel_pass("observe", lambda: run(lo, lo + kp), kp)
    # algorithmic bytes per launch, averaged over the timed steps: the 168 x 168 x 3 window of
    # every screen, the three kept frames of the games that go on, the 4-frame state and its
    # replay record (twice when the record lands in slot 0, which slot N repeats), the side
    # fields (read 4 + 1 + 1 bytes, write 3)
    FB = 84 * 84
    win = (84 * F) ** 2 * 3
    steps = np.arange(lo, lo + kp)
    kept = 3 * FB * (1 - term_h[lo:lo + kp]).sum(axis=1)
    mirror = ((steps + 1) % N == 0) * E * 4 * FB
    per = E * (win + 2 * 4 * FB + 9) + kept + mirror
    work = {"observe": (0, int(round(per.mean())))}
    out = base_record(K, W, ms)
    out["timed_runs_ms"] = [round(x, 3) for x in runs]
    out["metric"] = "observe steps/sec (raw RGB screens -> phi -> 4-frame states + replay); HBM GB/s"
    out["dtype"] = "u8"
    out["config"] = {
        "workload": f"phi of {E} raw {H}x{Wd} RGB screens per step (BT.601 gray, {84 * F}x{84 * F} crop at "
                    f"({TOP},{LEFT}), {F}x{F} mean) into {E} 4-frame states and a replay of {N} states per game; "
                    f"10% of the games restart per step; {K} steps (median of {R} timed runs)",
        "games": E, "screen": [H, Wd, 3], "factor": F, "replay_states": E * N}
    out["screens_per_s"] = round(out["value"] * E, 1)
    out["roofline"] = roofline(work, "observe", dom_us, used, 1, raw_us, "observe")
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle observe loop for about {args.cpu_seconds:.0f}s")
        orp = oracle.SegmentedReplay(E, N)
        ost = oracle.stack_frames(np.zeros((E, 4, 84, 84), np.uint8),
                                  oracle.preprocess(screens_host[0], TOP, LEFT, F), None, -1)
        orp.append(-1, ost)
        n, c0 = 0, time.perf_counter()
        while True:
            x = oracle.preprocess(screens_host[(n + 1) % POOL], TOP, LEFT, F)
            ost = oracle.stack_frames(ost, x, term_h[n], n)
            orp.append(n, ost, acts_h[n], rew_h[n].astype(np.float32), term_h[n])
            n += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds or n >= total:
                break
        out["cpu_baseline"] = {"value": round(n / el, 3), "unit": "steps/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {n} steps of the same loop ({E} screens each), {el:.1f}s wall"}
    return out


def host_u64(t, i):
    return t[i].cpu().numpy()


def bench_replica_sweep(args):
    """The server-bottleneck study on one GPU (Sec. IV.D.1, Fig. 3's
    question): updates/s of the replica schedule for P worker replicas and
    batch B, against the paper's model min(P/T, 1/tau) with T the time of
    one worker gradient and tau of one server update, both measured here
    alone.  Staleness is min(4, P - 1).  AdaGrad, small network, the
    100,000-transition replay."""
    import torch
    import dqn_inputs as di
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    net, shape = _small_setup(dev)
    SIZE, SEED, LR, EPS, GAMMA = 100_000, 1002, 0.01, 1e-8, 0.99
    U = args.steps or 1000
    log(f"replay: generating {SIZE} transitions (seed {SEED})")
    rp = _filled_replay(dev, SIZE, shape.n_actions, SEED)
    th0 = torch.from_numpy(di.xavier_theta(shape, SEED)).to(dev)
    P = dq.dqn_param_count(net)
    RS = dq.dqn_train_ring_stride(net)
    prof = Profiler(HipEvents())
    rows = []
    for B in (32, 128, 512):
        idx = torch.from_numpy(di.index_stream(U, B, SIZE, SEED + B)).to(dev)
        # T and tau alone
        g = torch.empty(P, dtype=torch.float32, device=dev)
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        G = torch.zeros(P, dtype=torch.float32, device=dev)
        tws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)
        th = th0.clone()
        Tt = worker_server_times(
            prof, lambda i: dq.dqn_td_gradient_replay(net, th, th, rp, idx[i], GAMMA, g, loss, ws=tws),
            lambda i: dq.ps_apply_update(dq.PS_ADAGRAD, th, th, G, g, LR, 0.0, EPS))
        T_us, tau_us = Tt["T_us"], Tt["tau_us"]
        del tws
        for R in (1, 2, 4, 8, 16, 32):
            S = min(4, R - 1)
            ring = torch.empty((S + 1) * RS, dtype=torch.float32, device=dev)
            ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, R), dtype=torch.uint8, device=dev)
            hs = dq.HipStreams(R + 1)

            def run(n):
                ring[:P].copy_(th0)
                G.zero_()
                torch.cuda.synchronize()
                dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA, rp, idx[:n], R, S,
                                      hs.handles, ws=ws)
            run(min(50, U))
            ring[:P].copy_(th0)
            G.zero_()
            ms = time_region(torch.cuda.synchronize,
                             lambda: dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA, rp,
                                                           idx, R, S, hs.handles, ws=ws))
            hs.close()
            ups = U / (ms * 1e-3)
            model = min(R / (T_us * 1e-6), 1.0 / (tau_us * 1e-6))
            rows.append({"batch": B, "replicas": R, "staleness": S, "updates_per_s": round(ups, 1),
                         "transitions_per_s": round(ups * B, 1), "T_us": round(T_us, 2),
                         "tau_us": round(tau_us, 2), "model_updates_per_s": round(model, 1)})
            log(f"B={B} P={R} S={S}: {ups:.0f} updates/s (T {T_us:.1f} us, tau {tau_us:.1f} us, "
                f"model {model:.0f})")
            del ring, ws
    best = max(rows, key=lambda x: x["transitions_per_s"])
    out = base_record(U, 0, U / best["updates_per_s"] * 1e3)
    out["config"] = {"workload": "server-bottleneck sweep: small Q-network, AdaGrad, replicas P in 1..32 on "
                                 "streams, batch B in 32/128/512, 100,000-transition device replay",
                     "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "replay_transitions": SIZE}
    out["note"] = "value is the best updates/s over the sweep; every point is in sweep"
    out["sweep"] = rows
    return out


def bench_replicas(args):
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    net, shape = _small_setup(dev)
    B, SIZE, SEED, LR, EPS, GAMMA, R_, S = 32, 100_000, 1002, 0.01, 1e-8, 0.99, 16, 4
    U = args.steps or 5000
    W = args.warmup if args.warmup is not None else 100
    log(f"replay: generating {SIZE} transitions (seed {SEED})")
    hr = di.host_replay(SIZE, shape.n_actions, SEED)
    rp = _filled_replay(dev, SIZE, shape.n_actions, SEED)
    th0 = di.xavier_theta(shape, SEED)
    idx_host = di.index_stream(U, B, SIZE, SEED)
    idx = torch.from_numpy(idx_host).to(dev)
    P = dq.dqn_param_count(net)
    RS = dq.dqn_train_ring_stride(net)
    ring = torch.empty((S + 1) * RS, dtype=torch.float32, device=dev)
    G = torch.zeros(P, dtype=torch.float32, device=dev)
    losses = torch.empty(U, dtype=torch.float32, device=dev)
    ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, R_), dtype=torch.uint8, device=dev)
    hs = dq.HipStreams(R_ + 1)

    def run(n):
        ring[:P].copy_(torch.from_numpy(th0).to(dev))
        G.zero_()
        torch.cuda.synchronize()
        dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA, rp, idx[:n], R_, S,
                              hs.handles, losses_out=losses[:n], ws=ws)

    run(W)
    torch.cuda.synchronize()
    hip = HipEvents()
    prof = Profiler(hip)
    work = kernel_work(shape, B, rule="adagrad")
    nb = min(args.breakdown_steps, U)
    bd = prof.breakdown(lambda: run(nb), nb, list(work))
    dom = max((k for k in bd if k in ROOFLINE_KERNELS), key=lambda k: bd[k][0] * bd[k][1])
    # timed: all U updates from the initial parameters, R times (the setup
    # copies are outside the timed regions)
    R = args.repeats
    runs = []
    for _ in range(R):
        ring[:P].copy_(torch.from_numpy(th0).to(dev))
        G.zero_()
        runs.append(time_region(torch.cuda.synchronize,
                                lambda: dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA,
                                                              rp, idx, R_, S, hs.handles, losses_out=losses,
                                                              ws=ws)))
    ms = float(np.median(runs))
    final_loss = float(losses[U - 1].item())
    # the dominant kernel's launch time over a separate run of the first updates
    kp = min(U, KERNEL_PASS_STEPS)
    ring[:P].copy_(torch.from_numpy(th0).to(dev))
    G.zero_()
    dom_us, raw_us, used = prof.kernel_pass(
        dom, lambda: dq.dqn_train_replicas(net, ring, G, dq.PS_ADAGRAD, LR, 0.0, EPS, GAMMA, rp, idx[:kp], R_, S,
                                           hs.handles, ws=ws), kp * max(1, round(bd[dom][1] / nb)))
    hs.close()
    log(f"timed {R} x {U} updates, median {ms:.1f} ms")
    # T and tau (paper Sec. IV.D.1): one worker gradient, one server update
    g = torch.empty(P, dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    tws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)
    th = ring[:P].clone()
    G2 = G.clone()
    Tt = worker_server_times(
        prof, lambda i: dq.dqn_td_gradient_replay(net, th, th, rp, idx[i], GAMMA, g, loss, ws=tws),
        lambda i: dq.ps_apply_update(dq.PS_ADAGRAD, th, th, G2, g, LR, 0.0, EPS))

    out = base_record(U, W, ms)
    out["config"] = {
        "workload": "config 2: 16 small-Q-network worker replicas on 16 streams + server stream, "
                    f"AdaGrad (lr 0.01, eps 1e-8), staleness <= 4, {U} updates of batch 32, "
                    f"100,000-transition device replay (median of {R} timed runs)",
        "net": "conv16@8x8/4-conv32@4x4/2-fc256-fc6", "batch": B, "replicas": R_, "staleness": S,
        "replay_transitions": SIZE, "update": "adagrad", "lr": LR, "gamma": GAMMA,
        "parallelism": "16 replicas + 1 server on one GPU (streams)"}
    out["transitions_per_s"] = round(out["value"] * B, 1)
    out["step_tflops"] = round(step_flop(shape, B) * out["value"] / 1e12, 4)
    out["final_loss"] = final_loss
    out["roofline"] = roofline(work, dom, dom_us, used, 1, raw_us, "2")
    out["roofline"]["note"] = ("kernels of up to five updates run concurrently on the replica "
                               "streams, so the event-bracketed launch time (a separate run of the "
                               "first updates) includes sharing the GPU with them")
    out["timed_runs_ms"] = [round(x, 3) for x in runs]
    out["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()}, **Tt}
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle stale-schedule updates for about {args.cpu_seconds:.0f}s")
        n_try = 8
        c0 = time.perf_counter()
        oracle.stale_replica_training(shape, th0, hr, idx_host[:n_try], float(F32(GAMMA)),
                                      float(F32(LR)), S, rule="adagrad", eps=float(F32(EPS)))
        per = (time.perf_counter() - c0) / n_try
        n = max(1, min(U, int(args.cpu_seconds / per)))
        c0 = time.perf_counter()
        oracle.stale_replica_training(shape, th0, hr, idx_host[:n], float(F32(GAMMA)),
                                      float(F32(LR)), S, rule="adagrad", eps=float(F32(EPS)))
        el = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": round(n / el, 3), "unit": "steps/s",
                               "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"first {n} updates of the same schedule, {el:.1f}s wall"}
        si, sni, ai, ri, ti = oracle.gather_from_host_replay(hr, idx_host[0])
        res = oracle.td_gradient(shape, th0, None, si, sni, ai, ri, ti, float(F32(GAMMA)))
        G0 = np.zeros_like(th0)
        out["cpu_baseline"]["single_thread"] = single_thread_baseline(
            lambda b: oracle.td_gradient(shape, th0, None, si[:b], sni[:b], ai[:b], ri[:b], ti[:b],
                                         float(F32(GAMMA))),
            lambda: oracle.apply_update("adagrad", th0, G0, res["grad"], float(F32(LR)), eps=float(F32(EPS))),
            B, B)
    return out


# ---------------------------------------------------------------------------
# configs 3, 4a and 4b (large network, 1,000,000-transition replay)

def _filled_replay(dev, size, n_actions, seed):
    """Device replay of `size` stacked 4 x 84 x 84 records and side arrays,
    written on the device by replay_fill_synthetic (the same bytes as the
    host generator dqn_inputs.host_replay)."""
    import torch
    import paper_1508_04186_amd as dq
    rec = torch.empty((size, 4, 84, 84), dtype=torch.uint8, device=dev)
    a = torch.empty(size, dtype=torch.uint8, device=dev)
    r = torch.empty(size, dtype=torch.int8, device=dev)
    t = torch.empty(size, dtype=torch.uint8, device=dev)
    rp = dq.Replay(rec, a, r, t, size)
    dq.replay_fill_synthetic(rp, n_actions, seed)
    torch.cuda.synchronize()
    return rp


def _large_replay(dev, size, seed):
    import dqn_inputs as di
    import paper_1508_04186_amd as dq
    t0 = time.time()
    log(f"replay: generating {size} transitions (seed {seed}) into device memory")
    rp = _filled_replay(dev, size, di.NET_L.n_actions, seed)
    log(f"replay ready in {time.time() - t0:.1f}s ({rp.frames.numel() / 2**30:.2f} GiB on device)")
    return rp


def bench_large(args):
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    hip = HipEvents()
    prof = Profiler(hip)
    bf16 = args.precision == "bf16"
    net, shape = (dq.NET_LARGE_BF16 if bf16 else dq.NET_LARGE), di.NET_L
    SIZE, SEED, LR, GAMMA = 1_000_000, 1003, 2.5e-4, 0.99
    if args.config == "3":
        B, C = 256, 1000
        K = args.steps or 3000
        W = args.warmup if args.warmup is not None else 20
    else:
        B, C = 2048, 0
        K = args.steps or 100
        W = args.warmup if args.warmup is not None else 5
    R = args.repeats
    nb = min(args.breakdown_steps, K, 20)
    kp = KERNEL_PASS_STEPS
    total = W + nb + R * K + kp
    rp = _large_replay(dev, SIZE, SEED)
    th0 = di.xavier_theta(shape, SEED)
    idx_host = di.index_stream(total, B, SIZE, SEED)
    idx = torch.from_numpy(idx_host).to(dev)
    theta = torch.from_numpy(th0).to(dev)
    tgt = torch.empty_like(theta) if C else None
    losses = torch.empty(total, dtype=torch.float32, device=dev)
    ws = torch.empty(dq.dqn_train_workspace_bytes(net, B, 1), dtype=torch.uint8, device=dev)

    def run(lo, hi):
        dq.dqn_train_steps(net, theta, tgt, None, dq.PS_SGD, LR, 0.9, 0.0, GAMMA, rp, idx[lo:hi],
                           step0=lo, target_period=C, losses_out=losses[lo:hi], ws=ws)

    run(0, W)
    torch.cuda.synchronize()
    work = kernel_work(shape, B)
    bd = prof.breakdown(lambda: run(W, W + nb), nb, list(work))
    dom = max((k for k in bd if k in ROOFLINE_KERNELS), key=lambda k: bd[k][0] * bd[k][1])
    lps = max(1, round(bd[dom][1] / nb))          # launches of the kernel per step
    ms, runs, lo = timed_runs(run, W + nb, K, R)
    final_loss = float(losses[lo - 1].item())
    dom_us, raw_us, used = prof.kernel_pass(dom, lambda: run(lo, lo + kp), kp * lps)
    log(f"timed {R} x {K} steps, median {ms:.1f} ms; dominant kernel {dom} {dom_us:.2f} us/launch")
    # the paper's T (worker gradient) and tau (server update) on the GPU clock
    g = torch.empty(dq.dqn_param_count(net), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    tws = dq.workspace(net, B, dq.DQN_OP_TD_GRADIENT, dev)
    th_copy = theta.clone()
    Tt = worker_server_times(
        prof, lambda i: dq.dqn_td_gradient_replay(net, th_copy, th_copy, rp, idx[i], GAMMA, g, loss, ws=tws),
        lambda i: dq.ps_apply_update(dq.PS_SGD, th_copy, th_copy, None, g, LR), n=20)
    del tws
    out = base_record(K, W, ms)
    name = "config 3" if args.config == "3" else "config 4b"
    out["config"] = {
        "workload": f"{name}: large Q-network, batch {B}, 1,000,000-transition device replay, "
                    f"{K} sequential gather + TD-gradient + SGD steps (median of {R} timed runs)"
                    + (f", target network refreshed every {C} steps" if C else "")
                    + (", bf16-input MFMA contractions with fp32 accumulation" if bf16 else ""),
        "net": "conv32@8x8/4-conv64@4x4/2-conv64@3x3/1-fc512-fc18", "batch": B,
        "replay_transitions": SIZE, "update": "sgd", "lr": LR, "gamma": GAMMA,
        "target": f"refresh every {C}" if C else "theta"}
    if bf16:
        out["dtype"] = "bf16"
        out["config"]["accumulate"] = "f32"
    out["timed_runs_ms"] = [round(x, 3) for x in runs]
    out["transitions_per_s"] = round(out["value"] * B, 1)
    out["step_tflops"] = round(step_flop(shape, B) * out["value"] / 1e12, 4)
    out["final_loss"] = final_loss
    out["roofline"] = roofline(work, dom, dom_us, used, lps, raw_us,
                               args.config + (" bf16" if bf16 else ""),
                               PEAK_BF16_MFMA if bf16 else PEAK_BF16_MFMA if dom in SPLIT_PRODUCTS else PEAK_FP32_MFMA,
                               1 if bf16 else SPLIT_PRODUCTS.get(dom, 1))
    out["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()},
                        "per_layer_tflops": {k: round(work[k][0] / (v[0] * (v[1] / nb) * 1e-6) / 1e12, 3)
                                             for k, v in bd.items() if work[k][0] > 0}, **Tt}
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle steps for about {args.cpu_seconds:.0f}s")
        th = th0.copy()
        n, c0 = 0, time.perf_counter()
        while True:
            s, sn, a, r, t = di.transitions_at(SEED, idx_host[n], shape.n_actions, SIZE)
            res = oracle.td_gradient(shape, th, None, s, sn, a, r, t, float(F32(GAMMA)), bf16=bf16)
            th, _ = oracle.apply_update("sgd", th, None, res["grad"], float(F32(LR)))
            n += 1
            el = time.perf_counter() - c0
            if el >= args.cpu_seconds or n >= total:
                break
        out["cpu_baseline"] = {"value": round(n / el, 4), "unit": "steps/s",
                               "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"first {n} step(s) of the same run (batch {B}), fp64 TD "
                                         f"gradient{' (bf16-input variant)' if bf16 else ''} + SGD, "
                                         f"{el:.1f}s wall"}
        s, sn, a, r, t = di.transitions_at(SEED, idx_host[0][:32], shape.n_actions, SIZE)
        out["cpu_baseline"]["single_thread"] = single_thread_baseline(
            lambda b: oracle.td_gradient(shape, th0, None, s[:b], sn[:b], a[:b], r[:b], t[:b],
                                         float(F32(GAMMA)), bf16=bf16),
            lambda: oracle.apply_update("sgd", th0, None, res["grad"], float(F32(LR))), B, 32)
    return out


def bench_forward(args):
    import torch
    import dqn_inputs as di
    import oracle
    import paper_1508_04186_amd as dq
    dev = torch.device("cuda:0")
    hip = HipEvents()
    prof = Profiler(hip)
    bf16 = args.precision == "bf16"
    net, shape = (dq.NET_LARGE_BF16 if bf16 else dq.NET_LARGE), di.NET_L
    SIZE, SEED, B, EPS = 1_000_000, 1004, 8192, F32(0.05)
    K = args.steps or 200
    W = args.warmup if args.warmup is not None else 10
    R = args.repeats
    nb = min(args.breakdown_steps, K, 20)
    kp = KERNEL_PASS_STEPS
    total = W + nb + R * K + kp
    rp = _large_replay(dev, SIZE, SEED)
    th0 = di.xavier_theta(shape, SEED)
    rng = np.random.default_rng(SEED)
    idx_host = rng.integers(0, SIZE, size=(total, B), dtype=np.int64)
    idx = torch.from_numpy(idx_host).to(dev)
    draws = torch.from_numpy(di.egreedy_draws(B, SEED)).to(dev)
    theta = torch.from_numpy(th0).to(dev)
    q = torch.empty((B, net.n_actions), dtype=torch.float32, device=dev)
    act = torch.empty(B, dtype=torch.int32, device=dev)
    ws = dq.workspace(net, B, dq.DQN_OP_FORWARD, dev)

    def run(lo, hi):
        for i in range(lo, hi):
            dq.dqn_forward_replay(net, theta, rp, idx[i], float(EPS), draws, q, act, ws=ws)

    run(0, W)
    torch.cuda.synchronize()
    work = kernel_work(shape, B, forward_only=True)
    work.pop("gather")
    bd = prof.breakdown(lambda: run(W, W + nb), nb, list(work))
    dom = max((k for k in bd if k in ROOFLINE_KERNELS), key=lambda k: bd[k][0] * bd[k][1])
    lps = max(1, round(bd[dom][1] / nb))
    ms, runs, lo = timed_runs(run, W + nb, K, R)
    dom_us, raw_us, used = prof.kernel_pass(dom, lambda: run(lo, lo + kp), kp * lps)
    log(f"timed {R} x {K} forward passes, median {ms:.1f} ms; dominant kernel {dom} {dom_us:.2f} us/launch")
    out = base_record(K, W, ms)
    out["config"] = {
        "workload": f"config 4a: large Q-network, epsilon-greedy (eps 0.05) forward pass over 8,192 "
                    f"states read in place from a 1,000,000-transition device replay, {K} passes "
                    f"(median of {R} timed runs)"
                    + (", bf16-input MFMA contractions with fp32 accumulation" if bf16 else ""),
        "net": "conv32@8x8/4-conv64@4x4/2-conv64@3x3/1-fc512-fc18", "batch": B,
        "replay_transitions": SIZE, "epsilon": float(EPS)}
    if bf16:
        out["dtype"] = "bf16"
        out["config"]["accumulate"] = "f32"
    out["timed_runs_ms"] = [round(x, 3) for x in runs]
    out["states_per_s"] = round(out["value"] * B, 1)
    out["step_tflops"] = round(step_flop(shape, B, forward_only=True) * out["value"] / 1e12, 4)
    out["roofline"] = roofline(work, dom, dom_us, used, lps, raw_us, "4a" + (" bf16" if bf16 else ""),
                               PEAK_BF16_MFMA if bf16 else PEAK_BF16_MFMA if dom in SPLIT_PRODUCTS else PEAK_FP32_MFMA,
                               1 if bf16 else SPLIT_PRODUCTS.get(dom, 1))
    out["breakdown"] = {"us_per_launch": {k: round(v[0], 2) for k, v in bd.items()},
                        "per_layer_tflops": {k: round(work[k][0] / (v[0] * (v[1] / nb) * 1e-6) / 1e12, 3)
                                             for k, v in bd.items() if work[k][0] > 0}}
    if not args.no_cpu_baseline:
        n = 512
        s, _, _, _, _ = di.transitions_at(SEED, idx_host[0][:n], shape.n_actions, SIZE)
        c0 = time.perf_counter()
        qr = oracle.forward_q(shape, th0, s, bf16=bf16)
        oracle.select_actions(qr, float(EPS), di.egreedy_draws(B, SEED)[:n])
        el = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": round(n / el / B, 5), "unit": "steps/s",
                               "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"fp64 forward + epsilon-greedy choice on {n} of the "
                                         f"8,192 states ({el:.1f}s wall), scaled to 8,192"}
        out["cpu_baseline"]["single_thread"] = single_thread_baseline(
            lambda b: oracle.forward_q(shape, th0, s[:b], bf16=bf16), None, B, 32)
    return out


if __name__ == "__main__":
    main()
