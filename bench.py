#!/usr/bin/env python3
"""InPlace-ABN training forward + backward throughput on one MI355X.

One step is the whole hot path over one batch of synthetic input: for every
layer of the workload the training forward (batch statistics, then
normalise + affine + leaky ReLU written over x) and, in reverse layer order,
the backward (recover y and xhat from z, reduce dy and dy*xhat, then dx
written over dz), all through libiabn's C entry points.  Each layer has its
own activation and gradient buffers, so a step streams the whole working set
through HBM the way a network does.

Default workload: the ResNet-101-like backbone sweep (N=8, 512x512 input,
output stride 8; 33 BN layers in four shape groups, fp16 storage, fp32
arithmetic), 1.14e9 elements per tensor.

Output: one JSON line (see the keys below).  ``value`` is elements/s of the
whole fwd+bwd step (elements = sum over layers of N*C*H*W).  ``roofline``
covers the kernel with the largest share of the step, timed live with HIP
events on the stream it runs on, in a separate pass that calls the two
phases of each entry point with events between them.  ``cpu_baseline`` is the
double-precision oracle on the host's cores over whole layers of the same
workload, bounded in time.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "IABN fwd+bwd elements/s and achieved HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBPS = 8000.0

# Algorithmic HBM bytes per element of each kernel, in units of the storage
# size b: what the kernel must read and write once.
KERNEL_BYTES_PER_ELEM = {"fwd_stats": 1, "fwd_apply": 2, "bwd_reduce": 2, "bwd_apply": 3}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload index (1-5)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the oracle baseline (0 disables it)")
    ap.add_argument("--no-kernel-pass", action="store_true",
                    help="skip the per-kernel event pass (no roofline object)")
    ap.add_argument("--phase-kernels", action="store_true",
                    help="also time the phase entry points (the streaming kernels)")
    return ap.parse_args()


class Layer:
    pass


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if os.environ.get("WORLD_SIZE", "1") != "1":
        print("bench.py runs as a single process on one GPU", file=sys.stderr)
        sys.exit(2)

    import paper_1712_02616_amd as iabn

    print(json.dumps(measure(iabn.load(), args)), flush=True)


def measure(lib, args):
    """Run the benchmark with a loaded libiabn handle; returns the JSON record."""
    import numpy as np
    import torch

    import paper_1712_02616_amd as iabn
    import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = workloads.WORKLOADS[args.config]
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[w.dtype]
    code = iabn.DTYPE_CODES[tdt]
    b = workloads.ELEM_BYTES[w.dtype]
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)

    # ---------------------------------------------------------------- inputs
    t0 = time.time()
    host_layers = []
    layers = []
    ws_bytes = max(lib.iabn_workspace_size(n, c, hw, code) for n, c, hw in w.layers)
    workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    wsp = ctypes.c_void_p(workspace.data_ptr())
    for li, (N, C, HW) in enumerate(w.layers):
        inp = workloads.workload_layer(w, li)
        host_layers.append(inp)
        L = Layer()
        L.shape = (N, C, HW)
        L.E = N * C * HW

        def dev_tensor(a):
            if w.dtype == "bf16":
                return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
            return torch.from_numpy(a).to(dev)
        L.x0 = dev_tensor(inp.x)       # pristine copies, restored between passes
        L.dz0 = dev_tensor(inp.dz)
        L.x = torch.empty_like(L.x0)
        L.dz = torch.empty_like(L.dz0)
        L.gamma = torch.from_numpy(inp.gamma).to(dev)
        L.beta = torch.from_numpy(inp.beta).to(dev)
        L.rm = torch.zeros(C, device=dev)
        L.rv = torch.ones(C, device=dev)
        L.sm = torch.empty(C, device=dev)
        L.sv = torch.empty(C, device=dev)
        L.dg = torch.empty(C, device=dev)
        L.db = torch.empty(C, device=dev)
        p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        L.fwd = (p(L.x), code, p(L.gamma), p(L.beta), p(L.rm), p(L.rv), p(L.sm), p(L.sv),
                 w.eps, w.momentum, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.stats = (p(L.x), code, N, C, HW, wsp, ws_bytes, sp)
        L.bwd = (p(L.x), p(L.dz), code, p(L.gamma), p(L.beta), p(L.sv), p(L.dg), p(L.db),
                 w.eps, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.reduce = (p(L.x), p(L.dz), code, p(L.gamma), p(L.beta), w.slope, N, C, HW, wsp,
                    ws_bytes, sp)
        layers.append(L)
    torch.cuda.synchronize()
    E_total = sum(L.E for L in layers)
    log("inputs ready: %d layers, %.3g elements per tensor, %.1f s" % (len(layers), E_total,
                                                                       time.time() - t0))

    def check(rc, what):
        if rc != 0:
            raise RuntimeError("%s failed: %s" % (what, lib.iabn_last_error().decode()))

    def refresh():
        for L in layers:
            L.x.copy_(L.x0)
            L.dz.copy_(L.dz0)
            L.rm.zero_()
            L.rv.fill_(1.0)

    fwd_train, backward = lib.iabn_forward_train, lib.iabn_backward

    def step():
        for L in layers:
            check(fwd_train(*L.fwd), "iabn_forward_train")
        for L in reversed(layers):
            check(backward(*L.bwd), "iabn_backward")

    # ---------------------------------------------------------------- timed steps
    refresh()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    refresh()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    ev_ms_per_step = ev0.elapsed_time(ev1) / args.steps
    value = E_total / (ms_per_step * 1e-3)
    sched_bytes = 8 * E_total * b
    floor_bytes = 5 * E_total * b
    finite = all(bool(torch.isfinite(L.dz).all()) and bool(torch.isfinite(L.x).all())
                 for L in layers)
    log("timed %d steps: %.3f ms/step (events %.3f), %.3g elements/s, finite=%s"
        % (args.steps, ms_per_step, ev_ms_per_step, value, finite))

    # ---------------------------------------------------------------- per-kernel pass
    # The step's two entry points timed one by one with HIP events on the
    # stream they run on.  On this workload each entry point is a single
    # kernel (the channel-resident forward / backward); its algorithmic bytes
    # are what the operation must move at least once: forward reads x and
    # writes z (2 E b), backward reads z and dz and writes dx (3 E b).
    roofline = None
    kernels = None
    phase_kernels = None

    def timed_pass(calls):
        """calls: list of (name, fn, args, bytes_per_elem) per layer in step order."""
        tot_ms, tot_bytes, launches = {}, {}, {}
        refresh()
        torch.cuda.synchronize()
        for _ in range(args.steps):
            evs = []
            for name, fn, cargs, bpe, E in calls:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                check(fn(*cargs), name)
                e1.record(stream)
                evs.append((name, e0, e1, bpe * E * b))
            torch.cuda.synchronize()
            for name, e0, e1, nbytes in evs:
                tot_ms[name] = tot_ms.get(name, 0.0) + e0.elapsed_time(e1)
                tot_bytes[name] = tot_bytes.get(name, 0) + nbytes
                launches[name] = launches.get(name, 0) + 1
        out = {}
        for name in tot_ms:
            out[name] = {"avg_us": round(tot_ms[name] / launches[name] * 1e3, 3),
                         "launches": launches[name],
                         "alg_bytes_per_launch": tot_bytes[name] // launches[name],
                         "achieved_gbps": round(tot_bytes[name] / (tot_ms[name] * 1e-3) / 1e9, 1),
                         "share_of_pass": tot_ms[name]}
        total = sum(tot_ms.values())
        for name in out:
            out[name]["share_of_pass"] = round(out[name]["share_of_pass"] / total, 4)
        return out

    if not args.no_kernel_pass:
        entry = ([("iabn_forward_train", fwd_train, L.fwd, 2, L.E) for L in layers] +
                 [("iabn_backward", backward, L.bwd, 3, L.E) for L in reversed(layers)])
        kernels = timed_pass(entry)
        dom = max(kernels, key=lambda n: kernels[n]["share_of_pass"])
        k = kernels[dom]
        roofline = {"bound": "hbm", "kernel": dom, "achieved": k["achieved_gbps"],
                    "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": round(k["achieved_gbps"] / HBM_PEAK_GBPS, 4), "traffic": None}
        log("entry points: " + json.dumps(kernels))
    if args.phase_kernels:
        phases = ([x for L in layers for x in (("iabn_forward_stats", lib.iabn_forward_stats, L.stats, 1, L.E),
                                                ("iabn_forward_apply", lib.iabn_forward_apply, L.fwd, 2, L.E))] +
                  [x for L in reversed(layers) for x in (("iabn_backward_reduce", lib.iabn_backward_reduce, L.reduce, 2, L.E),
                                                          ("iabn_backward_apply", lib.iabn_backward_apply, L.bwd, 3, L.E))])
        phase_kernels = timed_pass(phases)
        log("phase entry points: " + json.dumps(phase_kernels))

    # ---------------------------------------------------------------- CPU baseline
    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        oracle.build(force=False)
        # Whole layers of the same workload, one shape group after another,
        # until the time budget is spent.
        order = []
        groups = {}
        for li, shp in enumerate(w.layers):
            groups.setdefault(shp, []).append(li)
        for r in range(max(len(v) for v in groups.values())):
            for v in groups.values():
                if r < len(v):
                    order.append(v[r])
        spent = 0.0
        done = 0
        used = []
        for li in order:
            inp = host_layers[li]
            x = workloads.storage_to_f64(inp.x, w.dtype)
            dz = workloads.storage_to_f64(inp.dz, w.dtype)
            c0 = time.perf_counter()
            fw = oracle.forward_train(x, inp.gamma, inp.beta, inp.running_mean, inp.running_var,
                                      w.eps, w.momentum, w.slope)
            oracle.backward_i(fw["z"], dz, inp.gamma, inp.beta, fw["var"], w.eps, w.slope)
            spent += time.perf_counter() - c0
            done += x.size
            used.append(li)
            del x, dz, fw
            if spent >= args.cpu_seconds:
                break
        cpu = {"value": round(done / spent, 1), "unit": "elements/s", "cores": oracle.num_threads(),
               "kind": "oracle",
               "sample": "oracle fp64 forward_train + backward_i over whole layers %s of %s "
                         "(%.3g elements, %.1f s), inputs already in fp64" % (used, w.name, done,
                                                                           spent)}
        log("cpu baseline: %.3g elements/s on %d threads" % (cpu["value"], cpu["cores"]))

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded, per-channel Gaussian activations, Gaussian gradients)",
        "config": {"workload": w.name, "storage": w.dtype, "layers": len(w.layers),
                   "elements_per_tensor": E_total, "slope": w.slope, "eps": w.eps,
                   "momentum": w.momentum},
        # floor: every tensor crosses HBM once (x in, z out, z and dz in, dx
        # out); schedule: the two-pass streaming schedule (x, z, dz read twice).
        "hbm": {"schedule_bytes_per_step": sched_bytes,
                "schedule_gbps": round(sched_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                "schedule_frac_of_peak": round(sched_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                "floor_bytes_per_step": floor_bytes,
                "floor_gbps": round(floor_bytes / (ms_per_step * 1e-3) / 1e9, 1)},
        "event_ms_per_step": round(ev_ms_per_step, 4),
        "outputs_finite": finite,
        "activation_memory": {"iabn_stored_bytes": E_total * b,
                              "store_x_baseline_bytes": 2 * E_total * b},
        "kernels": kernels,
        "phase_kernels": phase_kernels,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    return out


if __name__ == "__main__":
    main()
