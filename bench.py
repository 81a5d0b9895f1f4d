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
arithmetic), 1.14e9 elements per tensor.  A workload whose x and dz together
hold less than 1 GiB (the single-layer ones, --config 1-4) is replicated
into distinct buffers up to that size (``config.replicas``), so that its
passes read from HBM rather than from the 256 MB Infinity Cache.

Output: one JSON line (see the keys below).  ``value`` is elements/s of the
whole fwd+bwd step (elements = sum over layers of N*C*H*W).  ``kernels``
gives each entry point's average launch duration, from HIP events recorded
on the stream inside the timed steps (at each step's start, between its
forward and backward passes, and at its end; timing-only events, see
``TimingEvent``), with its algorithmic bytes
(forward: read x, write z; backward: read z and dz, write dx).
``roofline`` covers the one with the larger share of the step; its
``traffic`` is the HBM bytes per launch that rocprofv3's FETCH_SIZE and
WRITE_SIZE counters measured for the same kernels (scaled by a copy of
known size), read from the committed profile summary and reported only
while the kernel sources are unchanged since.  ``cpu_baseline`` is the
double-precision oracle on the host's cores over whole layers of the same
workload, bounded in time.

``ceiling_gbps`` is what this part sustains over the same buffers for each
access mix of the kernels (read only; one read and one in-place write, the
forward's; two reads and one in-place write, the backward's), measured by
the bandwidth probes of ``libiabn_probe.so`` (16-byte non-temporal accesses,
no arithmetic; streaming grid-stride loops over several grid sizes, and the
channel-resident load / barrier / store pattern), the best rate per mix.
``activation_memory`` is measured: each block's training forward runs over
the layers with the buffers it keeps for the backward allocated through
torch's allocator (InPlace-ABN: z over x; the standard block: x and a new z;
the checkpointing: xhat over x, z transient), and the peak of allocated
device memory above the starting point is recorded.
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
# Working set (x and dz of every layer) below which a workload is replicated.
REPLICA_BYTES = 1 << 30
MAX_REPLICAS = 64

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
    ap.add_argument("--shape", default=None, metavar="N,C,H,W,DTYPE",
                    help="instead of --config: one layer of this shape (dtype f32, f16 or bf16) "
                         "with the ResNet layer's value distributions")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the oracle baseline (0 disables it)")
    ap.add_argument("--no-arms", action="store_true",
                    help="skip timing the other blocks of Sec. 3.2 (InPlace-ABN II, standard, "
                         "checkpointing) on the same workload")
    ap.add_argument("--no-probes", action="store_true",
                    help="skip the bandwidth-ceiling probes and the activation-memory measurement")
    ap.add_argument("--phase-kernels", action="store_true",
                    help="also time the phase entry points (the streaming kernels), pass by pass")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device three times and exit (a kernel of "
                         "known traffic, to scale hardware byte counters)")
    return ap.parse_args()


def kernel_source_digest() -> str:
    """sha256 of the sources libiabn.so is built from (csrc/ and the header)."""
    import glob
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1712_02616_amd", "csrc")
    files = sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h")))
    for path in files + [os.path.join(ROOT, "include", "iabn.h")]:
        h.update(os.path.relpath(path, ROOT).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _profile(name):
    return os.path.join(ROOT, "profiles", name)


# The committed counter summaries, by workload index.
TRAFFIC_SUMMARIES = {2: _profile("resnet_32x256x56x56_f32_hbm_traffic.md"),
                     3: _profile("segcrop_4x256x192x192_f16_hbm_traffic.md"),
                     4: _profile("wide_16x2048x28x28_bf16_hbm_traffic.md"),
                     5: _profile("backbone_r101_os8_n8_f16_hbm_traffic.md")}


def measured_traffic(entry_point, config):
    """HBM bytes per launch of an entry point's kernel, from the committed
    rocprofv3 counter summary of the workload (FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy of known size), or None when no summary covers
    this workload or it was taken from other kernel sources."""
    path = TRAFFIC_SUMMARIES.get(config)
    if path is None or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            key, val = line[2:].split(": ", 1)
            fields[key.strip()] = val.strip().strip("`")
    if fields.get("source_sha256") != kernel_source_digest():
        return None
    val = fields.get("traffic_bytes_per_launch." + entry_point)
    return int(val) if val else None


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence.
    A default event's record ends with a system-scope fence that writes back
    and invalidates the GPU's caches, so the kernel after it starts cold and
    an apply pass placed after one no longer re-reads what its reduction
    pass left in the caches; this one records the same timestamps without
    that fence.  Same use as torch.cuda.Event(enable_timing=True): record on
    a torch stream, elapsed_time in ms after a synchronisation.  The HIP
    runtime is the one torch loaded (one runtime per process)."""

    DISABLE_SYSTEM_FENCE = 0x20000000
    _rt = None

    @classmethod
    def runtime(cls):
        if cls._rt is None:
            import torch
            path = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
            rt = ctypes.CDLL(path if os.path.exists(path) else "libamdhip64.so.7")
            vp = ctypes.c_void_p
            rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            rt.hipEventRecord.argtypes = [vp, vp]
            rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
            rt.hipEventDestroy.argtypes = [vp]
            for f in (rt.hipEventCreateWithFlags, rt.hipEventRecord, rt.hipEventElapsedTime,
                      rt.hipEventDestroy):
                f.restype = ctypes.c_int
            cls._rt = rt
        return cls._rt

    def __init__(self):
        self._h = ctypes.c_void_p()
        rc = self.runtime().hipEventCreateWithFlags(ctypes.byref(self._h), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError("hipEventCreateWithFlags failed (%d)" % rc)

    def record(self, stream):
        rc = self.runtime().hipEventRecord(self._h, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError("hipEventRecord failed (%d)" % rc)

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        rc = self.runtime().hipEventElapsedTime(ctypes.byref(ms), self._h, end._h)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed (%d)" % rc)
        return ms.value

    def __del__(self):
        if self._h and self._rt is not None:
            self._rt.hipEventDestroy(self._h)


def time_phases(lib, layers, refresh, check, stream, steps, b):
    """The four phase entry points (the streaming kernels) in a step's order
    (forward: statistics then apply per layer; backward in reverse: reduce
    then apply), with one timing event between consecutive calls: each
    call's time is the interval between the events around it.  Each step
    starts from the pristine inputs (refreshed before its first event, which
    also queues work ahead of the host); one untimed step first."""
    calls = ([(name, fn, L, attr, bpe) for L in layers
              for name, fn, attr, bpe in (("iabn_forward_stats", lib.iabn_forward_stats, "stats", 1),
                                          ("iabn_forward_apply", lib.iabn_forward_apply, "fwd", 2))] +
             [(name, fn, L, attr, bpe) for L in reversed(layers)
              for name, fn, attr, bpe in (("iabn_backward_reduce", lib.iabn_backward_reduce, "reduce", 2),
                                          ("iabn_backward_apply", lib.iabn_backward_apply, "bwd", 3))])
    import torch
    tot_ms, tot_bytes, launches = {}, {}, {}
    ev = [TimingEvent() for _ in range(len(calls) + 1)]
    for step in range(steps + 1):
        refresh()
        ev[0].record(stream)
        for i, (name, fn, L, attr, _) in enumerate(calls):
            check(fn(*getattr(L, attr)), name)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        if step == 0:
            continue
        for i, (name, _, L, _, bpe) in enumerate(calls):
            tot_ms[name] = tot_ms.get(name, 0.0) + ev[i].elapsed_time(ev[i + 1])
            tot_bytes[name] = tot_bytes.get(name, 0) + bpe * L.E * b
            launches[name] = launches.get(name, 0) + 1
    out = {name: {"avg_us": round(tot_ms[name] / launches[name] * 1e3, 3),
                  "launches": launches[name],
                  "alg_bytes_per_launch": tot_bytes[name] // launches[name],
                  "achieved_gbps": round(tot_bytes[name] / (tot_ms[name] * 1e-3) / 1e9, 1)}
           for name in tot_ms}
    out["note"] = ("each interval holds one call and one event marker; the kernels' own "
                   "durations are rocprofv3's")
    return out


# Bandwidth probes (bench_probe.hip): mix code, tensors read, tensors written
# (per element, units of the storage size b), whether the grid is chosen.
PROBE_MIXES = {"read": (0, 2, 0, True), "rw_1r1w": (1, 1, 1, True), "rmw_2r1w": (2, 2, 1, True),
               "resident_rw_1r1w": (3, 1, 1, False), "resident_rmw_2r1w": (4, 2, 1, False)}
PROBE_GRIDS = (2048, 4096, 8192, 16384, 32768)


def load_probe():
    """libiabn_probe.so (the benchmark's bandwidth probes), built by build()."""
    from paper_1712_02616_amd import build as hip_build
    if not os.path.exists(hip_build.PROBE_LIB):
        hip_build.build_probe()
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    lib.iabn_probe_launch.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_size_t, ctypes.c_int, ctypes.c_uint,
                                      ctypes.c_void_p, ctypes.c_void_p]
    lib.iabn_probe_launch.restype = ctypes.c_int
    return lib


def time_probes(layers, stream, reps, b):
    """Attainable HBM rate of each access mix over the layers' own x and dz
    buffers (the same working set, in the same order as the passes), chained
    layer after layer and timed with HIP events on the stream; for the
    streaming mixes, the best of several grid sizes."""
    import torch
    probe = load_probe()
    sink = torch.zeros(64, dtype=torch.int32, device=layers[0].x.device)
    sp = ctypes.c_void_p(stream.cuda_stream)
    out = {}
    for name, (mix, nread, nwrite, gridded) in PROBE_MIXES.items():
        best = None
        for grid in (PROBE_GRIDS if gridded else (1,)):
            def one_pass():
                for L in layers:
                    rc = probe.iabn_probe_launch(mix, L.x.data_ptr(), L.dz.data_ptr(),
                                                 L.E * b, grid, 0, sink.data_ptr(), sp)
                    if rc != 0:
                        raise RuntimeError("iabn_probe_launch(%s) failed: %d" % (name, rc))
            one_pass()
            e0 = TimingEvent()
            e1 = TimingEvent()
            e0.record(stream)
            for _ in range(reps):
                one_pass()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            nbytes = (nread + nwrite) * sum(L.E for L in layers) * b * reps
            gbps = nbytes / (ms * 1e-3) / 1e9
            if best is None or gbps > best[0]:
                best = (gbps, grid if gridded else None, ms / (reps * len(layers)) * 1e3)
        out[name] = {"gbps": round(best[0], 1), "grid": best[1], "avg_us_per_layer": round(best[2], 3),
                     "reads_per_elem": nread, "writes_per_elem": nwrite}
    return out


def measure_activation_memory(lib, layers, check, dev, code, w, wsp, ws_bytes, sp):
    """Peak device memory above the starting point while each block's
    training forward runs over the layers, keeping what that block keeps for
    its backward; every kept buffer is a fresh allocation through torch's
    allocator.  InPlace-ABN: the layer's input x (as a convolution would
    deliver it) becomes z in place.  Standard: x is kept and z is a second
    buffer.  Checkpointing: x becomes xhat in place, z is written to a buffer
    that is released after the layer (the next layer's input would be made
    from it).  Also the change of the device's free memory (hipMemGetInfo) with
    torch's cache emptied first."""
    import torch
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731

    def forward_keeping(block):
        """The block's forward over every layer; returns what it keeps."""
        kept = []
        for L in layers:
            N, C, HW = L.shape
            x = torch.empty_like(L.x0)
            x.copy_(L.x0)
            stats = (p(L.gamma), p(L.beta), p(L.rm), p(L.rv), p(L.sm), p(L.sv), w.eps, w.momentum,
                     w.slope, N, C, HW, wsp, ws_bytes, sp)
            if block == "inplace_abn":
                check(lib.iabn_forward_train(p(x), code, *stats), block)
                kept.append(x)
            elif block == "standard":
                z = torch.empty_like(x)
                check(lib.iabn_std_forward_train(p(x), p(z), code, *stats), block)
                kept += [x, z]
            else:
                z = torch.empty_like(x)
                check(lib.iabn_ckpt_forward_train(p(x), p(z), code, *stats), block)
                kept.append(x)
                del z  # the stream orders its reuse after the forward
        return kept

    out = {}
    for block in ("inplace_abn", "standard", "checkpointing"):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats(dev)
        base = torch.cuda.memory_allocated(dev)
        free0 = torch.cuda.mem_get_info(dev)[0]
        kept = forward_keeping(block)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated(dev) - base
        held = torch.cuda.memory_allocated(dev) - base
        free_delta = free0 - torch.cuda.mem_get_info(dev)[0]
        out[block] = {"peak_allocated_bytes": int(peak), "kept_bytes": int(held),
                      "device_free_delta_bytes": int(free_delta)}
        del kept
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    for block in ("standard", "checkpointing"):
        out["inplace_abn_peak_vs_" + block] = round(
            out["inplace_abn"]["peak_allocated_bytes"] / out[block]["peak_allocated_bytes"], 4)
    return out


class Layer:
    pass


def cpu_model() -> str:
    """The host CPU's model name (Linux), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_arms(lib, layers, refresh, check, stream, args, E_total, b, iabn_kernels, dev, sp, code,
              w, wsp, ws_bytes):
    """The same step for the other blocks of Sec. 3.2, each through its own
    entry points over the same layers: InPlace-ABN II (backward from z in
    terms of y), the standard block (keeps x and z; backward from x with the
    signs of z) and the proposed checkpointing (keeps xhat; the backward
    recomputes z from xhat, then runs from xhat).  Per block: ms per step,
    average forward / backward time per layer, algorithmic bytes per element
    (units of the storage size b); the activation memory each block keeps is
    measured by measure_activation_memory."""
    import torch
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    zmax = max(L.E for L in layers)
    ztmp = torch.empty(zmax, dtype=layers[0].x.dtype, device=dev)  # checkpointing's transient z
    for L in layers:
        N, C, HW = L.shape
        L.zs = torch.empty_like(L.x)  # the standard block's stored z
        common = (w.eps, w.momentum, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.std_fwd = (p(L.x), p(L.zs), code, p(L.gamma), p(L.beta), p(L.rm), p(L.rv), p(L.sm),
                     p(L.sv)) + common
        L.std_bwd = (p(L.x), p(L.zs), p(L.dz), code, p(L.gamma), p(L.beta), p(L.sm), p(L.sv),
                     p(L.dg), p(L.db), w.eps, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.ck_fwd = (p(L.x), p(ztmp), code, p(L.gamma), p(L.beta), p(L.rm), p(L.rv), p(L.sm),
                    p(L.sv)) + common
        L.ck_rec = (p(L.x), p(ztmp), code, p(L.gamma), p(L.beta), w.slope, N, C, HW, sp)
        L.ck_bwd = (p(L.x), p(L.dz), code, p(L.gamma), p(L.beta), p(L.sv), p(L.dg), p(L.db),
                    w.eps, w.slope, N, C, HW, wsp, ws_bytes, sp)
    blocks = {
        "inplace_abn_ii": ([(lib.iabn_forward_train, "fwd")],
                           [(lib.iabn_backward_ii, "bwd")], 2, 3),
        "standard": ([(lib.iabn_std_forward_train, "std_fwd")],
                     [(lib.iabn_std_backward, "std_bwd")], 2, 4),
        "checkpointing": ([(lib.iabn_ckpt_forward_train, "ck_fwd")],
                          [(lib.iabn_ckpt_recompute, "ck_rec"), (lib.iabn_ckpt_backward, "ck_bwd")],
                          3, 5),
    }
    out = {}
    for name, (fcalls, bcalls, fb, bb) in blocks.items():
        def fwd_pass():
            for L in layers:
                for fn, attr in fcalls:
                    check(fn(*getattr(L, attr)), name)

        def bwd_pass():
            for L in reversed(layers):
                for fn, attr in bcalls:
                    check(fn(*getattr(L, attr)), name)
        refresh()
        for _ in range(args.warmup):
            fwd_pass()
            bwd_pass()
        torch.cuda.synchronize()
        refresh()
        torch.cuda.synchronize()
        marks = [TimingEvent() for _ in range(2 * args.steps + 1)]
        t0 = time.perf_counter()
        for i in range(args.steps):
            marks[2 * i].record(stream)
            fwd_pass()
            marks[2 * i + 1].record(stream)
            bwd_pass()
        marks[-1].record(stream)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        fwd_ms = sum(marks[2 * i].elapsed_time(marks[2 * i + 1]) for i in range(args.steps))
        bwd_ms = sum(marks[2 * i + 1].elapsed_time(marks[2 * i + 2]) for i in range(args.steps))
        n = args.steps * len(layers)
        out[name] = {"ms_per_step": round(ms, 4), "value": round(E_total / (ms * 1e-3), 1),
                     "forward_avg_us": round(fwd_ms / n * 1e3, 3),
                     "backward_avg_us": round(bwd_ms / n * 1e3, 3),
                     "alg_bytes_per_elem_b": {"forward": fb, "backward": bb},
                     "alg_gbps": round((fb + bb) * E_total * b * args.steps / ((fwd_ms + bwd_ms) * 1e-3) / 1e9, 1)}
    iabn_us = (iabn_kernels["iabn_forward_train"]["avg_us"] + iabn_kernels["iabn_backward"]["avg_us"])
    std_us = out["standard"]["forward_avg_us"] + out["standard"]["backward_avg_us"]
    out["inplace_abn_time_vs_standard"] = round(iabn_us / std_us - 1.0, 4)
    for L in layers:
        del L.zs
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if os.environ.get("WORLD_SIZE", "1") != "1":
        print("bench.py runs as a single process on one GPU", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 3}), flush=True)
        return

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
    if getattr(args, "shape", None):
        n, c, h, wd, dt = args.shape.split(",")
        w = workloads.single_layer(int(n), int(c), int(h), int(wd), dt)
        args.config = 0
    else:
        w = workloads.WORKLOADS[args.config]
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[w.dtype]
    code = iabn.DTYPE_CODES[tdt]
    b = workloads.ELEM_BYTES[w.dtype]
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)

    # ---------------------------------------------------------------- inputs
    t0 = time.time()
    host_layers = [workloads.workload_layer(w, li) for li in range(len(w.layers))]
    layers = []
    ws_bytes = max(lib.iabn_workspace_size(n, c, hw, code) for n, c, hw in w.layers)
    workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    wsp = ctypes.c_void_p(workspace.data_ptr())
    # A workload whose x and dz fit in the Infinity Cache (the single-layer
    # ones) is replicated into distinct buffers until they do not, so that
    # every pass reads from HBM as in a network; each replica is a copy of
    # the same synthetic input.
    set_bytes = sum(2 * n * c * hw * b for n, c, hw in w.layers)
    replicas = min(MAX_REPLICAS, max(1, -(-REPLICA_BYTES // set_bytes)))
    for li, (N, C, HW) in [(li, shp) for _ in range(replicas) for li, shp in enumerate(w.layers)]:
        inp = host_layers[li]
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
        L.rv0 = torch.zeros(C, device=dev)  # inference statistics: mean 0, variance 1
        L.rv1 = torch.ones(C, device=dev)
        L.db = torch.empty(C, device=dev)
        p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        L.fwd = (p(L.x), code, p(L.gamma), p(L.beta), p(L.rm), p(L.rv), p(L.sm), p(L.sv),
                 w.eps, w.momentum, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.stats = (p(L.x), code, N, C, HW, wsp, ws_bytes, sp)
        L.bwd = (p(L.x), p(L.dz), code, p(L.gamma), p(L.beta), p(L.sv), p(L.dg), p(L.db),
                 w.eps, w.slope, N, C, HW, wsp, ws_bytes, sp)
        L.reduce = (p(L.x), p(L.dz), code, p(L.gamma), p(L.beta), w.slope, N, C, HW, wsp,
                    ws_bytes, sp)
        L.eval = (p(L.x), code, p(L.gamma), p(L.beta), p(L.rv0), p(L.rv1), w.eps, w.slope, N, C,
                  HW, sp)
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
    # HIP events on the stream the kernels run on: at the start of each step,
    # between its forward pass and its backward pass, and at the end.  Each
    # pass is back-to-back launches of one entry point, so pass time / layers
    # is that entry point's average launch duration over the timed region.
    refresh()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    refresh()
    torch.cuda.synchronize()
    marks = [TimingEvent() for _ in range(2 * args.steps + 1)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        marks[2 * i].record(stream)
        for L in layers:
            check(fwd_train(*L.fwd), "iabn_forward_train")
        marks[2 * i + 1].record(stream)
        for L in reversed(layers):
            check(backward(*L.bwd), "iabn_backward")
    marks[-1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    fwd_ms = sum(marks[2 * i].elapsed_time(marks[2 * i + 1]) for i in range(args.steps))
    bwd_ms = sum(marks[2 * i + 1].elapsed_time(marks[2 * i + 2]) for i in range(args.steps))
    ev_ms_per_step = (fwd_ms + bwd_ms) / args.steps
    value = E_total / (ms_per_step * 1e-3)
    sched_bytes = 8 * E_total * b
    floor_bytes = 5 * E_total * b
    finite = all(bool(torch.isfinite(L.dz).all()) and bool(torch.isfinite(L.x).all())
                 for L in layers)
    log("timed %d steps: %.3f ms/step (events %.3f), %.3g elements/s, finite=%s"
        % (args.steps, ms_per_step, ev_ms_per_step, value, finite))

    launches = args.steps * len(layers)
    kernels = {}
    for name, tot_ms, bpe in (("iabn_forward_train", fwd_ms, 2), ("iabn_backward", bwd_ms, 3)):
        nbytes = bpe * E_total * b * args.steps
        kernels[name] = {"avg_us": round(tot_ms / launches * 1e3, 3), "launches": launches,
                         "alg_bytes_per_launch": bpe * E_total * b // len(layers),
                         "achieved_gbps": round(nbytes / (tot_ms * 1e-3) / 1e9, 1),
                         "share_of_step": round(tot_ms / (fwd_ms + bwd_ms), 4)}
    dom = max(kernels, key=lambda n: kernels[n]["share_of_step"])
    k = kernels[dom]
    roofline = {"bound": "hbm", "kernel": dom, "achieved": k["achieved_gbps"],
                "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(k["achieved_gbps"] / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(dom, args.config)}
    if roofline["traffic"]:
        # The counted bytes over the same average launch duration.
        roofline["traffic_gbps"] = round(roofline["traffic"] / (k["avg_us"] * 1e-6) / 1e9, 1)
    log("entry points: " + json.dumps(kernels))

    # ---------------------------------------------------------------- copy reference
    # A plain device-to-device copy of every layer's x and dz (torch's copy_,
    # the runtime's copy kernel), chained over the same buffers: the same
    # read-write mix and working set as the passes, with no arithmetic.
    torch.cuda.synchronize()
    c0 = TimingEvent()
    c1 = TimingEvent()
    reps = max(1, args.steps // 2)
    c0.record(stream)
    for _ in range(reps):
        for L in layers:
            L.x.copy_(L.x0)
            L.dz.copy_(L.dz0)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * 2 * E_total * b * reps / (c0.elapsed_time(c1) * 1e-3) / 1e9
    copy_ref = {"gbps": round(copy_gbps, 1),
                "what": "device-to-device copy of every layer's x and dz (read + write), chained",
                "iabn_forward_train_frac": round(kernels["iabn_forward_train"]["achieved_gbps"] / copy_gbps, 4),
                "iabn_backward_frac": round(kernels["iabn_backward"]["achieved_gbps"] / copy_gbps, 4)}
    log("copy reference: %.1f GB/s" % copy_gbps)

    # ---------------------------------------------------------------- bandwidth ceilings
    # The probes over the same x and dz buffers (they leave the data as they
    # found it), and each entry point's rate against the ceiling of its mix.
    ceiling = None
    if not args.no_probes:
        ceiling = time_probes(layers, stream, max(2, args.steps // 2), b)
        log("bandwidth ceilings: " + json.dumps(ceiling))
        mixes = {"iabn_forward_train": ("1R:1W", ("rw_1r1w", "resident_rw_1r1w")),
                 "iabn_backward": ("2R:1W", ("rmw_2r1w", "resident_rmw_2r1w"))}
        for name, (mix, probes) in mixes.items():
            best = max(probes, key=lambda q: ceiling[q]["gbps"])
            kernels[name]["ceiling"] = {"mix": mix, "probe": best, "gbps": ceiling[best]["gbps"],
                                        "frac": round(kernels[name]["achieved_gbps"] /
                                                      ceiling[best]["gbps"], 4)}
        roofline["ceiling"] = kernels[dom]["ceiling"]

    # ---------------------------------------------------------------- inference forward
    # The inference forward (running statistics, in place) over the same
    # layers: one read and one write per element.
    refresh()
    torch.cuda.synchronize()
    ev = [TimingEvent() for _ in range(args.steps + 1)]
    for L in layers:
        check(lib.iabn_forward_eval(*L.eval), "iabn_forward_eval")
    ev[0].record(stream)
    for i in range(args.steps):
        for L in layers:
            check(lib.iabn_forward_eval(*L.eval), "iabn_forward_eval")
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    eval_ms = ev[0].elapsed_time(ev[-1])
    kernels["iabn_forward_eval"] = {
        "avg_us": round(eval_ms / launches * 1e3, 3), "launches": launches,
        "alg_bytes_per_launch": 2 * E_total * b // len(layers),
        "achieved_gbps": round(2 * E_total * b * args.steps / (eval_ms * 1e-3) / 1e9, 1),
        "share_of_step": None}
    log("inference forward: %.3f us per layer, %.1f GB/s" % (kernels["iabn_forward_eval"]["avg_us"],
                                                             kernels["iabn_forward_eval"]["achieved_gbps"]))

    # ---------------------------------------------------------------- other blocks
    arms = None
    if not args.no_arms:
        arms = time_arms(lib, layers, refresh, check, stream, args, E_total, b, kernels, dev, sp,
                         code, w, wsp, ws_bytes)
        log("blocks: " + json.dumps(arms))

    # ---------------------------------------------------------------- activation memory
    memory = None
    if not args.no_probes:
        memory = measure_activation_memory(lib, layers, check, dev, code, w, wsp, ws_bytes, sp)
        log("activation memory: " + json.dumps(memory))

    # ---------------------------------------------------------------- phase kernels
    phase_kernels = None
    if args.phase_kernels:
        phase_kernels = time_phases(lib, layers, refresh, check, stream, args.steps, b)
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
        # Passes over the layers repeat until the budget is spent (the whole
        # sweep can take less than the budget).
        spent = 0.0
        done = 0
        used = []
        f64 = {}
        while spent < args.cpu_seconds:
            for li in order:
                inp = host_layers[li]
                if li not in f64:
                    f64[li] = (workloads.storage_to_f64(inp.x, w.dtype),
                               workloads.storage_to_f64(inp.dz, w.dtype))
                x, dz = f64[li]
                c0 = time.perf_counter()
                fw = oracle.forward_train(x, inp.gamma, inp.beta, inp.running_mean,
                                          inp.running_var, w.eps, w.momentum, w.slope)
                oracle.backward_i(fw["z"], dz, inp.gamma, inp.beta, fw["var"], w.eps, w.slope)
                spent += time.perf_counter() - c0
                done += x.size
                used.append(li)
                del fw
                if spent >= args.cpu_seconds:
                    break
        del f64
        passes = len(used) / len(order)
        cpu = {"value": round(done / spent, 1), "unit": "elements/s", "cores": oracle.num_threads(),
               "kind": "oracle", "cpu_model": cpu_model(),
               "sample": "oracle fp64 forward_train + backward_i over %.2f passes of the %d layers "
                         "of %s, shape groups interleaved (%.3g elements, %.1f s of oracle time); "
                         "inputs converted to fp64 outside the timing" % (passes, len(order),
                                                                          w.name, done, spent)}
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
                   "replicas": replicas,
                   "elements_per_tensor": E_total, "slope": w.slope, "eps": w.eps,
                   "momentum": w.momentum},
        # floor: every tensor crosses HBM once (x in, z out, z and dz in, dx
        # out), which is what the channel-resident kernels move; the two-pass
        # streaming schedule (x, z and dz read twice) is not what runs, its
        # bytes over the step time are only an equivalent rate.
        "hbm": {"floor_bytes_per_step": floor_bytes,
                "floor_gbps": round(floor_bytes / (ms_per_step * 1e-3) / 1e9, 1),
                "floor_frac_of_peak": round(floor_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                "two_pass_schedule_bytes_per_step": sched_bytes,
                "two_pass_schedule_equivalent_gbps": round(sched_bytes / (ms_per_step * 1e-3) / 1e9, 1)},
        "event_ms_per_step": round(ev_ms_per_step, 4),
        "outputs_finite": finite,
        # Measured (see measure_activation_memory); one workspace serves
        # every layer and call.
        "activation_memory": None if memory is None else dict(memory, workspace_bytes=ws_bytes),
        "kernels": kernels,
        "blocks": arms,
        "phase_kernels": phase_kernels,
        "roofline": roofline,
        "ceiling_gbps": None if ceiling is None else {k: v["gbps"] for k, v in ceiling.items()},
        "ceiling_probes": ceiling,
        "copy_reference": copy_ref,
        "cpu_baseline": cpu,
    }
    return out


if __name__ == "__main__":
    main()
