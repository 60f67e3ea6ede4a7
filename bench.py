#!/usr/bin/env python3
"""Throughput of the quadratic-neuron layer (arXiv 2204.01701, eq:2ndneuron3) on one MI355X.

One step = forward (saving T_a, T_b), input gradient and weight/bias gradients
of each of the 13 quadratic 3x3 conv layers of a CIFAR VGG-16 at batch 128,
bf16 inputs with fp32 accumulation, every layer on its own seeded synthetic
input (X ~ N(0,1), He-scaled weights, biases ~ N(0, 0.01), G ~ N(0,1)).  All
tensors are resident in HBM before the timed region.

Algorithmic work per layer: 9U flops, U = 2*N*Ho*Wo*O*C*KH*KW (every tap
counted, forward = input gradient = weight gradient = 3U; the elementwise
product and the prologue products are not counted).  value = total 9U over
the 13 layers / time per step, in TFLOP/s.

Prints ONE JSON line.  --gpus N > 1 is refused: this build runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing leg")
    ap.add_argument("--no-extra", action="store_true", help="skip the single-layer and dense workloads")
    ap.add_argument("--cpu-target-s", type=float, default=15.0, help="approximate oracle sample time")
    ap.add_argument("--profile-summary", metavar="KERNEL_STATS_CSV",
                    help="instead of running: summarise a rocprofv3 --stats kernel table per entry point")
    ap.add_argument("--trace", metavar="KERNEL_TRACE_CSV",
                    help="with --profile-summary: the run's kernel trace, to average the last --last-calls calls")
    ap.add_argument("--last-calls", type=int, default=0,
                    help="with --trace: entry calls per family in the roofline region")
    ap.add_argument("--skip-calls", type=int, default=0,
                    help="with --trace: entry calls per family after the roofline region (the timed steps)")
    ap.add_argument("--copy-calibration", type=int, metavar="BYTES",
                    help="instead of running: one elementwise device copy of BYTES bytes (for counter scaling)")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH_CSV", "CAL_WRITE_CSV"),
                    help="instead of running: HBM bytes per entry call from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE "
                         "counter tables of the benchmark and of --copy-calibration")
    ap.add_argument("--leg", choices=("depthwise", "epilogue", "neuron_types", "kernels", "resnet20", "cold"),
                    help="instead of the benchmark: run one extra leg alone and print its JSON (for profiling); "
                         "'kernels' runs every pass of the VGG-16 layers, the large layer and the dense layer "
                         "KERNEL_REPS times in a fixed order, for counter collection")
    ap.add_argument("--counter-summary", nargs="+", metavar="COUNTER_CSV",
                    help="instead of running: per-pass counter table (MFMA busy, VALU per MFMA, LDS) from "
                         "rocprofv3 --pmc counter_collection tables of the 'kernels' leg")
    return ap.parse_args()


class Layer:
    """Device tensors and call wrappers of one quadratic conv layer."""

    def __init__(self, ql, torch, L, cfg_id, layer_id, dev, bf16=True, neuron=0, depthwise=False):
        import numpy as np
        import synth

        self.L = L
        self.ql = ql
        self.neuron = neuron
        nt = ql.NEURON_TERMS[neuron]
        dt = torch.bfloat16 if bf16 else torch.float32
        if depthwise:  # groups = C = O: one KH x KW filter per channel and term
            inp = synth.random_dwconv_case([cfg_id, layer_id], L.n, L.c, L.h, L.w, L.k, L.k, L.stride, L.pad,
                                           bf16=bf16)
        else:
            inp = synth.conv_inputs(cfg_id, layer_id, L, bf16=bf16)
        cw = 1 if depthwise else L.c

        def nhwc(a):
            return torch.from_numpy(np.ascontiguousarray(a)).permute(0, 2, 3, 1).contiguous().to(dev, dt)

        self.desc = ql.conv_desc(L.n, L.c, L.h, L.w, L.o, L.k, L.k, L.stride, L.pad,
                                 ql.QL_BF16 if bf16 else ql.QL_F32, neuron, groups=L.c if depthwise else 1)
        self.x = nhwc(inp["x"])
        self.w = [nhwc(inp[k]) if i < nt else None for i, k in enumerate(("wa", "wb", "wc"))]
        self.b = [torch.from_numpy(inp[k]).to(dev) if i < nt else None for i, k in enumerate(("ba", "bb", "bc"))]
        self.gy = nhwc(inp["gy"])
        self.y = torch.empty((L.n, L.ho, L.wo, L.o), device=dev, dtype=dt)
        # the saved maps of the neuron type (T2 saves none: its input gradient takes X)
        self.ta = torch.empty_like(self.y) if neuron != ql.QL_NEURON_T2 else None
        self.tb = torch.empty_like(self.y) if nt >= 2 else None
        self.dx = torch.empty_like(self.x)
        self.dw = [torch.empty((L.o, L.k, L.k, cw), device=dev, dtype=torch.float32) if i < nt else None
                   for i in range(3)]
        self.db = [torch.empty(L.o, device=dev, dtype=torch.float32) if i < nt else None for i in range(3)]
        # forward and input gradient share one workspace (same stream); the weight
        # gradient has its own, so that it may run concurrently on a second stream
        need = max(ql.qlayer_conv2d_fwd_workspace_size(self.desc),
                   ql.qlayer_conv2d_bwd_data_workspace_size(self.desc))
        self.ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
        self.wsp = (self.ws.data_ptr(), self.ws.numel())
        need_w = ql.qlayer_conv2d_bwd_weight_workspace_size(self.desc)
        self.ws_w = torch.empty(max(need_w, 256), dtype=torch.uint8, device=dev)
        self.wsp_w = (self.ws_w.data_ptr(), self.ws_w.numel())
        self.inp = inp

    def fwd(self, st):
        self.ql.qlayer_conv2d_fwd(self.desc, self.x, *self.w, *self.b, self.y, self.ta, self.tb,
                                  workspace=self.wsp, stream=st)

    def bwd_data(self, st):
        ta = self.x if self.neuron == self.ql.QL_NEURON_T2 else self.ta
        self.ql.qlayer_conv2d_bwd_data(self.desc, self.gy, ta, self.tb, *self.w, self.dx,
                                       workspace=self.wsp, stream=st)

    def bwd_weight(self, st):
        self.ql.qlayer_conv2d_bwd_weight(self.desc, self.x, self.gy, self.ta, self.tb, *self.dw, *self.db,
                                         workspace=self.wsp_w, stream=st)


class DevEvent:
    """A HIP event recorded with device-scope release and acquire
    (hipEventDisableSystemFence), created on the HIP runtime that torch loaded.

    The benchmark's events only order kernels on one GPU and time them; a
    system-scope fence (what torch's events use) makes every record write the
    caches back for the host, an idle gap of several microseconds between two
    launches.  The host reads results only after torch.cuda.synchronize()."""
    _hip = None
    DISABLE_TIMING = 0x2
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, timing=True):
        import ctypes
        if DevEvent._hip is None:
            DevEvent._hip = ctypes.CDLL("libamdhip64.so.7")   # same soname as torch's runtime: same instance
        self._ct = ctypes
        self.ev = ctypes.c_void_p()
        flags = self.DISABLE_SYSTEM_FENCE | (0 if timing else self.DISABLE_TIMING)
        self._check(DevEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.ev), ctypes.c_uint(flags)),
                    "hipEventCreateWithFlags")

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed with HIP error {rc}")

    def record(self, stream):
        self._check(DevEvent._hip.hipEventRecord(self.ev, self._ct.c_void_p(stream.cuda_stream)), "hipEventRecord")

    def wait(self, stream):
        """Make `stream` wait for this event (device side)."""
        self._check(DevEvent._hip.hipStreamWaitEvent(self._ct.c_void_p(stream.cuda_stream), self.ev,
                                                      self._ct.c_uint(0)), "hipStreamWaitEvent")

    def elapsed_time(self, end):
        """Milliseconds from this event to `end` (both complete)."""
        ms = self._ct.c_float()
        self._check(DevEvent._hip.hipEventElapsedTime(self._ct.byref(ms), self.ev, end.ev), "hipEventElapsedTime")
        return ms.value

    def __del__(self):
        hip = getattr(type(self), "_hip", None)   # (None once the interpreter tears the module down)
        if hip is not None and self.ev:
            hip.hipEventDestroy(self.ev)


def unit_flops(L):
    return 2 * L.n * L.ho * L.wo * L.o * L.c * L.k * L.k


def time_calls(torch, calls, steps, warmup, stream, timed_families=None):
    """Run `calls` (list of (family, fn)) warmup + steps times.

    Returns (device ms per step, wall ms per step, {family: summed event ms}, {family: launches}).
    HIP events (device-scope, DevEvent) bracket every launch whose family is in
    `timed_families` (all when None); the events are recorded on `stream`, the stream
    the library launches on.
    """
    for _ in range(warmup):
        for _, fn in calls:
            fn(stream)
    torch.cuda.synchronize()
    evs = []
    t0 = time.perf_counter()
    start = DevEvent()
    stop = DevEvent()
    ntimed = steps * sum(1 for fam, _ in calls if timed_families is None or fam in timed_families)
    pool = [(DevEvent(), DevEvent()) for _ in range(ntimed)]  # created before the timed loop
    start.record(stream)
    for _ in range(steps):
        for fam, fn in calls:
            if timed_families is None or fam in timed_families:
                e0, e1 = pool.pop()
                e0.record(stream)
                fn(stream)
                e1.record(stream)
                evs.append((fam, e0, e1))
            else:
                fn(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    ms_step = start.elapsed_time(stop) / steps
    fam_ms = {}
    fam_n = {}
    for fam, e0, e1 in evs:
        fam_ms[fam] = fam_ms.get(fam, 0.0) + e0.elapsed_time(e1)
        fam_n[fam] = fam_n.get(fam, 0) + 1
    return ms_step, wall, fam_ms, fam_n


def time_each(torch, calls, reps, stream):
    """Device time per call of each (key, fn) in `calls`: the call repeated `reps`
    times back to back (after one untimed call), HIP events at the two ends only,
    so that the host's launch time between calls stays hidden behind the GPU's
    work; the median of three such trials.  Returns {key: ms per call}."""
    out = {}
    for key, fn in calls:
        fn(stream)
        # three trials, the median kept: one host stall (the GPU idling between
        # two launches) inside a trial does not reach the figure
        trials = []
        for _ in range(3):
            a, b = DevEvent(), DevEvent()
            a.record(stream)
            for _ in range(reps):
                fn(stream)
            b.record(stream)
            torch.cuda.synchronize()
            trials.append(a.elapsed_time(b) / reps)
        out[key] = sorted(trials)[1]
    return out


def time_family_runs(torch, calls, family, steps, stream):
    """Roofline timing of one entry point: `steps` single-stream steps, each running
    the step's other calls first and then the calls of `family` back to back between
    two HIP events (device scope, on the library's stream), so that an event record
    lands between launches only once per step.  Returns (ms per launch, launches)."""
    pool = [(DevEvent(), DevEvent()) for _ in range(steps)]  # created before the timed loop
    mine = [fn for fam, fn in calls if fam[0] == family]
    rest = [fn for fam, fn in calls if fam[0] != family]
    for e0, e1 in pool:
        for fn in rest:
            fn(stream)
        e0.record(stream)
        for fn in mine:
            fn(stream)
        e1.record(stream)
    torch.cuda.synchronize()
    return sum(e0.elapsed_time(e1) for e0, e1 in pool) / (steps * len(mine)), steps * len(mine)


def time_overlapped(torch, layers, steps, warmup, s1, s2, group=2):
    """Run the step `warmup` + `steps` times with the weight gradients on a second
    stream: a layer's weight gradient depends only on its forward (T_a, T_b), so it
    overlaps with the input gradients on the first stream.  The weight gradients of
    `group` consecutive layers are released together by one device-scope event
    (DevEvent) recorded after the last of their forwards: each record leaves the
    first stream idle for a few microseconds, and two layers per event measured
    faster than one or three.  Returns (device ms per step, wall ms per step), timed
    with events on s1 at the two ends of the timed steps."""
    fwd_done = [DevEvent(timing=False) for _ in layers]
    s2_done = DevEvent(timing=False)

    def step():
        pend = []
        for i, (ly, ev) in enumerate(zip(layers, fwd_done)):
            ly.fwd(s1)
            pend.append(ly)
            if len(pend) == group or i == len(layers) - 1:
                ev.record(s1)
                ev.wait(s2)
                for p in pend:
                    p.bwd_weight(s2)
                pend = []
            ly.bwd_data(s1)
        s2_done.record(s2)
        s2_done.wait(s1)  # the next step's forward overwrites T_a, T_b

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start = DevEvent()
    stop = DevEvent()
    t0 = time.perf_counter()
    start.record(s1)
    for _ in range(steps):
        step()
    stop.record(s1)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    return start.elapsed_time(stop) / steps, wall


def cpu_baseline(layers_geom, target_s):
    """Time the fp64 oracle on a bounded sample of the same workload: every layer's
    forward + backward at a reduced batch, seeded exactly like the GPU inputs."""
    import dataclasses

    import oracle
    import synth

    def run(nimg):
        t = 0.0
        flops = 0
        for li, L in enumerate(layers_geom):
            Ls = dataclasses.replace(L, n=nimg)
            inp = synth.conv_inputs(2, li, Ls, bf16=True)
            t0 = time.perf_counter()
            oracle.conv2d_fwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"],
                              Ls.stride, Ls.pad)
            oracle.conv2d_bwd(inp["x"], inp["wa"], inp["wb"], inp["wc"], inp["ba"], inp["bb"], inp["bc"],
                              inp["gy"], Ls.stride, Ls.pad)
            t += time.perf_counter() - t0
            flops += 9 * unit_flops(Ls)
        return t, flops

    t1, f1 = run(1)
    n = 1
    if t1 < target_s / 2:
        n = int(min(layers_geom[0].n, max(1, math.floor(target_s / max(t1, 1e-3)))))
        if n > 1:
            t1, f1 = run(n)
    return {"value": f1 / t1 / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"all 13 layers, forward + backward, batch {n} of 128 (fp64 direct summation; "
                      f"{t1:.1f} s for {f1 / 1e9:.1f} GFLOP)"}


# Kernel symbol -> (entry point that launches it, whether it is that entry's one main kernel).
# Every entry call launches exactly one main kernel, so main-kernel calls count entry calls.
_KERNEL_FAMILY = [
    (r"qconv_fwd_kernel<", "fwd", True),
    (r"qconv_fwd_generic_kernel<", "fwd", True),
    (r"qconv_fwd_smallc_kernel<", "fwd", True),
    (r"qconv_fwd_narrow_kernel<", "fwd", True),
    (r"qconv_fwd_ksplit_kernel<", "fwd", True),
    (r"qconv_fwd_combine_kernel<", "fwd", False),
    (r"qconv_pad_channels_kernel<[^,>]+, 4>", "fwd", False),
    (r"qconv_bwd_data_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_generic_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_wide_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_cols_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_cols_fused_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_narrow_kernel<", "bwd_data", True),
    (r"qconv_bwd_data_col2im_kernel<", "bwd_data", False),
    (r"qconv_sum_splits_kernel<", "bwd_data", False),
    (r"qconv_weight_transpose_kernel<", "bwd_data", False),
    (r"qconv_bwd_weight_kernel<", "bwd_weight", True),
    (r"qconv_bwd_weight16_kernel<", "bwd_weight", True),
    (r"qconv_bwd_weight_generic_kernel<", "bwd_weight", True),
    (r"qconv_bwd_weight_narrow_kernel<", "bwd_weight", True),
    (r"qconv_bwd_weight_reduce_kernel<", "bwd_weight", False),
    (r"qconv_bwd_weight_reduce2d_kernel<", "bwd_weight", False),
    (r"qconv_bwd_weight_reduce2dv_kernel[<(]", "bwd_weight", False),
    (r"qconv_pad_channels_kernel<[^,>]+, 1>", "bwd_weight", False),
]


def profile_summary(path, trace=None, last_calls=0, skip_calls=0):
    """Markdown summary of a rocprofv3 kernel statistics table (--stats, csv output):
    every kernel with its calls and average duration, then per entry point the total
    kernel time divided by the number of entry calls (= calls of its main kernels)."""
    import csv
    import re

    rows = list(csv.DictReader(open(path)))
    fam_ns, fam_calls = {}, {}
    lines = ["| kernel | entry point | calls | avg us | total ms |", "|---|---|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name, calls, tot = r["Name"], int(r["Calls"]), float(r["TotalDurationNs"])
        fam, main = "-", False
        for pat, f, m in _KERNEL_FAMILY:
            if re.search(pat, name):
                fam, main = f, m
                break
        if fam != "-":
            fam_ns[fam] = fam_ns.get(fam, 0.0) + tot
            if main:
                fam_calls[fam] = fam_calls.get(fam, 0) + calls
        short = name if len(name) < 110 else name[:107] + "..."
        lines.append(f"| `{short}` | {fam} | {calls} | {tot / calls / 1e3:.1f} | {tot / 1e6:.2f} |")
    lines += ["", "| entry point | entry calls | kernel time per call, us |", "|---|---:|---:|"]
    for fam in ("fwd", "bwd_data", "bwd_weight"):
        if fam_calls.get(fam):
            lines.append(f"| qlayer_conv2d_{fam} | {fam_calls[fam]} | {fam_ns[fam] / fam_calls[fam] / 1e3:.1f} |")
    if trace and last_calls:
        where = f"before its last {skip_calls}" if skip_calls else "its last"
        lines += ["", f"One region only ({last_calls} calls of each entry point, {where}, from the kernel trace):", "",
                  "| entry point | entry calls | kernel time per call, us |", "|---|---:|---:|"]
        for fam, (n, ns) in region_times(trace, last_calls, skip_calls).items():
            lines.append(f"| qlayer_conv2d_{fam} | {n} | {ns / n / 1e3:.1f} |")
    print("\n".join(lines))


def region_times(trace_csv, last_calls, skip_calls=0):
    """Per family: kernel time of `last_calls` entry calls in a rocprofv3 kernel trace, those
    that precede the family's last `skip_calls` calls (every kernel of the family from the
    first selected call's main-kernel dispatch up to the next unselected one)."""
    import csv
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Dispatch_Id"]))
    out = {}
    for fam in ("fwd", "bwd_data", "bwd_weight"):
        mains = [i for i, r in enumerate(rows) if _family(r["Kernel_Name"]) == (fam, True)]
        if len(mains) < last_calls + skip_calls:
            continue
        first = mains[len(mains) - skip_calls - last_calls]
        end = mains[len(mains) - skip_calls] if skip_calls else len(rows)
        ns = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in rows[first:end]
                 if _family(r["Kernel_Name"])[0] == fam)
        out[fam] = (last_calls, ns)
    return out


def _family(name):
    import re
    for pat, f, m in _KERNEL_FAMILY:
        if re.search(pat, name):
            return f, m
    return None, False


def _counter_rows(path, counter):
    """(kernel name, value) per dispatch of one counter in a rocprofv3 counter_collection table."""
    import csv
    out = []
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def sources_digest():
    """sha256 of the kernel and host sources of the library (identifies the code counters were taken on)."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2204_01701_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".h", ".hip")):
            h.update(f.encode())
            h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_summary(fetch_csv, write_csv, cal_fetch_csv, cal_write_csv, cal_bytes):
    """Markdown: HBM bytes per entry call per pass, from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch) scaled so that the plain copy reads and writes exactly its size."""
    # the calibration's multiply-by-one kernel (its buffer fill is another kernel)
    cf = sum(v for k, v in _counter_rows(cal_fetch_csv, "FETCH_SIZE") if "MulFunctor" in k)
    cw = sum(v for k, v in _counter_rows(cal_write_csv, "WRITE_SIZE") if "MulFunctor" in k)
    sf = cal_bytes / (cf * 1024.0)
    sw = cal_bytes / (cw * 1024.0)
    lines = [f"copy calibration: {cal_bytes} bytes read and written; FETCH_SIZE read {cf:.0f} KiB, "
             f"WRITE_SIZE {cw:.0f} KiB; scale factors fetch {sf:.4f}, write {sw:.4f}", "",
             "| entry point | entry calls | read MB per call | written MB per call | traffic bytes per call |",
             "|---|---:|---:|---:|---:|"]
    tot = {}
    for path, cnt, scale, key in ((fetch_csv, "FETCH_SIZE", sf, "r"), (write_csv, "WRITE_SIZE", sw, "w")):
        for name, v in _counter_rows(path, cnt):
            f, main = _family(name)
            if f is None:
                continue
            d = tot.setdefault(f, {"r": 0.0, "w": 0.0, "calls_r": 0, "calls_w": 0})
            d[key] += v * 1024.0 * scale
            if main:
                d["calls_" + key] += 1
    for f in ("fwd", "bwd_data", "bwd_weight"):
        if f in tot and tot[f]["calls_r"] and tot[f]["calls_w"]:
            d = tot[f]
            r, w = d["r"] / d["calls_r"], d["w"] / d["calls_w"]
            lines.append(f"| qlayer_conv2d_{f} | {d['calls_r']} | {r / 1e6:.1f} | {w / 1e6:.1f} | {r + w:.0f} |")
    lines += ["", f"sources: {sources_digest()}"]
    print("\n".join(lines))


def read_traffic(family):
    """Traffic bytes per call of `family` from the committed counter summary, or None when
    the summary is missing or was taken on other sources."""
    import re
    path = os.path.join(ROOT, "profiles", "vgg16_bf16_b128_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m = re.search(r"^sources: (\w+)$", txt, re.M)
    if not m or m.group(1) != sources_digest():
        return None
    m = re.search(r"^\| qlayer_conv2d_%s \| \d+ \| [\d.]+ \| [\d.]+ \| (\d+) \|$" % family, txt, re.M)
    return int(m.group(1)) if m else None


KERNEL_REPS = 3  # calls of each pass in the 'kernels' leg


def kernel_leg_sequence():
    """(workload, layer, pass) of the 'kernels' leg's entry calls in issue order (no GPU needed)."""
    import synth
    seq = []
    for i in range(len(synth.vgg16_layers(128))):
        for f in ("fwd", "bwd_data", "bwd_weight"):
            seq += [("vgg16", i + 1, f)] * KERNEL_REPS
    for f in ("fwd", "bwd_data", "bwd_weight"):
        seq += [("large", 0, f)] * KERNEL_REPS
    seq += [("dense", 0, "fwd")] * KERNEL_REPS
    seq += [("dense", 0, "bwd_data"), ("dense", 0, "bwd_weight")] * KERNEL_REPS  # one call, two main kernels
    return seq


def kernel_leg(ql, torch, dev, stream):
    """Every pass of the 13 VGG-16 layers, the large layer and the dense layer,
    KERNEL_REPS calls each, in the order kernel_leg_sequence() gives."""
    import synth
    calls = {}
    for i, L in enumerate(synth.vgg16_layers(128)):
        ly = Layer(ql, torch, L, 2, i, dev)
        for f in ("fwd", "bwd_data", "bwd_weight"):
            for _ in range(KERNEL_REPS):
                getattr(ly, f)(stream)
        torch.cuda.synchronize()
        del ly
    ly = Layer(ql, torch, synth.LARGE_BF16, 4, 0, dev)
    for f in ("fwd", "bwd_data", "bwd_weight"):
        for _ in range(KERNEL_REPS):
            getattr(ly, f)(stream)
    torch.cuda.synchronize()
    del ly
    D = synth.DENSE_BF16
    inp = synth.dense_inputs(5, 0, D, bf16=True)
    dt = torch.bfloat16
    d = ql.linear_desc(D.batch, D.inp, D.out, ql.QL_BF16)
    x = torch.from_numpy(inp["x"]).to(dev, dt)
    w = [torch.from_numpy(inp[k]).to(dev, dt) for k in ("wa", "wb", "wc")]
    b = [torch.from_numpy(inp[k]).to(dev) for k in ("ba", "bb", "bc")]
    gy = torch.from_numpy(inp["gy"]).to(dev, dt)
    y = torch.empty((D.batch, D.out), device=dev, dtype=dt)
    ta, tb, dx = torch.empty_like(y), torch.empty_like(y), torch.empty_like(x)
    dw = [torch.empty((D.out, D.inp), device=dev) for _ in range(3)]
    db = [torch.empty(D.out, device=dev) for _ in range(3)]
    need = max(ql.qlayer_linear_fwd_workspace_size(d), ql.qlayer_linear_bwd_workspace_size(d))
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    wsp = (ws.data_ptr(), ws.numel())
    for _ in range(KERNEL_REPS):
        ql.qlayer_linear_fwd(d, x, *w, *b, y, ta, tb, workspace=wsp, stream=stream)
    for _ in range(KERNEL_REPS):
        ql.qlayer_linear_bwd(d, x, gy, ta, tb, *w, dx, *dw, *db, workspace=wsp, stream=stream)
    torch.cuda.synchronize()
    calls["calls"] = len(kernel_leg_sequence())
    return calls


def counter_summary(paths):
    """Markdown table of the 'kernels' leg's counters: per pass (averaged over its
    calls, main kernel only): the kernel duration and the shader clock it ran at
    (GRBM_GUI_ACTIVE, which reads the sum over the 8 XCDs, / 8 / duration); MFMA
    busy = SQ_VALU_MFMA_BUSY_CYCLES (32 per 32x32x16 bf16 MFMA, 16 per 16x16x32,
    summed over the SIMDs) / (GRBM_GUI_ACTIVE / 8 x 256 CUs x 4 SIMDs), the
    fraction of the MFMA peak at the clock the kernel ran at (GRBM_GUI_ACTIVE also
    counts the dispatch's own overhead outside the kernel's timestamps, which on
    kernels of a few tens of microseconds reads as a clock above 2.4 GHz and a
    busy fraction too low); the same busy cycles over the kernel's duration at
    the nominal 2.4 GHz, the fraction of the published peak; non-MFMA VALU
    instructions per MFMA instruction, and per 32 MFMA busy cycles (the work of
    one 32x32x16 bf16 MFMA, which compares kernels of either MFMA shape); LDS
    instructions per MFMA; LDS bank-conflict cycles per LDS instruction."""
    import csv
    per = {}  # (file, dispatch id) -> {counter: value}; kernel names and durations
    names, durs = {}, {}
    for p in paths:
        for r in csv.DictReader(open(p)):
            did = (p, int(r["Dispatch_Id"]))
            per.setdefault(did, {})
            per[did][r["Counter_Name"]] = per[did].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            names[did] = r["Kernel_Name"]
            durs[did] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    # counters of separate runs: dispatches matched by their order among the main kernels
    seq = kernel_leg_sequence()
    rows = {}
    for p in paths:
        mains = [(p, d) for d in sorted({int(r["Dispatch_Id"]) for r in csv.DictReader(open(p))})
                 if _family(names[(p, d)])[1]]
        if len(mains) != len(seq):
            raise SystemExit(f"{p}: {len(mains)} main-kernel dispatches, the leg makes {len(seq)} calls")
        for d, key in zip(mains, seq):
            rows.setdefault(key, {"kernel": names[d], "dur_ns": [], "grbm": []})
            for c, v in per[d].items():
                rows[key][c] = rows[key].get(c, 0.0) + v / KERNEL_REPS
            if "GRBM_GUI_ACTIVE" in per[d]:
                rows[key]["dur_ns"].append(durs[d])
                rows[key]["grbm"].append(per[d]["GRBM_GUI_ACTIVE"])
    lines = ["| workload | layer | pass | main kernel | us (profiled) | clock GHz | MFMA busy % | MFMA busy % at 2.4 GHz "
             "| VALU / MFMA | VALU / 32 MFMA cycles | LDS / MFMA | LDS bank conflict cycles / LDS instr |",
             "|---|---:|---|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    nxcd = 8
    for (wl, layer, f), r in rows.items():
        g = r.get("GRBM_GUI_ACTIVE")
        g = g / nxcd if g is not None else None
        us = sum(r["dur_ns"]) / len(r["dur_ns"]) / 1e3 if r["dur_ns"] else None
        ghz = sum(gg / nxcd / dd for gg, dd in zip(r["grbm"], r["dur_ns"])) / len(r["dur_ns"]) if r["dur_ns"] else None
        busy = r.get("SQ_VALU_MFMA_BUSY_CYCLES")
        mf = r.get("SQ_INSTS_MFMA") or r.get("SQ_INSTS_VALU_MFMA_BF16")
        va = r.get("SQ_INSTS_VALU")
        lds = r.get("SQ_INSTS_LDS")
        bc = r.get("SQ_LDS_BANK_CONFLICT")
        cell = lambda v: "-" if v is None else v
        b = f"{100 * busy / (g * 256 * 4):.1f}" if busy is not None and g else "-"
        b24 = f"{100 * busy / (us * 1e3 * 2.4 * 256 * 4):.1f}" if busy is not None and us else "-"
        vpm = f"{(va - mf) / mf:.1f}" if va is not None and mf else "-"
        vpc = f"{(va - mf) / (busy / 32):.1f}" if va is not None and mf and busy else "-"
        lpm = f"{lds / mf:.2f}" if lds is not None and mf else "-"
        bpl = f"{bc / lds:.3f}" if bc is not None and lds else "-"
        k = r["kernel"]
        k = k[k.find("qconv"):][:60] if "qconv" in k else k[:60]
        t = f"{us:.1f}" if us is not None else "-"
        c = f"{ghz:.2f}" if ghz is not None else "-"
        lines.append(f"| {wl} | {cell(layer)} | {f} | `{k}` | {t} | {c} | {b} | {b24} | {vpm} | {vpc} | {lpm} | {bpl} |")
    lines += ["", f"sources: {sources_digest()}"]
    print("\n".join(lines))


def copy_calibration(nbytes):
    import torch
    dev = torch.device("cuda:0")
    n = nbytes // 4
    src = torch.ones(n, device=dev, dtype=torch.float32)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)  # one elementwise kernel: reads and writes nbytes
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4}))


def main():
    args = parse()
    if args.profile_summary:
        profile_summary(args.profile_summary, args.trace, args.last_calls, args.skip_calls)
        return
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary, cal_bytes=int(os.environ.get("QL_COPY_BYTES", 1 << 30)))
        return
    if args.counter_summary:
        counter_summary(args.counter_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this build runs on one GPU only; multi-GPU runs are not supported",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    import paper_2204_01701_amd as ql
    import synth

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    ql.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    if args.leg:
        legs = {"depthwise": depthwise, "epilogue": epilogue_cost, "neuron_types": neuron_types, "cold": cold_cache,
                "kernels": kernel_leg, "resnet20": resnet20_step_leg}
        print(json.dumps({args.leg: legs[args.leg](ql, torch, dev, stream)}), flush=True)
        return

    geoms = synth.vgg16_layers(128)
    layers = [Layer(ql, torch, L, 2, i, dev) for i, L in enumerate(geoms)]
    calls = []
    for i, ly in enumerate(layers):
        calls.append((("fwd", i), ly.fwd))
        calls.append((("bwd_data", i), ly.bwd_data))
        calls.append((("bwd_weight", i), ly.bwd_weight))

    # Diagnostic pass (not the timed region): each call repeated back to back with
    # events at the ends, for the per-layer table and to find the family that takes
    # the most time.
    for _ in range(args.warmup):  # warm-up steps
        for _, fn in calls:
            fn(stream)
    diag = time_each(torch, calls, 10, stream)
    per_layer = []
    fam_tot = {"fwd": 0.0, "bwd_data": 0.0, "bwd_weight": 0.0}
    for i, L in enumerate(geoms):
        row = {"layer": i + 1, "shape": f"{L.c}->{L.o} {L.h}x{L.w}"}
        for fam in ("fwd", "bwd_data", "bwd_weight"):
            ms = diag[(fam, i)]
            fam_tot[fam] += ms
            row[f"{fam}_us"] = round(ms * 1e3, 1)
            row[f"{fam}_tflops"] = round(3 * unit_flops(L) / (ms * 1e-3) / 1e12, 1)
        per_layer.append(row)
    dom = max(fam_tot, key=fam_tot.get)

    # Single-stream steps, then the roofline region: K more steps, the dominant family's
    # 13 launches of each step back to back between two events, after the step's other
    # calls.  Both run before the timed region, so that it
    # starts on a GPU that has been busy for a while (the first tens of steps after
    # start-up run several per cent slower).
    ms_serial, _, _, _ = time_calls(torch, calls, args.steps, 1, stream, timed_families=set())
    dom_avg_ms, dom_launches = time_family_runs(torch, calls, dom, args.steps, stream)

    # Timed region: W warm-up steps, then K steps with events only at its two ends (an
    # event between two launches serialises them); each layer's weight gradient runs on
    # a second stream beside its input gradient.
    stream2 = torch.cuda.Stream(dev)  # default priority
    ms_step, wall = time_overlapped(torch, layers, args.steps, args.warmup, stream, stream2)

    total_flops = sum(9 * unit_flops(L) for L in geoms)
    value = total_flops / (ms_step * 1e-3) / 1e12
    dom_flops = sum(3 * unit_flops(L) for L in geoms) / len(geoms)   # algorithmic flops per launch
    achieved = dom_flops / (dom_avg_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": read_traffic(dom),
                "kernel": f"qlayer_conv2d_{dom} over the 13 layers (avg {dom_avg_ms * 1e3:.1f} us per launch, "
                          f"{dom_flops / 1e9:.2f} GFLOP per launch)"}

    extra = {}
    if not args.no_extra:
        extra = extra_workloads(ql, torch, dev, stream)

    result = {
        "metric": "quadratic-layer fwd+bwd TFLOP/s and % of bf16 MFMA peak on one MI355X",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "VGG-16 stack of 13 quadratic 3x3 conv layers, bf16, batch 128, 3x32x32, "
                               "fwd + bwd_data + bwd_weight per layer",
                   "global_batch": 128, "layers": 13, "gflop_per_step": round(total_flops / 1e9, 1)},
        "pct_of_bf16_peak": round(100 * value / BF16_PEAK_TFLOPS, 2),
        "wall_ms_per_step": round(wall, 4),
        "ms_per_step_one_stream": round(ms_serial, 4),
        "roofline": roofline,
        "per_family_us": {k: round(v * 1e3, 1) for k, v in fam_tot.items()},
        "per_layer": per_layer,
    }
    if extra:
        result["extra"] = extra
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(geoms, args.cpu_target_s)
    print(json.dumps(result), flush=True)


def conv_bytes(L, fam, esize=2):
    """Algorithmic HBM bytes of one pass of a dense quadratic conv layer (every
    input and output tensor once): fwd (X + 3 W + 3 P) eb, bwd_data
    (3 P + 3 W + X) eb, bwd_weight (X + 3 P) eb + 4 (3 W + 3 O)."""
    X = L.n * L.h * L.w * L.c
    P = L.n * L.ho * L.wo * L.o
    W = L.o * L.c * L.k * L.k
    if fam == "fwd":
        return esize * (X + 3 * W + 3 * P)
    if fam == "bwd_data":
        return esize * (3 * P + 3 * W + X)
    return esize * (X + 3 * P) + 4 * (3 * W + 3 * L.o)


def cold_cache(ql, torch, dev, stream, reps=20):
    """The layers below the MFMA ridge, each pass hot and cold: the VGG-16 stem
    (3 -> 64, 32 x 32) and the 2 x 2 layers 11-13 (512 -> 512, one shape), and
    the large depthwise layer (N=64, C=256, 56 x 56).  Hot: `reps` calls back to
    back between two device-scope events, per call (the GPU runs ahead of the
    host, so host launch time stays hidden); cold: the median of single calls,
    each after a 512 MB scratch write, so that the MALL holds none of the
    layer's tensors (the write is outside the timed interval and keeps the GPU
    busy while the call is submitted).  GB/s: algorithmic bytes over the time,
    and the fraction of the 8 TB/s HBM spec."""
    import synth
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    geoms = synth.vgg16_layers(128)
    cases = [("vgg16_L1", Layer(ql, torch, geoms[0], 2, 0, dev), conv_bytes),
             ("vgg16_L11_13", Layer(ql, torch, geoms[10], 2, 10, dev), conv_bytes),
             ("large_dw", Layer(ql, torch, synth.ConvLayer(n=64, c=256, h=56, w=56, o=256, k=3, stride=1, pad=1),
                                9, 0, dev, depthwise=True), dw_bytes)]
    out = {}
    for name, ly, nbytes in cases:
        ly.fwd(stream)
        r = {"shape": f"N={ly.L.n} {ly.L.c}->{ly.L.o} {ly.L.h}x{ly.L.w}" + (" depthwise" if name == "large_dw" else "")}
        for f in ("fwd", "bwd_data", "bwd_weight"):
            fn = getattr(ly, f)
            for _ in range(3):
                fn(stream)
            torch.cuda.synchronize()
            a, b = DevEvent(), DevEvent()
            a.record(stream)
            for _ in range(reps):
                fn(stream)
            b.record(stream)
            torch.cuda.synchronize()
            th = a.elapsed_time(b) / reps
            cold = []
            for _ in range(reps):
                with torch.cuda.stream(stream):
                    flush.fill_(1)
                a, b = DevEvent(), DevEvent()
                a.record(stream)
                fn(stream)
                b.record(stream)
                torch.cuda.synchronize()
                cold.append(a.elapsed_time(b))
            tc = sorted(cold)[reps // 2]
            nb = nbytes(ly.L, f)
            r[f"{f}_us_hot"] = round(th * 1e3, 1)
            r[f"{f}_us_cold"] = round(tc * 1e3, 1)
            r[f"{f}_gbs_hot"] = round(nb / (th * 1e-3) / 1e9, 1)
            r[f"{f}_gbs_cold"] = round(nb / (tc * 1e-3) / 1e9, 1)
            r[f"{f}_hbm_frac_cold"] = round(nb / (tc * 1e-3) / 1e9 / 8000.0, 3)
        out[name] = r
        del ly
    del flush
    return out


def extra_workloads(ql, torch, dev, stream, reps=10):
    """The large single layer (N=64, 256->256, 56x56) and the dense layer (8192 x 4096 -> 4096),
    each pass timed separately (reported beside the main metric)."""
    import synth

    out = {}
    L = synth.LARGE_BF16
    ly = Layer(ql, torch, L, 4, 0, dev)
    calls = [("fwd", ly.fwd), ("bwd_data", ly.bwd_data), ("bwd_weight", ly.bwd_weight)]
    ms, _, fam_ms, fam_n = time_calls(torch, calls, reps, 3, stream)
    u = unit_flops(L)
    out["large_conv_bf16"] = {
        "shape": "N=64 C=256 56x56 -> 256, 3x3",
        **{f"{f}_us": round(fam_ms[f] / fam_n[f] * 1e3, 1) for f in ("fwd", "bwd_data", "bwd_weight")},
        **{f"{f}_tflops": round(3 * u / (fam_ms[f] / fam_n[f] * 1e-3) / 1e12, 1)
           for f in ("fwd", "bwd_data", "bwd_weight")},
        "fwd_bwd_tflops": round(9 * u / (ms * 1e-3) / 1e12, 1)}
    del ly

    D = synth.DENSE_BF16
    inp = synth.dense_inputs(5, 0, D, bf16=True)
    dt = torch.bfloat16
    d = ql.linear_desc(D.batch, D.inp, D.out, ql.QL_BF16)
    x = torch.from_numpy(inp["x"]).to(dev, dt)
    w = [torch.from_numpy(inp[k]).to(dev, dt) for k in ("wa", "wb", "wc")]
    b = [torch.from_numpy(inp[k]).to(dev) for k in ("ba", "bb", "bc")]
    gy = torch.from_numpy(inp["gy"]).to(dev, dt)
    y = torch.empty((D.batch, D.out), device=dev, dtype=dt)
    ta, tb, dx = torch.empty_like(y), torch.empty_like(y), torch.empty_like(x)
    dw = [torch.empty((D.out, D.inp), device=dev) for _ in range(3)]
    db = [torch.empty(D.out, device=dev) for _ in range(3)]
    need = max(ql.qlayer_linear_fwd_workspace_size(d), ql.qlayer_linear_bwd_workspace_size(d))
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    wsp = (ws.data_ptr(), ws.numel())
    calls = [("fwd", lambda st: ql.qlayer_linear_fwd(d, x, *w, *b, y, ta, tb, workspace=wsp, stream=st)),
             ("bwd", lambda st: ql.qlayer_linear_bwd(d, x, gy, ta, tb, *w, dx, *dw, *db, workspace=wsp,
                                                     stream=st))]
    ms, _, fam_ms, fam_n = time_calls(torch, calls, reps, 3, stream)
    u = D.unit_flops()
    out["dense_bf16"] = {
        "shape": "8192 x 4096 -> 4096",
        "fwd_us": round(fam_ms["fwd"] / fam_n["fwd"] * 1e3, 1),
        "bwd_us": round(fam_ms["bwd"] / fam_n["bwd"] * 1e3, 1),
        "fwd_tflops": round(3 * u / (fam_ms["fwd"] / fam_n["fwd"] * 1e-3) / 1e12, 1),
        "bwd_tflops": round(6 * u / (fam_ms["bwd"] / fam_n["bwd"] * 1e-3) / 1e12, 1),
        "fwd_bwd_tflops": round(9 * u / (ms * 1e-3) / 1e12, 1)}
    out["neuron_types"] = neuron_types(ql, torch, dev, stream, reps)
    out["depthwise"] = depthwise(ql, torch, dev, stream, reps)
    out["epilogue"] = epilogue_cost(ql, torch, dev, stream, reps)
    out["resnet20"] = resnet20_step_leg(ql, torch, dev, stream, reps)
    out["cold_cache"] = cold_cache(ql, torch, dev, stream)
    out["hybrid_bp_memory"] = hybrid_bp_memory(torch, dev)
    return out


def resnet20_step_leg(ql, torch, dev, stream, reps=10, drift=True):
    """The CIFAR ResNet-20 training step (batch 256, 3x32x32; section 4.2 model
    construction; paper_2204_01701_amd/resnet.py) in fp32 and bf16: forward to
    the logits and backward to every weight gradient, all in the library's
    kernels.  Per precision: the step time hot (steps back to back) and cold
    (a 512 MB buffer written before each step, so that the MALL holds none of
    the step's tensors; the write is outside the timed interval), the share of
    the 19 quadratic layers' calls (each call timed on its own, summed), the
    algorithmic TFLOP/s of the step (the 19 layers' 9U, less the 3U of the
    stem's input gradient, which the step does not compute; the dense head's
    and the glue's few flops are not counted) against the precision's
    dense MFMA peak, the quadratic layers' algorithmic GB/s, and the end-to-end
    drift of the logits and weight gradients from the fp64 network oracle."""
    import numpy as np
    import synth
    from paper_2204_01701_amd.resnet import ResNet20Step

    geoms = synth.resnet20_layers(256)
    # every layer's three passes, except the stem's input gradient, which the step does not compute
    flops = sum(9 * unit_flops(L) for L in geoms) - 3 * unit_flops(geoms[0])

    def qbytes(L, esize):
        X = L.n * L.h * L.w * L.c
        P = L.n * L.ho * L.wo * L.o
        W = L.o * L.c * L.k * L.k
        return esize * ((X + 3 * W + 3 * P) + (3 * P + 3 * W + X) + (X + 3 * P)) + 4 * (3 * W + 3 * L.o)

    out = {"shape": "CIFAR ResNet-20, batch 256, 3x32x32, 19 quadratic 3x3 convs + BN/ReLU/shortcuts + GAP + "
                    "quadratic FC 64->10", "gflop_per_step": round(flops / 1e9, 1)}
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    for name, dt, peak in (("fp32", torch.float32, 157.3), ("bf16", torch.bfloat16, BF16_PEAK_TFLOPS)):
        params, x, g = synth.resnet20_network(256, bf16=dt == torch.bfloat16)
        net = ResNet20Step(params, x, g, dtype=dt, device=dev)
        for _ in range(3):
            net.step(stream)
        torch.cuda.synchronize()
        a, b = DevEvent(), DevEvent()
        a.record(stream)
        for _ in range(reps):
            net.step(stream)
        b.record(stream)
        torch.cuda.synchronize()
        hot = a.elapsed_time(b) / reps
        # the step as one HIP graph (about 130 launches; from Python each launch
        # costs more host time than most of these kernels take on the GPU)
        net.capture()
        with torch.cuda.stream(stream):
            for _ in range(3):
                net.replay()
            torch.cuda.synchronize()
            a, b = DevEvent(), DevEvent()
            a.record(stream)
            for _ in range(reps):
                net.replay()
            b.record(stream)
            torch.cuda.synchronize()
            graph_hot = a.elapsed_time(b) / reps
            colds = []
            for _ in range(reps):
                flush.fill_(1)
                a, b = DevEvent(), DevEvent()
                a.record(stream)
                net.replay()
                b.record(stream)
                torch.cuda.synchronize()
                colds.append(a.elapsed_time(b))
        cold = sorted(colds)[len(colds) // 2]
        each = time_each(torch, net.qconv_calls(), reps, stream)
        qshare = sum(each.values()) / graph_hot
        esize = 2 if dt == torch.bfloat16 else 4
        r = {"step_ms_hot": round(graph_hot, 4), "step_ms_cold": round(cold, 4), "step_ms_eager": round(hot, 4),
             "tflops_hot": round(flops / (graph_hot * 1e-3) / 1e12, 1), "peak_tflops": peak,
             "pct_of_peak_hot": round(100 * flops / (graph_hot * 1e-3) / 1e12 / peak, 2),
             "quadratic_layer_share": round(qshare, 3),
             "quadratic_layers_gbs": round(sum(qbytes(L, esize) for L in geoms) / (sum(each.values()) * 1e-3) / 1e9, 1)}
        if drift:
            import oracle
            from oracle import network as onet
            f64 = {k: {n: np.asarray(v, np.float64) for n, v in p.items()} for k, p in params.items()}
            logits, grads, _ = onet.resnet20_step(
                f64, np.asarray(x, np.float64), np.asarray(g, np.float64), geoms,
                lambda xx, p, s_, pd: oracle.conv2d_fwd(xx, p["wa"], p["wb"], p["wc"], p["ba"], p["bb"], p["bc"],
                                                        s_, pd),
                lambda xx, p, gy, s_, pd: oracle.conv2d_bwd(xx, p["wa"], p["wb"], p["wc"], p["ba"], p["bb"],
                                                            p["bc"], gy, s_, pd),
                oracle.linear_fwd, oracle.linear_bwd)

            def rel(a_, b_):
                return float(np.linalg.norm(a_ - b_) / np.linalg.norm(b_))
            errs = [rel(net.layers[i]["dw"][t].permute(0, 3, 1, 2).double().cpu().numpy(), grads[i][k])
                    for i in range(len(geoms)) for t, k in enumerate(("dwa", "dwb", "dwc"))]
            r["drift_logits"] = round(rel(net.logits.double().cpu().numpy(), logits), 6)
            r["drift_weight_grad_median"] = round(float(np.median(errs)), 6)
            r["drift_weight_grad_max"] = round(float(np.max(errs)), 6)
        out[name] = r
        del net
    del flush
    # the small fp32 layer (N=2, 16 -> 16, 8x8): microseconds per call of each pass,
    # `reps` calls recorded as one HIP graph and replayed (a call from Python costs
    # more host time than this layer's kernels take on the GPU)
    L = synth.SMALL_FP32
    ly = Layer(ql, torch, L, 1, 0, dev, bf16=False)
    ly.fwd(stream)
    torch.cuda.synchronize()
    res = {}
    for f in ("fwd", "bwd_data", "bwd_weight"):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            cur = torch.cuda.current_stream(dev)
            for _ in range(reps):
                getattr(ly, f)(cur)
        with torch.cuda.stream(stream):
            g.replay()
            torch.cuda.synchronize()
            a, b = DevEvent(), DevEvent()
            a.record(stream)
            for _ in range(5):
                g.replay()
            b.record(stream)
            torch.cuda.synchronize()
        res[f] = round(a.elapsed_time(b) / (5 * reps) * 1e3, 2)
    out["small_fp32_layer_us"] = res
    return out


def neuron_types(ql, torch, dev, stream, reps=10):
    """The proposed neuron and the earlier types of Table 1 (T4, T4 + identity,
    T3, T2) on the large layer (N=64, 256->256, 56x56, bf16), each pass timed
    separately.  Algorithmic flops per pass: one first-order convolution (2 N
    Ho Wo O C KH KW) per weighted term (3, 2, 2, 1, 1); the elementwise work
    (products, the square of X for T2, the shortcut) is not counted."""
    import synth

    L = synth.LARGE_BF16
    u = unit_flops(L)
    names = {ql.QL_NEURON_QUADRA: "quadra", ql.QL_NEURON_T4: "t4", ql.QL_NEURON_T4_IDENTITY: "t4_identity",
             ql.QL_NEURON_T3: "t3", ql.QL_NEURON_T2: "t2"}
    res = {"shape": "N=64 C=256 56x56 -> 256, 3x3, bf16", "flops": "terms x 2 N Ho Wo O C KH KW per pass"}
    for ne, name in names.items():
        ly = Layer(ql, torch, L, 4, 0, dev, neuron=ne)
        calls = [("fwd", ly.fwd), ("bwd_data", ly.bwd_data), ("bwd_weight", ly.bwd_weight)]
        ms, _, fam_ms, fam_n = time_calls(torch, calls, reps, 3, stream)
        nt = ql.NEURON_TERMS[ne]
        r = {f"{f}_us": round(fam_ms[f] / fam_n[f] * 1e3, 1) for f in ("fwd", "bwd_data", "bwd_weight")}
        r["fwd_bwd_tflops"] = round(3 * nt * u / (ms * 1e-3) / 1e12, 1)
        res[name] = r
        del ly
    return res


def dw_bytes(L, fam, esize=2, nterms=3):
    """Algorithmic HBM bytes of one pass of a depthwise layer of the proposed
    neuron: every input and output tensor once (X, the maps Y / T_a / T_b or G /
    T_a / T_b, dX; the fp32 weight and bias gradients), nothing re-read."""
    X = L.n * L.h * L.w * L.c
    P = L.n * L.ho * L.wo * L.o
    Wt = nterms * L.c * L.k * L.k
    if fam == "fwd":
        return esize * (X + 3 * P + Wt) + 4 * nterms * L.c
    if fam == "bwd_data":
        return esize * (3 * P + X + Wt)
    return esize * (X + 3 * P) + 4 * (Wt + nterms * L.c)


def depthwise(ql, torch, dev, stream, reps=10):
    """Depthwise quadratic layers (groups = C, the pair layers of MobileNet-V1,
    section 4.2 and Table 3), bf16, the proposed neuron: the 13 depthwise /
    pointwise pairs of a CIFAR MobileNet-V1 at batch 128 (summed over the
    layers), and one large depthwise layer (N=64, C=256, 56x56, 3x3) where the
    direct kernels meet the HBM roofline; each pass timed separately (each call
    repeated back to back, events at the ends: time_each)."""
    import synth

    fams = ("fwd", "bwd_data", "bwd_weight")
    res = {}
    pairs = synth.mobilenet_v1_pairs(128)
    dws = [Layer(ql, torch, d, 7, i, dev, depthwise=True) for i, (d, _) in enumerate(pairs)]
    pws = [Layer(ql, torch, p, 8, i, dev) for i, (_, p) in enumerate(pairs)]
    calls = [((f, "dw", i), getattr(ly, f)) for i, ly in enumerate(dws) for f in fams]
    calls += [((f, "pw", i), getattr(ly, f)) for i, ly in enumerate(pws) for f in fams]
    ms, _, _, _ = time_calls(torch, calls, reps, 3, stream, timed_families=set())
    each = time_each(torch, calls, reps, stream)
    r = {"shape": "CIFAR MobileNet-V1, batch 128, 13 pairs of 3x3 depthwise + 1x1 pointwise, bf16",
         "pair_step_us": round(ms * 1e3, 1)}
    for kind, lys in (("dw", dws), ("pw", pws)):
        for f in fams:
            t = sum(each[(f, kind, i)] for i in range(len(lys)))
            r[f"{kind}_{f}_us"] = round(t * 1e3, 1)
            if kind == "dw":
                r[f"{kind}_{f}_gbs"] = round(sum(dw_bytes(ly.L, f) for ly in lys) / (t * 1e-3) / 1e9, 1)
            else:
                r[f"{kind}_{f}_tflops"] = round(3 * sum(unit_flops(ly.L) for ly in lys) / (t * 1e-3) / 1e12, 1)
    res["mobilenet_v1_cifar_b128"] = r
    del dws, pws, calls

    L = synth.ConvLayer(n=64, c=256, h=56, w=56, o=256, k=3, stride=1, pad=1)
    ly = Layer(ql, torch, L, 9, 0, dev, depthwise=True)
    calls = [(f, getattr(ly, f)) for f in fams]
    ly.fwd(stream)
    each = time_each(torch, calls, reps, stream)
    r = {"shape": "N=64 C=256 56x56, 3x3 depthwise, bf16", "peak_gbs": HBM_PEAK_GBS}
    for f in fams:
        t = each[f]
        gbs = dw_bytes(L, f) / (t * 1e-3) / 1e9
        r[f"{f}_us"] = round(t * 1e3, 1)
        r[f"{f}_gbs"] = round(gbs, 1)
        r[f"{f}_frac"] = round(gbs / HBM_PEAK_GBS, 3)
    res["large_dw"] = r
    return res


def epilogue_cost(ql, torch, dev, stream, reps=10):
    """The fused forward epilogue on the 13 VGG-16 layers (bf16, batch 128), the
    forward of each layer summed: plain; with the batch-normalization sums of
    Y (training); with a per-channel scale / shift and ReLU (a batch
    normalization with fixed statistics, then the activation; section 4.2).
    For comparison, the sums taken by a separate torch reduction over the
    stored Y (torch.var_mean over N, H, W)."""
    import synth

    geoms = synth.vgg16_layers(128)
    layers = [Layer(ql, torch, L, 2, i, dev) for i, L in enumerate(geoms)]
    stats, affs, wss = [], [], []
    for ly in layers:
        O = ly.L.o
        ssum, ssq = torch.empty(O, device=dev), torch.empty(O, device=dev)
        sc, sh = torch.rand(O, device=dev) + 0.5, torch.randn(O, device=dev)
        e_stat = ql.epilogue(None, None, False, ssum, ssq)
        e_aff = ql.epilogue(sc, sh, True)
        need = max(ql.qlayer_conv2d_fwd_ex_workspace_size(ly.desc, e_stat), 256)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        stats.append((e_stat, ssum, ssq))
        affs.append((e_aff, sc, sh))
        wss.append(ws)

    def fwd_ex(i, e):
        ly = layers[i]
        return lambda st: ql.qlayer_conv2d_fwd_ex(ly.desc, ly.x, *ly.w, *ly.b, ly.y, ly.ta, ly.tb, epi=e,
                                                  workspace=(wss[i].data_ptr(), wss[i].numel()), stream=st)

    def torch_stats(i):
        ly = layers[i]
        return lambda st: torch.var_mean(ly.y.float(), dim=(0, 1, 2), unbiased=False)

    res = {"shape": "13 VGG-16 layers, bf16, batch 128, forward only, us summed over the layers"}
    for name, calls in (("plain", [(i, layers[i].fwd) for i in range(len(layers))]),
                        ("bn_sums", [(i, fwd_ex(i, stats[i][0])) for i in range(len(layers))]),
                        ("scale_shift_relu", [(i, fwd_ex(i, affs[i][0])) for i in range(len(layers))]),
                        ("plain_then_torch_sums", [c for i in range(len(layers))
                                                   for c in ((i, layers[i].fwd), (("t", i), torch_stats(i)))])):
        each = time_each(torch, calls, reps, stream)
        res[f"{name}_us"] = round(sum(each.values()) * 1e3, 1)
    del layers
    return res


def hybrid_bp_memory(torch, dev, batch=256, reps=5):
    """Peak device memory of one training step (forward + backward) of a small
    quadratic ConvNet in the two memory modes of section 4.3: T_a, T_b saved by
    the forward, or regenerated in the backward (hybrid back-propagation).  The
    network stands in for the paper's memory experiment (3 quadratic conv layers
    + 2 quadratic FC layers, batch 256, 32 x 32 inputs): qconv 3->64, 64->128,
    128->256 (3x3, pad 1), each followed by ReLU and 2x2 max-pool, then qFC
    4096->512, ReLU, qFC 512->10; bf16, synthetic N(0,1) inputs, He-scaled weights."""
    from paper_2204_01701_amd.autograd import quad_conv2d, quad_linear

    g = torch.Generator(device=dev).manual_seed(0)

    def weights(shape, fan_in):
        return [(torch.randn(shape, device=dev, generator=g) * (2.0 / fan_in) ** 0.5).to(torch.bfloat16)
                .requires_grad_(True) for _ in range(3)]

    convs = [weights((64, 3, 3, 3), 27), weights((128, 64, 3, 3), 576), weights((256, 128, 3, 3), 1152)]
    fcs = [weights((512, 4096), 4096), weights((10, 512), 512)]
    x = torch.randn(batch, 3, 32, 32, device=dev, generator=g).to(torch.bfloat16)
    x = x.contiguous(memory_format=torch.channels_last)
    gl = torch.randn(batch, 10, device=dev, generator=g).to(torch.bfloat16)

    def step(recompute):
        h = x
        for w in convs:
            h = torch.nn.functional.max_pool2d(torch.relu(quad_conv2d(h, *w, stride=1, pad=1, recompute=recompute)), 2)
        h = h.flatten(1)
        h = torch.relu(quad_linear(h, *fcs[0], recompute=recompute))
        quad_linear(h, *fcs[1], recompute=recompute).backward(gl)

    res = {"network": "qconv 3-64-128-256 (3x3, ReLU, max-pool) + qFC 4096-512-10, bf16, batch 256, 32x32"}
    for mode in ("save", "recompute"):
        rc = mode == "recompute"
        for _ in range(3):  # warm-up (allocator growth, first launches)
            step(rc)
        torch.cuda.synchronize()
        for ws in convs + fcs:
            for w in ws:
                w.grad = None
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats(dev)
        base = torch.cuda.memory_allocated(dev)
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(reps):
            step(rc)
        t1.record()
        torch.cuda.synchronize()
        res[f"{mode}_peak_mb"] = round((torch.cuda.max_memory_allocated(dev) - base) / 2**20, 1)
        res[f"{mode}_step_ms"] = round(t0.elapsed_time(t1) / reps, 3)
        for ws in convs + fcs:
            for w in ws:
                w.grad = None
    res["memory_saving_pct"] = round(100 * (1 - res["recompute_peak_mb"] / res["save_peak_mb"]), 1)
    return res


if __name__ == "__main__":
    main()
