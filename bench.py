#!/usr/bin/env python3
"""Benchmark of the PVConv forward on one MI355X.

Layer workloads (1, 2, 5): a step is one call of pvconv_forward on the whole
batch: normalisation and voxelisation, the 3x3x3 convolutions with batch norm
and leaky ReLU, trilinear devoxelisation and the point-branch MLP whose
epilogue adds the two branches (Section 4 of the PVCNN paper).
Network workloads (3, 4): a step is one forward of the PVCNN segmentation
network (Section 5.1): PVConv blocks, point MLPs, max-pool, head. Workload 6:
one forward of PVCNN++ (Section 5.2: PointNet++'s set abstraction and feature
propagation levels around PVConv layers) on 4 x 8192 room points.
Inputs (coordinates, features, weights) are resident in device memory before
the timed region starts.

Default workload: the part-segmentation-scale layer, 16 clouds x 2048 points,
64 -> 128 channels, R = 32, bf16 operands with fp32 accumulation.

Printed: ONE JSON line with the headline throughput (points/s), ms per layer,
the roofline of the dominant kernel (the convolution, MFMA-bound, timed on
weights packed beforehand as the forward runs it), per-step timings of the
same chain (back to back, and cold: after a 512 MiB write that evicts the
caches), including the fused devoxelisation + point MLP kernel the forward
runs, the peak device memory of one forward, the device's measured peaks (a
dense bf16 MFMA loop and a 16-byte copy) as a second denominator next to the
published ones, the CPU oracle timed on a bounded sample of the same workload
(which also checks the GPU output on that sample), and for the default
workload a compact `workloads` summary of the four others.

The per-step breakdown runs before the headline's warmup and timed steps, so
that those run at the clock the GPU settles to under load.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "PVConv fwd points/sec + ms/layer (N=2048,R=32,C=64→128); % HBM/MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps first (the clock settles under load within ~50 ms)")
    ap.add_argument("--workload", type=int, default=2, choices=(1, 2, 3, 4, 5, 6),
                    help="1 fp32 layer R=8, 2 part-seg layer R=32, 3 part-seg network, "
                         "4 scene-seg network, 5 stress layer R=64, 6 PVCNN++ scene-seg "
                         "network")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="lower bound of CPU work for the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-workloads", action="store_true",
                    help="headline workload only (no `workloads` summary of the others)")
    ap.add_argument("--workload-cpu-seconds", type=float, default=2.0,
                    help="lower bound of CPU work for each other workload's oracle sample")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured-peak probes (MFMA loop, copy)")
    ap.add_argument("--variants", action="store_true",
                    help="instead of the headline: the layer variants the paper discusses "
                         "(R 16/24/32, one to three convolutions, channel widths, nearest-"
                         "neighbour devoxelisation) on the part-seg layer's clouds, one JSON "
                         "line each")
    ap.add_argument("--backward", action="store_true",
                    help="instead of the headline: the backward entry points (input and "
                         "conv weight gradients) at the part-seg layer's shapes, one JSON "
                         "line each")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-MiB buffer 3 times (a plain copy kernel of known "
                         "size, to calibrate the HBM byte counters) and exit")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pv_conv3d_bf16_partseg_B16_R32_traffic.txt")
CONV_SOURCE = os.path.join(ROOT, "paper_1907_03739_amd", "csrc", "conv3d.hip")


def measured_traffic():
    """HBM bytes per conv launch from the committed counter summary, or None
    when the summary is missing or the conv source has changed since the
    counters were taken (its sha256 is recorded in the summary)."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE).read()
        src = hashlib.sha256(open(CONV_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    fields = dict(l.split("=", 1) for l in text.splitlines() if "=" in l and not l.startswith("#"))
    if fields.get("conv3d_source_sha256", "").strip() != src:
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {mib} MiB x 3", flush=True)


PEAK_LIB = os.path.join(ROOT, "paper_1907_03739_amd", "libpvpeak.so")


def measured_peaks(stream):
    """The device's measured peaks: dense bf16 MFMA (v_mfma_f32_32x32x16_bf16
    on random operands, three waves per SIMD, ~16 ms per launch after ~0.1 s
    of the same load) and HBM (a 16-byte copy of 1 GiB, read + write bytes);
    best of five launches each."""
    import ctypes
    import torch
    lib = ctypes.CDLL(PEAK_LIB)
    lib.pv_peak_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.pv_peak_mfma_flop.restype = ctypes.c_double
    lib.pv_peak_mfma_flop.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.pv_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                 ctypes.c_void_p]
    h = ctypes.c_void_p(stream.cuda_stream)

    def best(launch, warm, reps):
        for _ in range(warm):
            launch()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return min(ts)

    blocks = 3 * torch.cuda.get_device_properties(stream.device).multi_processor_count
    iters = 100000
    out = torch.empty(blocks * 256, dtype=torch.float32, device=stream.device)

    def mfma():
        if lib.pv_peak_mfma(blocks, iters, ctypes.c_void_p(out.data_ptr()), h) != 0:
            raise RuntimeError("MFMA probe launch failed")
    t_mfma = best(mfma, 6, 5)
    n = 1 << 30
    src = torch.ones(n // 4, dtype=torch.float32, device=stream.device)
    dst = torch.empty_like(src)

    def copy():
        if lib.pv_peak_copy(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                            n // 16, h) != 0:
            raise RuntimeError("copy probe launch failed")
    t_copy = best(copy, 3, 5)
    del src, dst, out
    return {"mfma_bf16_tflops": round(lib.pv_peak_mfma_flop(blocks, iters) / t_mfma / 1e12, 1),
            "hbm_copy_gbs": round(2 * n / t_copy / 1e9, 1),
            "how": f"MFMA loop {blocks} workgroups x 4 waves, {iters} rounds of 4 "
                   f"32x32x16 bf16 MFMAs; streaming 16-byte copy of 1 GiB (2 GiB moved); "
                   f"best of 5 launches"}


def conv_flops(B, R, cin, cout):
    return 2.0 * 27 * cin * cout * B * R ** 3


def distinct_corners(pn, R):
    """Number of distinct (cloud, cell) pairs the trilinear gather touches,
    from the normalised coordinates the GPU wrote (for the algorithmic byte
    count of devoxelisation)."""
    import numpy as np
    B = pn.shape[0]
    t = np.clip(pn.astype(np.float64) * R - 0.5, 0.0, R - 1)
    i0 = np.floor(t).astype(np.int64)
    i1 = np.minimum(i0 + 1, R - 1)
    total = 0
    for b in range(B):
        cells = []
        for a in (i0[b], i1[b]):
            for e in (i0[b], i1[b]):
                for g in (i0[b], i1[b]):
                    cells.append((a[:, 0] * R + e[:, 1]) * R + g[:, 2])
        total += np.unique(np.concatenate(cells)).size
    return total


def cpu_baseline(wl, gpu_out, seconds):
    """The oracle on the workload's clouds, one per call, in order (again from
    the first once all are done) until at least `seconds` of CPU work; also
    compares the GPU output on those clouds against it (the bf16 chain bound
    of the parity tests)."""
    import numpy as np
    import oracle
    L = wl.layers[0]
    oracle.pvconv_forward(wl.coords[:1, :8], wl.feats[:1, :8], L)  # load the library
    done, worst, t_total = 0, 0.0, 0.0
    while t_total < seconds:
        b = done % wl.B
        t0 = time.perf_counter()
        ref = oracle.pvconv_forward(wl.coords[b:b + 1], wl.feats[b:b + 1], L)[0]
        t_total += time.perf_counter() - t0
        if done < wl.B:
            rms = float(np.sqrt(np.mean(ref ** 2)))
            worst = max(worst, float(np.max(np.abs(gpu_out[b] - ref) / (np.abs(ref) + rms))))
        done += 1
    checked = min(done, wl.B)
    tol = 2e-2 if wl.dtype == "bf16" else 1e-5
    return ({"value": done * wl.N / t_total, "unit": "points/s", "cores": oracle.threads(),
             "kind": "oracle",
             "sample": f"{done} oracle calls of one cloud ({done * wl.N} points) over the "
                       f"{wl.B} clouds in order, fp64, {t_total:.1f} s"},
            {"clouds": checked, "max_err": worst, "bound": tol, "ok": worst <= tol})


def network_flops(wl):
    """MFMA flops of one network forward, per step name."""
    B, N = wl.B, wl.N
    fl = {}
    for i, L in enumerate(wl.layers):
        c, f = L.cin, 0.0
        for _ in range(L.n_convs):
            f += conv_flops(B, L.R, c, L.cout)
            c = L.cout
        fl[f"pvconv{i + 1}"] = f + 2.0 * B * N * L.cin * L.cout
    for j, lp in enumerate(wl.mlps):
        fl[f"mlp{j + 1}"] = 2.0 * B * N * lp.w.shape[0] * lp.w.shape[1]
    cg = wl.mlps[-1].w.shape[0] if wl.mlps else wl.layers[-1].cout
    h0 = wl.head[0].w
    fl["global"] = 2.0 * B * cg * h0.shape[0]
    fl["head"] = 2.0 * B * N * (h0.shape[0] * (h0.shape[1] - cg)) + sum(
        2.0 * B * N * lp.w.shape[0] * lp.w.shape[1] for lp in wl.head[1:])
    return fl


def pvcnn2_work(wl):
    """Work of each step of the PVCNN++ forward: MFMA flops of the PVConv
    layers, the shared MLPs and the head (bf16), and for the sampling steps
    the fp32 operations of farthest point sampling and ball query (about 9
    per distance: three differences, three products, two sums and a
    comparison), which run as sequential steps per cloud."""
    B = wl.B
    npts = [wl.N] + [lev.npoint for lev in wl.sa]
    work = {}
    c = wl.feats.shape[2]
    c_feat = []
    for l, lev in enumerate(wl.sa):
        if lev.pvconvs:
            f = 0.0
            for L in lev.pvconvs:
                ci = L.cin
                for _ in range(L.n_convs):
                    f += conv_flops(B, L.R, ci, L.cout)
                    ci = L.cout
                f += 2.0 * B * npts[l] * L.cin * L.cout
            work[f"pvconv{l + 1}"] = ("TFLOP/s", f)
            c = lev.pvconvs[-1].cout
        c_feat.append(c)
        work[f"sample{l + 1}"] = ("fp32 TFLOP/s", 9.0 * B * npts[l] * (lev.npoint + lev.npoint))
        rows = B * lev.npoint * lev.nsample
        work[f"group_mlp{l + 1}"] = ("TFLOP/s", sum(2.0 * rows * m.w.shape[0] * m.w.shape[1]
                                                   for m in lev.mlps))
        c = lev.mlps[-1].w.shape[0]
    for k, lev in enumerate(wl.fp):
        l = len(wl.sa) - 1 - k
        work[f"fp{k + 1}"] = ("TFLOP/s", sum(2.0 * B * npts[l] * m.w.shape[0] * m.w.shape[1]
                                            for m in lev.mlps))
    work["head"] = ("TFLOP/s", sum(2.0 * B * wl.N * m.w.shape[0] * m.w.shape[1]
                                   for m in wl.head))
    return work


def bench_network(args, wl, dev, peaks=True, cpu_seconds=None):
    """A step is one whole segmentation-network forward on the batch: PVCNN
    (PVConv blocks, point MLPs, max-pool, head) or PVCNN++ (set abstraction
    and feature propagation levels around PVConv layers, head). Returns the
    JSON line (a dict)."""
    import numpy as np
    import torch
    from paper_1907_03739_amd.network import DeviceNetwork, DevicePVCNN2

    B, N = wl.B, wl.N
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats(dev)
    base = torch.cuda.memory_allocated(dev)
    if wl.is_pvcnn2:
        net = DevicePVCNN2(wl.sa, wl.fp, wl.head, B, N, wl.feats.shape[2], dev)
    else:
        net = DeviceNetwork(wl.layers, wl.mlps, wl.head, B, N, dev)
    coords = torch.as_tensor(wl.coords).to(dev)
    feats = torch.as_tensor(wl.feats).to(dev)
    net.forward(coords, feats)
    torch.cuda.synchronize()
    memory = {"peak_bytes": int(torch.cuda.max_memory_allocated(dev) - base),
              "how": "torch.cuda.max_memory_allocated over building the network (weights, "
                     "activation and workspace buffers), the inputs and one forward"}
    stream = torch.cuda.current_stream(dev)

    # per-step breakdown first (events between the steps of whole forwards),
    # so that the headline's steps run at the settled clock
    names = net.steps()
    per = {n: [] for n in names}
    for _ in range(max(args.steps, 10)):
        marks = []

        def mark(name, marks=marks):
            e = torch.cuda.Event(enable_timing=True)
            e.record(stream)
            marks.append(e)

        net.forward_timed(coords, feats, mark)
        torch.cuda.synchronize()
        for j, n in enumerate(names):
            per[n].append(marks[j].elapsed_time(marks[j + 1]))

    # two events around the K steps only: an event recorded between steps
    # leaves the GPU idle for a few microseconds
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    quiet_host()
    for _ in range(args.warmup):
        net.forward(coords, feats)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        net.forward(coords, feats)
    ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gc.enable()
    ev_ms = ev[0].elapsed_time(ev[1]) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    gpu_out = net.logits.double().cpu().numpy()

    work = pvcnn2_work(wl) if wl.is_pvcnn2 else {n: ("TFLOP/s", f)
                                                 for n, f in network_flops(wl).items()}
    kernels = {}
    for n in names:
        unit, amount = work[n]
        peak = PEAK_F32_TFLOPS if unit.startswith("fp32") else PEAK_BF16_TFLOPS
        ms = statistics.mean(per[n])
        rate = amount / (ms * 1e-3) / 1e12
        kernels[n] = {"ms": round(ms, 4), "ms_min": round(min(per[n]), 4),
                      "achieved": round(rate, 2), "unit": "TFLOP/s",
                      "frac": round(rate / peak, 4), "algorithmic": amount}
        if unit.startswith("fp32"):
            kernels[n]["bound"] = "alu (sequential per cloud)"
    dom = max(names, key=lambda n: kernels[n]["ms"])
    dom_f32 = work[dom][0].startswith("fp32")
    roofline = {"bound": "alu" if dom_f32 else "mfma", "achieved": kernels[dom]["achieved"],
                "peak": PEAK_F32_TFLOPS if dom_f32 else PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": kernels[dom]["frac"], "traffic": None,
                "kernel": f"network step {dom}", "flop_per_launch": work[dom][1],
                "avg_launch_ms": kernels[dom]["ms"]}
    pk = measured_peaks(stream) if peaks else None
    if pk and not dom_f32:
        roofline["frac_measured_peak"] = round(kernels[dom]["achieved"] /
                                               pk["mfma_bf16_tflops"], 4)
    total_fl = sum(a for u, a in work.values() if not u.startswith("fp32"))
    line = {
        "metric": METRIC, "value": round(B * N / (ms_per_step * 1e-3), 1), "unit": "points/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": ({"workload": wl.name, "B": B, "N": N,
                    "sa": [{"pvconv": [[L.cin, L.cout, L.R] for L in lev.pvconvs],
                            "npoint": lev.npoint, "radius": lev.radius,
                            "nsample": lev.nsample, "mlp": [int(m.w.shape[0]) for m in lev.mlps]}
                           for lev in wl.sa],
                    "fp": [[int(m.w.shape[0]) for m in lev.mlps] for lev in wl.fp],
                    "head": [int(h.w.shape[0]) for h in wl.head], "points_per_step": B * N}
                   if wl.is_pvcnn2 else
                   {"workload": wl.name, "B": B, "N": N,
                    "blocks": [[L.cin, L.cout, L.R] for L in wl.layers],
                    "mlps": [int(m.w.shape[0]) for m in wl.mlps],
                    "head": [int(h.w.shape[0]) for h in wl.head], "points_per_step": B * N}),
        "ms_per_step_events": round(ev_ms, 4),
        "network_tflops": round(total_fl / (ms_per_step * 1e-3) / 1e12, 2),
        "roofline": roofline,
        "kernels": kernels,
        "memory": memory,
        "peaks_measured": pk,
        "inputs_sha256": wl.sha256(),
    }
    if cpu_seconds:
        import oracle
        done, worst, t_total = 0, 0.0, 0.0
        while t_total < cpu_seconds and done < B:
            one = synth_one(wl, done)
            t1 = time.perf_counter()
            ref = (oracle.pvcnn2_forward(one, stage_dtype="bf16") if wl.is_pvcnn2 else
                   oracle.network_forward(one, stage_dtype="bf16"))[0]
            t_total += time.perf_counter() - t1
            rms = float(np.sqrt(np.mean(ref ** 2)))
            worst = max(worst, float(np.max(np.abs(gpu_out[done] - ref) /
                                            (np.abs(ref) + rms))))
            done += 1
        line["cpu_baseline"] = {
            "value": done * N / t_total, "unit": "points/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": f"first {done} of {B} clouds ({done * N} points), one cloud per oracle "
                      f"call, fp64 with bf16 stage storage, {t_total:.1f} s"}
        # end-to-end bound of the network parity tests: sqrt(S) x the chain bound
        if wl.is_pvcnn2:
            stages = sum(len(lev.pvconvs) + 1 + len(lev.mlps) for lev in wl.sa) + sum(
                1 + len(lev.mlps) for lev in wl.fp) + len(wl.head) - 1
        else:
            stages = len(wl.layers) + len(wl.mlps) + len(wl.head) - 1
        bound = 2e-2 * stages ** 0.5
        line["parity_sample"] = {"clouds": done, "max_err": worst, "bound": round(bound, 4),
                                 "ok": worst <= bound}
    return line


# Layer variants on the default workload's clouds (16 x 2048 points): the
# resolution sweep of the resolution table (R = 16, 24, 32), the number of
# convolutions per PVConv of the ablation table (1, 2, 3), narrower layers
# (the width multipliers of the scene-segmentation table, down to 0.125 x C:
# 8 -> 16 channels, a convolution tile half of zero weights) and the
# nearest-neighbour devoxelisation the ablation compares with trilinear.
VARIANTS = [
    # name, R, n_convs, width, devox
    ("base", 32, 2, 1.0, "trilinear"),
    ("R16", 16, 2, 1.0, "trilinear"),
    ("R24", 24, 2, 1.0, "trilinear"),
    ("convs1", 32, 1, 1.0, "trilinear"),
    ("convs3", 32, 3, 1.0, "trilinear"),
    ("width0.5", 32, 2, 0.5, "trilinear"),
    ("width0.25", 32, 2, 0.25, "trilinear"),
    ("width0.125", 32, 2, 0.125, "trilinear"),
    ("nearest", 32, 2, 1.0, "nearest"),
    ("R16_width0.25", 16, 2, 0.25, "trilinear"),
    ("R16_width0.125", 16, 2, 0.125, "trilinear"),
]


def bench_variants(args, dev):
    import numpy as np
    import torch

    import synth
    from paper_1907_03739_amd import binding as pv

    wl = synth.make_workload(2)
    B, N = wl.B, wl.N
    coords = torch.as_tensor(wl.coords).to(dev)
    stream = torch.cuda.current_stream(dev)
    REPS = 10
    for name, R, n_convs, width, devox in VARIANTS:
        cin, cout = int(64 * width), int(128 * width)
        rng = np.random.default_rng(7000 + R + 10 * n_convs + int(100 * width))
        L = synth.draw_pvconv(rng, cin, cout, R, n_convs, bf16=True)
        L.devox = devox
        layer = pv.DeviceLayer(L, dev, torch.bfloat16)
        feats = torch.as_tensor(wl.feats[..., :cin]).to(dev).contiguous()
        out = torch.empty((B, N, cout), dtype=torch.float32, device=dev)
        ws = torch.empty(max(pv.pvconv_forward_workspace_size(B, N, layer), 256),
                         dtype=torch.uint8, device=dev)
        fn = lambda: pv.pvconv_forward(coords, feats, layer, out=out, workspace=ws)
        for _ in range(max(1, args.warmup // 5)):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(REPS):
                fn()
        g.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(max(3, args.steps // REPS)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / REPS)
        del g
        ms = statistics.median(times)
        flops = sum(conv_flops(B, R, cin if i == 0 else cout, cout) for i in range(n_convs))
        print(json.dumps({
            "variant": name, "R": R, "n_convs": n_convs, "cin": cin, "cout": cout,
            "devox": devox, "B": B, "N": N, "ms_per_layer": round(ms, 4),
            "ms_min": round(min(times), 4), "points_per_s": round(B * N / (ms * 1e-3), 1),
            "conv_tflop_per_layer": round(flops / 1e12, 4), "dtype": "bf16",
            "data": "synthetic"}), flush=True)


def bench_backward(args, dev):
    """Gradients of the part-seg layer's steps (inputs, and the convolutions'
    weights), in reverse order, each timed as the average of 10 back-to-back
    calls captured in a graph."""
    import numpy as np
    import torch

    import synth
    from paper_1907_03739_amd import binding as pv

    wl = synth.make_workload(2)
    L = wl.layers[0]
    B, N, R, cin, cout = wl.B, wl.N, L.R, L.cin, L.cout
    V = R ** 3
    stream = torch.cuda.current_stream(dev)
    layer = pv.DeviceLayer(L, dev, torch.bfloat16)
    coords = torch.as_tensor(wl.coords).to(dev)
    feats = torch.as_tensor(wl.feats).to(dev)
    grid, counts, ids, pn = pv.pvconv_voxelize(coords, feats, R, grid_dtype=torch.bfloat16)
    gen = torch.Generator(device=dev).manual_seed(5)
    dout = torch.randn((B, N, cout), device=dev, generator=gen)
    dgrid = torch.empty((B, V, cout), dtype=torch.float32, device=dev)
    y = torch.randn((B, V, cout), device=dev, generator=gen).to(torch.bfloat16)
    dz = torch.empty((B, V, cout), dtype=torch.float32, device=dev)
    dy16 = torch.randn((B, V, cout), device=dev, generator=gen).to(torch.bfloat16)
    dx2 = torch.empty((B, V, cout), dtype=torch.bfloat16, device=dev)
    dx1 = torch.empty((B, V, cin), dtype=torch.bfloat16, device=dev)
    dvox = torch.randn((B, V, cin), device=dev, generator=gen).to(torch.bfloat16)
    dfeats = torch.empty((B, N, cin), dtype=torch.float32, device=dev)
    wsz = max(pv._lib.pvconv_conv3d_backward_data_workspace_size(c, cout, 1) for c in (cin, cout))
    ws = torch.empty(wsz, dtype=torch.uint8, device=dev)
    bn2 = layer.conv_bn[1]
    dw1 = torch.empty((cout, 3, 3, 3, cin), dtype=torch.float32, device=dev)
    dw2 = torch.empty((cout, 3, 3, 3, cout), dtype=torch.float32, device=dev)
    wws = torch.empty(max(pv._lib.pvconv_conv3d_backward_weight_workspace_size(B, R, c, cout)
                          for c in (cin, cout)), dtype=torch.uint8, device=dev)
    dws = torch.empty(pv._lib.pvconv_devoxelize_backward_workspace_size(B, N, cout, R),
                      dtype=torch.uint8, device=dev)
    s_g = 2
    steps = [
        # name, call, unit, algorithmic amount per call
        ("devoxelize_backward", lambda: pv.pvconv_devoxelize_backward(dout, R, pn, out=dgrid,
                                                                      workspace=dws),
         "GB/s", B * N * (12 + 4 * cout) + B * V * cout * 4),
        ("act_bn_backward", lambda: pv.pvconv_act_bn_backward(dgrid, y, bn=bn2, out=dz),
         "GB/s", B * V * cout * (4 + s_g + 4)),
        ("conv2_backward_data", lambda: pv.pvconv_conv3d_backward_data(
            dy16, layer.conv_w[1], R, out_dtype=torch.bfloat16, out=dx2, workspace=ws),
         "TFLOP/s", conv_flops(B, R, cout, cout)),
        ("conv1_backward_data", lambda: pv.pvconv_conv3d_backward_data(
            dy16, layer.conv_w[0], R, out_dtype=torch.bfloat16, out=dx1, workspace=ws),
         "TFLOP/s", conv_flops(B, R, cin, cout)),
        ("conv2_backward_weight", lambda: pv.pvconv_conv3d_backward_weight(
            dy16, y, R, out=dw2, workspace=wws), "TFLOP/s", conv_flops(B, R, cout, cout)),
        ("conv1_backward_weight", lambda: pv.pvconv_conv3d_backward_weight(
            dy16, grid, R, out=dw1, workspace=wws), "TFLOP/s", conv_flops(B, R, cin, cout)),
        ("voxelize_backward", lambda: pv.pvconv_voxelize_backward(dvox, R, ids, counts,
                                                                   out=dfeats),
         "GB/s", B * N * (4 + 4 + 4 * cin) + int((counts > 0).sum().item()) * cin * s_g),
    ]
    REPS = 10
    for name, fn, unit, amount in steps:
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(REPS):
                fn()
        g.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(max(3, args.steps // REPS)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / REPS)
        del g
        ms = statistics.median(times)
        if unit == "GB/s":
            rate, peak = amount / (ms * 1e-3) / 1e9, PEAK_HBM_GBS
        else:
            rate, peak = amount / (ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS
        print(json.dumps({"step": name, "workload": wl.name, "ms": round(ms, 4),
                          "ms_min": round(min(times), 4), "achieved": round(rate, 2),
                          "unit": unit, "peak": peak, "frac": round(rate / peak, 4),
                          "algorithmic": amount, "dtype": "bf16 in, fp32 gradients",
                          "data": "synthetic"}), flush=True)


def synth_one(wl, b):
    """Workload wl restricted to its cloud b (the networks are per cloud)."""
    import copy
    one = copy.copy(wl)
    one.B, one.coords, one.feats = 1, wl.coords[b:b + 1], wl.feats[b:b + 1]
    return one


def cpu_model():
    """The host CPU's model name and the cores this process may use."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": name, "cores_available": len(os.sched_getaffinity(0))}


def quiet_host():
    """Before a timed region: collect the garbage the breakdown left (graphs
    among it, whose destruction can block the host) and keep the collector
    off until the region ends (the caller enables it again)."""
    import torch
    gc.collect()
    torch.cuda.synchronize()
    gc.disable()


# The per-step breakdown: each step captured BREAKDOWN_REPS times back to back
# in one graph, replayed BREAKDOWN_ROUNDS times (independent of --steps: it is
# diagnostics around the headline, not the headline).
BREAKDOWN_REPS = 10
BREAKDOWN_ROUNDS = 10


def captured(fn, stream, reps, rounds):
    """The graph of `reps` back-to-back calls of fn (so that host submission
    cannot leave the GPU idle between them) and its ms per call over
    `rounds` replays, all enqueued before one synchronisation, between HIP
    events on the stream the kernels run on."""
    import torch
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    g.replay()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(max(1, rounds) + 1)]
    ev[0].record(stream)
    for i in range(max(1, rounds)):
        g.replay()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    return g, [ev[i].elapsed_time(ev[i + 1]) / reps for i in range(max(1, rounds))]


def graph_times(fn, stream, reps, rounds):
    """ms per call of fn, as captured() measures it (the graph is freed)."""
    g, times = captured(fn, stream, reps, rounds)
    del g
    return times


def cold_times(fn, stream, reps, rounds, dev):
    """ms per call from cold caches: a graph of `reps` (flush, call) pairs
    against a graph of `reps` flushes alone, where a flush is a 512 MiB write
    that evicts the L2s and the 256 MB Infinity Cache."""
    import torch
    scratch = torch.empty(512 << 18, dtype=torch.float32, device=dev)

    def flush():
        scratch.fill_(1.0)

    def both():
        flush()
        fn()

    t_flush = graph_times(flush, stream, reps, rounds)
    t_both = graph_times(both, stream, reps, rounds)
    del scratch
    return [b - f for b, f in zip(t_both, t_flush)]


def bench_layer(args, wl, dev, cold=True, peaks=True, cpu_seconds=None):
    """A step is one pvconv_forward call on the whole batch. Returns the JSON
    line (a dict) and the output of the last timed step."""
    import numpy as np
    import torch

    from paper_1907_03739_amd import binding as pv

    L = wl.layers[0]
    bf16 = wl.dtype == "bf16"
    cdt = torch.bfloat16 if bf16 else torch.float32
    B, N, R, cin, cout = wl.B, wl.N, L.R, L.cin, L.cout
    V = R ** 3
    stream = torch.cuda.current_stream(dev)

    # ---- device memory of one layer forward: inputs, weights, workspace,
    # output (the library allocates nothing itself) ------------------------
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats(dev)
    base = torch.cuda.memory_allocated(dev)
    layer = pv.DeviceLayer(L, dev, cdt)
    coords = torch.as_tensor(wl.coords).to(dev)
    feats = torch.as_tensor(wl.feats).to(dev)
    out = torch.empty((B, N, cout), dtype=torch.float32, device=dev)
    ws = torch.empty(max(pv.pvconv_forward_workspace_size(B, N, layer), 256), dtype=torch.uint8,
                     device=dev)
    pv.pvconv_forward(coords, feats, layer, out=out, workspace=ws)
    torch.cuda.synchronize()
    memory = {"peak_bytes": int(torch.cuda.max_memory_allocated(dev) - base),
              "workspace_bytes": int(ws.numel()),
              "how": "torch.cuda.max_memory_allocated over allocating the inputs, weights, "
                     "output and workspace and one forward"}

    # ---- per-step breakdown, run before the headline so that the headline's
    # steps run at the settled clock: the forward's kernels called one C-ABI
    # step at a time on the same data. Convolutions run on weights packed
    # beforehand (the forward packs them inside the voxelisation launch). ---
    grid = torch.empty((B, V, cin), dtype=cdt, device=dev)
    counts = torch.empty((B, V), dtype=torch.int32, device=dev)
    ids = torch.empty((B, N), dtype=torch.int32, device=dev)
    pn = torch.empty((B, N, 3), dtype=torch.float32, device=dev)
    vws = torch.empty(max(pv._lib.pvconv_voxelize_workspace_size(B, N, R), 256),
                      dtype=torch.uint8, device=dev)
    hs = [torch.empty((B, V, cout), dtype=cdt, device=dev) for _ in range(L.n_convs)]
    packed = [pv.pvconv_conv3d_pack_weights(w) for w in layer.conv_w] if bf16 else None
    dv = torch.empty((B, N, cout), dtype=torch.float32, device=dev)
    out2 = torch.empty_like(out)
    fused = bf16 and L.devox == "trilinear"
    # the forward hands a sparse grid to its first convolution for bf16 clouds
    # of up to 4096 points (the single-launch voxeliser's range)
    sparse_fwd = bf16 and N <= 4096
    steps = ["voxelize"] + [f"conv{i + 1}" for i in range(L.n_convs)]
    steps += ["devox_point_mlp", "devoxelize", "point_mlp"] if fused else ["devoxelize",
                                                                           "point_mlp"]

    def step_fn(name):
        if name == "voxelize":
            return lambda: pv.pvconv_voxelize(coords, feats, R, grid_dtype=cdt, grid=grid,
                                              counts=counts, ids=ids, norm=pn, workspace=vws)
        if name.startswith("conv"):
            i = int(name[4:]) - 1
            src = grid if i == 0 else hs[i - 1]
            if bf16:
                return lambda: pv.pvconv_conv3d_packed(src, packed[i], cout, R,
                                                       bn=layer.conv_bn[i], act="leaky",
                                                       slope=L.slope, out=hs[i])
            return lambda: pv.pvconv_conv3d(src, layer.conv_w[i], R, bn=layer.conv_bn[i],
                                            act="leaky", slope=L.slope, out=hs[i])
        if name == "devox_point_mlp":
            return lambda: pv.pvconv_devoxelize_point_mlp(hs[-1], R, pn, feats, layer.mlp_w,
                                                          bias=layer.mlp_b, bn=layer.mlp_bn,
                                                          act="relu", out=out2)
        if name == "devoxelize":
            return lambda: pv.pvconv_devoxelize(hs[-1], R, pn, out=dv)
        return lambda: pv.pvconv_point_mlp(feats, layer.mlp_w, bias=layer.mlp_b, bn=layer.mlp_bn,
                                           act="relu", residual=dv, out=out2)

    for n in steps:  # one eager pass fills every intermediate
        step_fn(n)()
    torch.cuda.synchronize()
    per = {n: graph_times(step_fn(n), stream, BREAKDOWN_REPS, BREAKDOWN_ROUNDS) for n in steps}
    cold_ms = {n: cold_times(step_fn(n), stream, BREAKDOWN_REPS, BREAKDOWN_ROUNDS, dev)
               for n in steps} if cold else None
    pn_host = pn.cpu().numpy()
    # two events around the K steps only: an event recorded between steps
    # leaves the GPU idle for a few microseconds
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    quiet_host()
    # the whole forward, BREAKDOWN_REPS steps per graph (no host launch cost
    # between kernels), last in the breakdown: about 50 ms of back-to-back
    # steps, followed by the headline without a pause (the GPU's clock drops
    # within milliseconds of idling and takes tens of milliseconds of load to
    # come back). The graph is freed after the headline.
    fwd = lambda: pv.pvconv_forward(coords, feats, layer, out=out, workspace=ws)
    fwd_graph, graph_ms = captured(fwd, stream, BREAKDOWN_REPS, BREAKDOWN_ROUNDS)

    # ---- headline: W untimed steps, then exactly K timed steps -------------
    for _ in range(args.warmup):
        pv.pvconv_forward(coords, feats, layer, out=out, workspace=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        pv.pvconv_forward(coords, feats, layer, out=out, workspace=ws)
    ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    del fwd_graph
    gc.enable()
    ev_ms = ev[0].elapsed_time(ev[1]) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    gpu_out = out.double().cpu().numpy()

    pk = measured_peaks(stream) if peaks else None

    # ---- algorithmic work per step ---------------------------------------
    s_g = 2 if bf16 else 4
    corners = distinct_corners(pn_host, R)
    work = {
        "voxelize": ("GB/s", B * N * (12 + 4 * cin + 4) + B * V * (cin * s_g + 4)),
        "devoxelize": ("GB/s", B * N * (12 + 4 * cout) + corners * cout * s_g),
        "point_mlp": ("GB/s", B * N * (4 * cin + 8 * cout)),
        # read: coordinates, features, the grid rows the points touch, the
        # weights; write: the output
        "devox_point_mlp": ("GB/s", B * N * (12 + 4 * cin + 4 * cout) + corners * cout * 2 +
                            cout * cin * 2),
    }
    c = cin
    for i in range(L.n_convs):
        work[f"conv{i + 1}"] = ("TFLOP/s", conv_flops(B, R, c, cout))
        c = cout
    kernels = {}
    for n in steps:
        unit, amount = work[n]
        ms = statistics.mean(per[n])
        if unit == "GB/s":
            rate, peak = amount / (ms * 1e-3) / 1e9, PEAK_HBM_GBS
        else:
            rate = amount / (ms * 1e-3) / 1e12
            peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
        k = {"ms": round(ms, 4), "ms_min": round(min(per[n]), 4), "achieved": round(rate, 2),
             "unit": unit, "frac": round(rate / peak, 4), "algorithmic": amount,
             "in_forward": not (fused and n in ("devoxelize", "point_mlp"))}
        if n == "voxelize" and sparse_fwd:
            k["in_forward"] = False
            k["forward_form"] = ("the forward runs the same kernel without the empty voxels' "
                                 "zero rows (its first convolution reads them as zero through "
                                 "the counts) and with the weight packing in extra workgroups")
        if cold_ms:
            ms_cold = statistics.median(cold_ms[n])
            rate_cold = amount / (ms_cold * 1e-3) / (1e9 if unit == "GB/s" else 1e12)
            k.update({"ms_cold": round(ms_cold, 4), "achieved_cold": round(rate_cold, 2),
                      "frac_cold": round(rate_cold / peak, 4)})
        if pk:
            mp = pk["hbm_copy_gbs"] if unit == "GB/s" else (
                pk["mfma_bf16_tflops"] if bf16 else None)
            if mp:
                k["frac_measured_peak"] = round(rate / mp, 4)
        kernels[n] = k

    # dominant kernel: the convolution (one kernel, L.n_convs launches per step)
    conv_names = [f"conv{i + 1}" for i in range(L.n_convs)]
    conv_ms = statistics.mean([kernels[n]["ms"] for n in conv_names])
    conv_work = statistics.mean([work[n][1] for n in conv_names])
    conv_peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    achieved = conv_work / (conv_ms * 1e-3) / 1e12
    roofline = {"bound": "mfma" if bf16 else "alu", "achieved": round(achieved, 2),
                "peak": conv_peak, "unit": "TFLOP/s", "frac": round(achieved / conv_peak, 4),
                "traffic": measured_traffic() if (bf16 and wl.index == 2) else None,
                "kernel": "pv_conv3d_bf16_kernel" if bf16 else "pv_conv3d_f32_kernel",
                "flop_per_launch": conv_work, "avg_launch_ms": round(conv_ms, 4),
                "timed": "pvconv_conv3d_packed (weights packed beforehand)" if bf16 else
                         "pvconv_conv3d"}
    if pk and bf16:
        roofline["frac_measured_peak"] = round(achieved / pk["mfma_bf16_tflops"], 4)

    line = {
        "metric": METRIC, "value": round(B * N / (ms_per_step * 1e-3), 1), "unit": "points/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if bf16 else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "N": N, "R": R, "cin": cin, "cout": cout,
                   "n_convs": L.n_convs, "points_per_step": B * N},
        "ms_per_layer": round(ms_per_step, 4),
        "ms_per_step_events": round(ev_ms, 4),
        "ms_per_step_graph": {"median": round(statistics.median(graph_ms), 4),
                              "min": round(min(graph_ms), 4),
                              "how": f"the forward captured {BREAKDOWN_REPS} times in one HIP "
                                     f"graph, replayed {BREAKDOWN_ROUNDS} times"},
        "roofline": roofline,
        "kernels": kernels,
        "memory": memory,
        "peaks_measured": pk,
        "inputs_sha256": wl.sha256(),
    }
    if cpu_seconds:
        cb, parity = cpu_baseline(wl, gpu_out, cpu_seconds)
        line["cpu_baseline"] = cb
        line["parity_sample"] = parity
    return line


def compact(line):
    """The summary of one workload's line kept in the headline's `workloads`."""
    ks = {n: k for n, k in line["kernels"].items() if k.get("in_forward", True)}
    dom = max(ks, key=lambda n: ks[n]["ms"])
    out = {"workload": line["config"]["workload"], "dtype": line["dtype"],
           "points_per_step": line["config"]["points_per_step"],
           "ms_per_step": line["ms_per_step"], "points_per_s": line["value"],
           "dominant": {"step": dom, "ms": ks[dom]["ms"], "achieved": ks[dom]["achieved"],
                        "unit": ks[dom]["unit"], "frac": ks[dom]["frac"]},
           "steps": {n: {"ms": k["ms"], "frac": k["frac"], "unit": k["unit"]}
                     for n, k in ks.items()},
           "memory_peak_bytes": line["memory"]["peak_bytes"]}
    if "cpu_baseline" in line:
        out["cpu_oracle"] = line["cpu_baseline"]
        out["parity_sample"] = line["parity_sample"]
    return out


def oracle_one_thread(wl, seconds):
    """The oracle on the workload's first cloud with one thread, repeated for
    at least `seconds`."""
    import oracle
    before = oracle.threads()
    oracle.set_threads(1)
    try:
        L = wl.layers[0]
        done, t_total = 0, 0.0
        while t_total < seconds:
            t0 = time.perf_counter()
            oracle.pvconv_forward(wl.coords[:1], wl.feats[:1], L)
            t_total += time.perf_counter() - t0
            done += 1
    finally:
        oracle.set_threads(before)
    return {"value": round(done * wl.N / t_total, 1), "unit": "points/s", "cores": 1,
            "kind": "oracle", "sample": f"cloud 0 ({wl.N} points) {done} times, fp64, "
                                        f"one thread, {t_total:.2f} s"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the PVConv forward here is a single-GPU "
              "build (the batch would shard by cloud across GPUs, which is not built). "
              "Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        return copy_probe(args.copy_probe)

    import torch

    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.variants:
        return bench_variants(args, dev)
    if args.backward:
        return bench_backward(args, dev)
    wl = synth.make_workload(args.workload)
    cpu_s = None if args.no_cpu_baseline else args.cpu_seconds
    if wl.is_network:
        line = bench_network(args, wl, dev, peaks=not args.no_peaks, cpu_seconds=cpu_s)
    else:
        line = bench_layer(args, wl, dev, peaks=not args.no_peaks, cpu_seconds=cpu_s)
    if "cpu_baseline" in line:
        line["cpu_baseline"]["cpu"] = cpu_model()
    if args.workload == 2 and not args.no_workloads:
        # the other workloads, each a compact summary: the same step timing
        # (W warmup, K timed steps), per-step breakdown, memory and a bounded
        # oracle sample with its parity check
        wls = {}
        for idx in (1, 3, 4, 5, 6):
            w = synth.make_workload(idx)
            ws_cpu = None if args.no_cpu_baseline else args.workload_cpu_seconds
            if w.is_network:
                one = bench_network(args, w, dev, peaks=False, cpu_seconds=ws_cpu)
            else:
                one = bench_layer(args, w, dev, cold=False, peaks=False, cpu_seconds=ws_cpu)
            summary = compact(one)
            if idx == 1 and not args.no_cpu_baseline:
                summary["cpu_oracle_one_thread"] = oracle_one_thread(w, 1.0)
            wls[str(idx)] = summary
        line["workloads"] = wls
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
