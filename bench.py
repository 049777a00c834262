#!/usr/bin/env python3
"""Cascade frames/s on one MI355X, with roofline fractions and the oracle's CPU rate.

Workload: 100,000 synthetic fixed-camera frames of 640x480 RGB uint8, already
resident in HBM; area downsample to 50x50, global MSE against frame t-15,
delta_diff = 15; specialized CNN (2 x conv3x3 32 + ReLU + max-pool, dense 128,
bf16) on the frames that fire; c_low = 0.2, c_high = 0.8.  One step is one
nsc_cascade_run over all frames (downsample, detector, compaction, CNN,
decisions and label resolution).

With --workload fhd-stream it instead runs the 1,000,000-frame 1920x1080 video
(detector 100x100, 10x10 blocked logistic score against frame t-30, 4-layer
64-channel bf16 CNN) in chunks of 4096 through two frame buffers on two
streams, the synthetic generator filling one buffer while the cascade reads the
other.  Its `value` is the cascade-only rate (each chunk's cascade timed alone
with HIP events, generator time excluded, as the paper excludes decoding); the
overlapped wall-clock rate, bound by the generator, is reported beside it.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
AREA_KERNEL = "k_area_sums_wave"
AREA_SOURCES = ("paper_1703_02529_amd/csrc/area_diff.hip", "paper_1703_02529_amd/csrc/nsc_internal.h")
COPY_BYTES = 1 << 31           # plain copy of known size for counter calibration
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t handles (the library records them on its stream)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            rc = self.hip.hipEventCreate(ctypes.byref(e))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed ({rc})")
            out.append(e.value)
        return out

    def ms(self, a, b):
        f = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(f), ctypes.c_void_p(a), ctypes.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(f.value)

    def destroy(self, evs):
        for e in evs:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))


def measured_traffic(workload: str):
    """HBM bytes per launch of the area kernel from the committed counter
    summary, or None when there is none or the kernel's sources changed since."""
    from paper_1703_02529_amd.profsum import sources_hash

    path = os.path.join(ROOT, "profiles", f"traffic_{AREA_KERNEL}_{workload}.json")
    if not os.path.exists(path):
        return None, "no counter summary"
    with open(path) as fh:
        t = json.load(fh)
    now = sources_hash([os.path.join(ROOT, p) for p in AREA_SOURCES])
    if t.get("sources_sha256_16") != now:
        return None, "kernel sources changed since the counters were taken"
    return float(t["traffic_bytes"]), os.path.relpath(path, ROOT)


def copy_calibration(torch, dev):
    """A plain copy (negation) of COPY_BYTES bytes: the reference point that
    scales the FETCH_SIZE / WRITE_SIZE counters of a profiled run."""
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(2):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()
    log(f"copy calibration: 2 x neg over {COPY_BYTES} bytes")


def cnn_flops(spec) -> int:
    layers, flat, _ = spec.shapes()
    f = sum(2 * h * w * cin * cout * 9 for cin, cout, h, w, _ in layers)
    return f + 2 * flat * spec.dense + 2 * spec.dense


def cpu_baseline(wl, budget_s: float) -> dict:
    """The oracle, single-threaded, on a contiguous window of the same video."""
    import numpy as np

    import oracle
    import synth

    v = synth.Video(wl.video)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    cfg, keep = oracle.make_cfg(wl)
    occ = v.occupied
    start = int(np.flatnonzero(occ)[0]) if occ.any() else 0
    start = max(0, start - 200)
    # probe 40 frames to size the sample to the budget
    probe = v.frames(start, start + 40)
    t = time.perf_counter()
    oracle.cascade(cfg, wl.cnn, blob, probe, t0=0)
    per = (time.perf_counter() - t) / 40
    n = int(max(100, min(4000, budget_s / max(per, 1e-6))))
    log(f"cpu baseline: oracle ~{per * 1e3:.1f} ms/frame, sampling {n} frames from {start}")
    frames = v.frames(start, start + n)
    t = time.perf_counter()
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames, t0=0)
    dt = time.perf_counter() - t
    return {"value": n / dt, "unit": "frames/s", "cores": 1, "kind": "oracle",
            "sample": f"frames [{start}, {start + n}) of the same video run as their own video "
                      f"(first {wl.delta} forced to fire); {out['fired']} fired "
                      f"({out['fired'] / n:.1%}); {dt:.1f} s single-threaded fp64; "
                      f"host has {os.cpu_count()} logical CPUs"}


def bench_stream(args):
    """The chunked 1080p million-frame run (see the module docstring)."""
    import torch

    import synth
    from paper_1703_02529_amd.streaming import StreamingCascade
    from synth import workloads as W

    wl = W.FHD_STREAM
    n, fb, chunk = wl.video.n, wl.video.frame_bytes, wl.chunk
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    v = synth.Video(wl.video)
    tables = v.device_tables(dev)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    lr = synth.lr_weights(wl.grid[0] * wl.grid[1], wl.weight_seed, wl.lr_bias)[0]
    sc = StreamingCascade(wl, blob, chunk, lr_w=torch.from_numpy(lr).to(dev), device=dev)
    label = torch.empty(n, dtype=torch.uint8, device=dev)
    defer = torch.empty(n, dtype=torch.uint8, device=dev)
    fire = torch.empty(n, dtype=torch.uint8, device=dev)

    def produce(buf, t0, m, stream):
        v.render_device(buf, t0, m, tables, stream=stream)

    log(f"workload {wl.name}: {n} frames x {fb} bytes in chunks of {chunk}")
    for _ in range(args.warmup):
        sc.run(2 * chunk, produce, label, defer, fire=fire)
    torch.cuda.synchronize()
    alone, over = [], []
    for k in range(args.steps):
        alone.append(sc.run(n, produce, label, defer, fire=fire, timing=True, overlap=False))
        log(f"pass {k}: chunks run alone: {alone[-1]}")
        over.append(sc.run(n, produce, label, defer, fire=fire, timing=True, overlap=True))
        log(f"pass {k}: overlapped: {over[-1]}")
    fired = int(fire.sum().item())
    sc.close()
    casc_ms = sum(a["cascade_ms"] for a in alone) / len(alone)
    wall_ms = sum(o["wall_ms"] for o in over) / len(over)
    result = {
        "metric": "cascade frames/sec on 1 MI355X (chunked 1080p stream)",
        "value": n / (casc_ms * 1e-3),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": casc_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8 frames, i32/i64 detector, bf16 CNN (fp32 accumulate)",
        "data": "synthetic",
        "config": {"workload": wl.name, "frames": n, "frame": f"{wl.video.w}x{wl.video.h} RGB u8",
                   "chunk": chunk, "fired": fired},
        "cascade_only_ms": casc_ms,
        "overlapped_wall_ms": wall_ms,
        "overlapped_wall_fps": n / (wall_ms * 1e-3),
        "note": "value: each chunk's cascade timed alone with HIP events (generator excluded); "
                "overlapped: generator filling the other buffer concurrently, wall clock",
    }
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (20; fhd-stream: 1)")
    ap.add_argument("--warmup", type=int, default=None, help="warm-up steps (3; fhd-stream: 1)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="oracle time budget for the CPU baseline (0 disables it)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain copy of known size (for counter calibration)")
    ap.add_argument("--workload", choices=("vga", "fhd-stream"), default="vga")
    ap.add_argument("--check-stride", type=int, default=1,
                    help="frame skipping on the 640x480 workload: check every s-th frame "
                         "(s must divide 15); 1 is the headline configuration")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the cascade's frames are independent across "
              f"streams; see the design notes for how it would shard): got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    stream = args.workload == "fhd-stream"
    if args.steps is None:
        args.steps = 1 if stream else 20
    if args.warmup is None:
        args.warmup = 1 if stream else 3
    if stream:
        bench_stream(args)
        return

    import numpy as np
    import torch

    import synth
    from paper_1703_02529_amd.runner import CascadeRunner
    from synth import workloads as W

    wl = W.VGA.replace(check_stride=args.check_stride)
    n = wl.video.n
    fb = wl.video.frame_bytes
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {wl.name}: {n} frames x {fb} bytes = {n * fb / 1e9:.1f} GB")

    v = synth.Video(wl.video)
    frames = torch.empty(n * fb, dtype=torch.uint8, device=dev)
    tables = v.device_tables(dev)
    v.render_device(frames, 0, n, tables)
    torch.cuda.synchronize()
    del tables
    log("frames rendered on the device")

    if args.calibrate_copy:
        copy_calibration(torch, dev)

    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    run = CascadeRunner(wl, blob, max_frames=n, device=dev)
    stats = run.run(frames, n, t0=0, taps=False, want_stats=True)
    log(f"untimed run: {stats}")

    hip = HipEvents()
    for _ in range(args.warmup):
        run.run(frames, n, t0=0, taps=False)
    torch.cuda.synchronize()
    evs = [hip.create(6) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        run.run(frames, n, t0=0, taps=False, stage_events=evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    log(f"timed {args.steps} steps in {wall * 1e3:.1f} ms")

    stage = np.array([[hip.ms(e[i], e[i + 1]) for i in range(5)] for e in evs])
    step_gpu = np.array([hip.ms(e[0], e[5]) for e in evs])
    for e in evs:
        hip.destroy(e)
    area_ms = float(stage[:, 0].mean())
    checked = -(-n // wl.check_stride)        # frames the detector reads
    area_bytes = checked * fb                 # algorithmic: every checked frame's bytes once
    achieved = area_bytes / (area_ms * 1e-3) / 1e9
    traffic, traffic_src = measured_traffic(wl.name)
    if wl.check_stride != 1:
        traffic, traffic_src = None, "counters were taken without frame skipping"
    cnn_ms = float(stage[:, 3].mean())
    fired = int(stats["fired"])
    cnn_tflops = fired * cnn_flops(wl.cnn) / (cnn_ms * 1e-3) / 1e12 if cnn_ms > 0 else 0.0

    result = {
        "metric": "cascade frames/sec on 1 MI355X + % HBM roofline (diff) / % MFMA peak (CNN)",
        "value": n * args.steps / wall,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8 frames, i32/i64 detector, bf16 CNN (fp32 accumulate)",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "frames": n,
            "frame": f"{wl.video.w}x{wl.video.h} RGB u8",
            "detector": f"{wl.dd_w}x{wl.dd_h} area average, global MSE vs frame t-{wl.delta}, "
                        f"delta_diff {wl.delta_diff}",
            "check_stride": wl.check_stride,
            "cnn": "2 x (conv3x3 32 + ReLU + maxpool2), dense 128, sigmoid; bf16",
            "c_low": wl.c_low,
            "c_high": wl.c_high,
            "fired": fired,
            "deferred": int(stats["deferred"]),
            "positive": int(stats["positive"]),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": AREA_KERNEL,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "traffic_source": traffic_src,
            "bytes_per_launch": area_bytes,
            "avg_launch_ms": area_ms,
        },
        "stages_ms": {
            "area_sums": area_ms,
            "detector": float(stage[:, 1].mean()),
            "compaction": float(stage[:, 2].mean()),
            "cnn": cnn_ms,
            "resolve": float(stage[:, 4].mean()),
            "step_gpu": float(step_gpu.mean()),
        },
        "cnn_mfma": {
            "achieved_tflops": cnn_tflops,
            "peak_tflops": BF16_PEAK_TFLOPS,
            "frac": cnn_tflops / BF16_PEAK_TFLOPS,
            "flop_per_survivor": cnn_flops(wl.cnn),
            "survivors": fired,
        },
    }
    del frames
    run.close()
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
