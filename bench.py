#!/usr/bin/env python3
"""Cascade frames/s on one MI355X, with roofline fractions and the oracle's CPU rate.

Workload (default, the largest): 1,000,000 synthetic fixed-camera frames of
1920x1080 RGB uint8 in chunks of 4,096 through two frame buffers on two HIP
streams; area downsample to 100x100, 10x10 blocked logistic score against
frame t-30, delta_diff = 0; specialized CNN (4 x conv3x3 64, max-pool after
the second and fourth, dense 128, bf16) on the frames that fire; c_low = 0.2,
c_high = 0.8; 10 % of frames hold objects (--occupancy 0.01 / 0.5 give the
other two points of its occupancy sweep).  One step is one pass over the
whole video: each chunk is rendered on the device into a frame buffer, then
its nsc_cascade_run (downsample, detector, compaction, CNN, decisions and
label resolution) runs alone on the GPU and is timed with HIP events on the
cascade stream.  `value` is the cascade-only rate (generator time excluded,
as the paper excludes decoding); after the timed steps one more pass with the
generator filling the other buffer concurrently gives the overlapped
wall-clock rate, reported beside it.  The stage split comes from events at
the stage boundaries of every chunk.

--workload hd-ref / hd-blocked run the other chunked videos the same way:
  hd-ref      100,000 frames of 1280x720, MSE against a fixed median-background
              image, 4-layer 64-channel CNN (the CNN-heavy regime), chunks of 16,384;
  hd-blocked  200,000 frames of 1280x720, 10x10 blocked logistic score against
              frame t-1, 3-layer 64-channel CNN, chunks of 16,384.
--workload vga and tiny keep a whole video resident in HBM and time one
nsc_cascade_run over all its frames per step:
  vga         100,000 frames of 640x480, global MSE against frame t-15,
              delta_diff 15, 2 x conv3x3 32 + max-pool, dense 128, bf16;
  tiny        1,000 frames of 100x100 (30 MB, cache-resident and
              latency-bound), global MSE against frame t-1, delta_diff 20,
              fp32 CNN 2 x conv3x3 32, dense 32.

--workload vga-sweep measures the threshold search of the cost-based optimizer
(Sec. 6.3) on the 640x480 video: one cascade run with delta_diff = -inf logs
every frame's detector score and CNN confidence (and, from its stage events,
the per-frame costs T_MSE and T_SNN), the generator's object labels stand for
the reference network's, and nsc_threshold_sweep costs 64 candidate
thresholds at 1 % FP / FN targets; `value` is frames x candidates per second.
The cascade is then run with the chosen thresholds, and its measured time per
frame is reported beside the cost model's prediction.

--workload cameras runs a camera group (Sec. 8: batching frames of many
streams, each with its own model): 100 fixed 640x480 cameras, each with its
own video, weights and state, one second (30 frames) of every camera per
call through nsc_group_run; the same frames through one nsc_cascade_run per
camera are timed beside it (`per_camera_calls`), with their outputs checked
to be identical.

--metric sad / nrmse / psnr runs the 640x480 workload (--workload vga) with one
of the alternative detector metrics (Sec. 5), at a threshold matching MSE 15.

Every run also measures the peaks the roofline fractions are quoted against:
a streaming read of the resident frame buffer (HBM) and a loop of independent
bf16 MFMAs, next to the published 8 TB/s and 2.5 PFLOP/s.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
AREA_KERNEL = "k_area_sums_wave"


def area_kernel(wl) -> str:
    """The area kernel a workload's cascade runs: with fuse_prev set, against
    an earlier frame at least two frames back with the global MSE metric and
    16-byte lane chunks, the one with the detector fused in
    (k_area_prev_wave); otherwise k_area_sums_wave (which fuses the global
    detector against a fixed reference image)."""
    delta = wl.delta // max(1, getattr(wl, "check_stride", 1))  # in checked frames
    if getattr(wl, "fuse_prev", 0) and wl.ref_mode == 0 and delta >= 2 and \
            getattr(wl, "metric", 0) == 0 and tuple(wl.grid) == (1, 1) and \
            lane_chunk_bytes(wl.video.w, wl.dd_w) == 16:
        return "k_area_prev_wave"
    return AREA_KERNEL


def lane_chunk_bytes(w: int, wo: int) -> int:
    """Bytes one lane of the area kernel reads per source row for rows of w
    pixels (16-byte aligned) resampled to wo columns: 16, or 32 where whole
    periods of the column pattern in 16-byte chunks leave more than a fifth
    of a wave's lanes idle and 32-byte chunks fewer (the library's plan)."""
    import math
    px = w // math.gcd(w, wo)
    best_cb, best_used = 0, 0
    for cb in (16, 32):
        k = 1
        while (3 * px * k) % cb:
            k *= 2
        glanes = 3 * px * k // cb
        if glanes > 64 or w % (px * k):
            continue
        used = 64 // glanes * glanes
        if best_cb == 0 or (5 * best_used < 4 * 64 and used > best_used):
            best_cb, best_used = cb, used
    return best_cb
AREA_SOURCES = ("paper_1703_02529_amd/csrc/area_diff.hip", "paper_1703_02529_amd/csrc/nsc_internal.h")
COPY_BYTES = 1 << 31           # plain copy of known size for counter calibration
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
DTYPE_BF16 = ("u8 frames, i32/i64 detector; CNN: bf16 weights and input; fp16 activations on "
              "the fp16 matrix cores in the 64-channel and dense layers, bf16 hi/lo activation "
              "pairs in the others; fp32 accumulate")
DTYPE_FP32 = "u8 frames, i32/i64 detector; CNN: fp32 weights and activations, fp32 MFMA"
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


def measured_traffic(workload: str, kernel: str = AREA_KERNEL):
    """HBM bytes per launch of the area kernel from the committed counter
    summary, or None when there is none or the kernel's sources changed since."""
    from paper_1703_02529_amd.profsum import sources_hash

    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None, "no counter summary"
    with open(path) as fh:
        t = json.load(fh)
    now = sources_hash([os.path.join(ROOT, p) for p in AREA_SOURCES])
    if t.get("sources_sha256_16") != now:
        return None, "kernel sources changed since the counters were taken"
    return float(t["traffic_bytes"]), os.path.relpath(path, ROOT)


CNN_SOURCES = ("paper_1703_02529_amd/csrc/cnn.hip", "paper_1703_02529_amd/csrc/nsc_internal.h")
CNN_KERNELS = "k_conv,k_prep_input,k_pair64,k_band64,k_dense"


def measured_mfma_busy(workload: str):
    """Matrix-core busy fraction of the CNN stage (rocprofv3 counters: issued
    MFMA cycles over the stage's SIMD-cycles, hi / lo passes and K padding
    included) from the committed counter summary, or None when there is none
    or the kernels' sources changed since."""
    from paper_1703_02529_amd.profsum import sources_hash

    path = os.path.join(ROOT, "profiles", f"mfma_{workload}.json")
    if not os.path.exists(path):
        return None, "no counter summary"
    with open(path) as fh:
        t = json.load(fh)
    now = sources_hash([os.path.join(ROOT, p) for p in CNN_SOURCES])
    if t.get("sources_sha256_16") != now:
        return None, "kernel sources changed since the counters were taken"
    return float(t["stage_mfma_busy"]), os.path.relpath(path, ROOT)


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


def measured_peaks(torch, buf, nbytes: int) -> dict:
    """Streaming read of `nbytes` of the device buffer `buf` (HBM) and a loop of
    independent bf16 MFMAs, timed with events on torch's current stream (the
    probes are launched there): the best of three runs each."""
    import synth

    lib = ctypes.CDLL(synth.SYNTH_SO)
    lib.probe_read_launch.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_int32, ctypes.c_void_p]
    lib.probe_mfma_launch.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p]
    dev = buf.device
    out = torch.zeros(4, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream(dev)
    nbytes = nbytes // 16 * 16

    def timed(launch):
        best = None
        for rep in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            if launch() != 0:
                raise RuntimeError("probe launch failed")
            e1.record(st)
            e1.synchronize()
            if rep:
                ms = e0.elapsed_time(e1)
                best = ms if best is None else min(best, ms)
        return best

    read_ms = timed(lambda: lib.probe_read_launch(ctypes.c_void_p(buf.data_ptr()), nbytes,
                                                  ctypes.c_void_p(out.data_ptr()), 8192,
                                                  ctypes.c_void_p(st.cuda_stream)))
    iters, grid = 20000, 2048
    mfma_ms = timed(lambda: lib.probe_mfma_launch(iters, grid, ctypes.c_void_p(out.data_ptr()),
                                                  ctypes.c_void_p(st.cuda_stream)))
    flop = grid * 4 * iters * 8 * 16 * 16 * 32 * 2
    res = {"hbm_read_gbs": nbytes / (read_ms * 1e-3) / 1e9, "hbm_read_bytes": nbytes,
           "mfma_bf16_tflops": flop / (mfma_ms * 1e-3) / 1e12}
    log(f"measured peaks: {res}")
    return res


def cpu_model() -> str:
    """The host CPU's model name (first /proc/cpuinfo entry)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, budget_s: float, fire_frac: float, lr_w=None, ref_img=None,
                 n_video=None) -> dict:
    """The oracle, single-threaded, on a window of the same video whose share
    of frames with objects matches the video's, so that its detector fires on
    about as many frames as the GPU run's (fire_frac, used only to size the
    window: a fired frame costs the oracle the CNN as well).  The window is
    continued from the area sums of the frames before it (computed untimed;
    their decisions are taken as 0, which only labels inherited in the
    window's first frames), so no frame is forced to fire."""
    import numpy as np

    import oracle
    import synth

    v = synth.Video(wl.video)
    n_video = n_video or wl.video.n
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    ref_sums = oracle.area_sums(ref_img, wl.dd_h, wl.dd_w) if ref_img is not None else None
    cfg, keep = oracle.make_cfg(wl, lr_w=lr_w, ref_sums=ref_sums)
    D = oracle.history(cfg)

    def state_before(t0):
        if D == 0 or t0 == 0:
            return None
        S = np.stack([oracle.area_sums(v.frame(t), wl.dd_h, wl.dd_w).reshape(-1)
                      for t in range(t0 - D, t0)]).astype(np.int64)
        return S, np.zeros(D, np.uint8)

    def run(t0, m):
        st = state_before(t0)
        frames = v.frames(t0, t0 + m)
        t = time.perf_counter()
        out, _ = oracle.cascade(cfg, wl.cnn, blob, frames, t0=t0, state=st)
        return out, time.perf_counter() - t

    # cost of a frame that does not fire (area sums and score) and of one that
    # does (plus the CNN): frames [D, D + k) of an unoccupied stretch, then the
    # same with every frame firing (delta_diff = -inf)
    quiet = np.flatnonzero(~v.occupied[:n_video])
    t_q = int(quiet[quiet >= D][0]) if (quiet >= D).any() else D
    k = 4 if wl.video.w > 640 else 16
    o1, dt1 = run(t_q, k)
    cfg_all, keep2 = oracle.make_cfg(wl, lr_w=lr_w, ref_sums=ref_sums, delta_diff=-math.inf)
    st = state_before(t_q)
    t = time.perf_counter()
    oracle.cascade(cfg_all, wl.cnn, blob, v.frames(t_q, t_q + k), t0=t_q, state=st)
    dt_all = time.perf_counter() - t
    t_f = dt_all / k
    f1 = o1["fired"]
    t_nf = (dt1 - f1 * t_f) / (k - f1) if f1 < k else t_f
    t_nf = min(max(t_nf, 1e-6), t_f)
    per = (1 - fire_frac) * t_nf + fire_frac * t_f
    n = int(max(64, min(20000, budget_s / max(per, 1e-6))))
    n = min(n, n_video - D)
    # 8 windows of m frames, evenly spaced over the video, at the phase whose
    # share of frames with objects is closest to the video's
    n_win = 8
    m = max(8, n // n_win)
    occ = v.occupied[:n_video].astype(np.int64)
    target = occ.mean()
    csum = np.concatenate([[0], np.cumsum(occ)])
    spacing = (n_video - D - m) // n_win
    best = None
    for o in range(0, max(1, spacing), max(1, m // 4)):
        starts = D + o + spacing * np.arange(n_win)
        share = float((csum[starts + m] - csum[starts]).sum()) / (n_win * m)
        if best is None or abs(share - target) < abs(best[1] - target):
            best = (starts, share)
    starts, share = best
    log(f"cpu baseline: oracle {t_nf * 1e3:.1f} ms per quiet frame, {t_f * 1e3:.1f} ms per fired "
        f"frame; {n_win} windows of {m} frames (share with objects {share:.3f}, video "
        f"{target:.3f})")
    dt = 0.0
    fired = 0
    for s0 in starts:
        out, d = run(int(s0), m)
        dt += d
        fired += out["fired"]
    tot = n_win * m
    # the sample's time per frame, moved to the GPU run's fire fraction by the
    # oracle's own cost of a fired frame over a quiet one (probed above)
    per_frame = dt / tot + (fire_frac - fired / tot) * (t_f - t_nf)
    return {"value": 1.0 / per_frame, "unit": "frames/s", "cores": 1, "kind": "oracle",
            "sample_rate": tot / dt,
            "sample": f"{n_win} windows of {m} frames of the same video, {spacing} frames apart "
                      f"from frame {int(starts[0])}, each continued from the area sums of the {D} "
                      f"frames before it: {dt:.1f} s single-threaded fp64, {tot / dt:.1f} "
                      f"frames/s with {fired} fired ({fired / tot:.1%}; {share:.1%} of frames "
                      f"with objects, video {target:.1%}); value = 1 / (sample time per frame + "
                      f"(fire fraction of the GPU run {fire_frac:.2%} - the sample's) x (oracle "
                      f"time of a fired frame {t_f * 1e3:.1f} ms - of a quiet one "
                      f"{t_nf * 1e3:.1f} ms))",
            "cpu_model": cpu_model(), "host_logical_cpus": os.cpu_count()}


CHUNKED = ("hd-ref", "hd-blocked", "fhd-stream")
# chunks of the 1080p stream staged per batch: the CNN then sees the survivors
# of 8 x 4,096 frames together (about 1,600 at 10 % occupancy instead of 200)
DEFAULT_BATCH_CHUNKS = 8
T_FULL_NN = 1.0 / 80.0  # reference network per frame: YOLOv2 at 80 frames/s (Sec. 2)
# Detector metric -> (code, delta_diff) on the 640x480 workload: thresholds that
# match MSE 15 on the 50x50x3 = 7,500 values: -PSNR fires on the same frames
# (10 log10(15 / 255^2)); SAD on a uniform error of sqrt(15) levels (N sqrt(15),
# a subset of MSE's frames, since SAD <= N sqrt(MSE)); NRMSE on that error over
# a mid-grey compared image (sqrt(15) / 128).
METRIC_DD = {
    "mse": (0, 15.0),
    "sad": (1, 7500 * 15 ** 0.5),
    "nrmse": (2, 15 ** 0.5 / 128.0),
    "psnr": (3, 10.0 * math.log10(15.0 / 65025.0)),
}


CAMERAS = 100    # fixed cameras of the camera-group workload
CAM_BATCH = 30   # frames per camera per call: one second of 30 frames/s video


def bench_cameras(args):
    """Camera group: 100 cameras of 640x480, a second of each per call (see the
    module docstring); the same frames through one nsc_cascade_run per camera
    are timed beside it."""
    import dataclasses

    import numpy as np
    import torch

    import synth
    from paper_1703_02529_amd.runner import CascadeRunner, GroupRunner
    from synth import workloads as W

    steps, warm = args.steps, args.warmup
    calls = steps + warm
    base = W.VGA
    fb = base.video.frame_bytes
    wls = [base.replace(video=dataclasses.replace(base.video, seed=100 + c, n=calls * CAM_BATCH),
                        weight_seed=2000 + c, name=f"camera-{c}") for c in range(CAMERAS)]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    per_call = CAMERAS * CAM_BATCH * fb
    log(f"camera group: {CAMERAS} cameras x {CAM_BATCH} frames of {base.video.w}x{base.video.h} "
        f"per call, {calls} calls ({calls * per_call / 1e9:.1f} GB resident)")
    bufs = [torch.empty(per_call, dtype=torch.uint8, device=dev) for _ in range(calls)]
    for c, w in enumerate(wls):
        v = synth.Video(w.video)
        tables = v.device_tables(dev)
        for k in range(calls):
            off = c * CAM_BATCH * fb
            v.render_device(bufs[k][off:off + CAM_BATCH * fb], k * CAM_BATCH, CAM_BATCH, tables)
        del tables
    torch.cuda.synchronize()
    peaks = measured_peaks(torch, bufs[0], per_call)
    blobs = [synth.weight_blob(w.cnn, synth.cnn_weights(w.cnn, w.weight_seed)) for w in wls]
    hip = HipEvents()

    # grouped: one nsc_group_run per call
    grp = GroupRunner(wls, blobs, frames_per_cam=CAM_BATCH, device=dev)
    for k in range(warm):
        grp.run(bufs[k], CAM_BATCH, t0=k * CAM_BATCH, taps=False)
    evs = [hip.create(6) for _ in range(steps)]
    torch.cuda.synchronize()
    t = time.perf_counter()
    for i in range(steps):
        k = warm + i
        grp.run(bufs[k], CAM_BATCH, t0=k * CAM_BATCH, taps=i == steps - 1, stage_events=evs[i])
    torch.cuda.synchronize()
    wall_g = time.perf_counter() - t
    stage = np.array([[hip.ms(e[j], e[j + 1]) for j in range(5)] for e in evs])
    for e in evs:
        hip.destroy(e)
    m = CAMERAS * CAM_BATCH
    g_out = {k: getattr(grp, k)[:m].cpu().numpy().copy() for k in ("label", "defer", "fire")}
    fired = int(g_out["fire"].sum())
    log(f"grouped: {steps} calls in {wall_g * 1e3:.1f} ms; last call fired {fired} of {m}")

    # the same frames, one nsc_cascade_run per camera
    runs = [CascadeRunner(w, b, max_frames=CAM_BATCH, device=dev) for w, b in zip(wls, blobs)]

    def one_call(k, taps=False):
        for c, r in enumerate(runs):
            off = c * CAM_BATCH * fb
            r.run(bufs[k][off:off + CAM_BATCH * fb], CAM_BATCH, t0=k * CAM_BATCH, taps=taps)

    for k in range(warm):
        one_call(k)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for i in range(steps):
        one_call(warm + i, taps=i == steps - 1)
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t
    same = all(np.array_equal(np.concatenate([getattr(r, k)[:CAM_BATCH].cpu().numpy()
                                              for r in runs]), g_out[k])
               for k in ("label", "defer", "fire"))
    log(f"per camera: {steps} x {CAMERAS} calls in {wall_s * 1e3:.1f} ms; outputs identical: {same}")
    for r in runs:
        r.close()
    grp.close()

    area_ms = float(stage[:, 0].mean())
    achieved = per_call / (area_ms * 1e-3) / 1e9
    result = {
        "metric": "cascade frames/sec on 1 MI355X, 100 camera streams batched per call",
        "value": m * steps / wall_g,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warm,
        "ms_per_step": wall_g * 1e3 / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_BF16,
        "data": "synthetic",
        "config": {
            "workload": f"cameras-{CAMERAS}x{CAM_BATCH}-640x480-prev15-bf16",
            "cameras": CAMERAS,
            "frames_per_camera_per_call": CAM_BATCH,
            "frame": f"{base.video.w}x{base.video.h} RGB u8",
            "detector": "50x50 area average, global MSE vs frame t-15, delta_diff 15, per camera",
            "cnn": "2 x (conv3x3 32 + ReLU + maxpool2), dense 128, sigmoid; bf16; own weights "
                   "per camera",
            "fired_last_call": fired,
        },
        "per_camera_calls": {
            "value": m * steps / wall_s,
            "ms_per_step": wall_s * 1e3 / steps,
            "calls_per_step": CAMERAS,
            "outputs_identical": bool(same),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": AREA_KERNEL,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": None,
            "traffic_source": "counters were taken on the single-video workload",
            "bytes_per_launch": per_call,
            "avg_launch_ms": area_ms,
            "measured_peak": peaks["hbm_read_gbs"],
            "frac_of_measured": achieved / peaks["hbm_read_gbs"],
        },
        "stages_ms": {
            "area_sums": area_ms,
            "detector": float(stage[:, 1].mean()),
            "compaction": float(stage[:, 2].mean()),
            "cnn": float(stage[:, 3].mean()),
            "resolve_state": float(stage[:, 4].mean()),
        },
        "cpu_baseline": None,
    }
    del bufs
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        # camera 0's video, long enough for the sample
        w0 = wls[0].replace(video=dataclasses.replace(wls[0].video, n=base.video.n))
        result["cpu_baseline"] = cpu_baseline(w0, args.cpu_seconds, fired / m)
    print(json.dumps(result), flush=True)


def bench_sweep(args):
    """Threshold search on the 640x480 video (see the module docstring)."""
    import math

    import numpy as np
    import torch

    import paper_1703_02529_amd as nsc
    import synth
    from paper_1703_02529_amd.runner import CascadeRunner
    from synth import workloads as W

    wl = W.VGA
    n, fb = wl.video.n, wl.video.frame_bytes
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    v = synth.Video(wl.video)
    frames = torch.empty(n * fb, dtype=torch.uint8, device=dev)
    v.render_device(frames, 0, n, v.device_tables(dev))
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    hip = HipEvents()
    # 1. every frame through the detector and the CNN: the logged scores
    run = CascadeRunner(wl.replace(delta_diff=-math.inf), blob, max_frames=n, device=dev)
    run.run(frames, n, t0=0)
    evs = hip.create(6)
    run.run(frames, n, t0=0, stage_events=evs)
    torch.cuda.synchronize()
    st = [hip.ms(evs[i], evs[i + 1]) for i in range(5)]
    hip.destroy(evs)
    t_mse = (st[0] + st[1] + st[2]) * 1e-3 / n
    t_snn = st[3] * 1e-3 / n
    score = run.score[:n].clone()
    conf = torch.sigmoid(run.logit[:n].double()).float()
    run.close()
    truth = torch.from_numpy(v.occupied.astype(np.uint8)).to(dev)
    finite = score[torch.isfinite(score)]
    n_t = 64
    deltas = torch.quantile(finite[:: max(1, finite.numel() // 16384)].double(),
                            torch.linspace(0, 1, n_t - 1, dtype=torch.float64, device=dev))
    deltas = torch.cat([torch.tensor([-math.inf], dtype=torch.float64, device=dev), deltas])
    cfg = nsc.SweepCfg(wl.ref_mode, wl.delta, 0.01, 0.01, t_mse, t_snn, T_FULL_NN)
    rows = torch.zeros(n_t * nsc.SWEEP_ROW_BYTES, dtype=torch.uint8, device=dev)
    best = torch.zeros(1, dtype=torch.int32, device=dev)
    log(f"sweep: {n} frames x {n_t} candidates; T_MSE {t_mse * 1e9:.1f} ns, "
        f"T_SNN {t_snn * 1e9:.1f} ns per frame")
    # 2. timed searches
    for _ in range(args.warmup):
        nsc.nsc_threshold_sweep(cfg, score, conf, truth, deltas, rows, best)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        nsc.nsc_threshold_sweep(cfg, score, conf, truth, deltas, rows, best)
    e1.record()
    torch.cuda.synchronize()
    sweep_ms = e0.elapsed_time(e1) / args.steps
    bi = int(best.item())
    row_bytes = rows.cpu().numpy()
    fields = ("delta", "c_low", "c_high", "f_m", "f_c", "cost")
    r = {}
    if bi >= 0:
        rec = row_bytes[bi * nsc.SWEEP_ROW_BYTES:(bi + 1) * nsc.SWEEP_ROW_BYTES]
        r = dict(zip(fields, np.frombuffer(rec[:48].tobytes(), np.float64).tolist()))
        ints = np.frombuffer(rec[48:112].tobytes(), np.int64).tolist()
        r.update(zip(("fired", "deferred", "fn_dd", "fp_dd", "fn_cnn", "fp_cnn", "positives",
                      "negatives"), ints))
    # 3. the chosen cascade, measured against the cost model
    check = None
    if bi >= 0:
        chosen = wl.replace(delta_diff=r["delta"], c_low=r["c_low"], c_high=r["c_high"])
        run = CascadeRunner(chosen, blob, max_frames=n, device=dev)
        run.run(frames, n, t0=0, taps=False)
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(5):
            run.run(frames, n, t0=0, taps=False)
        c1.record()
        torch.cuda.synchronize()
        st2 = run.run(frames, n, t0=0, taps=False, want_stats=True)
        run.close()
        measured = c0.elapsed_time(c1) * 1e-3 / 5 / n
        predicted = t_mse + r["f_m"] * t_snn
        check = {"predicted_s_per_frame": predicted, "measured_s_per_frame": measured,
                 "ratio": measured / predicted, "fired_measured": int(st2["fired"]),
                 "fired_predicted": int(r["fired"]),
                 "note": "cost model without the reference network term (it is not run)"}
    del frames
    torch.cuda.empty_cache()
    result = {
        "metric": "threshold search: frames x candidate thresholds per second on 1 MI355X",
        "value": n * n_t / (sweep_ms * 1e-3),
        "unit": "frame-candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sweep_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64 scores and costs, f32 confidences, integer counts",
        "data": "synthetic",
        "config": {"workload": "vga-100k-640x480-prev15-bf16 threshold search", "frames": n,
                   "candidates": n_t, "fp_target": 0.01, "fn_target": 0.01,
                   "t_mse_s": t_mse, "t_snn_s": t_snn, "t_full_s": T_FULL_NN},
        "best": r,
        "cost_model_check": check,
    }
    if args.cpu_seconds > 0:
        import oracle

        sc, cf, tr = score.cpu().numpy(), conf.cpu().numpy(), truth.cpu().numpy()
        dl = deltas.cpu().numpy()
        t = time.perf_counter()
        oracle.threshold_sweep(sc, cf, tr, dl, ref_mode=wl.ref_mode, delta=wl.delta,
                               fp_target=0.01, fn_target=0.01, t_mse=t_mse, t_snn=t_snn,
                               t_full=T_FULL_NN)
        dt = time.perf_counter() - t
        result["cpu_baseline"] = {"value": n * n_t / dt, "unit": "frame-candidates/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"the same {n} frames x {n_t} candidates, "
                                            f"{dt:.2f} s single-threaded"}
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)



def bench_chunked(args):
    """A larger video in chunks through two frame buffers (see the module docstring)."""
    import numpy as np
    import torch

    import paper_1703_02529_amd as nsc
    import synth
    from paper_1703_02529_amd.streaming import StreamingCascade
    from synth import workloads as W

    wl = {"hd-ref": W.HD_REF, "hd-blocked": W.HD_BLOCKED, "fhd-stream": W.FHD_STREAM}[args.workload]
    if args.occupancy is not None and args.occupancy != wl.video.occupancy:
        wl = wl.with_occupancy(args.occupancy)
    chunk = args.chunk or wl.chunk or 16384
    batch_chunks = args.batch_chunks if args.batch_chunks is not None else (
        DEFAULT_BATCH_CHUNKS if args.workload == "fhd-stream" else 1)
    n, fb = wl.video.n, wl.video.frame_bytes
    if args.frames is not None:
        if not 0 < args.frames <= n:
            raise SystemExit(f"--frames must lie in 1..{n}")
        n = args.frames
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    v = synth.Video(wl.video)
    tables = v.device_tables(dev)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    lr = lr_d = None
    if wl.grid != (1, 1):
        lr = synth.lr_weights(wl.grid[0] * wl.grid[1], wl.weight_seed, wl.lr_bias)[0]
        lr_d = torch.from_numpy(lr).to(dev)
    ref_img = ref_d = None
    if wl.ref_mode == W.FIXED:
        # the median-background reference image (untimed setup): frames 0, 10, ..., 1000
        # rendered on the device, per-pixel median (odd count: the middle value)
        ts = list(range(0, 1001, 10))
        stack = torch.empty(len(ts), fb, dtype=torch.uint8, device=dev)
        for i, t in enumerate(ts):
            v.render_device(stack[i], t, 1, tables)
        med = stack.view(len(ts), -1).to(torch.int16).median(dim=0).values.to(torch.uint8)
        del stack
        ref_img = med.cpu().numpy().reshape(wl.video.h, wl.video.w, 3)
        ref_d = torch.empty(wl.dd_h * wl.dd_w * 3, dtype=torch.int32, device=dev)
        nsc.nsc_downsample(med, 1, wl.video.h, wl.video.w, wl.dd_h, wl.dd_w, ref_d)
    sc = StreamingCascade(wl, blob, chunk, lr_w=lr_d, ref_sums=ref_d, device=dev,
                          batch_chunks=batch_chunks)
    label = torch.empty(n, dtype=torch.uint8, device=dev)
    defer = torch.empty(n, dtype=torch.uint8, device=dev)
    fire = torch.empty(n, dtype=torch.uint8, device=dev)

    def produce(buf, t0, m, stream):
        v.render_device(buf, t0, m, tables, stream=stream)

    log(f"workload {wl.name}: {n} frames x {fb} bytes in chunks of {chunk}, "
        f"{batch_chunks} chunk(s) per batch")
    if args.calibrate_copy:
        copy_calibration(torch, dev)
    peaks = measured_peaks(torch, sc.bufs[0], chunk * fb)
    # a step: frames [0, n) in chunks, each chunk's cascade alone on the GPU
    # (its fill waits for the previous cascade), timed with events per chunk
    for _ in range(args.warmup):
        sc.run(n, produce, label, defer, fire=fire, overlap=False)
    torch.cuda.synchronize()
    hip = HipEvents()
    n_chunks = -(-n // chunk)
    n_batches = -(-n_chunks // batch_chunks)
    evs = [hip.create(6) for _ in range(n_batches)]
    alone, stage_tot = [], np.zeros(5)
    torch.cuda.synchronize()
    t_steps = time.perf_counter()
    for k in range(args.steps):
        alone.append(sc.run(n, produce, label, defer, fire=fire, timing=True, overlap=False,
                            stage_events=lambda j: evs[j]))
        split = np.array([[hip.ms(e[i], e[i + 1]) for i in range(5)] for e in evs]).sum(0)
        if batch_chunks > 1:
            split[0] = alone[-1]["stage_ms"]   # the chunks' area stages
        stage_tot += split
        log(f"step {k}: {alone[-1]}")
    torch.cuda.synchronize()
    steps_wall = time.perf_counter() - t_steps
    # the generator filling the other buffer while the cascade runs: wall clock of one pass
    over = None
    if not args.no_overlapped_pass:
        over = sc.run(n, produce, label, defer, fire=fire, timing=True, overlap=True)
        log(f"overlapped pass: {over}")
    for e in evs:
        hip.destroy(e)
    fired = int(fire[:n].sum().item())
    sc.close()
    stage = stage_tot / args.steps
    casc_ms = sum(a["cascade_ms"] for a in alone) / len(alone)
    wall_ms = over["wall_ms"] if over else None
    area_ms, cnn_ms = float(stage[0]), float(stage[3])
    achieved = n * fb / (area_ms * 1e-3) / 1e9
    diff_ms = float(stage[0] + stage[1] + stage[2])
    diff_gbs = (n * fb + n) / (diff_ms * 1e-3) / 1e9
    cnn_tflops = fired * cnn_flops(wl.cnn) / (cnn_ms * 1e-3) / 1e12 if cnn_ms > 0 else 0.0
    busy, busy_src = measured_mfma_busy(wl.name)
    # HBM bytes per area launch (the mean over the chunks, as avg_launch_ms);
    # the area kernel does not depend on the occupancy
    base = {"hd-ref": W.HD_REF, "hd-blocked": W.HD_BLOCKED, "fhd-stream": W.FHD_STREAM}[args.workload]
    kern = area_kernel(wl)
    traffic, traffic_src = measured_traffic(base.name, kern)
    if args.frames is not None and traffic is not None:
        traffic_src += " (counters of the whole video)"
    layers = ", ".join(f"{c}{'+pool' if p else ''}" for c, p in zip(wl.cnn.conv, wl.cnn.pool))
    result = {
        "metric": "cascade frames/sec on 1 MI355X + % HBM roofline (diff) / % MFMA peak (CNN)",
        "value": n / (casc_ms * 1e-3),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": casc_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_BF16,
        "data": "synthetic",
        "config": {"workload": wl.name + ("" if n == wl.video.n else f"-first{n}") +
                               ("" if chunk == (wl.chunk or 16384) else f"-chunk{chunk}"),
                   "frames": n, "frame": f"{wl.video.w}x{wl.video.h} RGB u8",
                   "chunk": chunk, "chunks": n_chunks, "batch_chunks": batch_chunks,
                   "occupancy": wl.video.occupancy,
                   "detector": f"{wl.dd_w}x{wl.dd_h}, " + (
                       "fixed median-background reference" if wl.ref_mode == W.FIXED else
                       f"frame t-{wl.delta}") + (
                       f", {wl.grid[0]}x{wl.grid[1]} blocked logistic score" if wl.grid != (1, 1)
                       else ", global MSE") + f", delta_diff {wl.delta_diff}",
                   "cnn": f"conv3x3 [{layers}], dense {wl.cnn.dense}, sigmoid; bf16",
                   "c_low": wl.c_low, "c_high": wl.c_high, "fired": fired,
                   "step": "one pass over all frames; each chunk rendered into one of two "
                           "frame buffers, then its cascade timed alone (HIP events on the "
                           "cascade stream); ms_per_step is the cascade time of a pass" + (
                               f"; with batches: each chunk's area sums staged, then detector, "
                               f"compaction, CNN and labels once per {batch_chunks} chunks "
                               f"({batch_chunks * chunk} frames: the added label latency)"
                               if batch_chunks > 1 else "")},
        "roofline": {
            "bound": "hbm",
            "kernel": kern,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "traffic_source": traffic_src,
            "bytes_per_launch": n * fb / n_chunks,
            "avg_launch_ms": area_ms / n_chunks,
            "measured_peak": peaks["hbm_read_gbs"],
            "frac_of_measured": achieved / peaks["hbm_read_gbs"],
        },
        "diff_compaction_stage": {
            "what": "area sums + detector + compaction (stages 1-3): raw frame bytes and fire "
                    "flags over the stages' summed time",
            "achieved": diff_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": diff_gbs / HBM_PEAK_GBS, "ms_per_step": diff_ms},
        "stages_ms": {"area_sums": area_ms, "detector": float(stage[1]),
                      "compaction": float(stage[2]), "cnn": cnn_ms, "resolve": float(stage[4])},
        "cnn_mfma": {"achieved_tflops": cnn_tflops, "peak_tflops": BF16_PEAK_TFLOPS,
                     "frac": cnn_tflops / BF16_PEAK_TFLOPS,
                     "measured_peak_tflops": peaks["mfma_bf16_tflops"],
                     "frac_of_measured": cnn_tflops / peaks["mfma_bf16_tflops"],
                     "flop_per_survivor": cnn_flops(wl.cnn), "survivors": fired,
                     "busy_counter": busy, "busy_source": busy_src},
        "cascade_only_ms": casc_ms,
        "overlapped_wall_ms": wall_ms,
        "overlapped_wall_fps": n / (wall_ms * 1e-3) if wall_ms else None,
        "steps_wall_s": steps_wall,
        "note": "value: each chunk's cascade timed alone with HIP events (generator excluded, as "
                "the paper excludes decoding); overlapped: one more pass with the generator "
                "filling the other buffer concurrently, wall clock",
    }
    torch.cuda.empty_cache()
    result["cpu_baseline"] = (cpu_baseline(wl, args.cpu_seconds, fired / n, lr_w=lr,
                                           ref_img=ref_img, n_video=n)
                              if args.cpu_seconds > 0 else None)
    print(json.dumps(result), flush=True)


def bench_resident(args):
    """A video resident in HBM, one nsc_cascade_run over all its frames per
    step: the 640x480 workload (vga) or the 1,000-frame 100x100 one (tiny)."""
    import numpy as np
    import torch

    import synth
    from paper_1703_02529_amd.runner import CascadeRunner
    from synth import workloads as W

    tiny = args.workload == "tiny"
    base = W.TINY if tiny else W.VGA
    wl = base.replace(check_stride=args.check_stride)
    if args.metric != "mse":
        code, dd = METRIC_DD[args.metric]
        wl = wl.replace(metric=code, delta_diff=dd, name=f"{wl.name}-{args.metric}")
    n = wl.video.n
    fb = wl.video.frame_bytes
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {wl.name}: {n} frames x {fb} bytes = {n * fb / 1e9:.2f} GB")

    v = synth.Video(wl.video)
    frames = torch.empty(n * fb, dtype=torch.uint8, device=dev)
    tables = v.device_tables(dev)
    v.render_device(frames, 0, n, tables)
    torch.cuda.synchronize()
    del tables
    log("frames rendered on the device")

    if args.calibrate_copy:
        copy_calibration(torch, dev)
    peaks = measured_peaks(torch, frames, n * fb)

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
    diff_ms = float(stage[:, 0:3].sum(1).mean())
    diff_gbs = (area_bytes + checked) / (diff_ms * 1e-3) / 1e9
    kern = area_kernel(wl)
    traffic, traffic_src = measured_traffic(base.name, kern)  # counters of the MSE run
    if kern != area_kernel(base):
        traffic, traffic_src = None, f"counters were taken of {area_kernel(base)}"
    if wl.check_stride != 1:
        traffic, traffic_src = None, "counters were taken without frame skipping"
    cnn_ms = float(stage[:, 3].mean())
    fired = int(stats["fired"])
    flop = cnn_flops(wl.cnn)
    cnn_tflops = fired * flop / (cnn_ms * 1e-3) / 1e12 if cnn_ms > 0 else 0.0
    busy, busy_src = measured_mfma_busy(base.name)  # the network does not depend on the metric
    peak_tf = BF16_PEAK_TFLOPS if wl.cnn.bf16 else FP32_PEAK_TFLOPS
    layers = ", ".join(f"{c}{'+pool' if p else ''}" for c, p in zip(wl.cnn.conv, wl.cnn.pool))

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
        "dtype": DTYPE_BF16 if wl.cnn.bf16 else DTYPE_FP32,
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "frames": n,
            "frame": f"{wl.video.w}x{wl.video.h} RGB u8",
            "detector": f"{wl.dd_w}x{wl.dd_h} area average, global "
                        f"{'-PSNR' if args.metric == 'psnr' else args.metric.upper()} vs frame "
                        f"t-{wl.delta}, delta_diff {wl.delta_diff:.6g}",
            "check_stride": wl.check_stride,
            "cnn": f"conv3x3 [{layers}], dense {wl.cnn.dense}, sigmoid; "
                   f"{'bf16' if wl.cnn.bf16 else 'fp32'}",
            "c_low": wl.c_low,
            "c_high": wl.c_high,
            "fired": fired,
            "deferred": int(stats["deferred"]),
            "positive": int(stats["positive"]),
            "step": "one nsc_cascade_run over all frames, resident in HBM",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": kern,
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "traffic_source": traffic_src,
            "bytes_per_launch": area_bytes,
            "avg_launch_ms": area_ms,
            "measured_peak": peaks["hbm_read_gbs"],
            "frac_of_measured": achieved / peaks["hbm_read_gbs"],
        },
        "diff_compaction_stage": {
            "what": "area sums + detector + compaction (stages 1-3): raw frame bytes and fire "
                    "flags over the stages' summed time",
            "achieved": diff_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": diff_gbs / HBM_PEAK_GBS, "ms_per_step": diff_ms},
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
            "peak_tflops": peak_tf,
            "frac": cnn_tflops / peak_tf,
            "measured_peak_tflops": peaks["mfma_bf16_tflops"] if wl.cnn.bf16 else None,
            "frac_of_measured": cnn_tflops / peaks["mfma_bf16_tflops"] if wl.cnn.bf16 else None,
            "flop_per_survivor": flop,
            "survivors": fired,
            "busy_counter": busy,
            "busy_source": busy_src,
        },
    }
    if tiny:
        result["roofline"]["note"] = (
            f"{n * fb / 1e6:.0f} MB of frames fit in the 256 MB MALL: the step is latency-bound "
            "(a few microseconds per launch), so its HBM fraction is not a meaningful roofline")
    del frames
    run.close()
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, fired / n)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (resident workloads 20; chunked 10)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="warm-up steps (resident 3; chunked 2)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="oracle time budget for the CPU baseline (0 disables it)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain copy of known size (for counter calibration)")
    ap.add_argument("--workload", choices=("tiny", "vga", "vga-sweep", "cameras") + CHUNKED,
                    default="fhd-stream")
    ap.add_argument("--frames", type=int, default=None,
                    help="chunked workloads: run only the first N frames of the video (for "
                         "profiling runs; the benchmark line runs all of them)")
    ap.add_argument("--no-overlapped-pass", action="store_true",
                    help="chunked workloads: skip the pass with the generator overlapped (for "
                         "profiling runs whose kernel statistics should hold the timed passes only)")
    ap.add_argument("--chunk", type=int, default=None,
                    help="chunked workloads: frames per chunk (default: the workload's own, "
                         "4,096 for the 1080p stream and 16,384 for the 720p videos)")
    ap.add_argument("--batch-chunks", type=int, default=None,
                    help="chunked workloads: chunks staged per batch before the detector, "
                         "CNN and labels run over them together (default: "
                         f"{DEFAULT_BATCH_CHUNKS} for the 1080p stream, 1 otherwise)")
    ap.add_argument("--metric", choices=tuple(METRIC_DD), default="mse",
                    help="detector metric on the 640x480 workload (Sec. 5 and the alternatives "
                         "it names), at the threshold matching MSE 15 (see METRIC_DD)")
    ap.add_argument("--occupancy", type=float, default=None,
                    help="fraction of frames with objects for the chunked workloads (the "
                         "1920x1080 stream is measured at 0.01, 0.1 and 0.5; default: the "
                         "workload's own)")
    ap.add_argument("--check-stride", type=int, default=1,
                    help="frame skipping on the 640x480 workload: check every s-th frame "
                         "(s must divide 15); 1 is the headline configuration")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the cascade's frames are independent across "
              f"streams; see the design notes for how it would shard): got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    if args.workload == "cameras":
        if args.steps is None:
            args.steps = 20
        if args.warmup is None:
            args.warmup = 2
        bench_cameras(args)
        return
    if args.workload == "vga-sweep":
        if args.steps is None:
            args.steps = 20
        if args.warmup is None:
            args.warmup = 2
        bench_sweep(args)
        return
    chunked = args.workload in CHUNKED
    if args.metric != "mse" and args.workload not in ("vga", "tiny"):
        raise SystemExit("--metric applies to the resident workloads (--workload vga or tiny)")
    if args.steps is None:
        args.steps = 10 if chunked else 20
    if args.warmup is None:
        args.warmup = 2 if chunked else 3
    if chunked:
        bench_chunked(args)
    else:
        bench_resident(args)


if __name__ == "__main__":
    main()
