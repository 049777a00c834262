"""Host-side checks of bench.py: the one-GPU contract and the algorithmic
FLOP count per survivor that the CNN's MFMA fraction is quoted on."""
import os
import subprocess
import sys
import types

import bench
from synth import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _conv(cin, cout, h, w):
    return 2 * h * w * cin * cout * 9


def test_cnn_flops_per_survivor():
    # conv layers at their input resolution (pooling halves it for the next),
    # then dense (flat -> D) and the output unit (D -> 1)
    tiny = _conv(3, 32, 50, 50) + _conv(32, 32, 25, 25) + 2 * (12 * 12 * 32) * 32 + 2 * 32
    vga = _conv(3, 32, 50, 50) + _conv(32, 32, 25, 25) + 2 * (12 * 12 * 32) * 128 + 2 * 128
    hd4 = (_conv(3, 64, 50, 50) + _conv(64, 64, 50, 50) + _conv(64, 64, 25, 25) +
           _conv(64, 64, 25, 25) + 2 * (12 * 12 * 64) * 128 + 2 * 128)
    hd3 = (_conv(3, 64, 50, 50) + _conv(64, 64, 25, 25) + _conv(64, 64, 12, 12) +
           2 * (6 * 6 * 64) * 64 + 2 * 64)
    assert bench.cnn_flops(W.TINY.cnn) == tiny == 16_134_976
    assert bench.cnn_flops(W.VGA.cnn) == vga == 17_019_904
    assert bench.cnn_flops(W.HD_REF.cnn) == hd4 == 287_479_552
    assert bench.cnn_flops(W.HD_BLOCKED.cnn) == hd3 == 65_631_872
    assert bench.cnn_flops(W.FHD_STREAM.cnn) == hd4


def test_cpu_baseline_window_and_fields():
    """The CPU baseline leg runs the oracle on a window continued from the
    frames before it (no forced firing) and names the host CPU."""
    r = bench.cpu_baseline(W.VGA, 1.0, 0.226)
    assert r["value"] > 0 and r["cores"] == 1 and r["kind"] == "oracle"
    assert r["cpu_model"] and "continued from the area sums of the 15 frames" in r["sample"]
    r = bench.cpu_baseline(W.TINY, 0.3, 0.3)
    assert r["value"] > 0


def test_area_kernel_names_match_the_library_plan():
    """The kernel whose launches the roofline figure times: 16-byte lane
    chunks unless they leave more than a fifth of a wave idle (then 32), and
    the fused earlier-frame kernel only when the workload asks for it."""
    assert bench.lane_chunk_bytes(640, 50) == 16     # 60 of 64 lanes busy
    assert bench.lane_chunk_bytes(1280, 100) == 16   # 48 of 64
    assert bench.lane_chunk_bytes(1920, 100) == 16   # 54 of 64
    assert bench.lane_chunk_bytes(1280, 50) == 32    # 48 of 64 at 16 bytes, 60 at 32
    for wl in W.ALL:
        assert bench.area_kernel(wl) == "k_area_sums_wave", wl.name
    fused = types.SimpleNamespace(**vars(W.VGA), fuse_prev=1)  # a description asking for it
    assert bench.area_kernel(fused) == "k_area_prev_wave"
