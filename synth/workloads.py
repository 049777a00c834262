"""The five cascade workloads, as plain data (shapes, thresholds, seeds).

Each names a synthetic fixed-camera video, a difference-detector setting
(Sec. 5: earlier frame or fixed reference image, global or blocked MSE,
firing threshold delta_diff) and a specialized CNN (Sec. 4: conv layers,
dense width, c_low / c_high).  Readings of unstated details are recorded in
the design notes.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

from . import CNNSpec, VideoSpec

PREV, FIXED = 0, 1
MSE, SAD, NRMSE, PSNR = 0, 1, 2, 3      # difference metric (Sec. 5 and its alternatives)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    video: VideoSpec
    dd_h: int
    dd_w: int
    cnn: CNNSpec
    ref_mode: int = PREV
    delta: int = 1
    grid: Tuple[int, int] = (1, 1)
    delta_diff: float = 15.0
    c_low: float = 0.2
    c_high: float = 0.8
    weight_seed: int = 1000
    lr_bias: float = -2.0
    chunk: Optional[int] = None
    check_stride: int = 1          # frame skipping: check frames t with t mod s = 0
    metric: int = MSE              # detector metric; PSNR reports -PSNR (larger = more different)

    def with_frames(self, n: int) -> "Workload":
        return dataclasses.replace(self, video=dataclasses.replace(self.video, n=n))

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def with_occupancy(self, occ: float) -> "Workload":
        """The same workload with another fraction of frames inside an object
        episode, named with a suffix such as "-occ50" (percent)."""
        return dataclasses.replace(self, name=f"{self.name}-occ{occ * 100:g}",
                                   video=dataclasses.replace(self.video, occupancy=occ))


def _cnn(conv, pool, dense, bf16, hw=50):
    return CNNSpec(in_h=hw, in_w=hw, conv=tuple(conv), pool=tuple(pool), dense=dense, bf16=bf16)


TINY = Workload(
    name="tiny-1k-100x100-prev1-fp32",
    video=VideoSpec(n=1000, h=100, w=100, seed=0, sigma=3.0, min_objects=1, max_objects=3,
                    obj_min=10, obj_max=25, occupancy=0.3, drift=False, vmax=2),
    dd_h=50, dd_w=50,
    cnn=_cnn((32, 32), (True, True), 32, bf16=False),
    ref_mode=PREV, delta=1, delta_diff=20.0, weight_seed=1001)

VGA = Workload(
    name="vga-100k-640x480-prev15-bf16",
    video=VideoSpec(n=100_000, h=480, w=640, seed=0, sigma=5.0, min_objects=1, max_objects=10,
                    obj_min=48, obj_max=120, occupancy=0.2, drift=True, vmax=6),
    dd_h=50, dd_w=50,
    cnn=_cnn((32, 32), (True, True), 128, bf16=True),
    ref_mode=PREV, delta=15, delta_diff=15.0, weight_seed=1002)

HD_REF = Workload(
    name="hd-100k-1280x720-fixedref-bf16",
    video=VideoSpec(n=100_000, h=720, w=1280, seed=0, sigma=5.0, min_objects=1, max_objects=10,
                    obj_min=72, obj_max=180, occupancy=0.5, drift=True, vmax=12),
    dd_h=50, dd_w=50,
    cnn=_cnn((64, 64, 64, 64), (False, True, False, True), 128, bf16=True),
    ref_mode=FIXED, delta=1, delta_diff=15.0, weight_seed=1003)

HD_BLOCKED = Workload(
    name="hd-200k-1280x720-blocked10x10-prev1-bf16",
    video=VideoSpec(n=200_000, h=720, w=1280, seed=0, sigma=5.0, min_objects=1, max_objects=10,
                    obj_min=72, obj_max=180, occupancy=0.05, drift=True, vmax=12),
    dd_h=100, dd_w=100,
    cnn=_cnn((64, 64, 64), (True, True, True), 64, bf16=True),
    ref_mode=PREV, delta=1, grid=(10, 10), delta_diff=0.0, weight_seed=1004)

FHD_STREAM = Workload(
    name="fhd-1m-1920x1080-blocked10x10-prev30-bf16-streamed",
    video=VideoSpec(n=1_000_000, h=1080, w=1920, seed=0, sigma=5.0, min_objects=1, max_objects=10,
                    obj_min=108, obj_max=270, occupancy=0.1, drift=True, vmax=19),
    dd_h=100, dd_w=100,
    cnn=_cnn((64, 64, 64, 64), (False, True, False, True), 128, bf16=True),
    ref_mode=PREV, delta=30, grid=(10, 10), delta_diff=0.0, weight_seed=1005, chunk=4096)

# the streamed workload's occupancy sweep: 1 %, 10 % (FHD_STREAM itself) and 50 %
FHD_OCCUPANCIES = (0.01, 0.1, 0.5)

ALL = [TINY, VGA, HD_REF, HD_BLOCKED, FHD_STREAM]
BY_NAME = {w.name: w for w in ALL}
