"""Seeded synthetic fixed-camera video, model parameters and workload table.

This module is input infrastructure shared by the oracle side and the HIP side.
It draws pixels, rectangles and weights; it holds none of the cascade's
arithmetic (no resampling, no difference metric, no network evaluation).

Video model (fixed camera, Sec. 8 notes the restriction to static cameras):
    pixel(t, y, x, c) = clamp(base(t, y, x, c) + drift[t] + noise(t, y, x, c), 0, 255)
    base  = colour of the last active rectangle covering (x, y), else bg[y, x, c]
    noise = T[(h >> 16c) & 0xFFFF],  h = splitmix64(key + (pix + 1) * GOLDEN)
with pix = (t*H + y)*W + x.  The mixing function is the SplitMix64 finaliser
(Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014, using Stafford's "Mix13" constants).  T is a 65,536-entry table of
rounded Gaussian quantiles.  All tables are built here on the host, in fp64,
once; the per-pixel rule is integer-only, so the host rendering below and the
device rendering in ``synth_kernel.hip`` are bit-identical.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
from typing import Optional

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
KEYMUL = 0xD1B54A32D192ED03
RECT_FIELDS = 8  # x0, y0, x1, y1 (half-open), r, g, b, active

_U64 = np.uint64


@dataclasses.dataclass(frozen=True)
class VideoSpec:
    n: int
    h: int
    w: int
    seed: int = 0
    sigma: float = 5.0
    min_objects: int = 1
    max_objects: int = 10
    obj_min: int = 48          # rectangle side range, pixels
    obj_max: int = 120
    occupancy: float = 0.2     # fraction of frames inside an object episode
    drift: bool = True         # slow illumination drift round(2 sin(2 pi t / 20000))
    vmax: int = 6              # max |velocity| per axis, pixels per frame

    @property
    def frame_bytes(self) -> int:
        return self.h * self.w * 3


def splitmix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 array (wrapping arithmetic)."""
    z = z.astype(_U64, copy=True)
    z ^= z >> _U64(30)
    z *= _U64(MIX1)
    z ^= z >> _U64(27)
    z *= _U64(MIX2)
    z ^= z >> _U64(31)
    return z


def _key(seed: int) -> int:
    return (seed * KEYMUL + 0x5851F42D4C957F2D) & 0xFFFFFFFFFFFFFFFF


def gaussian_table(sigma: float) -> np.ndarray:
    """T[u] = round(sigma * Phi^-1((u + 0.5) / 65536)) as int16."""
    from scipy.special import ndtri
    u = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
    return np.rint(sigma * ndtri(u)).astype(np.int16)


def background(spec: VideoSpec) -> np.ndarray:
    """Static smooth background: coarse uniform [64, 192] grid, bilinear upsample."""
    rng = np.random.default_rng([spec.seed, 11])
    gh = max(2, spec.h // 40 + 2)
    gw = max(2, spec.w // 40 + 2)
    coarse = rng.integers(64, 193, size=(gh, gw, 3)).astype(np.float64)
    ys = np.linspace(0.0, gh - 1.0, spec.h)
    xs = np.linspace(0.0, gw - 1.0, spec.w)
    y0 = np.minimum(np.floor(ys).astype(int), gh - 2)
    x0 = np.minimum(np.floor(xs).astype(int), gw - 2)
    fy = (ys - y0)[:, None, None]
    fx = (xs - x0)[None, :, None]
    c00 = coarse[y0][:, x0]
    c01 = coarse[y0][:, x0 + 1]
    c10 = coarse[y0 + 1][:, x0]
    c11 = coarse[y0 + 1][:, x0 + 1]
    img = (1 - fy) * ((1 - fx) * c00 + fx * c01) + fy * ((1 - fx) * c10 + fx * c11)
    return np.clip(np.rint(img), 0, 255).astype(np.uint8)


def drift_table(spec: VideoSpec) -> np.ndarray:
    if not spec.drift:
        return np.zeros(spec.n, np.int8)
    t = np.arange(spec.n, dtype=np.float64)
    return np.rint(2.0 * np.sin(2.0 * math.pi * t / 20000.0)).astype(np.int8)


def _reflect(p0: int, v: int, steps: np.ndarray, span: int) -> np.ndarray:
    """Positions of a point bouncing in [0, span] with integer velocity v."""
    if span <= 0:
        return np.zeros_like(steps)
    period = 2 * span
    q = np.mod(p0 + v * steps, period)
    return np.where(q <= span, q, period - q)


def rect_table(spec: VideoSpec) -> np.ndarray:
    """int32 [n, K, 8]: per-frame rectangles of the object episodes."""
    n, K = spec.n, spec.max_objects
    rects = np.zeros((n, max(K, 1), RECT_FIELDS), np.int32)
    occ = spec.occupancy
    if occ <= 0.0 or K == 0:
        return rects
    rng = np.random.default_rng([spec.seed, 23])
    t = 0
    on = occ >= 1.0
    lo = max(1, min(spec.obj_min, spec.w, spec.h))
    hi_w = max(lo, min(spec.obj_max, spec.w))
    hi_h = max(lo, min(spec.obj_max, spec.h))
    while t < n:
        if not on:
            t += int(round(rng.uniform(30, 300) * (1.0 - occ) / occ))
            on = True
            continue
        length = int(rng.integers(30, 301))
        k = int(rng.integers(spec.min_objects, K + 1))
        steps = np.arange(min(length, n - t), dtype=np.int64)
        for j in range(k):
            ow = int(rng.integers(lo, hi_w + 1))
            oh = int(rng.integers(lo, hi_h + 1))
            x0 = int(rng.integers(0, spec.w - ow + 1))
            y0 = int(rng.integers(0, spec.h - oh + 1))
            vx = int(rng.integers(1, spec.vmax + 1)) * int(rng.choice([-1, 1]))
            vy = int(rng.integers(1, spec.vmax + 1)) * int(rng.choice([-1, 1]))
            col = rng.integers(0, 256, size=3)
            xs = _reflect(x0, vx, steps, spec.w - ow)
            ys = _reflect(y0, vy, steps, spec.h - oh)
            sl = rects[t:t + len(steps), j]
            sl[:, 0] = xs
            sl[:, 1] = ys
            sl[:, 2] = xs + ow
            sl[:, 3] = ys + oh
            sl[:, 4:7] = col
            sl[:, 7] = 1
        t += length
        on = occ >= 1.0
    return rects


class Video:
    """Host-side tables of one synthetic video and a host renderer."""

    def __init__(self, spec: VideoSpec):
        self.spec = spec
        self.bg = background(spec)
        self.noise = gaussian_table(spec.sigma)
        self.drift = drift_table(spec)
        self.rects = rect_table(spec)
        self.key = _key(spec.seed)

    @property
    def occupied(self) -> np.ndarray:
        """Ground-truth presence of any object per frame."""
        return self.rects[:, :, 7].any(axis=1)

    def frame(self, t: int) -> np.ndarray:
        s = self.spec
        if not 0 <= t < s.n:
            raise IndexError(t)
        base = self.bg.astype(np.int32)
        for r in self.rects[t]:
            if r[7]:
                base[r[1]:r[3], r[0]:r[2], :] = r[4:7]
        pix = _U64(t * s.h * s.w) + np.arange(s.h * s.w, dtype=_U64)
        h = splitmix64(_U64(self.key) + (pix + _U64(1)) * _U64(GOLDEN))
        noise = np.stack([self.noise[((h >> _U64(16 * c)) & _U64(0xFFFF)).astype(np.int64)]
                          for c in range(3)], axis=-1).reshape(s.h, s.w, 3)
        v = base + int(self.drift[t]) + noise.astype(np.int32)
        return np.clip(v, 0, 255).astype(np.uint8)

    def frames(self, t0: int, t1: int) -> np.ndarray:
        return np.stack([self.frame(t) for t in range(t0, t1)]) if t1 > t0 else \
            np.zeros((0, self.spec.h, self.spec.w, 3), np.uint8)

    def median_background(self, t_end: int = 1000, step: int = 10) -> np.ndarray:
        """Per-pixel, per-channel median of frames 0, step, ..., t_end (odd count)."""
        ts = list(range(0, min(t_end, self.spec.n - 1) + 1, step))
        if len(ts) % 2 == 0:
            ts = ts[:-1]
        stack = self.frames_at(ts)
        return np.median(stack, axis=0).astype(np.uint8)

    def frames_at(self, ts) -> np.ndarray:
        return np.stack([self.frame(int(t)) for t in ts])

    # device rendering -----------------------------------------------------
    def device_tables(self, device="cuda"):
        import torch
        return dict(
            bg=torch.from_numpy(self.bg.copy()).to(device),
            noise=torch.from_numpy(self.noise.copy()).to(device),
            drift=torch.from_numpy(self.drift.copy()).to(device),
            rects=torch.from_numpy(self.rects.copy()).to(device),
        )

    def render_device(self, out, t0: int, n: int, tables=None, stream=None):
        """Render frames [t0, t0+n) into a uint8 CUDA tensor viewed as [n, H, W, 3]."""
        import torch
        s = self.spec
        if tables is None:
            tables = self.device_tables(out.device)
        if out.dtype != torch.uint8 or not out.is_contiguous() or out.numel() < n * s.frame_bytes:
            raise ValueError("out must be a contiguous uint8 tensor of n frames")
        if t0 < 0 or t0 + n > s.n:
            raise ValueError("frame range outside the video")
        lib = _device_lib()
        st = stream if stream is not None else torch.cuda.current_stream(out.device)
        rc = lib.synth_render(
            ctypes.c_void_p(out.data_ptr()), ctypes.c_int64(t0), ctypes.c_int64(n),
            ctypes.c_int32(s.h), ctypes.c_int32(s.w), ctypes.c_uint64(self.key),
            ctypes.c_void_p(tables["bg"].data_ptr()), ctypes.c_void_p(tables["noise"].data_ptr()),
            ctypes.c_void_p(tables["drift"].data_ptr()), ctypes.c_void_p(tables["rects"].data_ptr()),
            ctypes.c_int32(self.rects.shape[1]), ctypes.c_void_p(st.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"synth_render failed with HIP error {rc}")


_LIB: Optional[ctypes.CDLL] = None
SYNTH_SO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth.so")


def _device_lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(SYNTH_SO):
            raise RuntimeError(f"{SYNTH_SO} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(SYNTH_SO)
        lib.synth_render.restype = ctypes.c_int
        lib.synth_render.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        _LIB = lib
    return _LIB


# --------------------------------------------------------------------------
# Model parameters (passed to both sides as inputs)
# --------------------------------------------------------------------------

def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), returned as fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    r = ((bits + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return (r & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(np.float32)


@dataclasses.dataclass(frozen=True)
class CNNSpec:
    """Specialized CNN shape: conv3x3 'same' + ReLU (+ 2x2 max-pool), dense D, 1 logit."""
    in_h: int
    in_w: int
    conv: tuple            # output channels per conv layer
    pool: tuple            # bool per conv layer: 2x2/2 max-pool after it
    dense: int
    bf16: bool

    def shapes(self):
        """[(cin, cout, h_in, w_in, pooled)] and the flattened feature size."""
        out = []
        c, h, w = 3, self.in_h, self.in_w
        for co, p in zip(self.conv, self.pool):
            out.append((c, co, h, w, bool(p)))
            c = co
            if p:
                h, w = h // 2, w // 2
        return out, c * h * w, (c, h, w)


def cnn_weights(spec: CNNSpec, seed: int) -> dict:
    """He-normal conv/dense weights (fp64 draw, stored fp32, bf16-rounded for bf16 nets).

    Biases are drawn N(0, 0.05^2) so that the bias paths are exercised."""
    rng = np.random.default_rng([seed, 31])
    layers, flat, _ = spec.shapes()
    conv_w, conv_b = [], []
    for cin, cout, _, _, _ in layers:
        conv_w.append(rng.standard_normal((cout, cin, 3, 3)) * math.sqrt(2.0 / (9 * cin)))
        conv_b.append(rng.standard_normal(cout) * 0.05)
    w1 = rng.standard_normal((spec.dense, flat)) * math.sqrt(2.0 / flat)
    b1 = rng.standard_normal(spec.dense) * 0.05
    w2 = rng.standard_normal(spec.dense) * math.sqrt(2.0 / spec.dense)
    b2 = rng.standard_normal(1) * 0.05
    fix = (lambda a: round_to_bf16(a.astype(np.float32))) if spec.bf16 else \
        (lambda a: a.astype(np.float32))
    return dict(conv_w=[fix(a) for a in conv_w], conv_b=[fix(a) for a in conv_b],
                w1=fix(w1), b1=fix(b1), w2=fix(w2), b2=fix(b2))


def weight_blob(spec: CNNSpec, wts: dict) -> np.ndarray:
    """Canonical fp32 blob: per conv [Cout][Cin][3][3] then bias[Cout];
    dense1 [D][flat] (flatten order c, y, x) then bias[D]; dense2 [D] then bias[1]."""
    parts = []
    for w, b in zip(wts["conv_w"], wts["conv_b"]):
        parts += [w.ravel(), b.ravel()]
    parts += [wts["w1"].ravel(), wts["b1"].ravel(), wts["w2"].ravel(), wts["b2"].ravel()]
    return np.ascontiguousarray(np.concatenate(parts).astype(np.float32))


def lr_weights(n_blocks: int, seed: int, bias: float = -2.0):
    """Blocked detector logistic-regression weights: w ~ N(0, 1) stored fp32, bias b."""
    rng = np.random.default_rng([seed, 47])
    return rng.standard_normal(n_blocks).astype(np.float32), float(bias)
