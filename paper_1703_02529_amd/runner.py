"""Convenience owner of the device buffers one cascade stream needs.

Allocates (through torch) the workspace, the carried state and the per-frame
output buffers, creates the CNN handle, and calls nsc_cascade_run.  It reads a
workload description by attribute (video.h, video.w, dd_h, dd_w, cnn, ref_mode,
delta, grid, delta_diff, c_low, c_high, lr_bias; check_stride, metric and
fuse_prev if present) and imports nothing else.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import (NSC_METRIC_MSE, NSC_REF_FIXED, NSC_REF_PREV, Cnn, Group, make_cfg, make_desc,
               nsc_batch_workspace_bytes, nsc_cascade_finish, nsc_cascade_run,
               nsc_cascade_stage, nsc_cascade_workspace_bytes, nsc_group_run,
               nsc_group_state_bytes, nsc_group_workspace_bytes, nsc_state_bytes)


def _cfg_of(wl, lr_w=None, ref_sums=None, frame_stride=None):
    return make_cfg(in_h=wl.video.h, in_w=wl.video.w, dd_h=wl.dd_h, dd_w=wl.dd_w,
                    cnn_h=wl.cnn.in_h, cnn_w=wl.cnn.in_w, ref_mode=wl.ref_mode, delta=wl.delta,
                    grid=tuple(wl.grid), lr_w=lr_w, lr_b=wl.lr_bias, ref_sums=ref_sums,
                    delta_diff=wl.delta_diff, c_low=wl.c_low, c_high=wl.c_high,
                    frame_stride=frame_stride, check_stride=getattr(wl, "check_stride", 1),
                    metric=getattr(wl, "metric", NSC_METRIC_MSE),
                    fuse_prev=getattr(wl, "fuse_prev", 0))


class CascadeRunner:
    """batch=True sizes the workspace for staged batches of up to max_frames
    frames (stage() per chunk, then finish()); cnn_pass bounds the survivors
    of one CNN pass in a batch (0: the library's default)."""

    def __init__(self, wl, blob, max_frames: int, lr_w: Optional[torch.Tensor] = None,
                 ref_sums: Optional[torch.Tensor] = None, device="cuda", frame_stride=None,
                 batch: bool = False, cnn_pass: int = 0):
        self.wl = wl
        self.device = torch.device(device)
        self.lr_w = lr_w
        self.ref_sums = ref_sums
        self.cfg = _cfg_of(wl, lr_w, ref_sums, frame_stride)
        self.desc = make_desc(wl.cnn.conv, wl.cnn.pool, wl.cnn.dense, wl.cnn.in_h, wl.cnn.in_w,
                              wl.cnn.bf16)
        self.cnn = Cnn(self.desc, blob)
        self.max_frames = max_frames
        self.batch = batch
        self.cnn_pass = cnn_pass
        if batch:
            ws = nsc_batch_workspace_bytes(self.cfg, self.cnn, max_frames, cnn_pass)
        else:
            ws = nsc_cascade_workspace_bytes(self.cfg, self.cnn, max_frames)
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
        self.state = torch.zeros(max(nsc_state_bytes(self.cfg), 256), dtype=torch.uint8,
                                 device=self.device)
        self.label = torch.empty(max_frames, dtype=torch.uint8, device=self.device)
        self.defer = torch.empty(max_frames, dtype=torch.uint8, device=self.device)
        self.score = torch.empty(max_frames, dtype=torch.float64, device=self.device)
        self.fire = torch.empty(max_frames, dtype=torch.uint8, device=self.device)
        self.logit = torch.empty(max_frames, dtype=torch.float32, device=self.device)
        self.next_t = 0

    def run(self, frames: torch.Tensor, n: int, t0: Optional[int] = None, taps: bool = True,
            want_stats: bool = False, stage_events=None, stream=None):
        """Runs frames [t0, t0+n) (default: continue where the last call ended)."""
        if n > self.max_frames:
            raise ValueError(f"{n} frames exceed the workspace's {self.max_frames}")
        t0 = self.next_t if t0 is None else t0
        kw = dict(score=self.score[:n], fire=self.fire[:n], logit=self.logit[:n]) if taps else {}
        st = nsc_cascade_run(self.cfg, self.cnn, frames, n, t0, self.state, self.ws,
                             self.label[:n], self.defer[:n], want_stats=want_stats,
                             stage_events=stage_events, stream=stream, **kw)
        self.next_t = t0 + n
        return st

    def stage(self, frames: torch.Tensor, n: int, at: int, stream=None):
        """Area sums of n frames into batch slots [at, at + n)."""
        if not self.batch:
            raise ValueError("stage() needs a runner made with batch=True")
        nsc_cascade_stage(self.cfg, self.cnn, self.max_frames, self.cnn_pass, frames, n, at,
                          self.ws, stream=stream)

    def finish(self, n: int, t0: Optional[int] = None, label=None, defer=None, score=None,
               fire=None, logit=None, want_stats: bool = False, stage_events=None, stream=None):
        """Steps 2-5 on the n staged frames, frames [t0, t0 + n) (default:
        continue where the last call ended).  Per-frame outputs go to the
        given device tensors, else to the runner's own buffers."""
        if not self.batch:
            raise ValueError("finish() needs a runner made with batch=True")
        t0 = self.next_t if t0 is None else t0
        if label is None:
            label, defer = self.label[:n], self.defer[:n]
            score, fire, logit = self.score[:n], self.fire[:n], self.logit[:n]
        st = nsc_cascade_finish(self.cfg, self.cnn, self.max_frames, self.cnn_pass, n, t0,
                                self.state, self.ws, label, defer, score=score, fire=fire,
                                logit=logit, want_stats=want_stats, stage_events=stage_events,
                                stream=stream)
        self.next_t = t0 + n
        return st

    def close(self):
        self.cnn.close()


class GroupRunner:
    """Buffers of a camera group: one workload description per camera (same
    frame geometry and metric), each with its weight blob and its device LR
    weights / reference sums (None where unused).  Runs n frames of every
    camera per call, camera-major."""

    def __init__(self, wls, blobs, frames_per_cam: int, lr_ws=None, ref_sums=None,
                 device="cuda"):
        self.wls = list(wls)
        k = len(self.wls)
        self.device = torch.device(device)
        self.lr_ws = list(lr_ws) if lr_ws is not None else [None] * k
        self.ref_sums = list(ref_sums) if ref_sums is not None else [None] * k
        self.cfgs = [_cfg_of(w, l, r) for w, l, r in zip(self.wls, self.lr_ws, self.ref_sums)]
        self.cnns = [Cnn(make_desc(w.cnn.conv, w.cnn.pool, w.cnn.dense, w.cnn.in_h, w.cnn.in_w,
                                   w.cnn.bf16), b) for w, b in zip(self.wls, blobs)]
        self.group = Group(self.cfgs, self.cnns)
        self.frames_per_cam = frames_per_cam
        total = k * frames_per_cam
        ws = nsc_group_workspace_bytes(self.group, frames_per_cam)
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
        sb, self.slot_bytes = nsc_group_state_bytes(self.group)
        self.state = torch.zeros(max(sb, 256), dtype=torch.uint8, device=self.device)
        self.label = torch.empty(total, dtype=torch.uint8, device=self.device)
        self.defer = torch.empty(total, dtype=torch.uint8, device=self.device)
        self.score = torch.empty(total, dtype=torch.float64, device=self.device)
        self.fire = torch.empty(total, dtype=torch.uint8, device=self.device)
        self.logit = torch.empty(total, dtype=torch.float32, device=self.device)
        self.next_t = 0

    def run(self, frames: torch.Tensor, n: int, t0: Optional[int] = None, taps: bool = True,
            want_stats: bool = False, stage_events=None, stream=None):
        """Frames [t0, t0+n) of every camera: frames holds camera c's frame
        t0 + j at index c * n + j; outputs are [camera][n] in the first
        len(wls) * n entries of label / defer / score / fire / logit."""
        if n > self.frames_per_cam:
            raise ValueError(f"{n} frames per camera exceed the workspace's {self.frames_per_cam}")
        t0 = self.next_t if t0 is None else t0
        m = len(self.wls) * n
        kw = dict(score=self.score[:m], fire=self.fire[:m], logit=self.logit[:m]) if taps else {}
        st = nsc_group_run(self.group, frames, n, t0, self.state, self.ws, self.label[:m],
                           self.defer[:m], want_stats=want_stats, stage_events=stage_events,
                           stream=stream, **kw)
        self.next_t = t0 + n
        return st

    def close(self):
        self.group.close()
        for c in self.cnns:
            c.close()


__all__ = ["CascadeRunner", "GroupRunner", "NSC_REF_PREV", "NSC_REF_FIXED"]
