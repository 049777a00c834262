"""Python binding of libnsc, the NoScope cascade filter for MI355X (gfx950).

Argument marshalling only: every step of the path runs in the HIP kernels of
libnsc.so.  Torch supplies device memory and streams; the functions below
take torch tensors, pass their device pointers and the current stream to the
C ABI of include/nsc.h under the same names, and raise NscError on any
non-zero status.  There is no fallback: if libnsc.so is missing the import of
the library fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libnsc.so")

NSC_REF_PREV, NSC_REF_FIXED = 0, 1
NSC_METRIC_MSE, NSC_METRIC_SAD, NSC_METRIC_NRMSE, NSC_METRIC_PSNR = 0, 1, 2, 3
NSC_F32, NSC_BF16, NSC_BF16_PAIRS = 0, 1, 2
NSC_MAX_CONV = 8

_i32, _i64, _u32, _dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_double
_vp, _sz = ctypes.c_void_p, ctypes.c_size_t


NSC_OK, NSC_E_INVAL, NSC_E_SHAPE, NSC_E_DTYPE, NSC_E_WORKSPACE, NSC_E_HIP, NSC_E_NOMEM, \
    NSC_E_STATE = 0, -1, -2, -3, -4, -5, -6, -7


class NscError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str):
        super().__init__(f"{what}: {status_string(status)} ({status}): {detail}")
        self.status = status


class CascadeCfg(ctypes.Structure):
    _fields_ = [("in_h", _i32), ("in_w", _i32), ("frame_stride", _i64), ("dd_h", _i32),
                ("dd_w", _i32), ("cnn_h", _i32), ("cnn_w", _i32), ("ref_mode", _i32),
                ("delta", _i32), ("grid_h", _i32), ("grid_w", _i32), ("lr_w", _vp),
                ("lr_b", _dbl), ("ref_sums", _vp), ("delta_diff", _dbl), ("c_low", _dbl),
                ("c_high", _dbl), ("check_stride", _i32), ("metric", _i32), ("fuse_prev", _i32)]


class CnnDesc(ctypes.Structure):
    _fields_ = [("n_conv", _i32), ("conv_out", _i32 * NSC_MAX_CONV), ("pool_after_mask", _u32),
                ("dense", _i32), ("in_h", _i32), ("in_w", _i32), ("dtype", _i32)]


class FrameOutputs(ctypes.Structure):
    _fields_ = [("score", _vp), ("fire", _vp), ("logit", _vp)]


class SweepCfg(ctypes.Structure):
    _fields_ = [("ref_mode", _i32), ("delta", _i32), ("fp_target", _dbl), ("fn_target", _dbl),
                ("t_mse", _dbl), ("t_snn", _dbl), ("t_full", _dbl)]


# nsc_sweep_row, as numpy reads it from the bytes of the rows buffer
SWEEP_ROW_BYTES = 120


class RunStats(ctypes.Structure):
    _fields_ = [("frames", _i64), ("fired", _i64), ("positive", _i64), ("deferred", _i64)]


_LIB: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Loads libnsc.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_1703_02529_amd.build` or __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        sig = {
            "nsc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "nsc_last_error": (ctypes.c_char_p, []),
            "nsc_area_den": (_i64, [_i32, _i32, _i32, _i32]),
            "nsc_cfg_check": (ctypes.c_int, [_vp]),
            "nsc_cnn_check": (ctypes.c_int, [_vp]),
            "nsc_cnn_blob_floats": (_i64, [_vp]),
            "nsc_cnn_create": (ctypes.c_int, [_vp, _vp, _i64, _vp]),
            "nsc_cnn_destroy": (ctypes.c_int, [_vp]),
            "nsc_cascade_workspace_bytes": (ctypes.c_int, [_vp, _vp, _i64, _vp]),
            "nsc_state_bytes": (ctypes.c_int, [_vp, _vp]),
            "nsc_compact_workspace_bytes": (ctypes.c_int, [_i64, _vp]),
            "nsc_cnn_workspace_bytes": (ctypes.c_int, [_vp, _i64, _vp]),
            "nsc_downsample": (ctypes.c_int, [_vp, _i64, _i32, _i32, _i64, _i32, _i32, _vp, _vp]),
            "nsc_diff_detect": (ctypes.c_int, [_vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _vp]),
            "nsc_compact": (ctypes.c_int, [_vp, _i64, _vp, _vp, _vp, _sz, _vp]),
            "nsc_compact_noalloc": (ctypes.c_int, [_vp, _i64, _vp, _vp, _vp]),
            "nsc_threshold_sweep": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp, _i32, _vp, _vp,
                                                   _vp]),
            "nsc_specialized_cnn": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i64, _vp, _vp, _i64,
                                                   _vp, _vp, _vp, _sz, _vp]),
            "nsc_cascade_run": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i64, _vp, _vp, _sz, _vp, _vp,
                                               _vp, _vp, _vp, _vp]),
            "nsc_batch_workspace_bytes": (ctypes.c_int, [_vp, _vp, _i64, _i64, _vp]),
            "nsc_cascade_stage": (ctypes.c_int, [_vp, _vp, _i64, _i64, _vp, _i64, _i64, _vp, _sz,
                                                 _vp]),
            "nsc_cascade_finish": (ctypes.c_int, [_vp, _vp, _i64, _i64, _i64, _i64, _vp, _vp, _sz,
                                                  _vp, _vp, _vp, _vp, _vp, _vp]),
            "nsc_group_create": (ctypes.c_int, [_vp, _vp, _i32, _vp]),
            "nsc_group_destroy": (ctypes.c_int, [_vp]),
            "nsc_group_state_bytes": (ctypes.c_int, [_vp, _vp, _vp]),
            "nsc_group_workspace_bytes": (ctypes.c_int, [_vp, _i64, _vp]),
            "nsc_group_run": (ctypes.c_int, [_vp, _vp, _i64, _i64, _vp, _vp, _sz, _vp, _vp, _vp,
                                             _vp, _vp, _vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().nsc_status_string(status).decode()


def last_error() -> str:
    return lib().nsc_last_error().decode()


def _check(rc: int, what: str):
    if rc != 0:
        raise NscError(rc, what, last_error())


# ------------------------------------------------------------ marshalling

def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def make_cfg(*, in_h, in_w, dd_h, dd_w, cnn_h, cnn_w, ref_mode=NSC_REF_PREV, delta=1,
             grid=(1, 1), lr_w=None, lr_b=0.0, ref_sums=None, delta_diff=0.0, c_low=0.2,
             c_high=0.8, frame_stride=None, check_stride=1, metric=0, fuse_prev=0) -> CascadeCfg:
    """Builds a CascadeCfg; lr_w and ref_sums are device tensors (kept alive by the caller)."""
    c = CascadeCfg()
    c.in_h, c.in_w = in_h, in_w
    c.frame_stride = frame_stride if frame_stride is not None else in_h * in_w * 3
    c.dd_h, c.dd_w, c.cnn_h, c.cnn_w = dd_h, dd_w, cnn_h, cnn_w
    c.ref_mode, c.delta = ref_mode, delta
    c.grid_h, c.grid_w = grid
    c.lr_w = _ptr(lr_w)
    c.lr_b = lr_b
    c.ref_sums = _ptr(ref_sums)
    c.delta_diff, c.c_low, c.c_high = delta_diff, c_low, c_high
    c.check_stride = check_stride
    c.metric = metric
    c.fuse_prev = fuse_prev
    return c


def make_desc(conv, pool, dense, in_h, in_w, bf16, pairs=False) -> CnnDesc:
    """pairs: a bf16 network whose later activations enter the matrix cores as
    bf16 hi / lo pairs (NSC_BF16_PAIRS) instead of fp16 (NSC_BF16)."""
    d = CnnDesc()
    d.n_conv = len(conv)
    mask = 0
    for i, (co, p) in enumerate(zip(conv, pool)):
        d.conv_out[i] = co
        mask |= (1 << i) if p else 0
    d.pool_after_mask = mask
    d.dense, d.in_h, d.in_w = dense, in_h, in_w
    d.dtype = (NSC_BF16_PAIRS if pairs else NSC_BF16) if bf16 else NSC_F32
    return d


def nsc_area_den(in_h, in_w, out_h, out_w) -> int:
    v = lib().nsc_area_den(in_h, in_w, out_h, out_w)
    _check(v if v < 0 else 0, "nsc_area_den")
    return int(v)


def nsc_cfg_check(cfg: CascadeCfg) -> int:
    return lib().nsc_cfg_check(ctypes.byref(cfg))


def nsc_cnn_check(desc: CnnDesc) -> int:
    return lib().nsc_cnn_check(ctypes.byref(desc))


def nsc_cnn_blob_floats(desc: CnnDesc) -> int:
    v = lib().nsc_cnn_blob_floats(ctypes.byref(desc))
    _check(v if v < 0 else 0, "nsc_cnn_blob_floats")
    return int(v)


class Cnn:
    """Owns an nsc_cnn handle (packed device weights)."""

    def __init__(self, desc: CnnDesc, blob):
        import numpy as np
        b = np.ascontiguousarray(blob, dtype=np.float32)
        h = _vp()
        _check(lib().nsc_cnn_create(ctypes.byref(desc), b.ctypes.data_as(_vp), b.size,
                                    ctypes.byref(h)), "nsc_cnn_create")
        self.desc = desc
        self.handle = h

    def close(self):
        if self.handle:
            _check(lib().nsc_cnn_destroy(self.handle), "nsc_cnn_destroy")
            self.handle = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def nsc_cascade_workspace_bytes(cfg, cnn: Cnn, max_frames: int) -> int:
    b = _sz()
    _check(lib().nsc_cascade_workspace_bytes(ctypes.byref(cfg), cnn.handle, max_frames,
                                             ctypes.byref(b)), "nsc_cascade_workspace_bytes")
    return b.value


def nsc_state_bytes(cfg) -> int:
    b = _sz()
    _check(lib().nsc_state_bytes(ctypes.byref(cfg), ctypes.byref(b)), "nsc_state_bytes")
    return b.value


def nsc_compact_workspace_bytes(n: int) -> int:
    b = _sz()
    _check(lib().nsc_compact_workspace_bytes(n, ctypes.byref(b)), "nsc_compact_workspace_bytes")
    return b.value


def nsc_cnn_workspace_bytes(cnn: Cnn, max_count: int) -> int:
    b = _sz()
    _check(lib().nsc_cnn_workspace_bytes(cnn.handle, max_count, ctypes.byref(b)),
           "nsc_cnn_workspace_bytes")
    return b.value


def nsc_downsample(frames, n, in_h, in_w, out_h, out_w, sums_out, frame_stride=None, stream=None):
    stride = frame_stride if frame_stride is not None else in_h * in_w * 3
    _check(lib().nsc_downsample(_ptr(frames), n, in_h, in_w, stride, out_h, out_w, _ptr(sums_out),
                                _stream(stream)), "nsc_downsample")


def nsc_diff_detect(cfg, frames, n, t0, sums_out, fire_out, score_out=None, prev_sums=None,
                    stream=None):
    _check(lib().nsc_diff_detect(ctypes.byref(cfg), _ptr(frames), n, t0, _ptr(prev_sums),
                                 _ptr(sums_out), _ptr(score_out), _ptr(fire_out), _stream(stream)),
           "nsc_diff_detect")


def nsc_compact(fire, n, idx_out, count_out, ws, stream=None):
    _check(lib().nsc_compact(_ptr(fire), n, _ptr(idx_out), _ptr(count_out), _ptr(ws),
                             ws.numel() * ws.element_size() if ws is not None else 0,
                             _stream(stream)), "nsc_compact")


NSC_NOALLOC_MAX_FLAGS = 67108864


def nsc_compact_noalloc(fire, n, idx_out, count_out, stream=None):
    _check(lib().nsc_compact_noalloc(_ptr(fire), n, _ptr(idx_out), _ptr(count_out),
                                     _stream(stream)), "nsc_compact_noalloc")


def nsc_specialized_cnn(cnn: Cnn, sums, sums_h, sums_w, den, idx, count, max_count, logit_out,
                        ws, prob_out=None, stream=None):
    _check(lib().nsc_specialized_cnn(cnn.handle, _ptr(sums), sums_h, sums_w, den, _ptr(idx),
                                     _ptr(count), max_count, _ptr(logit_out), _ptr(prob_out),
                                     _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "nsc_specialized_cnn")


NSC_STAGE_EVENTS = 6


def nsc_cascade_run(cfg, cnn: Cnn, frames, n, t0, state, ws, label_out, defer_out, score=None,
                    fire=None, logit=None, want_stats=False, stage_events=None, stream=None):
    """stage_events: optional sequence of NSC_STAGE_EVENTS raw hipEvent_t handles (ints)."""
    outs = None
    if score is not None or fire is not None or logit is not None:
        outs = FrameOutputs(_ptr(score), _ptr(fire), _ptr(logit))
    st = RunStats() if want_stats else None
    ev = None
    if stage_events is not None:
        if len(stage_events) != NSC_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {NSC_STAGE_EVENTS} entries")
        ev = (_vp * NSC_STAGE_EVENTS)(*[e if e else None for e in stage_events])
    _check(lib().nsc_cascade_run(ctypes.byref(cfg), cnn.handle, _ptr(frames), n, t0, _ptr(state),
                                 _ptr(ws), ws.numel() * ws.element_size(), _ptr(label_out),
                                 _ptr(defer_out), ctypes.byref(outs) if outs else None,
                                 ctypes.byref(st) if st else None, ev, _stream(stream)),
           "nsc_cascade_run")
    if st is not None:
        return dict(frames=st.frames, fired=st.fired, positive=st.positive, deferred=st.deferred)
    return None


def nsc_batch_workspace_bytes(cfg, cnn: Cnn, batch_frames: int, cnn_pass: int = 0) -> int:
    b = _sz()
    _check(lib().nsc_batch_workspace_bytes(ctypes.byref(cfg), cnn.handle, batch_frames, cnn_pass,
                                           ctypes.byref(b)), "nsc_batch_workspace_bytes")
    return b.value


def nsc_cascade_stage(cfg, cnn: Cnn, batch_frames, cnn_pass, frames, n, at, ws, stream=None):
    _check(lib().nsc_cascade_stage(ctypes.byref(cfg), cnn.handle, batch_frames, cnn_pass,
                                   _ptr(frames), n, at, _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream(stream)), "nsc_cascade_stage")


def nsc_cascade_finish(cfg, cnn: Cnn, batch_frames, cnn_pass, n, t0, state, ws, label_out,
                       defer_out, score=None, fire=None, logit=None, want_stats=False,
                       stage_events=None, stream=None):
    """Arguments after cnn_pass as for nsc_cascade_run, without frames."""
    outs = None
    if score is not None or fire is not None or logit is not None:
        outs = FrameOutputs(_ptr(score), _ptr(fire), _ptr(logit))
    st = RunStats() if want_stats else None
    ev = None
    if stage_events is not None:
        if len(stage_events) != NSC_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {NSC_STAGE_EVENTS} entries")
        ev = (_vp * NSC_STAGE_EVENTS)(*[e if e else None for e in stage_events])
    _check(lib().nsc_cascade_finish(ctypes.byref(cfg), cnn.handle, batch_frames, cnn_pass, n, t0,
                                    _ptr(state), _ptr(ws), ws.numel() * ws.element_size(),
                                    _ptr(label_out), _ptr(defer_out),
                                    ctypes.byref(outs) if outs else None,
                                    ctypes.byref(st) if st else None, ev, _stream(stream)),
           "nsc_cascade_finish")
    if st is not None:
        return dict(frames=st.frames, fired=st.fired, positive=st.positive, deferred=st.deferred)
    return None


class Group:
    """Owns an nsc_group handle: cameras sharing a frame geometry, each with its
    own cfg (CascadeCfg) and network (Cnn).  The cfgs' device buffers and the
    networks must outlive the group."""

    def __init__(self, cfgs, cnns):
        if len(cfgs) != len(cnns) or not cfgs:
            raise ValueError("one cfg and one network per camera")
        self.n_cams = len(cfgs)
        self._cfgs = (CascadeCfg * self.n_cams)(*cfgs)
        self._cnns = (_vp * self.n_cams)(*[c.handle for c in cnns])
        self.cnns = list(cnns)
        h = _vp()
        _check(lib().nsc_group_create(self._cfgs, self._cnns, self.n_cams, ctypes.byref(h)),
               "nsc_group_create")
        self.handle = h

    def close(self):
        if self.handle:
            _check(lib().nsc_group_destroy(self.handle), "nsc_group_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def nsc_group_create_status(cfgs, cnn_handles) -> int:
    """Raw status of nsc_group_create (host-side validation tests); destroys
    the group when it was created."""
    n = len(cfgs)
    arr = (CascadeCfg * n)(*cfgs)
    hs = (_vp * n)(*cnn_handles)
    h = _vp()
    rc = lib().nsc_group_create(arr, hs, n, ctypes.byref(h))
    if rc == 0:
        lib().nsc_group_destroy(h)
    return rc


def nsc_group_state_bytes(group: Group) -> tuple:
    b, s = _sz(), _sz()
    _check(lib().nsc_group_state_bytes(group.handle, ctypes.byref(b), ctypes.byref(s)),
           "nsc_group_state_bytes")
    return b.value, s.value


def nsc_group_workspace_bytes(group: Group, frames_per_cam: int) -> int:
    b = _sz()
    _check(lib().nsc_group_workspace_bytes(group.handle, frames_per_cam, ctypes.byref(b)),
           "nsc_group_workspace_bytes")
    return b.value


def nsc_group_run(group: Group, frames, n, t0, state, ws, label_out, defer_out, score=None,
                  fire=None, logit=None, want_stats=False, stage_events=None, stream=None):
    """n frames of every camera (camera-major in frames and in every output)."""
    outs = None
    if score is not None or fire is not None or logit is not None:
        outs = FrameOutputs(_ptr(score), _ptr(fire), _ptr(logit))
    st = RunStats() if want_stats else None
    ev = None
    if stage_events is not None:
        if len(stage_events) != NSC_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {NSC_STAGE_EVENTS} entries")
        ev = (_vp * NSC_STAGE_EVENTS)(*[e if e else None for e in stage_events])
    _check(lib().nsc_group_run(group.handle, _ptr(frames), n, t0, _ptr(state), _ptr(ws),
                               ws.numel() * ws.element_size(), _ptr(label_out), _ptr(defer_out),
                               ctypes.byref(outs) if outs else None,
                               ctypes.byref(st) if st else None, ev, _stream(stream)),
           "nsc_group_run")
    if st is not None:
        return dict(frames=st.frames, fired=st.fired, positive=st.positive, deferred=st.deferred)
    return None


def nsc_threshold_sweep(cfg: SweepCfg, score, conf, truth, deltas, rows, best, stream=None):
    """rows: device uint8 tensor of len(deltas) * SWEEP_ROW_BYTES bytes; best:
    device int32 tensor of one element."""
    n, n_t = score.numel(), deltas.numel()
    if rows.numel() * rows.element_size() < n_t * SWEEP_ROW_BYTES:
        raise ValueError("rows holds fewer than one nsc_sweep_row per candidate")
    _check(lib().nsc_threshold_sweep(ctypes.byref(cfg), _ptr(score), _ptr(conf), _ptr(truth), n,
                                     _ptr(deltas), n_t, _ptr(rows), _ptr(best), _stream(stream)),
           "nsc_threshold_sweep")
