"""Host-side checks of libnsc: exports, validation paths, sizes (no GPU calls)."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import paper_1703_02529_amd as nsc
import synth
from synth import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nsc.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nsc_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert len(names) >= 17
    L = ctypes.CDLL(nsc.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def _cfg(**kw):
    base = dict(in_h=480, in_w=640, dd_h=50, dd_w=50, cnn_h=50, cnn_w=50, ref_mode=0, delta=15,
                grid=(1, 1), delta_diff=15.0, c_low=0.2, c_high=0.8)
    base.update(kw)
    return nsc.make_cfg(**base)


def test_valid_configs_pass():
    assert nsc.nsc_cfg_check(_cfg()) == 0
    for wl in W.ALL:
        c = nsc.make_cfg(in_h=wl.video.h, in_w=wl.video.w, dd_h=wl.dd_h, dd_w=wl.dd_w,
                         cnn_h=wl.cnn.in_h, cnn_w=wl.cnn.in_w, ref_mode=wl.ref_mode,
                         delta=wl.delta, grid=wl.grid, delta_diff=wl.delta_diff)
        # pointers the check requires are given as dummy non-null values
        c.lr_w = 16 if wl.grid != (1, 1) else None
        c.ref_sums = 16 if wl.ref_mode == 1 else None
        assert nsc.nsc_cfg_check(c) == 0, (wl.name, nsc.last_error())


@pytest.mark.parametrize("kw,code", [
    (dict(dd_h=600), -2),                 # grid larger than the frame
    (dict(dd_w=0), -2),
    (dict(cnn_h=30), -2),                 # does not divide the detector grid
    (dict(delta=0), -1),
    (dict(delta=257), -1),
    (dict(ref_mode=2), -1),
    (dict(ref_mode=1), -1),               # fixed reference without ref_sums
    (dict(grid=(10, 10)), -1),            # blocked without lr_w
    (dict(grid=(51, 1)), -2),
    (dict(delta_diff=math.nan), -1),
    (dict(c_low=0.9, c_high=0.1), -1),
    (dict(c_low=-0.1), -1),
    (dict(c_high=1.5), -1),
    (dict(check_stride=-1), -1),
    (dict(check_stride=4097), -1),
    (dict(check_stride=4), -1),           # delta 15 is not a multiple of the stride
    (dict(metric=-1), -1),
    (dict(metric=4), -1),
    (dict(fuse_prev=2), -1),
    (dict(fuse_prev=-1), -1),
])
def test_invalid_configs(kw, code):
    assert nsc.nsc_cfg_check(_cfg(**kw)) == code
    assert nsc.last_error() != ""


def test_detector_metrics():
    for m in (nsc.NSC_METRIC_MSE, nsc.NSC_METRIC_SAD, nsc.NSC_METRIC_NRMSE, nsc.NSC_METRIC_PSNR):
        assert nsc.nsc_cfg_check(_cfg(metric=m)) == 0
    for m in (nsc.NSC_METRIC_MSE, nsc.NSC_METRIC_SAD, nsc.NSC_METRIC_NRMSE):
        c = _cfg(metric=m, grid=(10, 10))
        c.lr_w = 16
        assert nsc.nsc_cfg_check(c) == 0
    # the blocked detector does not take PSNR (an unchanged block is -inf)
    c = _cfg(metric=nsc.NSC_METRIC_PSNR, grid=(10, 10))
    c.lr_w = 16
    assert nsc.nsc_cfg_check(c) == -1 and "PSNR" in nsc.last_error()


def test_group_arguments_are_checked_on_the_host():
    """nsc_group_create rejects bad camera sets before any device call (NULL
    network handles are only looked at once every cfg has passed)."""
    good = _cfg()
    assert nsc.nsc_group_create_status([good, good], [None, None]) == -1   # NULL handles
    assert "handle" in nsc.last_error()
    for kw in (dict(in_h=240, in_w=320), dict(dd_h=25, dd_w=25, cnn_h=25, cnn_w=25),
               dict(metric=nsc.NSC_METRIC_SAD), dict(check_stride=5)):
        assert nsc.nsc_group_create_status([good, _cfg(**kw)], [None, None]) == -1, kw
        assert "camera 1" in nsc.last_error()
    assert nsc.nsc_group_create_status([good, _cfg(delta=0)], [None, None]) == -1
    assert nsc.nsc_group_create_status([], []) == -1


def test_frame_skipping_sizes():
    # stride 0 and 1 mean every frame; a stride that divides delta is valid
    assert nsc.nsc_cfg_check(_cfg(check_stride=0)) == 0
    assert nsc.nsc_cfg_check(_cfg(check_stride=5)) == 0
    assert nsc.nsc_cfg_check(_cfg(ref_mode=1, check_stride=7, delta=1)) == -1  # no ref_sums
    base = nsc.nsc_state_bytes(_cfg())
    # delta / s = 3 checked frames of sums instead of 15, plus one decision byte
    skip = nsc.nsc_state_bytes(_cfg(check_stride=5))
    assert skip < base
    assert skip == nsc.nsc_state_bytes(_cfg(delta=3)) + 256


def test_frame_stride_and_overflow_limits():
    c = _cfg()
    c.frame_stride = 480 * 640 * 3 - 1
    assert nsc.nsc_cfg_check(c) == -1
    # 255 * den must fit 32-bit sums: 20000x20000 onto 1x1 has den 4e8
    assert nsc.lib().nsc_area_den(20000, 20000, 1, 1) == -2
    assert nsc.nsc_area_den(480, 640, 50, 50) == 3072
    with pytest.raises(nsc.NscError):
        nsc.nsc_area_den(10, 10, 20, 20)


@pytest.mark.parametrize("H,W,Ho,Wo", [(480, 640, 50, 50), (720, 1280, 100, 100), (100, 100, 50, 50),
                                       (1080, 1920, 100, 100), (7, 9, 3, 4)])
def test_area_den_formula(H, W, Ho, Wo):
    assert nsc.nsc_area_den(H, W, Ho, Wo) == (H // math.gcd(H, Ho)) * (W // math.gcd(W, Wo))


def test_cnn_desc_checks_and_blob_size():
    for wl in W.ALL:
        d = nsc.make_desc(wl.cnn.conv, wl.cnn.pool, wl.cnn.dense, wl.cnn.in_h, wl.cnn.in_w,
                          wl.cnn.bf16)
        assert nsc.nsc_cnn_check(d) == 0, nsc.last_error()
        blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, 1))
        assert nsc.nsc_cnn_blob_floats(d) == blob.size
    bad = [
        nsc.make_desc((24,), (True,), 32, 50, 50, True),            # 24 output channels
        nsc.make_desc((32, 40), (True, True), 32, 50, 50, True),    # 40 output channels
        nsc.make_desc((32,), (True,), 48, 50, 50, True),            # dense 48
        nsc.make_desc((), (), 32, 50, 50, True),                    # no conv
        nsc.make_desc((256, 256), (False, False), 32, 50, 50, True),  # LDS too large
    ]
    for d in bad:
        assert nsc.nsc_cnn_check(d) == -2, nsc.last_error()
    d = nsc.make_desc((32,), (True,), 32, 50, 50, True)
    d.dtype = 7
    assert nsc.nsc_cnn_check(d) == -3
    d.dtype = 3
    assert nsc.nsc_cnn_check(d) == -3
    for pairs in (False, True):
        d = nsc.make_desc((64, 64), (False, True), 32, 50, 50, True, pairs)
        assert d.dtype == (nsc.NSC_BF16_PAIRS if pairs else nsc.NSC_BF16)
        assert nsc.nsc_cnn_check(d) == 0


def test_status_strings():
    assert nsc.status_string(0) == "NSC_OK"
    assert nsc.status_string(-4) == "NSC_E_WORKSPACE"
    assert nsc.status_string(-99) == "NSC_E_UNKNOWN"


def test_compact_noalloc_validation():
    """nsc_compact_noalloc refuses bad arguments on the host, before any HIP call."""
    L = nsc.lib()
    big = nsc.NSC_NOALLOC_MAX_FLAGS + 1
    assert L.nsc_compact_noalloc(16, big, 16, 16, None) == nsc.NSC_E_WORKSPACE
    assert "exceeds" in nsc.last_error()
    assert L.nsc_compact_noalloc(16, -1, 16, 16, None) == nsc.NSC_E_INVAL
    assert L.nsc_compact_noalloc(16, 10, 16, None, None) == nsc.NSC_E_INVAL
    assert L.nsc_compact_noalloc(None, 10, 16, 16, None) == nsc.NSC_E_INVAL


def test_compact_workspace_size():
    assert nsc.nsc_compact_workspace_bytes(0) >= 4
    assert nsc.nsc_compact_workspace_bytes(4097) >= 2 * 4
    with pytest.raises(nsc.NscError):
        nsc.nsc_compact_workspace_bytes(-1)


def test_threshold_sweep_rejects_bad_arguments_on_the_host():
    # every check runs before any HIP call; the dummy addresses are never read
    L = nsc.lib()
    good = nsc.SweepCfg(0, 1, 0.01, 0.01, 1e-6, 1e-4, 1e-2)
    p = ctypes.c_void_p(16)
    args = lambda cfg, n=10, n_t=4, ptr=p: (ctypes.byref(cfg), ptr, ptr, ptr, n, ptr, n_t, ptr, ptr,
                                             None)
    E_INVAL = -1
    assert L.nsc_threshold_sweep(*args(good, ptr=None)) == E_INVAL
    assert L.nsc_threshold_sweep(*args(good, n=0)) == E_INVAL
    assert L.nsc_threshold_sweep(*args(good, n_t=0)) == E_INVAL
    assert L.nsc_threshold_sweep(*args(good, n_t=70000)) == E_INVAL
    for bad in (nsc.SweepCfg(2, 1, 0.01, 0.01, 0, 0, 0), nsc.SweepCfg(0, 0, 0.01, 0.01, 0, 0, 0),
                nsc.SweepCfg(0, 1, 1.5, 0.01, 0, 0, 0), nsc.SweepCfg(0, 1, 0.01, -0.1, 0, 0, 0),
                nsc.SweepCfg(0, 1, 0.01, 0.01, -1, 0, 0),
                nsc.SweepCfg(0, 1, 0.01, 0.01, 0, math.inf, 0)):
        assert L.nsc_threshold_sweep(*args(bad)) == E_INVAL
        assert nsc.last_error()


def test_staged_batch_calls_check_on_the_host():
    """nsc_batch_workspace_bytes, nsc_cascade_stage and nsc_cascade_finish
    refuse a bad cfg or a NULL network before any device call."""
    L = nsc.lib()
    b = ctypes.c_size_t()
    good, bad = _cfg(), _cfg(delta=0)
    assert L.nsc_batch_workspace_bytes(ctypes.byref(good), None, 64, 0, ctypes.byref(b)) == -1
    assert "cnn" in nsc.last_error()
    assert L.nsc_batch_workspace_bytes(ctypes.byref(bad), None, 64, 0, ctypes.byref(b)) == -1
    p = ctypes.c_void_p(256)
    assert L.nsc_cascade_stage(ctypes.byref(good), None, 64, 0, p, 8, 0, p, 1 << 20, None) == -1
    assert L.nsc_cascade_finish(ctypes.byref(bad), None, 64, 0, 8, 0, p, p, 1 << 20, p, p, None,
                                None, None, None) == -1
