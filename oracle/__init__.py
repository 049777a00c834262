"""Python view of the fp64 CPU oracle (oracle.cpp).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are its only users.  The product path
(``paper_1703_02529_amd``) never imports it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SO = os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "oracle.cpp")

_i32, _i64, _dbl, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (single-threaded, -O2, no fast-math)."""
    if force or not os.path.exists(SO):
        tmp = SO + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fPIC", "-shared",
                               SRC, "-o", tmp])
        os.replace(tmp, SO)
    return SO


class CnnDesc(ctypes.Structure):
    _fields_ = [("n_conv", _i32), ("conv_out", _i32 * 8), ("pool_after", _i32 * 8),
                ("dense", _i32), ("in_h", _i32), ("in_w", _i32), ("bf16", _i32)]


class Cfg(ctypes.Structure):
    _fields_ = [("H", _i32), ("W", _i32), ("Ho", _i32), ("Wo", _i32), ("Hc", _i32), ("Wc", _i32),
                ("ref_mode", _i32), ("delta", _i32), ("Gh", _i32), ("Gw", _i32),
                ("lr_w", _vp), ("lr_b", _dbl), ("ref_sums", _vp), ("delta_diff", _dbl),
                ("c_low", _dbl), ("c_high", _dbl), ("check_stride", _i32), ("metric", _i32)]


# detector metrics (oracle.cpp, metric_of)
MSE, SAD, NRMSE, PSNR = 0, 1, 2, 3


class SweepCfg(ctypes.Structure):
    _fields_ = [("ref_mode", _i32), ("delta", _i32), ("fp_target", _dbl), ("fn_target", _dbl),
                ("t_mse", _dbl), ("t_snn", _dbl), ("t_full", _dbl)]


SWEEP_ROW = np.dtype([("delta", "<f8"), ("c_low", "<f8"), ("c_high", "<f8"), ("f_m", "<f8"),
                      ("f_c", "<f8"), ("cost", "<f8"), ("fired", "<i8"), ("deferred", "<i8"),
                      ("fn_dd", "<i8"), ("fp_dd", "<i8"), ("fn_cnn", "<i8"), ("fp_cnn", "<i8"),
                      ("positives", "<i8"), ("negatives", "<i8"), ("feasible", "<i4"),
                      ("pad", "<i4")])


_LIB = None


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        build(force=False)
        L = ctypes.CDLL(SO)
        L.oracle_area_weights.restype = _i64
        L.oracle_area_weights.argtypes = [_i32, _i32, _vp]
        L.oracle_history.restype = _i64
        L.oracle_history.argtypes = [_vp]
        L.oracle_area_den.restype = _i64
        L.oracle_area_den.argtypes = [_i32] * 4
        L.oracle_area_sums.restype = None
        L.oracle_area_sums.argtypes = [_vp, _i32, _i32, _i32, _i32, _vp]
        L.oracle_global_mse.restype = _dbl
        L.oracle_global_mse.argtypes = [_vp, _vp, _i32, _i32, _i64, _vp]
        L.oracle_global_metric.restype = _dbl
        L.oracle_global_metric.argtypes = [_i32, _vp, _vp, _i32, _i32, _i64, _vp]
        L.oracle_blocked_metric.restype = _dbl
        L.oracle_blocked_metric.argtypes = [_i32, _vp, _vp, _i32, _i32, _i64, _i32, _i32, _vp,
                                            _dbl, _vp]
        L.oracle_blocked_score.restype = _dbl
        L.oracle_blocked_score.argtypes = [_vp, _vp, _i32, _i32, _i64, _i32, _i32, _vp, _dbl, _vp]
        L.oracle_round_bf16.restype = _dbl
        L.oracle_round_bf16.argtypes = [_dbl]
        L.oracle_cnn_blob_floats.restype = _i64
        L.oracle_cnn_blob_floats.argtypes = [_vp]
        L.oracle_conv3x3.restype = None
        L.oracle_conv3x3.argtypes = [_vp, _i32, _i32, _i32, _vp, _vp, _i32, _vp]
        L.oracle_cnn_logit.restype = _dbl
        L.oracle_cnn_logit.argtypes = [_vp, _vp, _vp, _i64, _vp, _vp]
        L.oracle_sigmoid.restype = _dbl
        L.oracle_sigmoid.argtypes = [_dbl]
        L.oracle_decide.restype = _i32
        L.oracle_decide.argtypes = [_dbl, _dbl, _dbl]
        L.oracle_threshold_sweep.restype = _i32
        L.oracle_threshold_sweep.argtypes = [_vp, _vp, _vp, _vp, _i64, _vp, _i32, _vp]
        L.oracle_cascade.restype = _i64
        L.oracle_cascade.argtypes = [_vp, _vp, _vp, _vp, _i64, _i64, _vp, _vp,
                                     _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        _LIB = L
    return _LIB


def _p(a: np.ndarray):
    return a.ctypes.data_as(_vp) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ------------------------------------------------------------------ wrappers

def area_weights(n_in: int, n_out: int):
    w = np.zeros((n_out, n_in), np.int64)
    p = lib().oracle_area_weights(n_in, n_out, _p(w))
    return w, int(p)


def area_den(H, W, Ho, Wo) -> int:
    return int(lib().oracle_area_den(H, W, Ho, Wo))


def area_sums(frame: np.ndarray, Ho: int, Wo: int) -> np.ndarray:
    f = _c(frame, np.uint8)
    H, W = f.shape[0], f.shape[1]
    S = np.zeros((Ho, Wo, 3), np.int64)
    lib().oracle_area_sums(_p(f), H, W, Ho, Wo, _p(S))
    return S


def global_mse(a: np.ndarray, b: np.ndarray, den: int):
    a, b = _c(a, np.int64), _c(b, np.int64)
    E = np.zeros(1, np.int64)
    m = lib().oracle_global_mse(_p(a), _p(b), a.shape[0], a.shape[1], den, _p(E))
    return m, int(E[0])


def global_metric(a: np.ndarray, b: np.ndarray, den: int, metric: int):
    """Whole-image metric of frame sums a against compared sums b: MSE, SAD,
    NRMSE or -PSNR (metric 0..3); returns (value, sum of squared differences)."""
    a, b = _c(a, np.int64), _c(b, np.int64)
    E = np.zeros(1, np.int64)
    m = lib().oracle_global_metric(int(metric), _p(a), _p(b), a.shape[0], a.shape[1], den, _p(E))
    return m, int(E[0])


def blocked_metric(a, b, den, grid, w, bias, metric: int):
    """Blocked detector score bias + sum_k w_k m_k with the per-block metric m_k
    (MSE, SAD or NRMSE; NaN for PSNR); returns (score, m)."""
    a, b = _c(a, np.int64), _c(b, np.int64)
    w = _c(w, np.float32)
    m = np.zeros(grid[0] * grid[1], np.float64)
    z = lib().oracle_blocked_metric(int(metric), _p(a), _p(b), a.shape[0], a.shape[1], den,
                                    grid[0], grid[1], _p(w), float(bias), _p(m))
    return z, m


def blocked_score(a, b, den, grid, w, bias):
    a, b = _c(a, np.int64), _c(b, np.int64)
    w = _c(w, np.float32)
    m = np.zeros(grid[0] * grid[1], np.float64)
    z = lib().oracle_blocked_score(_p(a), _p(b), a.shape[0], a.shape[1], den, grid[0], grid[1],
                                   _p(w), float(bias), _p(m))
    return z, m


def round_bf16(v: float) -> float:
    return lib().oracle_round_bf16(float(v))


def cnn_desc(spec) -> CnnDesc:
    d = CnnDesc()
    d.n_conv = len(spec.conv)
    for i, (co, p) in enumerate(zip(spec.conv, spec.pool)):
        d.conv_out[i] = co
        d.pool_after[i] = 1 if p else 0
    d.dense, d.in_h, d.in_w, d.bf16 = spec.dense, spec.in_h, spec.in_w, 1 if spec.bf16 else 0
    return d


def conv3x3(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """x [C][H][W], w [O][C][3][3], b [O] -> [O][H][W] (fp64)."""
    x, w, b = _c(x, np.float64), _c(w, np.float64), _c(b, np.float64)
    C, H, W = x.shape
    O = w.shape[0]
    out = np.zeros((O, H, W), np.float64)
    lib().oracle_conv3x3(_p(x), C, H, W, _p(w), _p(b), O, _p(out))
    return out


def cnn_logit(spec, blob: np.ndarray, S: np.ndarray, den: int, want_features=False,
              want_scale=False):
    """Logit of one image; optionally also the dense input and the logit's scale
    |b2| + sum_j |w2_j h_j|."""
    d = cnn_desc(spec)
    blob = _c(blob, np.float32)
    if blob.size != lib().oracle_cnn_blob_floats(ctypes.byref(d)):
        raise ValueError("weight blob size does not match the network")
    S = _c(S, np.int64)
    _, flat, _ = spec.shapes()
    feats = np.zeros(flat, np.float64) if want_features else None
    scale = np.zeros(1)
    z = lib().oracle_cnn_logit(ctypes.byref(d), _p(blob), _p(S), int(den), _p(feats), _p(scale))
    out = (z,) + ((feats,) if want_features else ()) + ((float(scale[0]),) if want_scale else ())
    return out if len(out) > 1 else z


def sigmoid(z: float) -> float:
    return lib().oracle_sigmoid(float(z))


def decide(p: float, c_low: float, c_high: float) -> int:
    return int(lib().oracle_decide(float(p), float(c_low), float(c_high)))


def make_cfg(wl, lr_w=None, ref_sums=None, **over) -> tuple:
    """Build a Cfg from a synth Workload; returns (cfg, keepalive list)."""
    keep = []
    c = Cfg()
    c.H, c.W = wl.video.h, wl.video.w
    c.Ho, c.Wo = wl.dd_h, wl.dd_w
    c.Hc, c.Wc = wl.cnn.in_h, wl.cnn.in_w
    c.ref_mode, c.delta = wl.ref_mode, wl.delta
    c.Gh, c.Gw = wl.grid
    if lr_w is not None:
        lw = _c(lr_w, np.float32)
        keep.append(lw)
        c.lr_w = lw.ctypes.data
    c.lr_b = wl.lr_bias
    if ref_sums is not None:
        rs = _c(ref_sums, np.int64)
        keep.append(rs)
        c.ref_sums = rs.ctypes.data
    c.delta_diff, c.c_low, c.c_high = wl.delta_diff, wl.c_low, wl.c_high
    c.check_stride = getattr(wl, "check_stride", 1)
    c.metric = getattr(wl, "metric", MSE)
    for k, v in over.items():
        setattr(c, k, v)
    return c, keep


def history(cfg: Cfg) -> int:
    """Frames before t0 whose sums and decisions a chunked run needs."""
    return int(lib().oracle_history(ctypes.byref(cfg)))


def cascade(cfg: Cfg, spec, blob, frames: np.ndarray, t0: int = 0, state=None):
    """Run the oracle cascade on frames [t0, t0+n); returns a dict of outputs
    and the new state (area sums and decisions of the last history(cfg)
    frames: delta for the earlier-frame detector, s - 1 for frame skipping)."""
    frames = _c(frames, np.uint8)
    n = frames.shape[0]
    d = cnn_desc(spec)
    blob = _c(blob, np.float32)
    D = history(cfg)
    cells = cfg.Ho * cfg.Wo * 3
    out = dict(score=np.zeros(n), fire=np.zeros(n, np.uint8), logit=np.zeros(n),
               prob=np.zeros(n), lscale=np.zeros(n), label=np.zeros(n, np.uint8),
               defer=np.zeros(n, np.uint8))
    sS = np.zeros((max(D, 1), cells), np.int64)
    sD = np.zeros(max(D, 1), np.uint8)
    inS, inD = (None, None) if state is None else (_c(state[0], np.int64), _c(state[1], np.uint8))
    fired = lib().oracle_cascade(ctypes.byref(cfg), ctypes.byref(d), _p(blob), _p(frames), n, t0,
                                 _p(inS), _p(inD), _p(out["score"]), _p(out["fire"]),
                                 _p(out["logit"]), _p(out["prob"]), _p(out["lscale"]),
                                 _p(out["label"]), _p(out["defer"]), _p(sS), _p(sD))
    if fired < 0:
        raise ValueError("oracle_cascade rejected its arguments")
    out["fired"] = int(fired)
    return out, (sS[:D].copy(), sD[:D].copy())


def threshold_sweep(score, conf, truth, deltas, *, ref_mode: int, delta: int, fp_target: float,
                    fn_target: float, t_mse: float, t_snn: float, t_full: float):
    """Threshold search of the cost-based optimizer on logged per-frame scores
    (oracle.cpp, oracle_threshold_sweep): one row per candidate delta_diff
    (structured array of SWEEP_ROW) and the index of the cheapest feasible
    one (-1 if none)."""
    score = _c(score, np.float64)
    conf = _c(conf, np.float32)
    truth = _c(truth, np.uint8)
    deltas = _c(deltas, np.float64)
    n, n_t = score.size, deltas.size
    if conf.size != n or truth.size != n:
        raise ValueError("score, conf and truth need one entry per frame")
    cfg = SweepCfg(ref_mode, delta, fp_target, fn_target, t_mse, t_snn, t_full)
    rows = np.zeros(n_t, SWEEP_ROW)
    best = lib().oracle_threshold_sweep(ctypes.byref(cfg), _p(score), _p(conf), _p(truth), n,
                                        _p(deltas), n_t, rows.ctypes.data)
    if best < -1:
        raise ValueError("oracle_threshold_sweep rejected its arguments")
    return rows, int(best)
