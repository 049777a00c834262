"""Shared helpers of the GPU parity tests: inputs, oracle runs and comparisons."""
from __future__ import annotations

import concurrent.futures
import math
import os

import numpy as np

import oracle
import synth
from synth import workloads as W

LOGIT_TOL = {True: 1e-3, False: 1e-5}   # bf16 / fp32 networks: max relative logit error
# -PSNR goes through log10, which the host library and the device round
# differently (each within a few ulp); every other score is bit-exact
PSNR_SCORE_TOL = 1e-13


def compare_scores(wl, g: np.ndarray, o: np.ndarray):
    """Detector scores of the GPU (g) against the oracle's (o): identical bits,
    except -PSNR within PSNR_SCORE_TOL (relative, infinities identical).  With
    PSNR no oracle score may lie within rounding of delta_diff, so that the
    fire flags are still pinned exactly."""
    if getattr(wl, "metric", W.MSE) != W.PSNR:
        assert np.array_equal(g, o, equal_nan=True), \
            f"scores differ at {np.flatnonzero(g != o)[:10]}"
        return
    same = (g == o) | (np.isnan(g) & np.isnan(o))
    fin = np.isfinite(g) & np.isfinite(o)
    diff = np.zeros(o.shape)
    diff[fin] = np.abs(g[fin] - o[fin])
    close = fin & (diff <= PSNR_SCORE_TOL * np.maximum(1.0, np.abs(o)))
    assert (same | close).all(), f"-PSNR scores differ at {np.flatnonzero(~(same | close))[:10]}"
    band = 2 * PSNR_SCORE_TOL * max(1.0, abs(wl.delta_diff))
    assert not (np.isfinite(o) & (np.abs(o - wl.delta_diff) <= band)).any(), \
        "a -PSNR score lies within rounding of delta_diff"


def logit_rel_err(g: np.ndarray, o: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """|g - o| / scale, scale = |b2| + sum_j |w2_j h_j| from the oracle: the error
    relative to the magnitude of the terms the output layer sums (equal to the
    plain relative error when they do not cancel).  This is the measure the
    tolerance is asserted on."""
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    if o.size == 0:
        return np.zeros(0)
    return np.abs(g - o) / np.maximum(np.asarray(scale, np.float64), 1e-300)


FLOOR_FRAC = 2.0 ** -10   # floored relative error: |g - o| / max(|o|, 2^-10 max_batch |o|)


class LogitErrors:
    """Worst logit errors of a test in three measures, side by side:
    - scale: |g - o| / (|b2| + sum_j |w2_j h_j|) (asserted against the tolerance);
    - plain: |g - o| / |o|;
    - floored: |g - o| / max(|o|, 2^-10 max |o| over the batch), with the
      number of logits whose denominator is the floor;
    plus the decision counts: `excluded` frames (an oracle confidence within
    1e-5 relative of c_low or c_high, and frames reusing their output) and
    `straddled` frames (outside that band, but the GPU and oracle logits lie on
    opposite sides of a threshold, so their decisions differ by the logit error
    alone; also excluded with the frames reusing their output)."""

    def __init__(self):
        self.n = 0
        self.scale = self.plain = self.floored = 0.0
        self.floor_hits = self.excluded = self.straddled = 0

    def add(self, g, o, scale):
        g = np.asarray(g, np.float64).reshape(-1)
        o = np.asarray(o, np.float64).reshape(-1)
        if o.size == 0:
            return self
        d = np.abs(g - o)
        self.n += int(o.size)
        self.scale = max(self.scale, float(logit_rel_err(g, o, scale).max()))
        ao = np.abs(o)
        with np.errstate(divide="ignore", invalid="ignore"):
            plain = np.where(ao > 0, d / np.where(ao > 0, ao, 1.0), np.where(d > 0, np.inf, 0.0))
        self.plain = max(self.plain, float(plain.max()))
        floor = FLOOR_FRAC * float(ao.max())
        den = np.maximum(ao, floor)
        with np.errstate(divide="ignore", invalid="ignore"):
            fl = np.where(den > 0, d / np.where(den > 0, den, 1.0), np.where(d > 0, np.inf, 0.0))
        self.floored = max(self.floored, float(fl.max()))
        self.floor_hits += int(np.sum(ao < floor))
        return self

    def merge(self, other: "LogitErrors"):
        self.n += other.n
        self.scale = max(self.scale, other.scale)
        self.plain = max(self.plain, other.plain)
        self.floored = max(self.floored, other.floored)
        self.floor_hits += other.floor_hits
        self.excluded += other.excluded
        self.straddled += other.straddled
        return self

    def as_dict(self):
        return dict(logits=self.n, max_logit_rel_scale=self.scale, max_logit_rel_plain=self.plain,
                    max_logit_rel_floored=self.floored, floor_hits=self.floor_hits,
                    excluded=self.excluded, straddled=self.straddled)

    def __repr__(self):
        return (f"logit errors over {self.n}: scale-relative {self.scale:.3g}, plain relative "
                f"{self.plain:.3g}, floored {self.floored:.3g} ({self.floor_hits} at the floor); "
                f"decisions excluded {self.excluded}, straddled {self.straddled}")


DECISION_BAND = 1e-5   # a confidence within 1e-5 relative of a threshold is not compared


def decision_excluded(p_oracle: float, c_low: float, c_high: float) -> bool:
    """A fired frame's decision is not pinned when the oracle's confidence lies
    within 1e-5 relative of c_low or c_high."""
    return any(abs(p_oracle - c) <= DECISION_BAND * c for c in (c_low, c_high))


def decision_of_logit(z: float, c_low: float, c_high: float) -> int:
    """label | defer << 1 that the decision rule gives a logit (the oracle's
    sigmoid and rule, in fp64)."""
    return oracle.decide(oracle.sigmoid(float(z)), c_low, c_high)


def oracle_decision(z: float, c_low: float, c_high: float) -> int:
    return oracle.decide(oracle.sigmoid(z), c_low, c_high)


def lr_weights_for(wl):
    return synth.lr_weights(wl.grid[0] * wl.grid[1], wl.weight_seed, wl.lr_bias)[0]


def compare_cascade(wl, gpu: dict, ref: dict, t0: int = 0, state_excluded=None):
    """Element-by-element comparison of a GPU cascade run with the oracle's.

    gpu / ref: dicts of numpy arrays score, fire, logit, label, defer over the
    same frames (ref also prob and lscale).  Scores (see compare_scores) and
    fire flags must be bit-identical; logits within the network's tolerance
    (scale-relative; the plain and floored relative errors are reported beside
    it); labels and defer flags identical outside the excluded frames: fired
    frames whose oracle confidence lies within 1e-5 relative of c_low or
    c_high, fired frames whose GPU and oracle logits straddle a threshold (the
    GPU's decision must then be the rule's decision on its own logit), and
    frames reusing their output.  Returns the report dict."""
    n = len(ref["fire"])
    s = max(getattr(wl, "check_stride", 1), 1)
    compare_scores(wl, gpu["score"], ref["score"])
    assert np.array_equal(gpu["fire"], ref["fire"]), "fire flags differ"
    fired = np.flatnonzero(ref["fire"])
    tol = LOGIT_TOL[wl.cnn.bf16]
    errs = LogitErrors().add(gpu["logit"][fired], ref["logit"][fired], ref["lscale"][fired])
    assert np.isnan(gpu["logit"][ref["fire"] == 0]).all()
    assert errs.scale <= tol, f"max logit rel err {errs.scale:.3g} > {tol} ({errs})"
    excluded = np.zeros(n, bool)
    for u in range(n):
        if (t0 + u) % s:  # not checked: inherits from its checked frame
            if u >= (t0 + u) % s:
                excluded[u] = excluded[u - (t0 + u) % s]
            elif state_excluded is not None:
                excluded[u] = state_excluded[u]
        elif ref["fire"][u]:
            if decision_excluded(ref["prob"][u], wl.c_low, wl.c_high):
                excluded[u] = True
            else:
                dg = decision_of_logit(gpu["logit"][u], wl.c_low, wl.c_high)
                if dg != decision_of_logit(ref["logit"][u], wl.c_low, wl.c_high):
                    excluded[u] = True
                    errs.straddled += 1
                    got = int(gpu["label"][u]) | (int(gpu["defer"][u]) << 1)
                    assert got == dg, f"frame {t0 + u}: decision {got}, its logit gives {dg}"
        elif wl.ref_mode == 0:
            if u >= wl.delta:
                excluded[u] = excluded[u - wl.delta]
            elif state_excluded is not None:
                excluded[u] = state_excluded[u]
    errs.excluded = int(excluded.sum())
    keep = ~excluded
    bad = np.flatnonzero(keep & ((gpu["label"] != ref["label"]) | (gpu["defer"] != ref["defer"])))
    assert bad.size == 0, f"labels differ at frames {bad[:10] + t0}"
    rep = dict(frames=n, fired=int(fired.size), max_logit_rel=errs.scale,
               near_delta=int(np.sum(np.abs(ref["score"] - wl.delta_diff) <=
                                     1e-5 * max(abs(wl.delta_diff), 1.0))))
    rep.update(errs.as_dict())
    return rep


# ------------------------------------------- sampled frames of long runs

SAMPLE_THREADS = min(16, os.cpu_count() or 1)


def oracle_frame(wl, v, blob, lr, ref_sums_o, t):
    """Oracle score of frame t and, when it fires, its logit, scale and decision
    (a frame between checks has score NaN and does not fire)."""
    if t % max(getattr(wl, "check_stride", 1), 1):
        return dict(score=math.nan, fire=False)
    den = oracle.area_den(wl.video.h, wl.video.w, wl.dd_h, wl.dd_w)
    cur = oracle.area_sums(v.frame(t), wl.dd_h, wl.dd_w)
    if wl.ref_mode == W.PREV:
        if t < wl.delta:
            score = math.inf
        else:
            ref = oracle.area_sums(v.frame(t - wl.delta), wl.dd_h, wl.dd_w)
            score = (oracle.global_mse(cur, ref, den)[0] if wl.grid == (1, 1) else
                     oracle.blocked_score(cur, ref, den, wl.grid, lr, wl.lr_bias)[0])
    else:
        score = (oracle.global_mse(cur, ref_sums_o, den)[0] if wl.grid == (1, 1) else
                 oracle.blocked_score(cur, ref_sums_o, den, wl.grid, lr, wl.lr_bias)[0])
    fires = score > wl.delta_diff or (wl.ref_mode == W.PREV and t < wl.delta)
    out = dict(score=score, fire=fires)
    if fires:
        Sc = oracle.area_sums(v.frame(t), wl.cnn.in_h, wl.cnn.in_w)
        den_c = oracle.area_den(wl.video.h, wl.video.w, wl.cnn.in_h, wl.cnn.in_w)
        z, sc = oracle.cnn_logit(wl.cnn, blob, Sc, den_c, want_scale=True)
        out.update(logit=z, scale=sc, dec=oracle.decide(oracle.sigmoid(z), wl.c_low, wl.c_high))
    return out


def check_properties(wl, g, t0=0):
    """Properties of a run over frames [t0, t0 + n) that hold at any size."""
    n = len(g["fire"])
    t = np.arange(t0, t0 + n)
    s = max(getattr(wl, "check_stride", 1), 1)
    checked = t % s == 0
    fire = g["fire"].astype(bool)
    assert not fire[~checked].any() and np.isnan(g["score"][~checked]).all()
    u = np.flatnonzero(~checked)
    src = u - t[u] % s             # the checked frame a skipped frame copies
    ok = src >= 0
    assert (g["label"][u[ok]] == g["label"][src[ok]]).all()
    assert (g["defer"][u[ok]] == g["defer"][src[ok]]).all()
    if wl.ref_mode == W.PREV:
        assert fire[checked & (t < wl.delta)].all()
        assert np.isfinite(g["score"][checked & (t >= wl.delta)]).all()
        nf = np.flatnonzero(~fire & checked)
        nf = nf[nf >= wl.delta]
        assert (g["label"][nf] == g["label"][nf - wl.delta]).all()
        assert (g["defer"][nf] == g["defer"][nf - wl.delta]).all()
    else:
        nf = ~fire & checked
        assert ((g["label"][nf] == 0) & (g["defer"][nf] == 0)).all()
    assert np.isnan(g["logit"][~fire]).all() and not np.isnan(g["logit"][fire]).any()
    assert not (g["label"].astype(bool) & g["defer"].astype(bool)).any()


def check_samples(wl, v, blob, lr, ref_o, g, ts, t0=0) -> LogitErrors:
    """Frames ts of a run over [t0, ...) against the oracle, one by one: scores
    and fire flags exactly, logits within the tolerance (the three error
    measures are returned), decisions as in compare_cascade (a sampled frame's
    decision is compared where it fired).  The oracle frames are computed on a
    thread pool: the oracle library's calls release the GIL, and so does most
    of the numpy frame rendering (no process is forked from one that has
    initialised the GPU)."""
    tol = LOGIT_TOL[wl.cnn.bf16]
    oracle.lib()  # loaded once, before the threads use it
    with concurrent.futures.ThreadPoolExecutor(max_workers=SAMPLE_THREADS) as ex:
        outs = list(ex.map(lambda t: oracle_frame(wl, v, blob, lr, ref_o, int(t)), ts))
    gz, oz, sc = [], [], []
    for t, o in zip(ts, outs):
        u = int(t) - t0
        assert g["score"][u] == o["score"] or (math.isnan(g["score"][u]) and math.isnan(o["score"])), \
            (t, g["score"][u], o["score"])
        assert bool(g["fire"][u]) == o["fire"], t
        if o["fire"]:
            err = float(logit_rel_err(np.array([g["logit"][u]]), np.array([o["logit"]]),
                                      np.array([o["scale"]]))[0])
            assert err <= tol, (t, g["logit"][u], o["logit"], err)
            gz.append(g["logit"][u])
            oz.append(o["logit"])
            sc.append(o["scale"])
    errs = LogitErrors().add(np.array(gz), np.array(oz), np.array(sc))
    for t, o in zip(ts, outs):
        u = int(t) - t0
        if not o["fire"]:
            continue
        dec = int(g["label"][u]) | (int(g["defer"][u]) << 1)
        if decision_excluded(oracle.sigmoid(o["logit"]), wl.c_low, wl.c_high):
            errs.excluded += 1
            continue
        dg = decision_of_logit(g["logit"][u], wl.c_low, wl.c_high)
        if dg != o["dec"]:
            errs.straddled += 1
            assert dec == dg, (t, dec, dg)
        else:
            assert dec == o["dec"], (t, dec, o["dec"])
    return errs
