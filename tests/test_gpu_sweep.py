"""GPU threshold search (Sec. 6.3 step 3, cost model of Sec. 6.2) against the
oracle, row by row and bit for bit: counts, thresholds, rates and costs.

Inputs are seeded synthetic logs (scores with forced frames, confidences with
ties, labels) and, for a real video window, the scores and confidences the
oracle's own cascade computes; none comes from the GPU path.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_1703_02529_amd as nsc
import synth
from synth import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"
COSTS = dict(t_mse=2.0e-7, t_snn=8.0e-5, t_full=1.25e-2)
FIELDS = ("delta", "c_low", "c_high", "f_m", "f_c", "cost", "fired", "deferred", "fn_dd", "fp_dd",
          "fn_cnn", "fp_cnn", "positives", "negatives", "feasible")


def gpu_sweep(score, conf, truth, deltas, ref_mode, delta, fp_t, fn_t, costs=COSTS):
    cfg = nsc.SweepCfg(ref_mode, delta, fp_t, fn_t, costs["t_mse"], costs["t_snn"], costs["t_full"])
    n_t = len(deltas)
    rows = torch.zeros(n_t * nsc.SWEEP_ROW_BYTES, dtype=torch.uint8, device=DEV)
    best = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    nsc.nsc_threshold_sweep(cfg, torch.from_numpy(np.ascontiguousarray(score, np.float64)).to(DEV),
                            torch.from_numpy(np.ascontiguousarray(conf, np.float32)).to(DEV),
                            torch.from_numpy(np.ascontiguousarray(truth, np.uint8)).to(DEV),
                            torch.from_numpy(np.ascontiguousarray(deltas, np.float64)).to(DEV),
                            rows, best)
    got = rows.cpu().numpy().view(oracle.SWEEP_ROW)  # same field order and widths
    return got, int(best.item())


def check(score, conf, truth, deltas, ref_mode, delta, fp_t, fn_t):
    got, gbest = gpu_sweep(score, conf, truth, deltas, ref_mode, delta, fp_t, fn_t)
    want, wbest = oracle.threshold_sweep(score, conf, truth, deltas, ref_mode=ref_mode, delta=delta,
                                         fp_target=fp_t, fn_target=fn_t, **COSTS)
    for k in range(len(deltas)):
        for f in FIELDS:
            g, w = got[k][f], want[k][f]
            assert g == w or (isinstance(w, float) and math.isnan(w) and math.isnan(g)), \
                (k, f, g, w, got[k], want[k])
    assert gbest == wbest
    return want, wbest


def synthetic_log(n, seed, p_obj=0.25, ties=False):
    """Scores of a noisy detector (higher with the object), confidences of a
    noisy classifier, labels in episodes."""
    r = np.random.default_rng([seed, 91])
    truth = np.zeros(n, np.uint8)
    t = 0
    while t < n:
        on = r.random() < p_obj
        ln = int(r.integers(5, 60))
        truth[t:t + ln] = on
        t += ln
    score = np.abs(r.normal(8.0, 4.0, n)) + 20.0 * truth * r.random(n)
    conf = 1.0 / (1.0 + np.exp(-(r.normal(0, 1.5, n) + 3.0 * (truth - 0.5))))
    conf = conf.astype(np.float32)
    if ties:
        conf = (np.round(conf * 16) / 16).astype(np.float32)
    return score, conf, truth


@pytest.mark.parametrize("n,seed,ref_mode,delta,ties", [
    (1, 0, W.FIXED, 1, False), (7, 1, W.PREV, 3, True), (1000, 2, W.PREV, 1, False),
    (5000, 3, W.PREV, 15, True), (5000, 4, W.FIXED, 1, True), (65537, 5, W.PREV, 30, False)])
def test_sweep_synthetic_logs(n, seed, ref_mode, delta, ties):
    score, conf, truth = synthetic_log(n, seed, ties=ties)
    if ref_mode == W.PREV:
        score[:delta] = np.inf
    qs = np.quantile(score[np.isfinite(score)], np.linspace(0, 1, 33)) if n > 1 else score[:1]
    deltas = np.concatenate([[-np.inf, np.inf], qs, [qs[5] if n > 1 else 0.0]])
    for fp_t, fn_t in ((0.01, 0.01), (0.05, 0.02), (0.0, 0.5), (1.0, 1.0)):
        check(score, conf, truth, deltas, ref_mode, delta, fp_t, fn_t)


def test_sweep_extremes():
    # confidences exactly 0 and 1 (and -0), every frame with the object, none
    n = 300
    r = np.random.default_rng(3)
    score = r.uniform(0, 5, n)
    conf = r.choice(np.array([0.0, -0.0, 1.0, 0.5], np.float32), n)
    for truth in (np.ones(n, np.uint8), np.zeros(n, np.uint8), (r.random(n) < 0.5).astype(np.uint8)):
        check(score, conf, truth, [-np.inf, 1.0, 2.5, np.inf], W.PREV, 2, 0.1, 0.1)


def test_sweep_on_oracle_cascade_outputs():
    """A window of the 640x480 video around an object episode: the oracle's
    cascade (delta_diff = -inf, every frame through the CNN) gives the scores
    and confidences; labels are the generator's ground truth."""
    wl = W.VGA
    v = synth.Video(wl.video)
    occ = np.flatnonzero(v.occupied)
    t0 = max(0, int(occ[0]) - 60)
    n = 240
    frames = v.frames(t0, t0 + n)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    cfg, keep = oracle.make_cfg(wl.replace(delta_diff=-math.inf))
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames, t0=0)
    score = out["score"]
    conf = out["prob"].astype(np.float32)
    truth = v.occupied[t0:t0 + n].astype(np.uint8)
    finite = score[np.isfinite(score)]
    deltas = np.concatenate([[-np.inf], np.quantile(finite, np.linspace(0, 1, 17)), [np.inf]])
    want, best = check(score, conf, truth, deltas, W.PREV, wl.delta, 0.05, 0.05)
    print(dict(frames=n, positives=int(want[0]["positives"]), best=best,
               feasible=int(want["feasible"].sum())))
