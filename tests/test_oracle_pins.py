"""Pins of the fp64 oracle against facts fixed outside it.

Each test checks the oracle against something other than itself: a hand-worked
fixture, a closed form, an invariant, brute force on tiny inputs, or an
independent library routine (torch CPU, numpy) for a special case.
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth
from synth import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(1234)


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


# ------------------------------------------------------------ area averaging

def test_area_5to2_hand_computed():
    rows = _read_golden("area_5to2.txt")
    frame = np.zeros((5, 5, 3), np.uint8)
    for j in range(5):
        for i in range(5):
            frame[j, i] = (10 * j + i, 1, 0)
    w, p = oracle.area_weights(5, 2)
    assert p == 5
    den = oracle.area_den(5, 5, 2, 2)
    S = oracle.area_sums(frame, 2, 2)
    for r in rows:
        if r[0] == "den":
            assert den == int(r[1])
        elif r[0] == "weights0":
            assert list(w[0]) == [int(x) for x in r[1:]]
        elif r[0] == "weights1":
            assert list(w[1]) == [int(x) for x in r[1:]]
        elif r[0] == "S":
            Y, X = int(r[1]), int(r[2])
            assert list(S[Y, X]) == [int(x) for x in r[3:]]


@pytest.mark.parametrize("n_in,n_out", [(640, 50), (480, 50), (1280, 50), (720, 50), (1280, 100),
                                        (720, 100), (1920, 100), (1080, 100), (100, 50), (7, 3),
                                        (13, 13)])
def test_area_weights_partition(n_in, n_out):
    """Every output cell receives p input units and every input pixel gives q units."""
    w, p = oracle.area_weights(n_in, n_out)
    g = math.gcd(n_in, n_out)
    assert p == n_in // g
    assert (w.sum(axis=1) == n_in // g).all()
    assert (w.sum(axis=0) == n_out // g).all()
    assert (w >= 0).all()


@pytest.mark.parametrize("H,W,Ho,Wo", [(12, 20, 3, 8), (15, 10, 6, 4), (9, 9, 9, 9), (16, 24, 5, 7)])
def test_area_sums_equal_replicated_block_sums(H, W, Ho, Wo):
    """Exact area averaging equals: replicate each pixel q_y x q_x times, then sum
    p_y x p_x blocks (a textbook definition, computed here with numpy)."""
    f = rng.integers(0, 256, size=(H, W, 3), dtype=np.uint8)
    gy, gx = math.gcd(H, Ho), math.gcd(W, Wo)
    py, qy, px, qx = H // gy, Ho // gy, W // gx, Wo // gx
    up = np.repeat(np.repeat(f.astype(np.int64), qy, axis=0), qx, axis=1)
    blocks = up.reshape(Ho, py, Wo, px, 3).sum(axis=(1, 3))
    assert (oracle.area_sums(f, Ho, Wo) == blocks).all()
    assert oracle.area_den(H, W, Ho, Wo) == py * px


def test_area_integer_ratio_is_box_sum():
    f = rng.integers(0, 256, size=(100, 100, 3), dtype=np.uint8)
    box = f.astype(np.int64).reshape(50, 2, 50, 2, 3).sum(axis=(1, 3))
    assert (oracle.area_sums(f, 50, 50) == box).all()
    assert oracle.area_den(100, 100, 50, 50) == 4


@pytest.mark.parametrize("H,W,Ho,Wo", [(480, 640, 50, 50), (720, 1280, 100, 100), (33, 17, 5, 4)])
def test_constant_frame(H, W, Ho, Wo):
    v = 173
    f = np.full((H, W, 3), v, np.uint8)
    den = oracle.area_den(H, W, Ho, Wo)
    assert (oracle.area_sums(f, Ho, Wo) == den * v).all()


def test_nesting_100_to_50():
    """2x2 sums of the 100-grid give exactly the 50-grid area average."""
    f = rng.integers(0, 256, size=(720, 1280, 3), dtype=np.uint8)
    S100 = oracle.area_sums(f, 100, 100)
    S50 = oracle.area_sums(f, 50, 50)
    d100, d50 = oracle.area_den(720, 1280, 100, 100), oracle.area_den(720, 1280, 50, 50)
    nest = S100.reshape(50, 2, 50, 2, 3).sum(axis=(1, 3))
    # value equality as exact rationals: nest / (4 d100) == S50 / d50
    assert (nest * d50 == S50 * 4 * d100).all()


# ------------------------------------------------------- difference detector

def test_mse_hand_computed_4x4():
    rows = _read_golden("mse_4x4.txt")
    a = np.full((4, 4, 3), 10, np.uint8)
    b = a.copy()
    b[0, 0] = (13, 14, 10)
    b[3, 3] = (10, 10, 0)
    for r in rows:
        g = int(r[1])
        den = oracle.area_den(4, 4, g, g)
        m, E = oracle.global_mse(oracle.area_sums(a, g, g), oracle.area_sums(b, g, g), den)
        assert E == int(r[4])
        assert m == pytest.approx(float(r[6]), rel=1e-15)
    assert float(rows[0][6]) == 125 / 48 and float(rows[1][6]) == 125 / 192


def test_identical_frames_mse_zero():
    f = rng.integers(0, 256, size=(480, 640, 3), dtype=np.uint8)
    S = oracle.area_sums(f, 50, 50)
    m, E = oracle.global_mse(S, S, oracle.area_den(480, 640, 50, 50))
    assert m == 0.0 and E == 0


@pytest.mark.parametrize("k", [1, 3, 17])
def test_mse_of_constant_offset(k):
    """MSE(F, F + k) = k^2 exactly when nothing clips."""
    f = rng.integers(20, 200, size=(480, 640, 3), dtype=np.uint8)
    den = oracle.area_den(480, 640, 50, 50)
    m, _ = oracle.global_mse(oracle.area_sums(f, 50, 50), oracle.area_sums(f + k, 50, 50), den)
    assert m == k * k


def test_blocked_mean_equals_global_and_unit_grid():
    f = rng.integers(0, 256, size=(100, 100, 3), dtype=np.uint8)
    g = rng.integers(0, 256, size=(100, 100, 3), dtype=np.uint8)
    den = oracle.area_den(100, 100, 100, 100)
    a, b = oracle.area_sums(f, 100, 100), oracle.area_sums(g, 100, 100)
    mse, _ = oracle.global_mse(a, b, den)
    # equal-size 10x10 blocks: the mean of the block MSEs is the global MSE
    z, m = oracle.blocked_score(a, b, den, (10, 10), np.zeros(100, np.float32), 0.0)
    assert m.mean() == pytest.approx(mse, rel=1e-13)
    assert z == 0.0
    # 1x1 grid with w = 1, b = 0 is the global detector
    z1, _ = oracle.blocked_score(a, b, den, (1, 1), np.ones(1, np.float32), 0.0)
    assert z1 == pytest.approx(mse, rel=1e-15)
    # bias and weights enter linearly
    w = rng.standard_normal(100).astype(np.float32)
    zb, mb = oracle.blocked_score(a, b, den, (10, 10), w, -2.0)
    assert zb == pytest.approx(-2.0 + float(np.dot(w.astype(np.float64), mb)), rel=1e-12)


def test_blocked_uneven_grid_bounds():
    """Block k covers rows floor(by*Ho/Gh)..floor((by+1)*Ho/Gh): checked by brute force."""
    a = rng.integers(0, 5000, size=(7, 11, 3)).astype(np.int64)
    b = rng.integers(0, 5000, size=(7, 11, 3)).astype(np.int64)
    den = 3
    z, m = oracle.blocked_score(a, b, den, (3, 4), np.ones(12, np.float32), 0.0)
    for by in range(3):
        for bx in range(4):
            ys = slice(by * 7 // 3, (by + 1) * 7 // 3)
            xs = slice(bx * 11 // 4, (bx + 1) * 11 // 4)
            d = (a[ys, xs] - b[ys, xs]).astype(np.float64) / den
            assert m[by * 4 + bx] == pytest.approx((d ** 2).mean(), rel=1e-13)


# --------------------------------------------- alternative detector metrics

def test_metrics_hand_computed_4x4():
    """SAD, NRMSE and PSNR of the worked 4x4 example, at both grids."""
    rows = _read_golden("metrics_4x4.txt")
    r = np.full((4, 4, 3), 10, np.uint8)
    f = r.copy()
    f[0, 0] = (13, 14, 10)
    f[3, 3] = (10, 10, 0)
    for row in rows:
        g = int(row[1])
        den = oracle.area_den(4, 4, g, g)
        a, b = oracle.area_sums(f, g, g), oracle.area_sums(r, g, g)
        assert oracle.global_metric(a, b, den, oracle.SAD)[0] == float(row[3])
        assert oracle.global_metric(a, b, den, oracle.NRMSE)[0] == pytest.approx(float(row[5]),
                                                                                 rel=1e-15)
        assert oracle.global_metric(a, b, den, oracle.PSNR)[0] == pytest.approx(-float(row[7]),
                                                                                rel=1e-15)
        # the MSE through the same entry point is the MSE
        assert oracle.global_metric(a, b, den, oracle.MSE)[0] == oracle.global_mse(a, b, den)[0]
    # NRMSE is relative to the compared frame: swapping the frames changes it
    # (sum of F's squares is 45*100 + 13^2 + 14^2 + 0 = 4865)
    a, b = oracle.area_sums(f, 4, 4), oracle.area_sums(r, 4, 4)
    assert oracle.global_metric(b, a, 1, oracle.NRMSE)[0] == pytest.approx(math.sqrt(125 / 4865),
                                                                           rel=1e-15)
    assert oracle.global_metric(b, a, 1, oracle.SAD)[0] == 17.0


@pytest.mark.parametrize("k", [1, 3, 51])
def test_metrics_of_constant_offset(k):
    """A uniform brightness change of k levels (no clipping): SAD = N k,
    PSNR = 20 log10(255 / k), and NRMSE = k / v over a uniform image of v."""
    den = oracle.area_den(480, 640, 50, 50)
    N = 50 * 50 * 3
    f = rng.integers(20, 200, size=(480, 640, 3), dtype=np.uint8)
    a, b = oracle.area_sums(f + k, 50, 50), oracle.area_sums(f, 50, 50)
    assert oracle.global_metric(a, b, den, oracle.SAD)[0] == N * k
    assert -oracle.global_metric(a, b, den, oracle.PSNR)[0] == pytest.approx(
        20 * math.log10(255 / k), rel=1e-14)
    u = np.full((480, 640, 3), 120, np.uint8)
    nr = oracle.global_metric(oracle.area_sums(u + k, 50, 50), oracle.area_sums(u, 50, 50), den,
                              oracle.NRMSE)[0]
    assert nr == pytest.approx(k / 120, rel=1e-15)
    if k == 51:  # a fifth of the range: 20 log10(5)
        assert -oracle.global_metric(a, b, den, oracle.PSNR)[0] == pytest.approx(
            13.979400086720377, rel=1e-15)


def test_metrics_special_cases():
    """Identical images, an all-zero compared image, and the PSNR of MSE = 1."""
    den = oracle.area_den(480, 640, 50, 50)
    f = rng.integers(0, 256, size=(480, 640, 3), dtype=np.uint8)
    S = oracle.area_sums(f, 50, 50)
    assert oracle.global_metric(S, S, den, oracle.SAD)[0] == 0.0
    assert oracle.global_metric(S, S, den, oracle.NRMSE)[0] == 0.0
    assert oracle.global_metric(S, S, den, oracle.PSNR)[0] == -math.inf
    Z = np.zeros_like(S)
    assert oracle.global_metric(S, Z, den, oracle.NRMSE)[0] == math.inf
    assert oracle.global_metric(Z, Z, den, oracle.NRMSE)[0] == 0.0
    # a black frame compared with a non-black one is off by all of it
    assert oracle.global_metric(Z, S, den, oracle.NRMSE)[0] == 1.0
    # MSE = 1 (every value one level off): PSNR = 20 log10(255) = 48.1308... dB
    one = np.ones((2, 2, 3), np.int64)
    assert -oracle.global_metric(one, 0 * one, 1, oracle.PSNR)[0] == pytest.approx(
        48.130803608679102, rel=1e-15)


def test_metrics_bounds_and_equality_cases():
    """(SAD / N)^2 <= MSE (Cauchy-Schwarz), with equality iff every |d| is equal;
    the reverse triangle inequality bounds NRMSE below; -PSNR rises with MSE."""
    N = 30 * 40 * 3
    for seed in range(20):
        r = np.random.default_rng(seed)
        den = int(r.integers(1, 50))
        b = r.integers(0, 255 * den + 1, size=(30, 40, 3)).astype(np.int64)
        a = r.integers(0, 255 * den + 1, size=(30, 40, 3)).astype(np.int64)
        mse = oracle.global_metric(a, b, den, oracle.MSE)[0]
        sad = oracle.global_metric(a, b, den, oracle.SAD)[0]
        nr = oracle.global_metric(a, b, den, oracle.NRMSE)[0]
        assert (sad / N) ** 2 <= mse * (1 + 1e-12)
        na, nb = np.linalg.norm(a.astype(np.float64)), np.linalg.norm(b.astype(np.float64))
        assert abs(na / nb - 1) <= nr * (1 + 1e-12)
        # equal magnitudes, mixed signs
        k = int(r.integers(1, 9)) * den
        sign = np.where(r.random((30, 40, 3)) < 0.5, -1, 1)
        c = b + k * sign
        assert oracle.global_metric(c, b, den, oracle.SAD)[0] == N * (k // den)
        assert oracle.global_metric(c, b, den, oracle.MSE)[0] == (k // den) ** 2
        # -PSNR is increasing in the MSE
        m2 = oracle.global_metric(2 * a - b, b, den, oracle.MSE)[0]  # differences doubled
        p1 = oracle.global_metric(a, b, den, oracle.PSNR)[0]
        p2 = oracle.global_metric(2 * a - b, b, den, oracle.PSNR)[0]
        assert m2 == pytest.approx(4 * mse, rel=1e-14)
        assert p2 == pytest.approx(p1 + 20 * math.log10(2), rel=1e-13)


def test_blocked_metrics_brute_force():
    """Per-block SAD and NRMSE on an uneven 3x4 grid, block by block; a 1x1 grid
    with weight 1 and bias 0 is the global metric; PSNR is not blocked."""
    a = rng.integers(0, 5000, size=(7, 11, 3)).astype(np.int64)
    b = rng.integers(1, 5000, size=(7, 11, 3)).astype(np.int64)
    den = 3
    w = rng.standard_normal(12).astype(np.float32)
    for metric in (oracle.SAD, oracle.NRMSE):
        z, m = oracle.blocked_metric(a, b, den, (3, 4), w, 0.25, metric)
        zz = 0.25
        for by in range(3):
            for bx in range(4):
                ys = slice(by * 7 // 3, (by + 1) * 7 // 3)
                xs = slice(bx * 11 // 4, (bx + 1) * 11 // 4)
                d = (a[ys, xs] - b[ys, xs]).astype(np.float64)
                exp = (np.abs(d).sum() / den if metric == oracle.SAD else
                       math.sqrt((d ** 2).sum() / (b[ys, xs].astype(np.float64) ** 2).sum()))
                assert m[by * 4 + bx] == pytest.approx(exp, rel=1e-13)
                zz += float(w[by * 4 + bx]) * m[by * 4 + bx]
        assert z == pytest.approx(zz, rel=1e-12, abs=1e-9)
        z1, _ = oracle.blocked_metric(a, b, den, (1, 1), np.ones(1, np.float32), 0.0, metric)
        assert z1 == oracle.global_metric(a, b, den, metric)[0]
    assert math.isnan(oracle.blocked_metric(a, b, den, (3, 4), w, 0.0, oracle.PSNR)[0])


def test_cascade_psnr_fires_like_mse_at_the_matching_threshold():
    """-PSNR > d  <=>  MSE > 255^2 10^(d/10): the PSNR detector fires on the same
    frames as the MSE detector at the matching threshold (frames within rounding
    of it aside); with every metric an unchanged frame never fires."""
    wl = _tiny_fast()
    v, blob = _small(wl, 300)
    frames = v.frames(200, 500)
    for d in (-35.0, -30.0, -25.0):
        cfg_p, _ = oracle.make_cfg(wl.replace(delta_diff=d), metric=oracle.PSNR)
        out_p, _ = oracle.cascade(cfg_p, wl.cnn, blob, frames)
        m_thr = 65025.0 * 10 ** (d / 10)
        cfg_m, _ = oracle.make_cfg(wl.replace(delta_diff=m_thr))
        out_m, _ = oracle.cascade(cfg_m, wl.cnn, blob, frames)
        near = np.abs(out_m["score"] - m_thr) <= 1e-9 * m_thr
        assert not near.any()
        assert 0 < out_p["fire"].sum() < len(frames)
        for k in ("fire", "label", "defer"):
            assert (out_p[k] == out_m[k]).all()
    still = np.repeat(frames[:1], 6, axis=0)
    for metric in (oracle.SAD, oracle.NRMSE, oracle.PSNR):
        cfg, _ = oracle.make_cfg(wl.replace(delta_diff=0.0), metric=metric)
        out, _ = oracle.cascade(cfg, wl.cnn, blob, still)
        assert list(np.flatnonzero(out["fire"])) == [0]   # only the forced first frame
    cfg, _ = oracle.make_cfg(wl.replace(grid=(2, 2)), lr_w=np.ones(4, np.float32),
                             metric=oracle.PSNR)
    with pytest.raises(ValueError):
        oracle.cascade(cfg, wl.cnn, blob, frames[:5])


# --------------------------------------------------------------- CNN pieces

def test_round_bf16_against_torch_and_ties():
    import torch
    x = (rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in x])
    assert (got == ref).all()
    # ties go to the even significand: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert oracle.round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert oracle.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert oracle.round_bf16(-(1.0 + 2.0 ** -8)) == -1.0
    # monotone, so it commutes with ReLU and with max-pooling
    s = np.sort(rng.standard_normal(5000))
    r = np.array([oracle.round_bf16(v) for v in s])
    assert (np.diff(r) >= 0).all()
    assert oracle.round_bf16(0.0) == 0.0


def test_conv3x3_against_torch():
    import torch
    import torch.nn.functional as F
    for (C, O, H, Wd) in [(3, 4, 5, 5), (2, 3, 7, 4), (5, 2, 1, 1)]:
        x = rng.standard_normal((C, H, Wd))
        w = rng.standard_normal((O, C, 3, 3))
        b = rng.standard_normal(O)
        ref = F.conv2d(torch.from_numpy(x)[None], torch.from_numpy(w), torch.from_numpy(b),
                       padding=1)[0].numpy()
        np.testing.assert_allclose(oracle.conv3x3(x, w, b), ref, rtol=1e-12, atol=1e-12)


def test_conv3x3_brute_force_tiny():
    """Six nested loops written out here on a 5x5x3 -> 4 filter case."""
    x = rng.standard_normal((3, 5, 5))
    w = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    ref = np.zeros((4, 5, 5))
    for o in range(4):
        for y in range(5):
            for xx in range(5):
                s = b[o]
                for c in range(3):
                    for dy in range(3):
                        for dx in range(3):
                            yy, x2 = y + dy - 1, xx + dx - 1
                            if 0 <= yy < 5 and 0 <= x2 < 5:
                                s += w[o, c, dy, dx] * x[c, yy, x2]
                ref[o, y, xx] = s
    np.testing.assert_allclose(oracle.conv3x3(x, w, b), ref, rtol=1e-13, atol=1e-13)


def _torch_net_logit(spec, wts, S, den, bf16):
    """The specialized CNN as a torch CPU fp64 network (independent library path)."""
    import torch
    import torch.nn.functional as F

    def rnd(t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64) if bf16 else t

    x = torch.from_numpy(S.astype(np.float64) / den).permute(2, 0, 1)[None] / 127.5 - 1.0
    x = rnd(x)  # a bf16 network rounds its input only
    for w, b, p in zip(wts["conv_w"], wts["conv_b"], spec.pool):
        x = F.conv2d(x, torch.from_numpy(w.astype(np.float64)), torch.from_numpy(b.astype(np.float64)),
                     padding=1)
        x = F.relu(x)
        if p:
            x = F.max_pool2d(x, 2)
    f = x.flatten(1)
    h = F.relu(f @ torch.from_numpy(wts["w1"].astype(np.float64)).T +
               torch.from_numpy(wts["b1"].astype(np.float64)))
    z = h @ torch.from_numpy(wts["w2"].astype(np.float64)) + float(wts["b2"][0])
    return float(z[0])


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("conv,pool,dense", [((8, 8), (True, True), 16),
                                             ((8, 8, 8), (False, True, True), 12)])
def test_cnn_against_torch(bf16, conv, pool, dense):
    spec = synth.CNNSpec(in_h=11, in_w=9, conv=conv, pool=pool, dense=dense, bf16=bf16)
    wts = synth.cnn_weights(spec, 7)
    blob = synth.weight_blob(spec, wts)
    for trial in range(3):
        den = 7
        S = rng.integers(0, 255 * den + 1, size=(11, 9, 3)).astype(np.int64)
        z = oracle.cnn_logit(spec, blob, S, den)
        ref = _torch_net_logit(spec, wts, S, den, bf16)
        assert z == pytest.approx(ref, rel=1e-9, abs=1e-12)


def test_cnn_zero_weights_and_center_tap():
    spec = synth.CNNSpec(in_h=4, in_w=4, conv=(2,), pool=(False,), dense=3, bf16=False)
    wts = synth.cnn_weights(spec, 3)
    zero = {k: ([np.zeros_like(a) for a in v] if isinstance(v, list) else np.zeros_like(v))
            for k, v in wts.items()}
    zero["b2"] = np.array([0.75], np.float32)
    S = rng.integers(0, 256, size=(4, 4, 3)).astype(np.int64)
    z, sc = oracle.cnn_logit(spec, synth.weight_blob(spec, zero), S, 1, want_scale=True)
    assert z == 0.75 and sc == 0.75
    # b2 = 0 gives p = 0.5, which defers under (0.2, 0.8)
    assert oracle.sigmoid(0.0) == 0.5 and oracle.decide(0.5, 0.2, 0.8) == 2
    # centre-tap-only conv: channel o of the conv output is a per-pixel linear map
    cw = np.zeros((2, 3, 3, 3), np.float32)
    cw[0, 0, 1, 1], cw[1, 2, 1, 1] = 2.0, -1.0
    t = dict(conv_w=[cw], conv_b=[np.array([0.5, 0.25], np.float32)],
             w1=np.zeros((3, 32), np.float32), b1=np.zeros(3, np.float32),
             w2=np.zeros(3, np.float32), b2=np.zeros(1, np.float32))
    t["w1"][0, 5] = 1.0    # feature (c=0, y=1, x=1)
    t["w1"][1, 16 + 6] = 1.0  # feature (c=1, y=1, x=2)
    t["w2"][:] = (1.0, 1.0, 0.0)
    _, feats = oracle.cnn_logit(spec, synth.weight_blob(spec, t), S, 1, want_features=True)
    x = S / 127.5 - 1.0
    assert feats[5] == pytest.approx(max(0.0, 2.0 * x[1, 1, 0] + 0.5), rel=1e-15)
    assert feats[16 + 6] == pytest.approx(max(0.0, -x[1, 2, 2] + 0.25), rel=1e-15)
    z, sc = oracle.cnn_logit(spec, synth.weight_blob(spec, t), S, 1, want_scale=True)
    assert z == pytest.approx(feats[5] + feats[16 + 6], rel=1e-15)
    # scale = |b2| + sum_j |w2_j h_j| with hidden units h = features picked by w1 (b1 = 0)
    assert sc == pytest.approx(abs(feats[5]) + abs(feats[16 + 6]), rel=1e-15)


def test_decision_rule_ties_defer():
    assert oracle.decide(0.1, 0.2, 0.8) == 0
    assert oracle.decide(0.9, 0.2, 0.8) == 1
    assert oracle.decide(0.2, 0.2, 0.8) == 2
    assert oracle.decide(0.8, 0.2, 0.8) == 2
    assert oracle.decide(0.5, 0.2, 0.8) == 2


def _ulp(x: float) -> float:
    return abs(np.nextafter(x, math.inf) - x)


def test_sigmoid_exact_rationals():
    """sigma(ln k) = k / (1 + k): the confidence at a logit whose odds are a
    rational number.  At ln 4 and -ln 4 these are exactly the workloads'
    c_high = 0.8 and c_low = 0.2; a sign error (1 / (1 + e^z)) swaps them."""
    assert abs(oracle.sigmoid(math.log(4.0)) - 0.8) <= _ulp(0.8)
    assert abs(oracle.sigmoid(-math.log(4.0)) - 0.2) <= _ulp(0.2)
    for k in (1.0, 2.0, 3.0, 9.0, 0.5, 0.1, 1000.0):
        want = k / (1.0 + k)
        assert abs(oracle.sigmoid(math.log(k)) - want) <= 2 * _ulp(want), k


def test_sigmoid_shape():
    """Symmetry sigma(z) + sigma(-z) = 1, strict increase, slope 1/4 at 0 and
    the limits 0 and 1: a dropped minus sign, a wrong offset or a missing
    reciprocal each break one of them."""
    zs = rng.normal(0.0, 4.0, 200)
    for z in zs:
        assert oracle.sigmoid(z) + oracle.sigmoid(-z) == pytest.approx(1.0, abs=5e-16)
    srt = np.unique(np.clip(zs, -30.0, 30.0))
    vals = [oracle.sigmoid(z) for z in srt]
    assert all(a < b for a, b in zip(vals, vals[1:]))
    h = 1e-5
    assert (oracle.sigmoid(h) - oracle.sigmoid(-h)) / (2 * h) == pytest.approx(0.25, rel=1e-9)
    assert oracle.sigmoid(-40.0) == pytest.approx(math.exp(-40.0), rel=1e-15)
    assert oracle.sigmoid(-800.0) == 0.0 and oracle.sigmoid(40.0) == 1.0
    assert 0.0 < oracle.sigmoid(-700.0) < 1e-300


def test_decision_at_threshold_logits():
    """decide(sigmoid(z)) on both sides of logit(c_low) = -ln 4 and
    logit(c_high) = ln 4: below c_low no object, between the two defer, above
    c_high object (ties defer, as the paper's open intervals leave them)."""
    lo, hi = -math.log(4.0), math.log(4.0)
    eps = 1e-9  # moves the confidence by about 1.6e-10, far beyond rounding
    assert oracle.decide(oracle.sigmoid(lo - eps), 0.2, 0.8) == 0
    assert oracle.decide(oracle.sigmoid(lo + eps), 0.2, 0.8) == 2
    assert oracle.decide(oracle.sigmoid(hi - eps), 0.2, 0.8) == 2
    assert oracle.decide(oracle.sigmoid(hi + eps), 0.2, 0.8) == 1
    assert oracle.decide(oracle.sigmoid(0.0), 0.2, 0.8) == 2
    assert oracle.decide(oracle.sigmoid(-5.0), 0.2, 0.8) == 0
    assert oracle.decide(oracle.sigmoid(5.0), 0.2, 0.8) == 1


# ------------------------------------------------------------------ cascade

def _small(wl, n):
    v = synth.Video(wl.video)
    wts = synth.cnn_weights(wl.cnn, wl.weight_seed)
    return v, synth.weight_blob(wl.cnn, wts)


def _tiny_fast(**kw):
    """TINY with a smaller CNN so the cascade pins run in seconds."""
    spec = synth.CNNSpec(in_h=50, in_w=50, conv=(4, 4), pool=(True, True), dense=8, bf16=False)
    return W.TINY.replace(cnn=spec, **kw)


def test_cascade_chain_rule_brute_force():
    for delta in (1, 3, 7):
        wl = _tiny_fast(delta=delta)
        v, blob = _small(wl, 300)
        frames = v.frames(150, 450)
        cfg, keep = oracle.make_cfg(wl)
        out, _ = oracle.cascade(cfg, wl.cnn, blob, frames, t0=0)
        n = len(frames)
        # recompute the outputs in plain Python from the oracle's scores and probs
        lab = np.zeros(n, np.uint8)
        dfr = np.zeros(n, np.uint8)
        for t in range(n):
            fires = t < delta or out["score"][t] > wl.delta_diff
            assert bool(out["fire"][t]) == fires
            if fires:
                p = out["prob"][t]
                assert p == pytest.approx(1 / (1 + math.exp(-out["logit"][t])), rel=1e-15)
                lab[t], dfr[t] = (0, 0) if p < wl.c_low else ((1, 0) if p > wl.c_high else (0, 1))
            else:
                lab[t], dfr[t] = lab[t - delta], dfr[t - delta]
        assert (lab == out["label"]).all() and (dfr == out["defer"]).all()


def test_cascade_delta1_forward_fill():
    wl = _tiny_fast(delta=1, c_low=0.45, c_high=0.55)
    v, blob = _small(wl, 400)
    frames = v.frames(100, 500)
    cfg, keep = oracle.make_cfg(wl)
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    last = None
    for t in range(len(frames)):
        if out["fire"][t]:
            last = t
        assert last is not None
        assert out["label"][t] == out["label"][last] and out["defer"][t] == out["defer"][last]


def test_survivors_monotone_in_threshold():
    wl = _tiny_fast()
    v, blob = _small(wl, 300)
    frames = v.frames(200, 500)
    prev = None
    for dd in [-1.0, 0.0, 4.5, 10.0, 20.0, 60.0, 1e9]:
        cfg, keep = oracle.make_cfg(wl.replace(delta_diff=dd))
        out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
        s = set(np.flatnonzero(out["fire"]))
        if prev is not None:
            assert s <= prev
        prev = s
    # delta_diff = +inf leaves only the forced frames t < delta
    cfg, keep = oracle.make_cfg(wl.replace(delta_diff=math.inf))
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    assert list(np.flatnonzero(out["fire"])) == list(range(wl.delta))
    cfg, keep = oracle.make_cfg(wl.replace(delta_diff=-math.inf))
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    assert out["fire"].all()


def test_compaction_is_ascending_fired_list():
    wl = _tiny_fast()
    v, blob = _small(wl, 300)
    cfg, keep = oracle.make_cfg(wl)
    out, _ = oracle.cascade(cfg, wl.cnn, blob, v.frames(300, 600))
    idx = np.flatnonzero(out["fire"])
    assert out["fired"] == len(idx) == int(out["fire"].sum())
    assert np.isnan(out["logit"][out["fire"] == 0]).all()
    assert not np.isnan(out["logit"][idx]).any()


def test_chunk_invariance_and_determinism():
    for delta in (1, 4):
        wl = _tiny_fast(delta=delta, c_low=0.45, c_high=0.55)
        v, blob = _small(wl, 300)
        frames = v.frames(180, 480)
        cfg, keep = oracle.make_cfg(wl)
        full, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
        again, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
        for k in ("score", "fire", "label", "defer"):
            assert (full[k] == again[k]).all()
        parts, state, t0 = [], None, 0
        for size in (37, 3, 1, 100, 159):
            o, state = oracle.cascade(cfg, wl.cnn, blob, frames[t0:t0 + size], t0=t0, state=state)
            parts.append(o)
            t0 += size
        for k in ("fire", "label", "defer"):
            assert (np.concatenate([p[k] for p in parts]) == full[k]).all()
        np.testing.assert_array_equal(np.concatenate([p["score"] for p in parts]), full["score"])


def test_fixed_reference_mode():
    wl = _tiny_fast(ref_mode=W.FIXED)
    v, blob = _small(wl, 200)
    frames = v.frames(0, 60)
    ref = oracle.area_sums(frames[10], wl.dd_h, wl.dd_w)
    cfg, keep = oracle.make_cfg(wl, ref_sums=ref)
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    assert out["score"][10] == 0.0 and out["fire"][10] == 0
    # a non-firing frame is labelled "no object" without deferring
    nf = out["fire"] == 0
    assert (out["label"][nf] == 0).all() and (out["defer"][nf] == 0).all()
    assert np.isfinite(out["score"]).all()


# ------------------------------------------------------------- frame skipping

def _brute_skip(wl, blob, frames, s, ref=None):
    """The cascade with check stride s in plain Python loops over the oracle's
    per-frame primitives (area sums, MSE, CNN logit, decision rule)."""
    n = len(frames)
    den = oracle.area_den(wl.video.h, wl.video.w, wl.dd_h, wl.dd_w)
    den_c = oracle.area_den(wl.video.h, wl.video.w, wl.cnn.in_h, wl.cnn.in_w)
    S = [oracle.area_sums(f, wl.dd_h, wl.dd_w) for f in frames]
    lab = np.zeros(n, np.uint8)
    dfr = np.zeros(n, np.uint8)
    fire = np.zeros(n, np.uint8)
    for t in range(n):
        if t % s:
            lab[t], dfr[t] = lab[t - t % s], dfr[t - t % s]
            continue
        if wl.ref_mode == W.PREV:
            score = math.inf if t < wl.delta else oracle.global_mse(S[t], S[t - wl.delta], den)[0]
        else:
            score = oracle.global_mse(S[t], ref, den)[0]
        fire[t] = score > wl.delta_diff or (wl.ref_mode == W.PREV and t < wl.delta)
        if fire[t]:
            z = oracle.cnn_logit(wl.cnn, blob, oracle.area_sums(frames[t], wl.cnn.in_h, wl.cnn.in_w),
                                 den_c)
            d = oracle.decide(oracle.sigmoid(z), wl.c_low, wl.c_high)
            lab[t], dfr[t] = d & 1, (d >> 1) & 1
        elif wl.ref_mode == W.PREV:
            lab[t], dfr[t] = lab[t - wl.delta], dfr[t - wl.delta]
    return lab, dfr, fire


@pytest.mark.parametrize("s,delta,ref_mode", [(3, 3, W.PREV), (4, 8, W.PREV), (5, 5, W.PREV),
                                              (4, 1, W.FIXED)])
def test_skipping_brute_force(s, delta, ref_mode):
    wl = _tiny_fast(delta=delta, ref_mode=ref_mode, c_low=0.45, c_high=0.55, check_stride=s)
    if ref_mode == W.FIXED:  # the reference is a noisy frame: a threshold at the noise level
        wl = wl.replace(delta_diff=4.4)
    v, blob = _small(wl, 200)
    frames = v.frames(150, 350)
    ref = oracle.area_sums(frames[7], wl.dd_h, wl.dd_w) if ref_mode == W.FIXED else None
    cfg, keep = oracle.make_cfg(wl, ref_sums=ref)
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    lab, dfr, fire = _brute_skip(wl, blob, frames, s, ref)
    assert (out["fire"] == fire).all() and (out["label"] == lab).all() and (out["defer"] == dfr).all()
    unchecked = np.arange(len(frames)) % s != 0
    assert np.isnan(out["score"][unchecked]).all() and np.isnan(out["logit"][unchecked]).all()
    assert np.isfinite(out["score"][~unchecked][delta if ref_mode == W.PREV else 0:]).all()
    assert fire.sum() > 0 and (fire[~unchecked] == 0).sum() > 0  # both branches exercised


@pytest.mark.parametrize("s,delta", [(3, 6), (2, 2)])
def test_skipping_equals_subsampled_video(s, delta):
    # checking every s-th frame is the cascade on the subsampled video (delta / s
    # checked frames back) with each skip block taking its checked frame's output
    wl = _tiny_fast(delta=delta, c_low=0.45, c_high=0.55, check_stride=s)
    v, blob = _small(wl, 200)
    frames = v.frames(120, 360)
    cfg, keep = oracle.make_cfg(wl)
    out, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    sub_wl = wl.replace(delta=delta // s, check_stride=1)
    cfg2, keep2 = oracle.make_cfg(sub_wl)
    sub, _ = oracle.cascade(cfg2, wl.cnn, blob, frames[::s])
    blk = np.arange(len(frames)) // s
    for k in ("label", "defer"):
        assert (out[k] == sub[k][blk]).all()
    for k in ("fire", "score", "logit"):
        np.testing.assert_array_equal(out[k][::s], sub[k])


def test_skipping_chunk_invariance():
    wl = _tiny_fast(delta=6, c_low=0.45, c_high=0.55, check_stride=3)
    v, blob = _small(wl, 200)
    frames = v.frames(150, 400)
    cfg, keep = oracle.make_cfg(wl)
    full, _ = oracle.cascade(cfg, wl.cnn, blob, frames)
    parts, state, t0 = [], None, 0
    for size in (37, 3, 1, 2, 100, 107):   # boundaries inside skip blocks
        o, state = oracle.cascade(cfg, wl.cnn, blob, frames[t0:t0 + size], t0=t0, state=state)
        parts.append(o)
        t0 += size
    for k in ("fire", "label", "defer"):
        assert (np.concatenate([p[k] for p in parts]) == full[k]).all()
    np.testing.assert_array_equal(np.concatenate([p["score"] for p in parts]), full["score"])


def test_skipping_stride_one_and_bad_delta():
    wl = _tiny_fast(delta=2, c_low=0.45, c_high=0.55)
    v, blob = _small(wl, 200)
    frames = v.frames(150, 230)
    a, _ = oracle.cascade(oracle.make_cfg(wl)[0], wl.cnn, blob, frames)
    for s in (0, 1):
        b, _ = oracle.cascade(oracle.make_cfg(wl.replace(check_stride=s))[0], wl.cnn, blob, frames)
        for k in ("fire", "label", "defer", "score"):
            np.testing.assert_array_equal(a[k], b[k])
    with pytest.raises(ValueError):   # reading: delta must be a multiple of the stride
        oracle.cascade(oracle.make_cfg(wl.replace(check_stride=3))[0], wl.cnn, blob, frames)


# ------------------------------------------------- threshold search (Sec. 6.3)

SWEEP_COSTS = dict(t_mse=1e-6, t_snn=1e-4, t_full=1e-2)


def test_sweep_hand_worked():
    rows = _read_golden("sweep_6.txt")
    score = np.array([np.inf, 5, 1, 3, 0.5, 2])
    conf = np.array([0.9, 0.1, 0.5, 0.7, 0.2, 0.95], np.float32)
    truth = np.array([1, 0, 0, 1, 0, 1], np.uint8)
    cands = [float(r[0]) for r in rows if r[0] != "best"]
    got, best = oracle.threshold_sweep(score, conf, truth, cands, ref_mode=W.PREV, delta=1,
                                       fp_target=0.5, fn_target=0.5, **SWEEP_COSTS)
    for g, r in zip(got, [r for r in rows if r[0] != "best"]):
        d, fired, fn_dd, fp_dd, cl, ch, deferred, fn_c, fp_c, feas, cost = r
        assert (g["fired"], g["fn_dd"], g["fp_dd"]) == (int(fired), int(fn_dd), int(fp_dd))
        assert g["c_low"] == float(np.float32(cl)) and g["c_high"] == float(np.float32(ch))
        assert (g["deferred"], g["fn_cnn"], g["fp_cnn"], g["feasible"]) == (
            int(deferred), int(fn_c), int(fp_c), int(feas))
        assert g["cost"] == pytest.approx(float(cost), rel=1e-12)
    assert best == int(rows[-1][1])


def _sweep_brute(score, conf, truth, cands, ref_mode, delta, fp_t, fn_t, costs):
    """Per-frame simulation of every threshold pair: the labels a cascade with
    thresholds (delta_diff, c_low, c_high) gives, counted against the reference
    labels; c_low is the largest candidate value meeting the false negative
    target, c_high the smallest (not below c_low) meeting the false positive
    target."""
    n = len(score)
    pos = int(truth.sum())
    neg = n - pos
    fn_b = fn_t * pos if pos else math.inf
    fp_b = fp_t * neg if neg else math.inf
    out = []
    for d in cands:
        fired = [t for t in range(n) if score[t] == math.inf or score[t] > d]
        fs = set(fired)
        fn_dd = fp_dd = 0
        for t in range(n):
            if t in fs:
                continue
            ref = truth[t - delta] if (ref_mode == W.PREV and t >= delta) else 0
            fn_dd += int(truth[t] == 1 and ref == 0)
            fp_dd += int(truth[t] == 0 and ref == 1)
        values = sorted({0.0, 1.0} | {float(conf[t]) for t in fired})

        def count(cl, ch):
            fn = fp = dfr = 0
            for t in fired:
                c = float(conf[t])
                if c < cl:
                    fn += int(truth[t] == 1)
                elif c > ch:
                    fp += int(truth[t] == 0)
                else:
                    dfr += 1
            return fn, fp, dfr

        feasible = fn_dd < fn_b and fp_dd < fp_b
        if feasible:
            cl = max(v for v in values if fn_dd + count(v, 2.0)[0] < fn_b)
            ch = min(v for v in values if v >= cl and fp_dd + count(cl, v)[1] < fp_b)
        else:
            cl, ch = 0.0, 1.0
        fn, fp, dfr = count(cl, ch)
        f_m = len(fired) / n
        f_c = dfr / len(fired) if fired else 0.0
        cost = costs["t_mse"] + f_m * costs["t_snn"] + (f_m * f_c) * costs["t_full"]
        out.append(dict(fired=len(fired), fn_dd=fn_dd, fp_dd=fp_dd, c_low=cl, c_high=ch,
                        deferred=dfr, fn_cnn=fn, fp_cnn=fp, feasible=int(feasible), cost=cost))
    feas = [k for k, o in enumerate(out) if o["feasible"]]
    best = min(feas, key=lambda k: (out[k]["cost"], k)) if feas else -1
    return out, best


@pytest.mark.parametrize("seed", range(60))
def test_sweep_against_brute_force(seed):
    r = np.random.default_rng([seed, 77])
    n = int(r.integers(1, 15))
    delta = int(r.integers(1, 4))
    ref_mode = W.PREV if seed % 3 else W.FIXED
    score = np.round(r.uniform(0, 10, n), 1)
    if ref_mode == W.PREV:
        score[:delta] = np.inf
    # few distinct confidences, so that ties occur; 0 and 1 included
    conf = r.choice(np.array([0.0, 0.125, 0.25, 0.5, 0.75, 1.0], np.float32), n)
    truth = (r.random(n) < r.uniform(0.1, 0.9)).astype(np.uint8)
    cands = np.concatenate([[-np.inf, np.inf], np.round(r.uniform(-1, 11, 6), 1), score[:3]])
    fp_t, fn_t = float(r.choice([0.05, 0.2, 0.34, 0.5, 1.0])), float(r.choice([0.05, 0.2, 0.5, 1.0]))
    got, best = oracle.threshold_sweep(score, conf, truth, cands, ref_mode=ref_mode, delta=delta,
                                       fp_target=fp_t, fn_target=fn_t, **SWEEP_COSTS)
    want, wbest = _sweep_brute(score, conf, truth, cands, ref_mode, delta, fp_t, fn_t,
                               SWEEP_COSTS)
    for g, w in zip(got, want):
        for k in ("fired", "fn_dd", "fp_dd", "deferred", "fn_cnn", "fp_cnn", "feasible"):
            assert int(g[k]) == w[k], (k, g, w)
        assert g["c_low"] == w["c_low"] and g["c_high"] == w["c_high"], (g, w)
        assert g["cost"] == w["cost"]
        if w["feasible"]:  # the chosen thresholds meet the targets
            pos, neg = int(truth.sum()), n - int(truth.sum())
            assert not pos or g["fn_dd"] + g["fn_cnn"] < fn_t * pos
            assert not neg or g["fp_dd"] + g["fp_cnn"] < fp_t * neg
    assert best == wbest


def test_sweep_monotone_in_delta():
    # raising delta_diff never adds fired frames and never removes detector errors
    r = np.random.default_rng(5)
    n = 400
    score = r.exponential(5, n)
    score[:3] = np.inf
    conf = r.random(n).astype(np.float32)
    truth = (r.random(n) < 0.3).astype(np.uint8)
    cands = np.sort(r.uniform(0, 20, 40))
    got, _ = oracle.threshold_sweep(score, conf, truth, cands, ref_mode=W.PREV, delta=3,
                                    fp_target=0.1, fn_target=0.1, **SWEEP_COSTS)
    assert (np.diff(got["fired"]) <= 0).all()
    assert (np.diff(got["fn_dd"]) >= 0).all() and (np.diff(got["fp_dd"]) >= 0).all()
    assert got["fired"][0] == int((score > cands[0]).sum())


def test_sweep_special_cases():
    n = 50
    r = np.random.default_rng(9)
    conf = r.random(n).astype(np.float32)
    truth = (r.random(n) < 0.4).astype(np.uint8)
    score = r.uniform(0, 1, n)
    # delta_diff = -inf: every frame fires, the detector makes no error; with
    # targets of 100 % every frame can be labelled, so only frames at exactly
    # c_low = c_high are deferred
    got, best = oracle.threshold_sweep(score, conf, truth, [-np.inf], ref_mode=W.FIXED, delta=1,
                                       fp_target=1.0, fn_target=1.0, **SWEEP_COSTS)
    g = got[0]
    assert g["fired"] == n and g["fn_dd"] == 0 and g["fp_dd"] == 0 and best == 0
    assert g["deferred"] == int((conf.astype(np.float64) == g["c_low"]).sum())
    # targets of 0: nothing may be labelled by the CNN, everything fired defers
    got, best = oracle.threshold_sweep(score, conf, truth, [-np.inf], ref_mode=W.FIXED, delta=1,
                                       fp_target=0.0, fn_target=0.0, **SWEEP_COSTS)
    assert got[0]["feasible"] == 0 and best == -1
    # fixed reference, delta_diff = +inf: nothing fires, every frame with the
    # object is a false negative of the detector
    got, _ = oracle.threshold_sweep(score, conf, truth, [np.inf], ref_mode=W.FIXED, delta=1,
                                    fp_target=1.0, fn_target=1.0, **SWEEP_COSTS)
    assert got[0]["fired"] == 0 and got[0]["fn_dd"] == int(truth.sum()) and got[0]["fp_dd"] == 0
    assert got[0]["cost"] == SWEEP_COSTS["t_mse"]
