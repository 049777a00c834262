"""The difference detector against a fixed reference image fused into the
area kernel (partial sums per wave, added up by a finishing kernel), as
nsc_cascade_run runs it, against the two-pass path of nsc_diff_detect (area
sums, then k_diff) and against the oracle: scores bit-identical, fire flags
identical, for every metric and every lane-chunk width of the area kernel."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_1703_02529_amd as nsc
import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
rng = np.random.default_rng(4321)

METRICS = {0: "mse", 1: "sad", 2: "nrmse", 3: "psnr"}


def _frames(n, H, W):
    f = rng.integers(0, 256, size=(n, H, W, 3), dtype=np.uint8)
    for k in range(1, n):  # similar consecutive frames, so scores spread around the threshold
        keep = rng.random((H, W, 1)) < 0.93
        f[k] = np.where(keep, f[k - 1], f[k])
    return f


def _oracle_metric(metric, cur, ref, den):
    return oracle.global_metric(cur, ref, den, metric)[0]


@pytest.mark.parametrize("H,W,Ho,Wo", [
    (480, 640, 50, 50),      # 16-byte lane chunks
    (720, 1280, 50, 50),     # 32-byte lane chunks
    (1080, 1920, 100, 100),  # 32-byte lane chunks, 10-row bands
    (100, 100, 50, 50),      # 4-byte lane chunks
])
@pytest.mark.parametrize("metric", sorted(METRICS), ids=lambda m: METRICS[m])
def test_fused_fixed_detector(H, W, Ho, Wo, metric):
    n = 21
    frames = _frames(n + 1, H, W)
    ref_img, vid = frames[0], frames[1:]
    den = oracle.area_den(H, W, Ho, Wo)
    ref_d = torch.empty(Ho * Wo * 3, dtype=torch.int32, device=DEV)
    nsc.nsc_downsample(torch.from_numpy(ref_img.reshape(-1)).to(DEV), 1, H, W, Ho, Wo, ref_d)
    dframes = torch.from_numpy(vid.reshape(-1)).to(DEV)
    # two-pass scores
    cfg = nsc.make_cfg(in_h=H, in_w=W, dd_h=Ho, dd_w=Wo, cnn_h=Ho, cnn_w=Wo, ref_mode=1,
                       ref_sums=ref_d, delta_diff=0.0, metric=metric)
    sums = torch.empty(n * Ho * Wo * 3, dtype=torch.int32, device=DEV)
    s2 = torch.empty(n, dtype=torch.float64, device=DEV)
    f2 = torch.empty(n, dtype=torch.uint8, device=DEV)
    nsc.nsc_diff_detect(cfg, dframes, n, 0, sums, f2, score_out=s2)
    two = s2.cpu().numpy()
    fin = two[np.isfinite(two)]
    thr = float(np.median(fin)) if fin.size else 0.0
    # fused, inside the cascade, at a threshold among the scores
    cfg = nsc.make_cfg(in_h=H, in_w=W, dd_h=Ho, dd_w=Wo, cnn_h=Ho, cnn_w=Wo, ref_mode=1,
                       ref_sums=ref_d, delta_diff=thr, metric=metric)
    spec = synth.CNNSpec(in_h=Ho, in_w=Wo, conv=(16,), pool=(True,), dense=16, bf16=False)
    blob = synth.weight_blob(spec, synth.cnn_weights(spec, 3))
    cnn = nsc.Cnn(nsc.make_desc(spec.conv, spec.pool, spec.dense, Ho, Wo, False), blob)
    ws = torch.empty(nsc.nsc_cascade_workspace_bytes(cfg, cnn, n), dtype=torch.uint8, device=DEV)
    state = torch.zeros(max(nsc.nsc_state_bytes(cfg), 256), dtype=torch.uint8, device=DEV)
    label = torch.empty(n, dtype=torch.uint8, device=DEV)
    defer = torch.empty(n, dtype=torch.uint8, device=DEV)
    score = torch.full((n,), math.nan, dtype=torch.float64, device=DEV)
    fire = torch.empty(n, dtype=torch.uint8, device=DEV)
    nsc.nsc_cascade_run(cfg, cnn, dframes, n, 0, state, ws, label, defer, score=score, fire=fire)
    torch.cuda.synchronize()
    fused = score.cpu().numpy()
    cnn.close()
    assert np.array_equal(fused, two, equal_nan=True), np.flatnonzero(fused != two)
    assert np.array_equal(fire.cpu().numpy(), (two > thr).astype(np.uint8))
    assert 0 < int(fire.sum()) < n or fin.size == 0
    # and the oracle, frame by frame
    ref_o = oracle.area_sums(ref_img, Ho, Wo)
    for t in (0, n // 2, n - 1):
        want = _oracle_metric(metric, oracle.area_sums(vid[t], Ho, Wo), ref_o, den)
        if metric == 3:
            assert fused[t] == pytest.approx(want, rel=1e-13)
        else:
            assert fused[t] == want, (t, fused[t], want)


# ------------------------------------------------------------ earlier frame

@pytest.mark.parametrize("H,W,Ho,Wo,grid,delta,chunks", [
    (480, 640, 50, 50, (1, 1), 2, [37, 9, 30]),         # 16-byte lane chunks, global: fused
    (1080, 1920, 100, 100, (1, 1), 7, [36, 22]),        # 16-byte lane chunks, global: fused
    (100, 100, 50, 50, (1, 1), 5, [64, 11, 25]),        # 4-byte lane chunks, global: fused
    (720, 1280, 50, 50, (1, 1), 3, [30, 20]),           # 32-byte lane chunks: two passes
    (480, 640, 50, 50, (5, 5), 3, [50, 26]),            # blocked: two passes
    (1080, 1920, 100, 100, (10, 10), 7, [36, 22]),      # blocked: two passes
    (720, 1280, 100, 100, (3, 7), 4, [40]),             # uneven block grid: two passes
])
def test_fused_prev_detector(H, W, Ho, Wo, grid, delta, chunks):
    """The MSE detector against frame t - delta as nsc_cascade_run runs it
    over consecutive calls with fuse_prev set: for a global score with 16- or
    4-byte lane chunks fused into the area kernel (chains of frames delta
    apart, partial sums; each chain's first frame from the sums), otherwise in
    two passes; against the two-pass scores of one nsc_diff_detect call over
    all frames and the oracle: bit-identical scores, identical fire flags."""
    n = sum(chunks)
    vid = _frames(n, H, W)
    dframes = torch.from_numpy(vid.reshape(-1)).to(DEV)
    G = grid[0] * grid[1]
    lr_w = rng.standard_normal(G).astype(np.float32) if G > 1 else None
    lr_d = torch.from_numpy(lr_w).to(DEV) if G > 1 else None
    kw = dict(in_h=H, in_w=W, dd_h=Ho, dd_w=Wo, cnn_h=Ho, cnn_w=Wo, ref_mode=0, delta=delta,
              grid=grid, lr_w=lr_d, lr_b=-2.0)
    cfg = nsc.make_cfg(delta_diff=0.0, **kw)
    sums = torch.empty(n * Ho * Wo * 3, dtype=torch.int32, device=DEV)
    s2 = torch.empty(n, dtype=torch.float64, device=DEV)
    f2 = torch.empty(n, dtype=torch.uint8, device=DEV)
    nsc.nsc_diff_detect(cfg, dframes, n, 0, sums, f2, score_out=s2)
    two = s2.cpu().numpy()
    fin = two[np.isfinite(two)]
    thr = float(np.median(fin))
    cfg = nsc.make_cfg(delta_diff=thr, fuse_prev=1, **kw)
    spec = synth.CNNSpec(in_h=Ho, in_w=Wo, conv=(16,), pool=(True,), dense=16, bf16=False)
    blob = synth.weight_blob(spec, synth.cnn_weights(spec, 3))
    cnn = nsc.Cnn(nsc.make_desc(spec.conv, spec.pool, spec.dense, Ho, Wo, False), blob)
    m = max(chunks)
    ws = torch.empty(nsc.nsc_cascade_workspace_bytes(cfg, cnn, m), dtype=torch.uint8, device=DEV)
    state = torch.zeros(max(nsc.nsc_state_bytes(cfg), 256), dtype=torch.uint8, device=DEV)
    label = torch.empty(m, dtype=torch.uint8, device=DEV)
    defer = torch.empty(m, dtype=torch.uint8, device=DEV)
    score = torch.full((m,), math.nan, dtype=torch.float64, device=DEV)
    fire = torch.empty(m, dtype=torch.uint8, device=DEV)
    fused = np.empty(n)
    fired = np.empty(n, dtype=np.uint8)
    fb = H * W * 3
    t0 = 0
    for c in chunks:
        nsc.nsc_cascade_run(cfg, cnn, dframes[t0 * fb:(t0 + c) * fb], c, t0, state, ws,
                            label[:c], defer[:c], score=score[:c], fire=fire[:c])
        torch.cuda.synchronize()
        fused[t0:t0 + c] = score[:c].cpu().numpy()
        fired[t0:t0 + c] = fire[:c].cpu().numpy()
        t0 += c
    cnn.close()
    assert np.array_equal(fused, two, equal_nan=True), np.flatnonzero(fused != two)
    assert np.array_equal(fired, ((two > thr) | ~np.isfinite(two)).astype(np.uint8))
    assert 0 < int(fired[delta:].sum()) < n - delta
    # and the oracle, frame by frame (frames t >= delta; earlier ones always fire)
    den = oracle.area_den(H, W, Ho, Wo)
    for t in sorted({delta, delta + 1, n // 2, n - 1}):
        a = oracle.area_sums(vid[t], Ho, Wo)
        b = oracle.area_sums(vid[t - delta], Ho, Wo)
        want = (oracle.global_metric(a, b, den, 0)[0] if G == 1
                else oracle.blocked_metric(a, b, den, grid, lr_w, -2.0, 0)[0])
        assert fused[t] == want, (t, fused[t], want)
