"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Every input is seeded and synthetic; every expected value comes from the
oracle on the host.  Integer and index outputs must match bit for bit; logits
within the network's tolerance (1e-3 bf16, 1e-5 fp32, relative to the logit's scale).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_1703_02529_amd as nsc
import synth
from paper_1703_02529_amd.runner import CascadeRunner
from paper_1703_02529_amd.streaming import StreamingCascade
from synth import workloads as W

from helpers import (LOGIT_TOL, LogitErrors, check_properties, check_samples, compare_cascade,
                     lr_weights_for)

pytestmark = pytest.mark.gpu
DEV = "cuda"
rng = np.random.default_rng(20240611)


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV) if dtype is None else t.to(DEV, dtype)


def _render(video, t0, n):
    out = torch.empty(max(n, 1) * video.spec.frame_bytes, dtype=torch.uint8, device=DEV)
    video.render_device(out, t0, n)
    return out


# ----------------------------------------------------------------- inputs

@pytest.mark.parametrize("wl", W.ALL, ids=lambda w: w.name.split("-")[0])
def test_device_renderer_matches_host(wl):
    v = synth.Video(wl.video)
    occ = np.flatnonzero(v.occupied)
    t0 = int(occ[0]) if occ.size else 0
    t0 = min(t0, wl.video.n - 3)
    d = _render(v, t0, 3).cpu().numpy().reshape(3, wl.video.h, wl.video.w, 3)
    assert np.array_equal(d, v.frames(t0, t0 + 3))


def test_device_renderer_odd_frame_size():
    # 33 x 17 x 3 = 1683 bytes per frame: frames start off 16-byte boundaries
    spec = synth.VideoSpec(n=600, h=33, w=17, seed=3, obj_min=4, obj_max=12, occupancy=0.6, vmax=3)
    v = synth.Video(spec)
    t0 = int(np.flatnonzero(v.occupied)[0])
    d = _render(v, t0, 7).cpu().numpy().reshape(7, 33, 17, 3)
    assert np.array_equal(d, v.frames(t0, t0 + 7))


# ------------------------------------------------------------- downsample

@pytest.mark.parametrize("H,W,Ho,Wo,pad", [
    (100, 100, 50, 50, 0),      # 4-byte chunks, integer ratio
    (480, 640, 50, 50, 0),      # 16-byte chunks, ratios 9.6 x 12.8
    (480, 640, 50, 50, 48),     # padded frame stride
    (720, 1280, 100, 100, 0),
    (720, 1280, 50, 50, 0),     # 32-byte lane chunks (two 16-byte loads per lane)
    (1080, 1920, 100, 100, 0),  # 16-byte lane chunks, 54 of 64 lanes
    (1080, 1920, 50, 50, 32),   # padded stride, 16-byte chunks
    (33, 17, 5, 4, 0),          # 1-byte chunks, ragged
    (600, 64, 2, 16, 0),        # 300 source rows per output row: unpacked sums
    (64, 64, 64, 64, 0),        # identity
])
def test_downsample_parity(H, W, Ho, Wo, pad):
    n = 7
    fb = H * W * 3
    stride = fb + pad
    host = rng.integers(0, 256, size=(n, stride), dtype=np.uint8)
    dev = _dev(host.reshape(-1))
    out = torch.empty(n * Ho * Wo * 3, dtype=torch.int32, device=DEV)
    nsc.nsc_downsample(dev, n, H, W, Ho, Wo, out, frame_stride=stride)
    got = out.cpu().numpy().reshape(n, Ho, Wo, 3)
    for f in range(n):
        ref = oracle.area_sums(host[f, :fb].reshape(H, W, 3), Ho, Wo)
        assert np.array_equal(got[f], ref), f"frame {f}"


def test_downsample_extremes():
    # all-255 frames reach the largest sums; all-0 frames give zeros
    H, W = 720, 1280
    for v in (0, 255):
        dev = torch.full((2 * H * W * 3,), v, dtype=torch.uint8, device=DEV)
        out = torch.empty(2 * 50 * 50 * 3, dtype=torch.int32, device=DEV)
        nsc.nsc_downsample(dev, 2, H, W, 50, 50, out)
        assert (out.cpu().numpy() == v * oracle.area_den(H, W, 50, 50)).all()


# --------------------------------------------------------------- detector

def _diff_case(H, W, Ho, Wo, ref_mode, delta, grid, n, t0, delta_diff):
    frames = rng.integers(0, 256, size=(n + delta, H, W, 3), dtype=np.uint8)
    # make consecutive frames similar so scores straddle the threshold
    for k in range(1, n + delta):
        keep = rng.random((H, W, 1)) < 0.9
        frames[k] = np.where(keep, frames[k - 1], frames[k])
    den = oracle.area_den(H, W, Ho, Wo)
    S = np.stack([oracle.area_sums(f, Ho, Wo) for f in frames])
    lr_w = rng.standard_normal(grid[0] * grid[1]).astype(np.float32)
    ref_img = frames[0]
    kw = dict(in_h=H, in_w=W, dd_h=Ho, dd_w=Wo, cnn_h=Ho, cnn_w=Wo, ref_mode=ref_mode,
              delta=delta, grid=grid, delta_diff=delta_diff, lr_b=-0.5)
    lr_dev = _dev(lr_w)
    ref_dev = _dev(S[0].astype(np.int32).reshape(-1))
    cfg = nsc.make_cfg(lr_w=lr_dev if grid != (1, 1) else None,
                       ref_sums=ref_dev if ref_mode == 1 else None, **kw)
    dframes = _dev(frames[delta:].reshape(-1))
    prev = _dev(S[:delta].astype(np.int32).reshape(-1)) if (ref_mode == 0 and t0 > 0) else None
    sums = torch.empty(n * Ho * Wo * 3, dtype=torch.int32, device=DEV)
    score = torch.empty(n, dtype=torch.float64, device=DEV)
    fire = torch.empty(n, dtype=torch.uint8, device=DEV)
    nsc.nsc_diff_detect(cfg, dframes, n, t0, sums, fire, score_out=score, prev_sums=prev)
    g_s, g_f = score.cpu().numpy(), fire.cpu().numpy()
    assert np.array_equal(sums.cpu().numpy().reshape(n, Ho, Wo, 3), S[delta:])
    for i in range(n):
        t = t0 + i
        cur = S[delta + i]
        ref = S[0] if ref_mode == 1 else S[i]
        if ref_mode == 0 and t < delta:
            exp = math.inf
        elif grid == (1, 1):
            exp = oracle.global_mse(cur, ref, den)[0]
        else:
            exp = oracle.blocked_score(cur, ref, den, grid, lr_w, -0.5)[0]
        assert g_s[i] == exp, (i, g_s[i], exp)
        assert g_f[i] == (1 if (exp > delta_diff or (ref_mode == 0 and t < delta)) else 0)
    return g_f


@pytest.mark.parametrize("case", [
    dict(H=480, W=640, Ho=50, Wo=50, ref_mode=0, delta=15, grid=(1, 1), n=40, t0=100, dd=400.0),
    dict(H=480, W=640, Ho=50, Wo=50, ref_mode=0, delta=3, grid=(1, 1), n=20, t0=0, dd=400.0),
    dict(H=100, W=100, Ho=50, Wo=50, ref_mode=1, delta=1, grid=(1, 1), n=20, t0=5, dd=600.0),
    dict(H=200, W=200, Ho=100, Wo=100, ref_mode=0, delta=1, grid=(10, 10), n=12, t0=9, dd=0.0),
    dict(H=90, W=120, Ho=50, Wo=50, ref_mode=0, delta=2, grid=(3, 4), n=12, t0=0, dd=0.0),
    dict(H=150, W=150, Ho=75, Wo=75, ref_mode=1, delta=1, grid=(1, 1), n=9, t0=0, dd=-math.inf),
])
def test_diff_detect_parity(case):
    c = dict(case)
    dd = c.pop("dd")
    _diff_case(delta_diff=dd, **c)


# ------------------------------------------------------------- compaction

@pytest.mark.parametrize("n", [0, 1, 63, 64, 65, 4095, 4096, 4097, 12345, 100_000, 4_194_305])
@pytest.mark.parametrize("density", [0.0, 0.013, 0.5, 1.0])
def test_compact_parity(n, density):
    fire = (rng.random(n) < density).astype(np.uint8)
    ws = torch.empty(max(nsc.nsc_compact_workspace_bytes(n), 4), dtype=torch.uint8, device=DEV)
    idx = torch.full((max(n, 1),), -7, dtype=torch.int32, device=DEV)
    cnt = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    nsc.nsc_compact(_dev(fire) if n else None, n, idx if n else None, cnt, ws if n else None)
    ref = np.flatnonzero(fire)
    assert int(cnt.item()) == ref.size
    assert np.array_equal(idx.cpu().numpy()[:ref.size], ref)


# -------------------------------------------------------------------- CNN

def _cnn_case(spec, n_frames, n_img, fy=1, seed=5, max_count=None, pairs=False):
    hs, ws_ = spec.in_h * fy, spec.in_w * fy
    den = 9
    S = rng.integers(0, 255 * den + 1, size=(n_frames, hs, ws_, 3)).astype(np.int32)
    idx = np.sort(rng.choice(n_frames, size=n_img, replace=False)).astype(np.int32)
    wts = synth.cnn_weights(spec, seed)
    blob = synth.weight_blob(spec, wts)
    desc = nsc.make_desc(spec.conv, spec.pool, spec.dense, spec.in_h, spec.in_w, spec.bf16, pairs)
    cnn = nsc.Cnn(desc, blob)
    max_count = n_img + 5 if max_count is None else max_count
    ws = torch.empty(nsc.nsc_cnn_workspace_bytes(cnn, max_count), dtype=torch.uint8, device=DEV)
    logit = torch.full((max_count,), math.nan, dtype=torch.float32, device=DEV)
    prob = torch.full((max_count,), math.nan, dtype=torch.float32, device=DEV)
    idx_d = torch.zeros(max_count, dtype=torch.int32, device=DEV)
    idx_d[:n_img] = _dev(idx)
    cnt = torch.tensor([n_img], dtype=torch.int32, device=DEV)
    nsc.nsc_specialized_cnn(cnn, _dev(S.reshape(-1)), hs, ws_, den, idx_d, cnt, max_count, logit,
                            ws, prob_out=prob)
    g = logit.cpu().numpy()
    p = prob.cpu().numpy()
    cnn.close()
    assert np.isnan(g[n_img:]).all(), "entries beyond count must not be written"
    ref = np.zeros(n_img)
    scale = np.zeros(n_img)
    for i, f in enumerate(idx):
        x = S[f].astype(np.int64)
        if fy > 1:
            x = x.reshape(spec.in_h, fy, spec.in_w, fy, 3).sum(axis=(1, 3))
        ref[i], scale[i] = oracle.cnn_logit(spec, blob, x, den * fy * fy, want_scale=True)
    errs = LogitErrors().add(g[:n_img], ref, scale)
    print(f"{spec}: {errs}")
    assert errs.scale <= LOGIT_TOL[spec.bf16], f"max rel err {errs.scale:.3g} ({errs})"
    np.testing.assert_allclose(p[:n_img], 1 / (1 + np.exp(-g[:n_img].astype(np.float64))),
                               rtol=1e-6, atol=1e-7)
    return errs


@pytest.mark.parametrize("wl", [W.TINY, W.VGA], ids=["tiny-fp32", "vga-bf16"])
def test_cnn_parity_small_nets(wl):
    _cnn_case(wl.cnn, n_frames=60, n_img=37)


@pytest.mark.parametrize("wl", [W.HD_REF, W.HD_BLOCKED], ids=["hd4conv", "hd3conv-nested"])
def test_cnn_parity_large_nets(wl):
    fy = wl.dd_h // wl.cnn.in_h
    _cnn_case(wl.cnn, n_frames=30, n_img=17, fy=fy)


def test_cnn_fp32_variants():
    # fp32 inner layers with 4-aligned channels, odd grid, no pooling on the last layer
    spec = synth.CNNSpec(in_h=13, in_w=11, conv=(16, 48), pool=(True, False), dense=16, bf16=False)
    _cnn_case(spec, n_frames=20, n_img=19)
    spec = synth.CNNSpec(in_h=9, in_w=21, conv=(32, 64), pool=(False, True), dense=64, bf16=True)
    _cnn_case(spec, n_frames=20, n_img=3)


def test_cnn_column_segments():
    # layers whose weights plus a full-width band exceed the LDS budget run in
    # column segments (ragged last segment): bf16 64 -> 64 on a 120-wide map,
    # and an fp32 64 -> 64 layer whose weights alone fill most of the LDS
    spec = synth.CNNSpec(in_h=10, in_w=120, conv=(64, 64), pool=(False, True), dense=32, bf16=True)
    _cnn_case(spec, n_frames=12, n_img=5)
    spec = synth.CNNSpec(in_h=12, in_w=40, conv=(16, 64, 64), pool=(False, False, True), dense=16,
                         bf16=False)
    _cnn_case(spec, n_frames=12, n_img=5)


@pytest.mark.parametrize("conv,pool,hw,fy", [
    ((32, 64, 32), (True, False, True), (23, 31), 1),   # fused pair + a layered third layer
    ((64, 16), (True, True), (20, 20), 1),              # 64 then 16 channels
    ((32, 32), (True, True), (50, 50), 2),              # nested 2x2 cells into the first layer
    ((32, 32), (True, False), (13, 9), 1),              # unpooled second layer, tiny odd map
])
def test_cnn_fused_pair_shapes(conv, pool, hw, fy):
    # bf16 nets whose pooled first layer fits in LDS run their first two layers fused
    spec = synth.CNNSpec(in_h=hw[0], in_w=hw[1], conv=conv, pool=pool, dense=32, bf16=True)
    _cnn_case(spec, n_frames=24, n_img=11, fy=fy)


@pytest.mark.parametrize("conv,pool,hw,fy", [
    ((64, 64), (False, True), (13, 9), 1),                 # fused 64-channel pair, ragged tiles
    ((64, 32, 64), (False, False, True), (23, 31), 1),     # fused pair into 32 channels
    ((64, 64, 64), (False, False, False), (7, 5), 1),      # map smaller than a band
    ((64, 64, 64, 64), (False, True, False, True), (50, 50), 2),  # the 4-layer net, nested cells
    ((32, 64, 64), (True, False, True), (30, 61), 1),      # banded layer after a layered one
    ((64, 64), (False, False), (6, 80), 1),                # pair band over 80 KB: 1 group per CU
    ((32, 64, 64), (True, False, False), (11, 200), 1),    # banded layer 100 wide (160 KB plan)
    ((64, 64), (True, True), (13, 9), 1),                  # pooled 64-channel first layer fused
    ((64, 32, 64), (True, False, True), (23, 31), 1),      # ... into 32 channels, odd map
    ((64, 64, 64), (True, True, True), (50, 50), 2),       # the 3-layer net, nested cells
    ((64, 64), (True, False), (10, 96), 1),                # ... 48-wide second layer
])
@pytest.mark.parametrize("pairs", [False, True], ids=["fp16-acts", "bf16-pairs"])
def test_cnn_banded_shapes(conv, pool, hw, fy, pairs):
    # bf16 layers with 64 input channels run banded, weights streamed in fragment
    # order: on the fp16 matrix cores (fp16 activations between banded layers),
    # or with hi / lo bf16 activation pairs
    spec = synth.CNNSpec(in_h=hw[0], in_w=hw[1], conv=conv, pool=pool, dense=32, bf16=True)
    _cnn_case(spec, n_frames=16, n_img=9, fy=fy, pairs=pairs)


@pytest.mark.parametrize("dense", [16, 32, 64, 128, 256])
@pytest.mark.parametrize("bf16", [True, False], ids=["bf16", "fp32"])
def test_cnn_dense_paths(dense, bf16):
    """The dense layer below 16,384 survivors' capacity (K split over
    workgroups, then a finishing pass) and from it on (row-blocked
    workgroups), at every dense width: a count of 1, 3 or 133 survivors in
    both."""
    spec = synth.CNNSpec(in_h=10, in_w=12, conv=(32, 32), pool=(True, False), dense=dense,
                         bf16=bf16)
    for n_img in (1, 3, 133):
        _cnn_case(spec, n_frames=140, n_img=n_img)
        _cnn_case(spec, n_frames=140, n_img=n_img, max_count=16400)


def test_cnn_zero_count():
    spec = W.VGA.cnn
    desc = nsc.make_desc(spec.conv, spec.pool, spec.dense, 50, 50, True)
    cnn = nsc.Cnn(desc, synth.weight_blob(spec, synth.cnn_weights(spec, 1)))
    ws = torch.empty(nsc.nsc_cnn_workspace_bytes(cnn, 8), dtype=torch.uint8, device=DEV)
    logit = torch.full((8,), 7.0, dtype=torch.float32, device=DEV)
    nsc.nsc_specialized_cnn(cnn, torch.zeros(50 * 50 * 3, dtype=torch.int32, device=DEV), 50, 50,
                            1, torch.zeros(8, dtype=torch.int32, device=DEV),
                            torch.zeros(1, dtype=torch.int32, device=DEV), 8, logit, ws)
    assert (logit.cpu().numpy() == 7.0).all()
    cnn.close()


# ---------------------------------------------------------------- cascade

def _prepare(wl, t0, n, need_ref=False):
    v = synth.Video(wl.video)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    lr = lr_weights_for(wl) if wl.grid != (1, 1) else None
    ref_img = v.median_background() if (need_ref or wl.ref_mode == 1) else None
    return v, blob, lr, ref_img


def _gpu_ref_sums(wl, ref_img):
    d = _dev(ref_img.reshape(-1))
    out = torch.empty(wl.dd_h * wl.dd_w * 3, dtype=torch.int32, device=DEV)
    nsc.nsc_downsample(d, 1, wl.video.h, wl.video.w, wl.dd_h, wl.dd_w, out)
    return out


def _run_and_compare(wl, n, chunks=None):
    """Frames [0, n) of the workload's video, optionally fed in chunks."""
    v, blob, lr, ref_img = _prepare(wl, 0, n)
    ref_o = oracle.area_sums(ref_img, wl.dd_h, wl.dd_w) if ref_img is not None else None
    cfg_o, keep = oracle.make_cfg(wl, lr_w=lr, ref_sums=ref_o)
    ref, _ = oracle.cascade(cfg_o, wl.cnn, blob, v.frames(0, n), t0=0)
    lr_d = _dev(lr) if lr is not None else None
    ref_d = _gpu_ref_sums(wl, ref_img) if ref_img is not None else None
    sizes = chunks or [n]
    run = CascadeRunner(wl, blob, max_frames=max(sizes), lr_w=lr_d, ref_sums=ref_d)
    dev_frames = _render(v, 0, n)
    fb = wl.video.frame_bytes
    outs = {k: [] for k in ("score", "fire", "logit", "label", "defer")}
    done = 0
    for s in sizes:
        run.run(dev_frames[done * fb:(done + s) * fb], s, t0=done)
        for k in outs:
            outs[k].append(getattr(run, k)[:s].cpu().numpy().copy())
        done += s
    gpu = {k: np.concatenate(vv) for k, vv in outs.items()}
    run.close()
    return compare_cascade(wl, gpu, ref, t0=0)


def test_cascade_tiny_full_video():
    wl = W.TINY
    rep = _run_and_compare(wl, wl.video.n)
    assert rep["fired"] > 100
    print(rep)
    rep = _run_and_compare(wl, 400, chunks=[100, 1, 99, 200])
    print(rep)


def _first_occupied(wl, lead):
    v = synth.Video(wl.video)
    occ = np.flatnonzero(v.occupied)
    return max(0, int(occ[0]) - lead) if occ.size else 0


def test_cascade_vga_window():
    wl = W.VGA
    rep = _run_and_compare(wl, 30)
    print(rep)
    t0 = _first_occupied(wl, 20)
    rep = _run_and_compare_from_zero_window(wl, t0, 120)
    print(rep)


@pytest.mark.parametrize("frac", [0.0, 0.25, 0.5, 0.9], ids=["start", "q1", "mid", "end"])
def test_cascade_vga_512_windows(frac):
    """Whole windows of 512 consecutive 640x480 frames at four offsets of the
    100k-frame video, every frame compared (the t - 15 label chains included)."""
    wl = W.VGA
    v = synth.Video(wl.video)
    occ = np.flatnonzero(v.occupied)
    t0 = int(occ[np.searchsorted(occ, int(frac * wl.video.n))]) if frac > 0 else 0
    t0 = max(0, min(t0 - 40, wl.video.n - 512))
    rep = _run_and_compare_from_zero_window(wl, t0, 512)
    print(t0, rep)
    assert rep["fired"] > 0


def _run_and_compare_from_zero_window(wl, t0, n):
    """Window [t0, t0+n) of a video whose frames before t0 are dropped: the
    window is treated as its own video (frame indices restart at 0)."""
    spec_v = wl.video
    v = synth.Video(spec_v)
    frames = v.frames(t0, t0 + n)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    lr = lr_weights_for(wl) if wl.grid != (1, 1) else None
    ref_img = v.median_background() if wl.ref_mode == 1 else None
    ref_o = oracle.area_sums(ref_img, wl.dd_h, wl.dd_w) if ref_img is not None else None
    cfg_o, keep = oracle.make_cfg(wl, lr_w=lr, ref_sums=ref_o)
    ref, _ = oracle.cascade(cfg_o, wl.cnn, blob, frames, t0=0)
    run = CascadeRunner(wl, blob, max_frames=n, lr_w=_dev(lr) if lr is not None else None,
                        ref_sums=_gpu_ref_sums(wl, ref_img) if ref_img is not None else None)
    dev_frames = _dev(frames.reshape(-1))
    run.run(dev_frames, n, t0=0)
    gpu = {k: getattr(run, k)[:n].cpu().numpy() for k in ("score", "fire", "logit", "label",
                                                          "defer")}
    run.close()
    return compare_cascade(wl, gpu, ref, t0=0)


@pytest.mark.parametrize("wl,lead,n", [(W.HD_REF, 4, 14), (W.HD_BLOCKED, 4, 16),
                                       (W.FHD_STREAM, 2, 40),
                                       (W.FHD_STREAM.with_occupancy(0.01), 2, 40),
                                       (W.FHD_STREAM.with_occupancy(0.5), 2, 40)],
                         ids=["hd-ref", "hd-blocked", "fhd-blocked", "fhd-blocked-occ1",
                              "fhd-blocked-occ50"])
def test_cascade_large_windows(wl, lead, n):
    t0 = _first_occupied(wl, lead)
    rep = _run_and_compare_from_zero_window(wl, t0, n)
    print(rep)


def test_chunked_equals_one_shot_and_oracle():
    wl = W.VGA
    t0 = _first_occupied(wl, 10)
    n = 90
    v = synth.Video(wl.video)
    frames = v.frames(t0, t0 + n)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    dev_frames = _dev(frames.reshape(-1))
    fb = wl.video.frame_bytes
    keys = ("score", "fire", "logit", "label", "defer")

    def run_chunks(sizes):
        run = CascadeRunner(wl, blob, max_frames=max(sizes))
        outs = {k: [] for k in keys}
        done = 0
        for s in sizes:
            run.run(dev_frames[done * fb:(done + s) * fb], s, t0=done)
            for k in keys:
                outs[k].append(getattr(run, k)[:s].cpu().numpy().copy())
            done += s
        run.close()
        return {k: np.concatenate(vv) for k, vv in outs.items()}

    one = run_chunks([n])
    for sizes in ([7, 15, 1, 40, 27], [14, 16, 60], [1] * 20 + [70]):
        ch = run_chunks(sizes)
        for k in keys:
            assert np.array_equal(np.nan_to_num(ch[k], nan=-9), np.nan_to_num(one[k], nan=-9)), k
    cfg_o, keep = oracle.make_cfg(wl)
    ref, _ = oracle.cascade(cfg_o, wl.cnn, blob, frames, t0=0)
    print(compare_cascade(wl, one, ref))


def test_threshold_extremes_and_tiny_calls():
    wl = W.TINY.replace(delta=2)
    v = synth.Video(wl.video)
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    frames = v.frames(300, 340)
    d = _dev(frames.reshape(-1))
    for dd in (-math.inf, math.inf):
        w2 = wl.replace(delta_diff=dd)
        run = CascadeRunner(w2, blob, max_frames=40)
        run.run(d, 40, t0=0)
        fire = run.fire[:40].cpu().numpy()
        run.close()
        if dd < 0:
            assert fire.all()
        else:
            assert list(np.flatnonzero(fire)) == [0, 1]
    # zero frames and a single frame
    run = CascadeRunner(wl, blob, max_frames=4)
    assert run.run(d, 0, t0=0, want_stats=True)["frames"] == 0
    st = run.run(d, 1, t0=0, want_stats=True)
    assert st == dict(frames=1, fired=1, positive=st["positive"], deferred=st["deferred"])
    run.close()


def test_state_required_and_workspace_checks():
    wl = W.TINY
    blob = synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))
    run = CascadeRunner(wl, blob, max_frames=8)
    d = torch.zeros(8 * wl.video.frame_bytes, dtype=torch.uint8, device=DEV)
    small = torch.empty(1024, dtype=torch.uint8, device=DEV)
    with pytest.raises(nsc.NscError) as e:
        nsc.nsc_cascade_run(run.cfg, run.cnn, d, 8, 0, run.state, small, run.label, run.defer)
    assert e.value.status == -4
    with pytest.raises(nsc.NscError) as e:
        nsc.nsc_cascade_run(run.cfg, run.cnn, d, 8, 0, None, run.ws, run.label, run.defer)
    assert e.value.status == -7
    run.close()


# --------------------------------------------------------------- streaming

def test_streamed_chunks_equal_one_shot():
    """Two frame buffers on two streams, ragged last chunk, reference frame
    t - 30 across chunk boundaries: every output equals a one-shot run."""
    wl = W.FHD_STREAM.with_frames(3 * 512 + 77)
    n, fb, chunk = wl.video.n, wl.video.frame_bytes, 512
    v, blob, lr, _ = _prepare(wl, 0, n)
    lr_d = _dev(lr)
    tables = v.device_tables(DEV)
    frames = torch.empty(n * fb, dtype=torch.uint8, device=DEV)
    v.render_device(frames, 0, n, tables)
    one = CascadeRunner(wl, blob, max_frames=n, lr_w=lr_d)
    one.run(frames, n, t0=0)
    keys = ("score", "fire", "logit", "label", "defer")
    ref = {k: getattr(one, k)[:n].cpu().numpy().copy() for k in keys}
    one.close()
    del frames
    out = {k: torch.full((n,), 77, dtype=getattr(one, k).dtype, device=DEV) for k in keys}
    sc = StreamingCascade(wl, blob, chunk, lr_w=lr_d)
    st = sc.run(n, lambda buf, t0, m, s: v.render_device(buf, t0, m, tables, stream=s),
                timing=True, **out)
    sc.close()
    assert st["chunks"] == 4
    g = {k: out[k].cpu().numpy() for k in keys}
    for k in keys:
        assert np.array_equal(np.nan_to_num(g[k], nan=-7), np.nan_to_num(ref[k], nan=-7)), k
    check_properties(wl, g)
    # oracle on frames around the chunk boundaries
    ts = [0, 29, 30, 511, 512, 541, 1024 + 13, n - 1]
    print(check_samples(wl, v, blob, lr, None, g, ts))
    torch.cuda.empty_cache()


# ---------------------------------------------------------- frame skipping

@pytest.mark.parametrize("s,delta,ref_mode", [(3, 3, W.PREV), (4, 8, W.PREV), (5, 1, W.FIXED)])
def test_skipping_tiny_full_video(s, delta, ref_mode):
    wl = W.TINY.replace(check_stride=s, delta=delta, ref_mode=ref_mode)
    rep = _run_and_compare(wl, wl.video.n)
    assert rep["fired"] > 10
    print(rep)
    # chunk boundaries inside skip blocks, a chunk with no checked frame
    rep = _run_and_compare(wl, 400, chunks=[101, 2, 1, 97, 199])
    print(rep)


def test_skipping_vga_window():
    # the benchmark configuration checking every 5th frame (delta 15 = 3 checks back)
    wl = W.VGA.replace(check_stride=5)
    t0 = _first_occupied(wl, 40)
    rep = _run_and_compare_from_zero_window(wl, t0, 160)
    assert rep["fired"] > 0
    print(rep)


def test_skipping_streamed_equals_one_shot():
    wl = W.HD_BLOCKED.with_frames(1300).replace(delta=2, check_stride=2)
    n, fb = wl.video.n, wl.video.frame_bytes
    v, blob, lr, _ = _prepare(wl, 0, n)
    lr_d = _dev(lr)
    tables = v.device_tables(DEV)
    frames = torch.empty(n * fb, dtype=torch.uint8, device=DEV)
    v.render_device(frames, 0, n, tables)
    one = CascadeRunner(wl, blob, max_frames=n, lr_w=lr_d)
    one.run(frames, n, t0=0)
    keys = ("score", "fire", "logit", "label", "defer")
    ref = {k: getattr(one, k)[:n].cpu().numpy().copy() for k in keys}
    one.close()
    del frames
    out = {k: torch.full((n,), 77, dtype=getattr(one, k).dtype, device=DEV) for k in keys}
    sc = StreamingCascade(wl, blob, 301, lr_w=lr_d)   # odd chunks: boundaries inside skip blocks
    sc.run(n, lambda buf, t0, m, st: v.render_device(buf, t0, m, tables, stream=st), **out)
    sc.close()
    g = {k: out[k].cpu().numpy() for k in keys}
    for k in keys:
        assert np.array_equal(np.nan_to_num(g[k], nan=-7), np.nan_to_num(ref[k], nan=-7)), k
    print(check_samples(wl, v, blob, lr, None, g, [0, 1, 2, 301, 302, 603, 1299]))
