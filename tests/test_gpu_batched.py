"""GPU parity of staged batches: the area sums of each chunk staged into a
batch (nsc_cascade_stage), then the detector, compaction, CNN and label
resolution once per batch of chunks (nsc_cascade_finish).

A batched run must give the outputs of one nsc_cascade_run call over the same
frames: scores and fire flags bit for bit, logits up to the rounding order of
the dense layer's sums (its split over the survivors depends on how many share
a pass), labels and defer flags exactly except where the probability lies
within 1e-5 relative of c_low or c_high.  One case is also compared with the
fp64 oracle element by element.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1703_02529_amd as nsc
import synth
from paper_1703_02529_amd.runner import CascadeRunner
from paper_1703_02529_amd.streaming import StreamingCascade
from synth import workloads as W

from helpers import check_properties, check_samples, compare_cascade, lr_weights_for

pytestmark = pytest.mark.gpu
DEV = "cuda"
KEYS = ("score", "fire", "logit", "label", "defer")


def _blob(wl):
    return synth.weight_blob(wl.cnn, synth.cnn_weights(wl.cnn, wl.weight_seed))


def _ref_sums(wl, v):
    if wl.ref_mode != W.FIXED:
        return None
    img = torch.from_numpy(v.median_background().reshape(-1)).to(DEV)
    out = torch.empty(wl.dd_h * wl.dd_w * 3, dtype=torch.int32, device=DEV)
    nsc.nsc_downsample(img, 1, wl.video.h, wl.video.w, wl.dd_h, wl.dd_w, out)
    return out


def _lr(wl):
    return torch.from_numpy(lr_weights_for(wl)).to(DEV) if wl.grid != (1, 1) else None


def _one_shot(wl, v, blob, lr_d, ref_d, n):
    frames = torch.empty(n * wl.video.frame_bytes, dtype=torch.uint8, device=DEV)
    v.render_device(frames, 0, n)
    one = CascadeRunner(wl, blob, max_frames=n, lr_w=lr_d, ref_sums=ref_d)
    one.run(frames, n, t0=0)
    ref = {k: getattr(one, k)[:n].cpu().numpy().copy() for k in KEYS}
    one.close()
    del frames
    return ref


def _outputs(n):
    return {k: torch.full((n,), 77, dtype=d, device=DEV)
            for k, d in zip(KEYS, (torch.float64, torch.uint8, torch.float32, torch.uint8,
                                   torch.uint8))}


def _same_as_one_shot(wl, g, ref):
    """Batched outputs g against the one-shot run's ref (see the module
    docstring); returns the number of frames whose decision was not compared."""
    assert np.array_equal(np.nan_to_num(g["score"], nan=-7), np.nan_to_num(ref["score"], nan=-7))
    assert np.array_equal(g["fire"], ref["fire"])
    fired = ref["fire"] != 0
    assert np.isnan(g["logit"][~fired]).all() and np.isnan(ref["logit"][~fired]).all()
    a, b = g["logit"][fired].astype(np.float64), ref["logit"][fired].astype(np.float64)
    err = np.abs(a - b) / np.maximum(np.abs(b), 1.0)
    assert err.size == 0 or err.max() <= 1e-5, err.max()
    p = 1.0 / (1.0 + np.exp(-ref["logit"].astype(np.float64)))
    near = np.zeros(len(p), bool)
    for c in (wl.c_low, wl.c_high):
        near |= np.abs(p - c) <= 1e-5 * c
    keep = ~near
    assert np.array_equal(g["label"][keep], ref["label"][keep])
    assert np.array_equal(g["defer"][keep], ref["defer"][keep])
    return int(near.sum())


def test_batched_stream_equals_one_shot():
    """The 1080p stream (blocked detector against frame t - 30) in 256-frame
    chunks, three chunks per batch: batches of 768, 768 and a ragged last
    one of 77 frames; frame t - 30 lies across chunk and batch boundaries."""
    wl = W.FHD_STREAM.with_frames(6 * 256 + 77)
    n, chunk = wl.video.n, 256
    v, blob, lr_d = synth.Video(wl.video), _blob(wl), _lr(wl)
    ref = _one_shot(wl, v, blob, lr_d, None, n)
    tables = v.device_tables(DEV)
    out = _outputs(n)
    sc = StreamingCascade(wl, blob, chunk, lr_w=lr_d, batch_chunks=3)
    st = sc.run(n, lambda buf, t0, m, s: v.render_device(buf, t0, m, tables, stream=s),
                timing=True, **out)
    sc.close()
    assert st["chunks"] == 7 and st["batches"] == 3
    g = {k: out[k].cpu().numpy() for k in KEYS}
    excluded = _same_as_one_shot(wl, g, ref)
    check_properties(wl, g)
    print(dict(frames=n, fired=int(g["fire"].sum()), excluded=excluded))


def test_batch_continues_plain_run_state():
    """A plain nsc_cascade_run call on frames [0, 300) hands its carried state
    to staged batches of the frames after it (odd chunk sizes, two chunks per
    batch): together they equal one call over all frames."""
    wl = W.FHD_STREAM.with_frames(300 + 5 * 200 + 13)
    n, first, chunk = wl.video.n, 300, 200
    v, blob, lr_d = synth.Video(wl.video), _blob(wl), _lr(wl)
    ref = _one_shot(wl, v, blob, lr_d, None, n)
    out = _outputs(n)
    plain = CascadeRunner(wl, blob, max_frames=first, lr_w=lr_d)
    frames = torch.empty(first * wl.video.frame_bytes, dtype=torch.uint8, device=DEV)
    v.render_device(frames, 0, first)
    plain.run(frames, first, t0=0)
    for k in KEYS:
        out[k][:first].copy_(getattr(plain, k)[:first])
    del frames
    tables = v.device_tables(DEV)
    sc = StreamingCascade(wl, blob, chunk, lr_w=lr_d, batch_chunks=2)
    assert sc.runner.state.numel() == plain.state.numel()
    sc.runner.state.copy_(plain.state)
    plain.close()
    sc.run(n - first, lambda buf, t0, m, s: v.render_device(buf, t0, m, tables, stream=s),
           t_start=first, **{k: t[first:] for k, t in out.items()})
    sc.close()
    g = {k: out[k].cpu().numpy() for k in KEYS}
    print(dict(frames=n, fired=int(g["fire"].sum()), excluded=_same_as_one_shot(wl, g, ref)))


def test_batched_fixed_reference_equals_fused_one_shot():
    """The 720p fixed-reference video (4 x conv64 network): the batched run's
    detector is a pass over the staged sums, the one-shot run's is fused into
    its area kernel; scores agree bit for bit."""
    wl = W.HD_REF.with_frames(600)
    n, chunk = wl.video.n, 128
    v, blob = synth.Video(wl.video), _blob(wl)
    ref_d = _ref_sums(wl, v)
    ref = _one_shot(wl, v, blob, None, ref_d, n)
    tables = v.device_tables(DEV)
    out = _outputs(n)
    sc = StreamingCascade(wl, blob, chunk, ref_sums=ref_d, batch_chunks=4)
    st = sc.run(n, lambda buf, t0, m, s: v.render_device(buf, t0, m, tables, stream=s),
                timing=True, **out)
    sc.close()
    assert st["chunks"] == 5 and st["batches"] == 2
    g = {k: out[k].cpu().numpy() for k in KEYS}
    excluded = _same_as_one_shot(wl, g, ref)
    assert int(g["fire"].sum()) > 100
    print(dict(frames=n, fired=int(g["fire"].sum()), excluded=excluded))


def test_batched_cnn_passes_against_oracle():
    """The 640x480 video with CNN passes of at most 64 survivors: each batch
    of 3 x 160 frames runs 8 passes, some of them empty.  Every frame against
    the fp64 oracle's cascade."""
    wl = W.VGA.with_frames(1000)
    n, chunk = wl.video.n, 160
    v, blob = synth.Video(wl.video), _blob(wl)
    tables = v.device_tables(DEV)
    out = _outputs(n)
    sc = StreamingCascade(wl, blob, chunk, batch_chunks=3, cnn_pass=64)
    st = sc.run(n, lambda buf, t0, m, s: v.render_device(buf, t0, m, tables, stream=s),
                timing=True, **out)
    sc.close()
    assert st["chunks"] == 7 and st["batches"] == 3
    g = {k: out[k].cpu().numpy() for k in KEYS}
    cfg_o, _ = oracle.make_cfg(wl)
    ref, _ = oracle.cascade(cfg_o, wl.cnn, blob, v.frames(0, n), t0=0)
    rep = compare_cascade(wl, g, ref, t0=0)
    assert rep["fired"] > 64
    print(rep)


def test_batched_million_frames():
    """1,048,583 frames of the 100x100 video staged in 17 chunks of up to
    65,536 and finished in one call: compaction over a million fire flags, the
    CNN in 65 passes of up to 16,384 survivors (most of them empty), label
    chains of the whole video.  Sampled frames against the oracle, properties
    over every frame."""
    chunk = 65536
    wl = W.TINY.with_frames(16 * chunk + 7)
    n, fb = wl.video.n, wl.video.frame_bytes
    v, blob = synth.Video(wl.video), _blob(wl)
    tables = v.device_tables(DEV)
    run = CascadeRunner(wl, blob, max_frames=n, batch=True)
    buf = torch.empty(chunk * fb, dtype=torch.uint8, device=DEV)
    for at in range(0, n, chunk):
        m = min(chunk, n - at)
        v.render_device(buf, at, m, tables)
        run.stage(buf, m, at)
    st = run.finish(n, t0=0, want_stats=True)
    g = {k: getattr(run, k)[:n].cpu().numpy() for k in KEYS}
    run.close()
    del buf
    fired = int(g["fire"].sum())
    assert st["fired"] == fired > 2 * 16384
    check_properties(wl, g)
    rng = np.random.default_rng(11)
    occ = np.flatnonzero(v.occupied)
    fired_at = np.flatnonzero(g["fire"])
    # random frames, occupied ones, the ends, and the fired frames that open
    # and close each CNN pass
    ts = set(rng.integers(0, n, 120).tolist()) | set(rng.choice(occ, 120, replace=False).tolist())
    ts |= {0, n - 1} | {int(fired_at[k]) for k in range(0, fired, 16384)}
    ts |= {int(fired_at[min(k + 16383, fired - 1)]) for k in range(0, fired, 16384)}
    errs = check_samples(wl, v, blob, None, None, g, sorted(ts))
    print(dict(frames=n, fired=fired, sampled=len(ts), **errs.as_dict()))
    torch.cuda.empty_cache()


def test_stage_and_finish_check_their_arguments():
    wl = W.TINY
    blob = _blob(wl)
    run = CascadeRunner(wl, blob, max_frames=64, batch=True)
    frames = torch.zeros(64 * wl.video.frame_bytes, dtype=torch.uint8, device=DEV)
    with pytest.raises(nsc.NscError, match="outside the batch"):
        run.stage(frames, 40, 30)
    with pytest.raises(nsc.NscError):
        run.finish(65, t0=0)
    small = torch.empty(256, dtype=torch.uint8, device=DEV)
    with pytest.raises(nsc.NscError, match="workspace"):
        nsc.nsc_cascade_stage(run.cfg, run.cnn, 64, 0, frames, 8, 0, small)
    skip = CascadeRunner(wl.replace(check_stride=2, delta=2), blob, max_frames=8)
    with pytest.raises(nsc.NscError, match="check_stride"):
        nsc.nsc_batch_workspace_bytes(skip.cfg, skip.cnn, 64)
    skip.close()
    # a plain run on a batch workspace: refused (sized differently), not run
    with pytest.raises(nsc.NscError):
        nsc.nsc_cascade_run(run.cfg, run.cnn, frames, 64, 0, run.state, small, run.label,
                            run.defer)
    run.close()
