"""Host-side checks of the seeded synthetic video generator (input infrastructure)."""
import numpy as np
import pytest

import synth
from synth import workloads as W


def test_splitmix64_reference_outputs():
    # First outputs of the SplitMix64 generator seeded with 0 (state advanced by
    # the golden gamma before each finalisation), as published with the method.
    z = np.array([synth.GOLDEN, 2 * synth.GOLDEN % 2**64, 3 * synth.GOLDEN % 2**64], np.uint64)
    got = [int(v) for v in synth.splitmix64(z)]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_frames_deterministic_and_seeded():
    v1 = synth.Video(W.TINY.video)
    v2 = synth.Video(W.TINY.video)
    assert (v1.frame(123) == v2.frame(123)).all()
    v3 = synth.Video(W.TINY.video.__class__(**{**W.TINY.video.__dict__, "seed": 5}))
    assert not (v1.frame(123) == v3.frame(123)).all()


def test_noise_table_statistics():
    t = synth.gaussian_table(5.0)
    assert t.dtype == np.int16 and t.size == 65536
    assert abs(t.mean()) < 1e-3 and abs(t.std() - 5.0) < 0.05
    assert (np.diff(t) >= 0).all()


def test_rects_inside_frame_and_occupancy():
    spec = W.VGA.video.__class__(**{**W.VGA.video.__dict__, "n": 20000})
    v = synth.Video(spec)
    r = v.rects
    act = r[:, :, 7] == 1
    assert (r[act][:, 0] >= 0).all() and (r[act][:, 2] <= spec.w).all()
    assert (r[act][:, 1] >= 0).all() and (r[act][:, 3] <= spec.h).all()
    assert (r[act][:, 2] > r[act][:, 0]).all()
    assert 0.08 < v.occupied.mean() < 0.35


def test_static_scene_between_episodes():
    v = synth.Video(W.TINY.video)
    empty = np.flatnonzero(~v.occupied)
    a, b = v.frame(int(empty[5])).astype(int), v.frame(int(empty[6])).astype(int)
    # only noise differs: per-pixel difference of two N(0, 3^2) draws
    assert abs((a - b).std() - 3.0 * np.sqrt(2)) < 0.3


def test_weights_bf16_exact_and_blob_layout():
    spec = W.VGA.cnn
    w = synth.cnn_weights(spec, 1002)
    for a in w["conv_w"] + [w["w1"], w["w2"]]:
        assert (synth.round_to_bf16(a) == a).all()
    blob = synth.weight_blob(spec, w)
    layers, flat, _ = spec.shapes()
    expect = sum(co * ci * 9 + co for ci, co, *_ in layers) + spec.dense * flat + 2 * spec.dense + 1
    assert blob.size == expect and flat == 32 * 12 * 12
