"""Seeded generator: determinism, centroid definition, occlusion order,
channel layout and noise statistics."""
import numpy as np
import pytest

from paper_2609_16874_amd import synth


def test_deterministic_and_frames_differ():
    a, b = synth.make_frame(0), synth.make_frame(0)
    assert np.array_equal(a.emb, b.emb) and np.array_equal(a.fg, b.fg) and np.array_equal(a.inst, b.inst)
    f0, f1 = synth.make_frame(4, 0), synth.make_frame(4, 1)
    assert not np.array_equal(f0.inst, f1.inst)
    cal = synth.make_frame(0, calibration=True)
    assert not np.array_equal(cal.inst, a.inst)


def test_centroids_are_means_of_visible_pixel_centres():
    f = synth.make_frame(0)
    H, W = f.inst.shape
    for k in range(1, len(f.kept) + 1):
        ii, jj = np.nonzero(f.inst == k)
        if len(ii) == 0:
            assert not f.kept[k - 1]
            continue
        assert abs(f.centroids[k - 1, 0] - (jj + 0.5).mean()) < 1e-9
        assert abs(f.centroids[k - 1, 1] - (ii + 0.5).mean()) < 1e-9


def test_later_instances_overwrite_earlier():
    f = synth.make_frame(1)
    H, W = f.inst.shape
    expect = np.zeros((H, W), np.int32)
    for k, shp in enumerate(f.meta["shapes"], start=1):
        single = np.zeros((H, W), np.int32)
        if shp[0] == "ellipse":
            synth._raster_ellipse(single, 1, *shp[1:])
        else:
            synth._raster_polygon(single, 1, *shp[1:])
        expect[single > 0] = k
    assert np.array_equal(expect, f.inst)


@pytest.mark.parametrize("cfg", [0, 1])
def test_layout_and_noise(cfg):
    f = synth.make_frame(cfg)
    fx, fy = f.spec.freqs()
    n = len(f.kept)
    table = np.zeros((n + 1, f.spec.D))
    table[1:] = synth.encode_positions(f.centroids[:, 0], f.centroids[:, 1], fx, fy)
    resid = f.emb.astype(np.float64) - table[f.inst]
    assert abs(resid.mean()) < 0.01
    assert abs(resid.std() - f.spec.sigma) < 0.01 * f.spec.sigma + 2e-3
    fgres = f.fg.astype(np.float64) - (f.inst > 0)
    assert abs(fgres.std() - 0.05) < 0.005


def test_shapes_and_dtypes():
    for c, (H, W, D, dt) in {0: (64, 64, 32, np.float32), 1: (256, 256, 32, np.float32),
                             4: (640, 640, 64, np.float16)}.items():
        f = synth.make_frame(c)
        assert f.emb.shape == (H, W, D) and f.emb.dtype == dt and f.fg.dtype == dt
        assert 0.05 < f.fg_fraction < 0.9


def test_outliers_encode_other_positions():
    spec = synth.FrameSpec("outlier check", 64, 64, 4, "f32", 64.0, 64.0, 0.0, fg_sigma=0.0,
                           outlier_frac=0.05, kind="ellipse", n_inst=(3, 3), radius=(8.0, 16.0), radius_law="semi")
    f = synth.make_frame(2, spec=spec)
    assert len(f.outliers) == round(0.05 * 64 * 64)
    assert len(np.unique(f.outliers)) == len(f.outliers)
    fx, fy = spec.freqs()
    table = np.zeros((len(f.kept) + 1, spec.D))
    table[1:] = synth.encode_positions(f.centroids[:, 0], f.centroids[:, 1], fx, fy)
    clean = table[f.inst].reshape(-1, spec.D)
    diff = np.abs(f.emb.reshape(-1, spec.D) - clean).max(-1)
    others = np.setdiff1d(np.arange(64 * 64), f.outliers)
    assert diff[others].max() < 1e-6
    assert np.all(np.abs(np.linalg.norm(f.emb.reshape(-1, spec.D)[f.outliers].astype(np.float64), axis=-1) ** 2 - 2 * spec.n_freq) < 1e-4)
