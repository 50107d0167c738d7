"""The seeded generators: determinism, validity, and the stated input densities."""

import numpy as np
import pytest

from workloads import CONFIGS, circle_sites, get_config, make_batch, make_paths

SITE_CONFIGS = [c for c in CONFIGS if c.generator != "paths"]
PATH_CONFIGS = [c for c in CONFIGS if c.generator == "paths"]


@pytest.mark.parametrize("cfg", PATH_CONFIGS, ids=lambda c: c.name)
def test_paths_are_valid_and_deterministic(cfg):
    a, b = make_paths(cfg, 0), make_paths(cfg, 0)
    np.testing.assert_array_equal(a.points, b.points)
    np.testing.assert_array_equal(a.stroke_begin, b.stroke_begin)
    assert a.stroke_begin[0] == 0 and a.stroke_begin[-1] == a.n_points and np.all(np.diff(a.stroke_begin) > 0)
    assert a.stroke_sample.min() >= 0 and a.stroke_sample.max() < cfg.batch
    lo = (cfg.grid - cfg.gen_args["box"]) // 2
    assert a.points.min() >= lo and a.points.max() < lo + cfg.gen_args["box"]
    assert not np.array_equal(make_paths(cfg, 1).points[:10], a.points[:10])
    with pytest.raises(ValueError):
        make_batch(cfg, 0)


@pytest.mark.parametrize("cfg", SITE_CONFIGS, ids=lambda c: c.name)
def test_batches_are_valid_and_deterministic(cfg):
    a = make_batch(cfg, 0)
    b = make_batch(cfg, 0)
    np.testing.assert_array_equal(a.coords, b.coords)
    np.testing.assert_array_equal(a.feats, b.feats)
    assert a.coords.dtype == np.int32 and a.feats.shape == (a.n, cfg.c_in)
    assert a.coords[:, 0].min() >= 0 and a.coords[:, 0].max() < cfg.batch
    assert a.coords[:, 1:].min() >= 0 and a.coords[:, 1:].max() < cfg.grid
    keys = (a.coords[:, 0].astype(np.int64) * cfg.grid + a.coords[:, 1]) * cfg.grid + a.coords[:, 2]
    assert np.unique(keys).size == a.n
    c = make_batch(cfg, 1)
    assert c.n != a.n or not np.array_equal(c.coords, a.coords)


def test_active_fractions():
    # stroke workloads: ~3-8% (96x96, 64x64 box), <3% (192x192); the RGB patch is 32*32/96^2 exactly
    f = {c.name: make_batch(c, 0).active_fraction() for c in SITE_CONFIGS}
    assert 0.03 <= f["deepcnet5_50_strokes_b100"] <= 0.08
    assert 0.03 <= f["deepcnet5_50_strokes_m8_b100"] <= 0.08
    assert f["deepcnet6_100_strokes_b64"] < 0.03
    assert abs(f["deepcnet5_100_rgbpatch_b128"] - 1024 / 96 ** 2) < 1e-12
    assert 0.01 < f["deepcnet4_20_strokes_b8"] < 0.08


def test_patch_stays_in_centred_region():
    cfg = get_config("deepcnet5_100_rgbpatch_b128")
    b = make_batch(cfg, 0)
    lo = (96 - 40) // 2
    assert b.coords[:, 1:].min() >= lo and b.coords[:, 1:].max() < lo + 40
    for s in range(cfg.batch):
        assert (b.coords[:, 0] == s).sum() == 1024


def test_circle_fixture():
    c = circle_sites(96, 32)
    assert c.batch == 1 and c.n > 80
    d = np.hypot(c.coords[:, 1] - 47.5, c.coords[:, 2] - 47.5)
    assert np.all(np.abs(d - 16) < 0.5)


def test_digit_pictures_shape():
    """Digit stand-ins (Section 2.5): about 150 grey-level pixels per sample, all inside the
    centred 28 x 28 frame of the 96 x 96 grid, grey levels in (0, 1]."""
    cfg = get_config("deepcnet5_10_digits_b1000")
    assert cfg.mode == "infer" and cfg.grid == 96 and (cfg.ell, cfg.k, cfg.n_classes) == (5, 10, 10)
    b = make_batch(cfg, 0)
    per = np.bincount(b.coords[:, 0], minlength=cfg.batch)
    assert 130 <= per.mean() <= 170 and per.min() > 0
    lo = (96 - 28) // 2
    assert b.coords[:, 1:].min() >= lo and b.coords[:, 1:].max() < lo + 28
    assert b.feats.min() > 0.0 and b.feats.max() <= 1.0
