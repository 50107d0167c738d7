"""Pins for the oracle's input encoding (Section 2.4: picture plus 8-direction histograms,
M = 9) and its SGD update.

Encoding: the raster against the classic integer Bresenham line wherever the rounding
has no tie, the raster's distance bound, a hand-worked stroke, the total histogram mass
against the closed-form length of the rasterised path, the transposition and
stroke-reversal symmetries, and the picture channel against the pictures of the same
paths drawn by the generator.  SGD: against the library optimiser (torch.optim.SGD) and
a loss that falls when the oracle network is trained on a fixed synthetic batch.
"""

import math

import numpy as np
import pytest
import torch

from oracle import SparseDeepCNet
from oracle.sgd import sgd_step
from oracle.strokes import DIRS, encode_strokes, raster_segment
from workloads import he_params, random_labels, stroke_paths
from workloads.synth import _bresenham


def _has_tie(y0, x0, y1, x1):
    dy, dx = y1 - y0, x1 - x0
    L = max(abs(dy), abs(dx))
    return L > 0 and any((2 * i * dm) % (2 * L) == L for i in range(L + 1) for dm in (dy, dx))


def test_raster_equals_bresenham_without_ties_and_stays_within_half_a_pixel():
    rng = np.random.default_rng(0)
    checked = 0
    for _ in range(3000):
        y0, x0, y1, x1 = (int(v) for v in rng.integers(-12, 13, 4))
        pix = raster_segment(y0, x0, y1, x1)
        L = max(abs(y1 - y0), abs(x1 - x0))
        assert len(pix) == L + 1 and pix[0] == (y0, x0) and pix[-1] == (y1, x1)
        for u, v in zip(pix[:-1], pix[1:]):
            assert (v[0] - u[0], v[1] - u[1]) in DIRS
        for i, (y, x) in enumerate(pix):
            t = i / L if L else 0.0
            assert abs(y - (y0 + t * (y1 - y0))) <= 0.5 + 1e-12 and abs(x - (x0 + t * (x1 - x0))) <= 0.5 + 1e-12
        if not _has_tie(y0, x0, y1, x1):
            assert pix == _bresenham(y0, x0, y1, x1)
            checked += 1
    assert checked > 1000


def test_hand_worked_stroke():
    """(2,2) -> (2,6) -> (5,6): four moves east, then three south (y grows downwards)."""
    coords, feats = encode_strokes([[2, 2], [2, 6], [5, 6]], [0, 3], [0], 1, 12)
    assert coords.tolist() == [[0, 2, 2], [0, 2, 3], [0, 2, 4], [0, 2, 5], [0, 2, 6], [0, 3, 6], [0, 4, 6], [0, 5, 6]]
    E, S = 1 + 0, 1 + 6
    want = np.zeros((8, 9))
    want[:, 0] = 1
    want[[0, 1, 2, 3, 4], E] = [0.5, 1, 1, 1, 0.5]
    want[[4, 5, 6, 7], S] = [0.5, 1, 1, 0.5]
    np.testing.assert_array_equal(feats, want)
    # one diagonal move: half of sqrt(2) at each end, direction NE (dy = -1, dx = +1)
    coords, feats = encode_strokes([[5, 5], [4, 6]], [0, 2], [0], 1, 12)
    assert coords.tolist() == [[0, 4, 6], [0, 5, 5]]
    np.testing.assert_allclose(feats[:, 1 + 1], [math.sqrt(2) / 2] * 2, rtol=0, atol=1e-15)
    assert feats[:, 1:].sum() == pytest.approx(math.sqrt(2))


def _paths(seed, batch=5, grid=48):
    return stroke_paths(np.random.default_rng(seed), batch, grid, (1, 6), (1, 25), 40, 2.5)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_histogram_mass_is_the_rasterised_path_length(seed):
    """Every move gives half its length to each end: per sample, the direction channels sum to
    the raster's length, which for a segment of extent L with minor-axis extent m is
    (L - m) + sqrt(2) m (m diagonal moves, L - m axis moves)."""
    p = _paths(seed)
    coords, feats = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
    want = np.zeros(p.batch)
    for s in range(p.n_strokes):
        pts = p.points[p.stroke_begin[s]:p.stroke_begin[s + 1]].astype(np.int64)
        for a, c in zip(pts[:-1], pts[1:]):
            d = np.abs(c - a)
            L, m = d.max(), d.min()
            want[p.stroke_sample[s]] += (L - m) + math.sqrt(2) * m
    got = np.bincount(coords[:, 0], weights=feats[:, 1:].sum(axis=1), minlength=p.batch)
    np.testing.assert_allclose(got, want, rtol=1e-12)
    assert np.all(feats[:, 0] == 1.0)


def test_transposition_and_reversal_symmetries():
    p = _paths(7)
    c, f = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
    # transpose the grid: (y, x) -> (x, y) maps direction (dy, dx) to (dx, dy)
    perm = [DIRS.index((dx, dy)) for dy, dx in DIRS]
    ct, ft = encode_strokes(p.points[:, ::-1], p.stroke_begin, p.stroke_sample, p.batch, p.grid)
    key = lambda cc: (cc[:, 0] * p.grid + cc[:, 1]) * p.grid + cc[:, 2]
    order = np.argsort(key(c[:, [0, 2, 1]]))
    np.testing.assert_array_equal(ct, c[:, [0, 2, 1]][order])
    np.testing.assert_allclose(ft[:, 1 + np.array(perm)], f[order][:, 1:], rtol=0, atol=0)
    # reverse every stroke: the same pixels, every move in the opposite direction
    pts = np.concatenate([p.points[p.stroke_begin[s]:p.stroke_begin[s + 1]][::-1] for s in range(p.n_strokes)])
    cr, fr = encode_strokes(pts, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
    np.testing.assert_array_equal(cr, c)
    np.testing.assert_array_equal(fr[:, 1:], np.roll(f[:, 1:], 4, axis=1))


def test_picture_channel_matches_generator_pictures_of_tie_free_paths():
    """Sites are the pen's picture: for paths whose segments round without ties, exactly the
    pixels the generator's Bresenham rasteriser draws."""
    p = _paths(11, batch=8)
    keep = []
    for s in range(p.n_strokes):
        pts = p.points[p.stroke_begin[s]:p.stroke_begin[s + 1]]
        keep.append(all(not _has_tie(int(a[0]), int(a[1]), int(b[0]), int(b[1])) for a, b in zip(pts[:-1], pts[1:])))
    sel = [s for s in range(p.n_strokes) if keep[s]]
    assert len(sel) >= 5
    pts = [p.points[p.stroke_begin[s]:p.stroke_begin[s + 1]] for s in sel]
    begin = np.concatenate([[0], np.cumsum([len(x) for x in pts])])
    coords, _ = encode_strokes(np.concatenate(pts), begin, p.stroke_sample[sel], p.batch, p.grid)
    want = set()
    for s, x in zip(sel, pts):
        b = int(p.stroke_sample[s])
        want.add((b, int(x[0][0]), int(x[0][1])))
        for a, c in zip(x[:-1], x[1:]):
            want.update((b, y, xx) for y, xx in _bresenham(int(a[0]), int(a[1]), int(c[0]), int(c[1])))
    assert sorted(want) == [tuple(r) for r in coords.tolist()]


def test_bad_paths_rejected():
    with pytest.raises(ValueError):
        encode_strokes([[0, 0], [0, 12]], [0, 2], [0], 1, 12)  # outside the grid
    with pytest.raises(ValueError):
        encode_strokes([[0, 0]], [0, 1], [1], 1, 12)  # sample outside the batch
    with pytest.raises(ValueError):
        encode_strokes([[0, 0], [1, 1]], [0, 2, 1], [0, 0], 1, 12)  # decreasing offsets
    c, f = encode_strokes(np.zeros((0, 2)), [0, 0], [0], 1, 12)  # an empty stroke draws nothing
    assert c.shape == (0, 3) and f.shape == (0, 9)


def test_sgd_matches_library_optimiser():
    rng = np.random.default_rng(3)
    shapes = [(6, 4), (4, 3)]
    W = [rng.normal(size=s) for s in shapes]
    b = [rng.normal(size=s[1]) for s in shapes]
    vW = [np.zeros(s) for s in shapes]
    vb = [np.zeros(s[1]) for s in shapes]
    tW = [torch.tensor(w, requires_grad=True) for w in W]
    tb = [torch.tensor(x, requires_grad=True) for x in b]
    lr, mom, wd = 0.05, 0.9, 1e-3
    opt = torch.optim.SGD([{"params": tW, "weight_decay": wd}, {"params": tb, "weight_decay": 0.0}], lr=lr,
                          momentum=mom)
    for step in range(4):
        dW = [rng.normal(size=s) for s in shapes]
        db = [rng.normal(size=s[1]) for s in shapes]
        W, _, b, vW, vb = sgd_step(W, b, dW, db, vW, vb, lr, mom, wd)
        for t, g in zip(tW + tb, dW + db):
            t.grad = torch.tensor(g)
        opt.step()
        for a, t in zip(W + b, tW + tb):
            np.testing.assert_allclose(a, t.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_training_the_oracle_lowers_the_loss():
    """The loop closes: SGD on the oracle's gradients fits a fixed synthetic batch."""
    ell, k, ncls, batch = 2, 4, 3, 6
    p = stroke_paths(np.random.default_rng(5), batch, 12, (1, 2), (2, 6), 10, 1.5)
    coords, feats = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, batch, 12)
    Ws, bs = he_params(ell, k, 9, ncls, 6)
    labels = random_labels(batch, ncls, 7)
    vW = [np.zeros_like(w) for w in Ws]
    vb = [np.zeros_like(x) for x in bs]
    losses = []
    for _ in range(40):
        o = SparseDeepCNet(ell, k, 9, ncls)
        o.build(coords, batch)
        losses.append(o.forward(feats, Ws, bs, labels)[1])
        dW, db, _ = o.backward()
        Ws, _, bs, vW, vb = sgd_step(Ws, bs, dW, db, vW, vb, 0.05, 0.9, 0.0, mode="f64")
    assert losses[-1] < 0.25 * losses[0], losses[::8]
