"""Seeded generators: pen strokes, digit pictures, RGB patch, circle fixture, weights, labels.

All randomness comes from numpy's PCG64 (``np.random.default_rng``).  Values are
returned in float64; callers convert to the storage dtype they test.
"""

from dataclasses import dataclass
from typing import List, Tuple

import numpy as np

from .configs import WorkloadConfig


@dataclass
class Batch:
    """A batch of sparse inputs: ``coords[i] = (b, y, x)``, ``feats[i]`` its M features.

    Sites are listed in generation order (not sorted); every (b, y, x) appears once.
    """

    coords: np.ndarray  # int32 [n, 3]
    feats: np.ndarray  # float64 [n, M]
    batch: int
    grid: int

    @property
    def n(self) -> int:
        return int(self.coords.shape[0])

    def active_fraction(self) -> float:
        return self.n / float(self.batch * self.grid * self.grid)


def _bresenham(y0: int, x0: int, y1: int, x1: int) -> List[Tuple[int, int]]:
    """8-connected integer line from (y0, x0) to (y1, x1), both ends included."""
    pts = []
    dy, dx = abs(y1 - y0), abs(x1 - x0)
    sy = 1 if y1 >= y0 else -1
    sx = 1 if x1 >= x0 else -1
    err = dx - dy
    y, x = y0, x0
    while True:
        pts.append((y, x))
        if y == y1 and x == x1:
            break
        e2 = 2 * err
        if e2 > -dy:
            err -= dy
            x += sx
        if e2 < dx:
            err += dx
            y += sy
    return pts


def _strokes_one(rng: np.random.Generator, grid: int, strokes, points, box, sigma) -> List[Tuple[int, int]]:
    lo = (grid - box) // 2
    hi = lo + box - 1
    seen = {}
    n_strokes = int(rng.integers(strokes[0], strokes[1] + 1))
    for _ in range(n_strokes):
        n_pts = int(rng.integers(points[0], points[1] + 1))
        y = int(rng.integers(lo, hi + 1))
        x = int(rng.integers(lo, hi + 1))
        steps = np.rint(rng.normal(0.0, sigma, size=(n_pts - 1, 2))).astype(np.int64)
        seen.setdefault((y, x), None)
        for sy, sx in steps:
            ny = min(max(y + int(sy), lo), hi)
            nx = min(max(x + int(sx), lo), hi)
            for p in _bresenham(y, x, ny, nx):
                seen.setdefault(p, None)
            y, x = ny, nx
    return list(seen.keys())


@dataclass
class Paths:
    """A batch of raw pen paths: stroke s is ``points[stroke_begin[s]:stroke_begin[s + 1]]``
    ((y, x) integer grid points, in drawing order) of sample ``stroke_sample[s]``."""

    points: np.ndarray  # int32 [P, 2]
    stroke_begin: np.ndarray  # int32 [S + 1]
    stroke_sample: np.ndarray  # int32 [S]
    batch: int
    grid: int

    @property
    def n_points(self) -> int:
        return int(self.points.shape[0])

    @property
    def n_strokes(self) -> int:
        return int(self.stroke_sample.shape[0])


def _walk(rng: np.random.Generator, n_pts: int, lo: int, hi: int, sigma: float) -> np.ndarray:
    """One random-walk stroke: a uniform start in [lo, hi]^2, then round(N(0, sigma^2)) steps, clamped."""
    y = int(rng.integers(lo, hi + 1))
    x = int(rng.integers(lo, hi + 1))
    steps = np.rint(rng.normal(0.0, sigma, size=(n_pts - 1, 2))).astype(np.int64)
    pts = [(y, x)]
    for sy, sx in steps:
        y = min(max(y + int(sy), lo), hi)
        x = min(max(x + int(sx), lo), hi)
        pts.append((y, x))
    return np.asarray(pts, dtype=np.int32)


def stroke_paths(rng: np.random.Generator, batch: int, grid: int, strokes=(1, 20), points=(10, 60), box=64,
                 sigma=2.0) -> Paths:
    """Random-walk pen paths as in ``stroke_batch``, left as point sequences (not rasterised):
    the input of the 8-direction histogram encoding of Section 2.4."""
    lo = (grid - box) // 2
    hi = lo + box - 1
    pts, begin, sample = [], [0], []
    for b in range(batch):
        for _ in range(int(rng.integers(strokes[0], strokes[1] + 1))):
            w = _walk(rng, int(rng.integers(points[0], points[1] + 1)), lo, hi, sigma)
            pts.append(w)
            begin.append(begin[-1] + w.shape[0])
            sample.append(b)
    points_arr = np.concatenate(pts, axis=0) if pts else np.zeros((0, 2), np.int32)
    return Paths(points=points_arr.astype(np.int32), stroke_begin=np.asarray(begin, np.int32),
                 stroke_sample=np.asarray(sample, np.int32), batch=batch, grid=grid)


def stroke_batch(rng: np.random.Generator, batch: int, grid: int, c_in: int, strokes=(1, 20),
                 points=(10, 60), box=64, sigma=2.0, features="ones") -> Batch:
    """Random-walk pen strokes rasterised 1 px wide inside a centred box.

    Per sample: the stroke count and each stroke's point count are uniform
    integers in the given closed ranges; a stroke starts uniformly in the box
    and each step adds round(N(0, sigma^2)) per axis, clamped to the box;
    consecutive points are joined by an 8-connected Bresenham line; repeated
    pixels are kept once.  Features are 1.0 (``"ones"``) or i.i.d. N(0, 1)
    (``"normal"``), ``c_in`` of them per pixel.
    """
    coords = []
    for b in range(batch):
        pix = _strokes_one(rng, grid, strokes, points, box, sigma)
        if pix:
            arr = np.asarray(pix, dtype=np.int32)
            coords.append(np.concatenate([np.full((len(pix), 1), b, np.int32), arr], axis=1))
    coords = np.concatenate(coords, axis=0) if coords else np.zeros((0, 3), np.int32)
    if features == "ones":
        feats = np.ones((coords.shape[0], c_in), np.float64)
    elif features == "normal":
        feats = rng.normal(0.0, 1.0, size=(coords.shape[0], c_in))
    else:
        raise ValueError(features)
    return Batch(coords=coords.astype(np.int32), feats=feats, batch=batch, grid=grid)


def digit_batch(rng: np.random.Generator, batch: int, grid: int, c_in: int = 1, strokes=(2, 4), points=(10, 18),
                box=20, sigma=2.5, brush=2) -> Batch:
    """Handwritten-digit stand-ins: grey-level strokes in the middle of the grid.

    Section 2.5 places 28 x 28 digit pictures (on average about 150 non-zero
    pixels on a zero background) in the middle of the 96 x 96 input layer.  Per
    sample: random-walk strokes as in ``stroke_batch`` inside a centred
    ``box x box`` square, each pixel widened to a ``brush x brush`` block (down
    and right), so the digit stays inside the centred 28 x 28 frame; the
    defaults give about 150 active pixels per sample.  Each active pixel gets
    ``c_in`` grey levels uniform in (0, 1].
    """
    coords = []
    for b in range(batch):
        pix = _strokes_one(rng, grid, strokes, points, box, sigma)
        seen = {}
        for (y, x) in pix:
            for dy in range(brush):
                for dx in range(brush):
                    seen.setdefault((y + dy, x + dx), None)
        if seen:
            arr = np.asarray(list(seen.keys()), dtype=np.int32)
            coords.append(np.concatenate([np.full((len(arr), 1), b, np.int32), arr], axis=1))
    coords = np.concatenate(coords, axis=0) if coords else np.zeros((0, 3), np.int32)
    feats = 1.0 - rng.random(size=(coords.shape[0], c_in))
    return Batch(coords=coords.astype(np.int32), feats=feats, batch=batch, grid=grid)


def patch_batch(rng: np.random.Generator, batch: int, grid: int, c_in: int = 3, patch=32, region=40) -> Batch:
    """A dense ``patch x patch`` block of U[0,1) features at a random offset.

    The block's top-left corner is ``lo + (oy, ox)`` with ``lo = (grid - region) // 2``
    and ``oy, ox`` uniform in ``0 .. region - patch``, so the block stays inside
    the centred ``region x region`` square.  Every pixel of the block is active.
    """
    lo = (grid - region) // 2
    coords = []
    for b in range(batch):
        oy = int(rng.integers(0, region - patch + 1))
        ox = int(rng.integers(0, region - patch + 1))
        yy, xx = np.meshgrid(np.arange(patch) + lo + oy, np.arange(patch) + lo + ox, indexing="ij")
        c = np.stack([np.full(yy.size, b), yy.ravel(), xx.ravel()], axis=1)
        coords.append(c)
    coords = np.concatenate(coords, axis=0).astype(np.int32)
    # shuffle the listing order: the interface takes sites in any order
    perm = rng.permutation(coords.shape[0])
    coords = coords[perm]
    feats = rng.random(size=(coords.shape[0], c_in))
    return Batch(coords=coords, feats=feats, batch=batch, grid=grid)


def circle_sites(grid: int = 96, diameter: int = 32) -> Batch:
    """A 1-px circle outline of the given diameter centred in the grid (one sample).

    Pixel (y, x) is on the outline when its centre lies within half a pixel of
    the circle of radius ``diameter / 2`` around the grid centre.
    """
    c = (grid - 1) / 2.0
    r = diameter / 2.0
    yy, xx = np.meshgrid(np.arange(grid), np.arange(grid), indexing="ij")
    d = np.sqrt((yy - c) ** 2 + (xx - c) ** 2)
    on = np.abs(d - r) < 0.5
    ys, xs = np.nonzero(on)
    coords = np.stack([np.zeros_like(ys), ys, xs], axis=1).astype(np.int32)
    feats = np.ones((coords.shape[0], 1), np.float64)
    return Batch(coords=coords, feats=feats, batch=1, grid=grid)


def _layer_shapes(ell: int, k: int, c_in: int, arch: str = "deepcnet"):
    """(fan_in_rows, c_out) of each convolution weight in stage order: 3x3 first, then
    2x2; conv n has n*k filters.  DeepCNiN adds a 1x1 layer of the same width after
    every pooling layer and after the last convolution."""
    shapes = [(9 * c_in, k)]
    for n in range(2, ell + 2):
        if arch == "deepcnin":
            shapes.append(((n - 1) * k, (n - 1) * k))
        shapes.append((4 * (n - 1) * k, n * k))
    if arch == "deepcnin":
        shapes.append(((ell + 1) * k, (ell + 1) * k))
    return shapes


def he_params(ell: int, k: int, c_in: int, n_classes: int, seed: int, arch: str = "deepcnet"):
    """Random parameters for DeepCNet(ell, k): U[-0.1, 0.1] biases; He-normal
    convolution weights (N(0, 2/fan_in), the usual choice before a ReLU) and a
    Glorot-normal softmax layer (N(0, 2/(fan_in + fan_out)), the usual choice for
    a linear output layer; it keeps fresh logits O(1) instead of saturating the
    softmax).

    Returns ``(Ws, bs)``: one matrix per convolution in stage order (``ell + 1`` for
    DeepCNet, ``2 ell + 2`` for DeepCNiN), each ``[F*F*C_in, C_out]``
    (rows ordered ``(dy*F + dx)*C_in + c``) followed by the softmax layer's
    ``[C_last, n_classes]``, and the matching bias vectors.  Biases are non-zero
    on purpose: with zero biases every ground state would be zero.
    """
    rng = np.random.default_rng(seed)
    shapes = _layer_shapes(ell, k, c_in, arch) + [((ell + 1) * k, n_classes)]
    Ws, bs = [], []
    for i, (rows, cols) in enumerate(shapes):
        var = 2.0 / rows if i < len(shapes) - 1 else 2.0 / (rows + cols)
        Ws.append(rng.normal(0.0, np.sqrt(var), size=(rows, cols)))
        bs.append(rng.uniform(-0.1, 0.1, size=cols))
    return Ws, bs


def random_labels(batch: int, n_classes: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_classes, size=batch).astype(np.int32)


def make_paths(cfg: WorkloadConfig, index: int = 0) -> Paths:
    """Pen-path batch number ``index`` of a workload whose input is encoded from paths."""
    if cfg.generator != "paths":
        raise ValueError(f"{cfg.name} does not draw pen paths")
    rng = np.random.default_rng([cfg.seed, index])
    return stroke_paths(rng, cfg.batch, cfg.grid, **cfg.gen_args)


def make_batch(cfg: WorkloadConfig, index: int = 0) -> Batch:
    """Batch number ``index`` of a workload (seeded by the workload seed and ``index``)."""
    if cfg.generator == "paths":
        raise ValueError(f"{cfg.name} draws pen paths: use make_paths and encode them")
    rng = np.random.default_rng([cfg.seed, index])
    if cfg.generator == "strokes":
        return stroke_batch(rng, cfg.batch, cfg.grid, cfg.c_in, **cfg.gen_args)
    if cfg.generator == "patch":
        return patch_batch(rng, cfg.batch, cfg.grid, cfg.c_in, **cfg.gen_args)
    if cfg.generator == "digits":
        return digit_batch(rng, cfg.batch, cfg.grid, cfg.c_in, **cfg.gen_args)
    raise ValueError(cfg.generator)


def make_batches(cfg: WorkloadConfig, count: int) -> List[Batch]:
    return [make_batch(cfg, i) for i in range(count)]
