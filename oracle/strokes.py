"""Input encoding of online pen strokes with 8-direction histograms (test infrastructure only).

Section 2.4 combines two representations of a handwritten character on one n x n
grid: the picture of the pen's path (one feature per square) and, per square, an
8-bin histogram of how much the pen moved in each of the 8 compass directions --
M = 1 + 8 = 9 features per site, all zero where the pen never went, so the input
stays sparse.

Readings (the paper gives no formula; each is listed in the design notes):

* strokes are sequences of integer grid points (y, x), y growing downwards;
  consecutive points are joined by the raster ``raster_segment``: with
  d = p1 - p0 and L = max(|dy|, |dx|), pixel i = 0 .. L is
  p0 + round_half_up(i * d / L), an exactly 8-connected line with both ends
  (a one-point stroke, or a repeated point, marks one pixel and no movement);
* each unit step of a raster (from pixel u to the next pixel v) is a move in
  one of the 8 compass directions E, NE, N, NW, W, SW, S, SE (indices 0..7,
  counter-clockwise, north = -y); its length is 1 (E, N, W, S) or sqrt(2)
  (diagonals) and it is shared equally by the two squares it joins: direction
  channel d of a site is (number of moves in direction d that start or end
  there) * length_d / 2;
* the picture channel (feature 0) is 1 at every site the pen touches; sites
  are the union of all raster pixels of the sample, listed in ascending
  (b, y, x) order.
"""

import math
from typing import Tuple

import numpy as np

# (dy, dx) of the 8 compass moves, counter-clockwise from east; y grows downwards
DIRS = ((0, 1), (-1, 1), (-1, 0), (-1, -1), (0, -1), (1, -1), (1, 0), (1, 1))
MOVE_LEN = tuple(1.0 if dy == 0 or dx == 0 else math.sqrt(2.0) for dy, dx in DIRS)
N_FEATURES = 9


def _round_half_up(num: int, den: int) -> int:
    """floor(num / den + 1/2) for integers, den > 0."""
    return (2 * num + den) // (2 * den)


def raster_segment(y0: int, x0: int, y1: int, x1: int):
    """The pixels of the segment p0 -> p1, p0 first and p1 last."""
    dy, dx = y1 - y0, x1 - x0
    L = max(abs(dy), abs(dx))
    if L == 0:
        return [(y0, x0)]
    return [(y0 + _round_half_up(i * dy, L), x0 + _round_half_up(i * dx, L)) for i in range(L + 1)]


def encode_strokes(points, stroke_begin, stroke_sample, batch: int, N: int) -> Tuple[np.ndarray, np.ndarray]:
    """Sites and M = 9 features of a batch of pen strokes (Section 2.4).

    ``points`` [P, 2] (y, x) integer grid points of all strokes, concatenated;
    stroke s is ``points[stroke_begin[s]:stroke_begin[s + 1]]`` and belongs to
    sample ``stroke_sample[s]``.  Returns coords [n, 3] (b, y, x) ascending and
    feats [n, 9] float64: the picture channel, then the 8 direction channels.
    """
    points = np.asarray(points, dtype=np.int64).reshape(-1, 2)
    begin = np.asarray(stroke_begin, dtype=np.int64)
    sample = np.asarray(stroke_sample, dtype=np.int64)
    if begin.size != sample.size + 1 or (begin.size and (begin[0] != 0 or begin[-1] != points.shape[0])):
        raise ValueError("stroke_begin must run from 0 to the point count, one entry per stroke plus one")
    if np.any(np.diff(begin) < 0):
        raise ValueError("stroke_begin must be non-decreasing")
    if points.size and (points.min() < 0 or points.max() >= N):
        raise ValueError("a point lies outside the grid")
    if sample.size and (sample.min() < 0 or sample.max() >= batch):
        raise ValueError("a stroke's sample lies outside the batch")
    counts = {}  # (b, y, x) -> move counts per direction

    def site(b, p):
        return counts.setdefault((b, p[0], p[1]), [0] * 8)

    for s in range(sample.size):
        b = int(sample[s])
        pts = points[begin[s]:begin[s + 1]]
        if len(pts) == 0:
            continue
        site(b, (int(pts[0][0]), int(pts[0][1])))
        for (y0, x0), (y1, x1) in zip(pts[:-1], pts[1:]):
            pix = raster_segment(int(y0), int(x0), int(y1), int(x1))
            for u, v in zip(pix[:-1], pix[1:]):
                d = DIRS.index((v[0] - u[0], v[1] - u[1]))
                site(b, u)[d] += 1
                site(b, v)[d] += 1
            site(b, pix[-1])
    keys = sorted(counts)
    coords = np.array(keys, dtype=np.int64).reshape(-1, 3)
    feats = np.zeros((len(keys), N_FEATURES))
    feats[:, 0] = 1.0
    for r, key in enumerate(keys):
        for d in range(8):
            feats[r, 1 + d] = counts[key][d] * MOVE_LEN[d] / 2.0
    return coords, feats
