"""The identity behind the per-layer bitmap kernel, on the CPU.

A valid F x F convolution marks an output site active when any input site of its
window is active, a 2 x 2 stride-2 pooling when any of its four is (Section 2.1).
Chained, layer s marks (Y, X) active exactly when an input site lies in the square
of side r_s from (a_s Y, a_s X), with a_s the product of the pooling strides and
r_s = r_{s-1} + a_{s-1} (F_s - 1) (a pooling counts as F = 2 and doubles a).  The
kernel computes every layer that way, straight from the input; this checks the
identity against the layer-by-layer definition for both network families.
"""

import numpy as np
import pytest


def _layers(ell, nin):
    ks = [("conv", 3)]
    for _ in range(ell):
        ks.append(("pool", 2))
        if nin:
            ks.append(("conv", 1))
        ks.append(("conv", 2))
    if nin:
        ks.append(("conv", 1))
    return ks


def _chain(g, ks):
    out, p = [], g
    for kind, F in ks:
        S = p.shape[0]
        if kind == "conv":
            So = S - F + 1
            o = np.zeros((So, So), bool)
            for dy in range(F):
                for dx in range(F):
                    o |= p[dy:dy + So, dx:dx + So]
        else:
            So = S // 2
            q = p[:2 * So, :2 * So]
            o = q[0::2, 0::2] | q[0::2, 1::2] | q[1::2, 0::2] | q[1::2, 1::2]
        out.append(o)
        p = o
    return out


def _composite(g, ks):
    N = g.shape[0]
    # prefix sums: "any site in a square" as a count > 0
    P = np.zeros((N + 1, N + 1), np.int64)
    P[1:, 1:] = g.astype(np.int64).cumsum(0).cumsum(1)
    out, a, r, S = [], 1, 1, N
    for kind, F in ks:
        r += a * (F - 1)
        if kind == "pool":
            a *= 2
            S //= 2
        else:
            S = S - F + 1
        Y = np.arange(S)[:, None] * a
        X = np.arange(S)[None, :] * a
        cnt = P[Y + r, X + r] - P[Y, X + r] - P[Y + r, X] + P[Y, X]
        out.append(cnt > 0)
    return out


@pytest.mark.parametrize("nin", [False, True])
@pytest.mark.parametrize("ell", [1, 2, 3, 4, 5])
def test_composite_window_equals_layer_chain(ell, nin):
    rng = np.random.default_rng(10 * ell + nin)
    N = 3 * 2 ** ell
    ks = _layers(ell, nin)
    for dens in (0.0, 0.002, 0.03, 0.3, 1.0):
        g = rng.random((N, N)) < dens
        for s, (want, got) in enumerate(zip(_chain(g, ks), _composite(g, ks)), start=1):
            assert want.shape == got.shape, (s, want.shape, got.shape)
            np.testing.assert_array_equal(got, want, err_msg=f"ell={ell} nin={nin} dens={dens} layer {s}")
