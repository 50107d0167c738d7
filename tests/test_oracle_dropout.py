"""Pins for the oracle's dropout (Section 2.1: one rate per convolution input and one for
the softmax layer's input; Section 2.2: none on the 1x1 network-in-network layers).

* the generator against its published known-answer vectors;
* the keep rate, independence across channels, layers and seeds (binomial bounds);
* the sparse network with dropout against the dense network (torch autograd) given
  the same multipliers as explicit grids -- 1 at inactive sites, whose shared ground
  state is never dropped, and keep/(1 - p) at active ones;
* rate 0 and inference passes reduce exactly to the network without dropout.
"""

import os

import numpy as np
import pytest

from oracle import SparseDeepCNet
from oracle.philox import drop_scale, drop_threshold, dropout_keep, philox4x32_10
from tests.dense_ref import DenseDeepCNet, dilate_reference
from tests.test_oracle import _check_grad_against_dense, _check_layer_against_dense, _random_sites
from workloads import he_params, random_labels

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([int(t, 16) for t in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat_rows())
def test_philox_known_answers(row):
    c, k, want = row[:4], row[4:6], row[6:]
    got = philox4x32_10(*c, *k)
    assert [int(w) for w in got] == want


def test_philox_vectorised_equals_scalar():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 2 ** 32, size=(4, 50), dtype=np.uint64)
    k = rng.integers(0, 2 ** 32, size=(2, 50), dtype=np.uint64)
    vec = philox4x32_10(*c, *k)
    for i in range(50):
        one = philox4x32_10(*(int(x[i]) for x in c), *(int(x[i]) for x in k))
        assert [int(v[i]) for v in vec] == [int(o) for o in one]


def test_keep_rate_and_independence():
    keys = np.arange(40000) * 7 + 3
    for p in (0.1, 0.5, 0.75):
        m = dropout_keep(keys, 8, 2, p, 99)
        n = m.size
        assert abs(m.mean() - (1 - p)) < 5 * np.sqrt(p * (1 - p) / n)
        # adjacent channels (same and different Philox words) are uncorrelated
        for a, b in ((0, 1), (3, 4), (0, 7)):
            r = np.corrcoef(m[:, a], m[:, b])[0, 1]
            assert abs(r) < 5 / np.sqrt(m.shape[0])
    base = dropout_keep(keys[:4000], 8, 2, 0.5, 99)
    for other in (dropout_keep(keys[:4000], 8, 3, 0.5, 99), dropout_keep(keys[:4000], 8, 2, 0.5, 100),
                  dropout_keep(keys[:4000], 8, 2, 0.5, 99 + (1 << 32)), dropout_keep(keys[1:4001], 8, 2, 0.5, 99)):
        agree = (base == other).mean()
        assert abs(agree - 0.5) < 5 * np.sqrt(0.25 / base.size)
    np.testing.assert_array_equal(base, dropout_keep(keys[:4000], 8, 2, 0.5, 99))


def test_threshold_and_scale():
    assert drop_threshold(0.0) == 0 and drop_threshold(0.5) == 2 ** 31 and drop_threshold(0.25) == 2 ** 30
    assert drop_scale(0.5) == 2.0 and drop_scale(0.0) == 1.0
    assert dropout_keep(np.arange(100), 5, 0, 0.0, 1).all()
    with pytest.raises(ValueError):
        drop_threshold(1.0)


def _mask_grids(o, coords, batch, rates, seed):
    """Dense multipliers for every dropout level, from active sets found by library dilation."""
    N = o.N
    active = np.zeros((batch, N, N), bool)
    if coords.shape[0]:
        active[coords[:, 0], coords[:, 1], coords[:, 2]] = True
    grids = []
    j = 0
    for st in o.stages:
        if st.kind == "conv" and st.F > 1:
            g = np.ones((batch, st.c_in, st.S_in, st.S_in))
            b, y, x = np.nonzero(active)
            if rates[j] > 0 and b.size:
                keys = (b * st.S_in + y) * st.S_in + x
                fac = np.where(dropout_keep(keys, st.c_in, j, rates[j], seed), drop_scale(rates[j]), 0.0)
                g[b, :, y, x] = fac
            grids.append(g if rates[j] > 0 else None)
            j += 1
        active = dilate_reference(active, st.kind, st.F)
    p = rates[-1]
    grids.append(np.where(dropout_keep(np.arange(batch), o.stages[-1].c_out, j, p, seed), drop_scale(p), 0.0)
                 if p > 0 else None)
    return grids


DROP_CASES = [
    # arch, ell, k, c_in, classes, batch, density, empty, rates, seed
    ("deepcnet", 1, 3, 2, 3, 3, 0.3, (1,), [0.3, 0.5, 0.4], 31),
    ("deepcnet", 2, 3, 1, 4, 2, 0.1, (), [0.2, 0.0, 0.5, 0.25], 32),
    ("deepcnet", 3, 2, 2, 3, 2, 0.03, (), [0.0, 0.1, 0.2, 0.3, 0.5], 33),
    ("deepcnin", 2, 2, 1, 3, 3, 0.08, (0,), [0.5, 0.3, 0.2, 0.4], 34),
]


@pytest.mark.parametrize("arch,ell,k,c_in,ncls,batch,density,empty,rates,seed", DROP_CASES)
def test_dropout_equals_dense_network_with_mask_grids(arch, ell, k, c_in, ncls, batch, density, empty, rates, seed):
    rng = np.random.default_rng(seed)
    coords, feats = _random_sites(rng, batch, 3 * 2 ** ell, density, c_in, empty)
    Ws, bs = he_params(ell, k, c_in, ncls, seed, arch)
    labels = random_labels(batch, ncls, seed + 1)
    dseed = 0x1234_5678_9ABC + seed
    o = SparseDeepCNet(ell, k, c_in, ncls, "f64", arch)
    o.build(coords, batch)
    o.set_dropout(rates, dseed)
    o.forward(feats, Ws, bs, labels)
    o.backward()
    masks = _mask_grids(o, coords, batch, rates, dseed)
    d = DenseDeepCNet(ell, k, c_in, ncls, arch).run(coords, feats, batch, Ws, bs, labels, masks)
    for s in range(1, len(o.layers)):
        _check_layer_against_dense(o.layers[s], d.Ys[s - 1].detach().numpy())
    np.testing.assert_allclose(o.logits, d.logits, rtol=1e-10, atol=1e-12)
    assert abs(o.loss - d.loss) < 1e-10 * max(1.0, abs(d.loss))
    for a, b in zip(o.dW + o.db, d.dW + d.db):
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-12 * max(1.0, np.abs(b).max()))
    for s in range(1, len(o.layers)):
        st = o.stages[s - 1]
        dg = d.Zs[s - 1].grad if st.kind == "conv" else d.Ys[s - 1].grad
        _check_grad_against_dense(o.layers[s], dg.numpy())
    _check_grad_against_dense(o.layers[0], d.x.grad.numpy())
    # dropout changed something, and the ground rows were left alone
    assert any("drop" in L.extra for L in o.layers)
    for si in o.dropout_stages():
        np.testing.assert_array_equal(o.layers[si + 1].extra["Xin"][0], o.layers[si].X[0])


def _run(arch, rates, labels_on=True, mode="f64"):
    ell, k, c_in, ncls, batch = 2, 3, 2, 4, 3
    rng = np.random.default_rng(5)
    coords, feats = _random_sites(rng, batch, 12, 0.15, c_in)
    Ws, bs = he_params(ell, k, c_in, ncls, 5, arch)
    o = SparseDeepCNet(ell, k, c_in, ncls, mode, arch)
    o.build(coords, batch)
    o.set_dropout(rates, 77)
    logits, loss = o.forward(feats, Ws, bs, random_labels(batch, ncls, 6) if labels_on else None)
    if labels_on:
        o.backward()
    return o, logits


@pytest.mark.parametrize("arch", ["deepcnet", "deepcnin"])
@pytest.mark.parametrize("mode", ["f64", "bf16"])
def test_rate_zero_is_no_dropout(arch, mode):
    a, la = _run(arch, None, mode=mode)
    b, lb = _run(arch, [0.0] * 4, mode=mode)
    np.testing.assert_array_equal(la, lb)
    for x, y in zip(a.dW + a.db, b.dW + b.db):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(a.dfeats, b.dfeats)


def test_inference_pass_ignores_dropout():
    a, la = _run("deepcnet", None, labels_on=False)
    b, lb = _run("deepcnet", [0.5] * 4, labels_on=False)
    np.testing.assert_array_equal(la, lb)
    c, lc = _run("deepcnet", [0.5] * 4, labels_on=True)
    assert not np.array_equal(la, lc)
    with pytest.raises(RuntimeError):
        b.backward()


def test_bad_rates_rejected():
    o = SparseDeepCNet(2, 2, 1, 3)
    with pytest.raises(ValueError):
        o.set_dropout([0.1, 0.2, 0.3], 1)
    with pytest.raises(ValueError):
        o.set_dropout([0.1, 0.2, 1.0, 0.3], 1)
