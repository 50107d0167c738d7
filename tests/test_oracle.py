"""Pins for the CPU oracle: it is checked against things other than itself.

* the dense network computed with torch's library routines and autograd
  (sparse features equal dense values at active sites and the ground state
  elsewhere; gradients equal dense autograd);
* closed forms the paper states: stage sizes, the DeepCNet(4,100) layer list,
  the parameter count, the path-count plateau;
* the translation property of Section 2.6;
* active sets from library dilation (torch conv2d / scipy.signal);
* central finite differences, textbook cross-entropy, torch's bfloat16 cast.
"""

import os

import numpy as np
import pytest
import scipy.signal
import torch
import torch.nn.functional as Fn

from oracle import OracleInputError, SparseDeepCNet, round_bf16, stage_plan
from tests.dense_ref import DenseDeepCNet, dilate_reference
from workloads import circle_sites, he_params, random_labels

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _random_sites(rng, batch, N, p, c_in, empty_samples=(), full_samples=()):
    coords = []
    for b in range(batch):
        if b in empty_samples:
            continue
        mask = np.ones((N, N), bool) if b in full_samples else rng.random((N, N)) < p
        ys, xs = np.nonzero(mask)
        coords.append(np.stack([np.full(ys.size, b), ys, xs], 1))
    coords = np.concatenate(coords) if coords else np.zeros((0, 3), np.int64)
    coords = coords[rng.permutation(coords.shape[0])]
    feats = rng.normal(size=(coords.shape[0], c_in))
    return coords.astype(np.int64), feats


def _run_pair(ell, k, c_in, n_classes, batch, coords, feats, seed, arch="deepcnet"):
    Ws, bs = he_params(ell, k, c_in, n_classes, seed, arch)
    labels = random_labels(batch, n_classes, seed + 1)
    o = SparseDeepCNet(ell, k, c_in, n_classes, "f64", arch)
    o.build(coords, batch)
    o.forward(feats, Ws, bs, labels)
    o.backward()
    d = DenseDeepCNet(ell, k, c_in, n_classes, arch).run(coords, feats, batch, Ws, bs, labels)
    return o, d


def _check_layer_against_dense(L, dense, tol=1e-10):
    """dense: [B, C, S, S]; active sites equal their rows, inactive sites equal row 0."""
    B, C, S, _ = dense.shape
    scale = max(np.abs(dense).max(), 1e-30)
    act = L.P != 0
    got = L.X[L.P]  # [B, S, S, C] -- row 0 (ground) wherever inactive
    np.testing.assert_allclose(got, dense.transpose(0, 2, 3, 1), atol=tol * scale, rtol=0)
    return act


def _check_grad_against_dense(L, dense_grad, tol=1e-9):
    """Active rows equal the dense gradient; row 0 equals its sum over inactive sites."""
    g = dense_grad.transpose(0, 2, 3, 1)  # [B, S, S, C]
    scale = max(np.abs(g).max(), 1e-30)
    act = L.P != 0
    np.testing.assert_allclose(L.grad[L.P[act]], g[act], atol=tol * scale, rtol=0)
    np.testing.assert_allclose(L.grad[0], g[~act].sum(axis=0), atol=tol * max(scale, np.abs(g[~act]).sum()), rtol=0)


CASES = [
    # ell, k, c_in, classes, batch, p, empty, full, seed
    (1, 2, 1, 3, 2, 0.2, (), (), 11),
    (1, 3, 3, 4, 3, 0.3, (1,), (), 12),
    (2, 2, 1, 5, 2, 0.1, (), (1,), 13),
    (2, 3, 3, 3, 3, 0.05, (0,), (), 14),
    (3, 2, 1, 4, 2, 0.03, (), (), 15),
    (3, 1, 2, 3, 1, 0.02, (), (), 16),
]


ARCH_CASES = [("deepcnet",) + c for c in CASES] + [
    # DeepCNiN (Section 2.2): 1x1 layers and the leaky rectifier
    ("deepcnin", 1, 2, 1, 3, 2, 0.2, (), (), 21),
    ("deepcnin", 2, 2, 2, 4, 3, 0.08, (1,), (), 22),
    ("deepcnin", 2, 3, 1, 3, 2, 0.1, (), (0,), 23),
    ("deepcnin", 3, 2, 1, 3, 1, 0.03, (), (), 24),
]


@pytest.mark.parametrize("arch,ell,k,c_in,ncls,batch,p,empty,full,seed", ARCH_CASES)
def test_oracle_equals_dense_network(arch, ell, k, c_in, ncls, batch, p, empty, full, seed):
    rng = np.random.default_rng(seed)
    coords, feats = _random_sites(rng, batch, 3 * 2 ** ell, p, c_in, empty, full)
    o, d = _run_pair(ell, k, c_in, ncls, batch, coords, feats, seed, arch)
    # forward: every layer, active and inactive sites
    for s in range(1, len(o.layers)):
        _check_layer_against_dense(o.layers[s], d.Ys[s - 1].detach().numpy())
    np.testing.assert_allclose(o.logits, d.logits, rtol=1e-10, atol=1e-12)
    assert abs(o.loss - d.loss) < 1e-10 * max(1.0, abs(d.loss))
    # parameter gradients
    for a, b in zip(o.dW, d.dW):
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-12 * max(1.0, np.abs(b).max()))
    for a, b in zip(o.db, d.db):
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-12 * max(1.0, np.abs(b).max()))
    # layer gradients: conv layers hold dL/dZ, pooling layers dL/dY
    for s in range(1, len(o.layers)):
        st = o.stages[s - 1]
        dg = d.Zs[s - 1].grad if st.kind == "conv" else d.Ys[s - 1].grad
        _check_grad_against_dense(o.layers[s], dg.numpy())
    # input gradient
    _check_grad_against_dense(o.layers[0], d.x.grad.numpy())


def test_oracle_all_active_is_dense_without_ground():
    """Fully active input: every layer is fully active below the 1x1 top, no window reads row 0."""
    rng = np.random.default_rng(3)
    ell, k, c_in = 2, 2, 2
    coords, feats = _random_sites(rng, 2, 12, 1.0, c_in, (), (0, 1))
    o, d = _run_pair(ell, k, c_in, 3, 2, coords, feats, 5)
    for s, L in enumerate(o.layers):
        assert L.n == 2 * L.S * L.S
        if s:
            assert (L.R[1:] != 0).all()


def test_oracle_zero_bias_ground_is_zero():
    rng = np.random.default_rng(4)
    ell, k, c_in, ncls = 2, 3, 1, 4
    coords, feats = _random_sites(rng, 2, 12, 0.1, c_in)
    Ws, bs = he_params(ell, k, c_in, ncls, 9)
    bs = [np.zeros_like(b) for b in bs]
    o = SparseDeepCNet(ell, k, c_in, ncls)
    o.build(coords, 2)
    o.forward(feats, Ws, bs, [0, 1])
    for L in o.layers:
        assert np.all(L.X[0] == 0)


def test_oracle_empty_batch_is_ground_everywhere():
    ell, k, c_in, ncls = 2, 2, 1, 3
    Ws, bs = he_params(ell, k, c_in, ncls, 2)
    o = SparseDeepCNet(ell, k, c_in, ncls)
    assert o.build(np.zeros((0, 3), np.int64), 2) == [0] * (2 * ell + 2)
    logits, loss = o.forward(np.zeros((0, 1)), Ws, bs, [0, 2])
    d = DenseDeepCNet(ell, k, c_in, ncls).run(np.zeros((0, 3), np.int64), np.zeros((0, 1)), 2, Ws, bs, [0, 2])
    np.testing.assert_allclose(logits, d.logits, rtol=1e-12)
    np.testing.assert_allclose(logits[0], logits[1])
    dW, db, _ = o.backward()
    for a, b in zip(dW, d.dW):
        np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-14)


@pytest.mark.parametrize("bad,kind", [
    ([[0, 1, 1], [0, 1, 1]], "duplicate"),
    ([[0, 12, 1]], "out_of_range"),
    ([[0, 1, -1]], "out_of_range"),
    ([[2, 1, 1]], "out_of_range"),
])
def test_oracle_rejects_undefined_inputs(bad, kind):
    o = SparseDeepCNet(2, 2, 1, 3)
    with pytest.raises(OracleInputError) as e:
        o.build(np.array(bad), 2)
    assert e.value.kind == kind


def test_stage_sizes_closed_form():
    # Section 2.1 / Figure 1: for ell = 5 the spatial sizes go from 96 down to 1
    sizes = [96] + [s.S for s in stage_plan(5, 10, 1)]
    assert sizes == [96, 94, 47, 46, 23, 22, 11, 10, 5, 4, 2, 1]
    for ell in range(1, 8):
        st = stage_plan(ell, 1, 1)
        assert st[0].S_in == 3 * 2 ** ell and st[-1].S == 1
        assert [s.kind for s in st] == ["conv"] + ["pool", "conv"] * ell


@pytest.mark.parametrize("arch,fname", [("deepcnet", "deepcnet_4_100_layer_list.txt"),
                                        ("deepcnin", "deepcnin_4_100_layer_list.txt")])
def test_layer_list_golden(arch, fname):
    # Section 2.1 gives DeepCNet(4,100)'s layer list, Section 2.2 DeepCNiN(4,100)'s
    with open(os.path.join(GOLDEN, fname)) as f:
        lines = [l.strip() for l in f if l.strip() and not l.startswith("#")]
    hdr = dict(kv.split("=") for kv in lines[0].split())
    ell, k = int(hdr["ell"]), int(hdr["k"])
    tokens = lines[1].split("-")
    assert tokens[0] == "input" and tokens[-1] == "output"
    expected = []
    for s in stage_plan(ell, k, 1, arch):
        expected.append(f"{s.c_out}C{s.F}" if s.kind == "conv" else "MP2")
    assert tokens[1:-1] == expected
    assert stage_plan(ell, k, 1, arch)[0].S_in == int(hdr["N"])


@pytest.mark.parametrize("ell,k,M", [(1, 3, 1), (4, 20, 1), (5, 50, 9), (6, 100, 1)])
def test_parameter_count_closed_form(ell, k, M):
    # Section 2.1: 3^2 M k + sum_{n=1..ell} 2^2 (n k)((n+1) k) weights (the n = 1 term read as 2^2 k (2k))
    o = SparseDeepCNet(ell, k, M, 10)
    conv = o.param_shapes()[:-1]
    total = sum(r * c for r, c in conv)
    assert total == 9 * M * k + sum(4 * (n * k) * ((n + 1) * k) for n in range(1, ell + 1))
    assert conv[0] == (9 * M, k)


def _path_counts(o):
    """Routes from every input site to the top layer, following the window lists downwards."""
    cnt = np.zeros(o.layers[-1].n + 1)
    cnt[1:] = 1.0
    for s in range(len(o.layers) - 1, 0, -1):
        L, below = o.layers[s], o.layers[s - 1]
        nxt = np.zeros(below.n + 1)
        R = L.R[1:]
        np.add.at(nxt, R.ravel(), np.repeat(cnt[1:], R.shape[1]))
        nxt[0] = 0.0  # the ground row is not a site
        cnt = nxt
    grid = cnt[o.layers[0].P[0]]
    return grid


def test_path_count_plateau_golden():
    with open(os.path.join(GOLDEN, "path_counts.txt")) as f:
        rows = [list(map(int, l.split())) for l in f if l.strip() and not l.startswith("#")]
    for ell, corner, central in rows:
        if ell > 4:
            continue  # keep the CPU suite quick; ell = 5 is covered by the GPU rulebook test
        N = 3 * 2 ** ell
        ys, xs = np.meshgrid(np.arange(N), np.arange(N), indexing="ij")
        coords = np.stack([np.zeros(N * N, int), ys.ravel(), xs.ravel()], 1)
        o = SparseDeepCNet(ell, 1, 1, 2)
        o.build(coords, 1)
        g = _path_counts(o)
        for y, x in [(0, 0), (0, N - 1), (N - 1, 0), (N - 1, N - 1)]:
            assert g[y, x] == corner
        c = g[N // 3: 2 * N // 3, N // 3: 2 * N // 3]
        assert c.shape == (N // 3, N // 3) and np.all(c == central)
        assert g.max() == central
        assert central == 9 * 4 ** (ell - 1)


@pytest.mark.parametrize("kshift", [1, 2, 3])
def test_translation_by_power_of_two_moves_pool_output_by_one(kshift):
    # Section 2.6: shifting a sparse input by 2^k shifts the k-th pooling layer's output by exactly one
    # the object keeps a margin of 2^(k+1) from the grid's edges so no layer up to the
    # k-th pooling level clips it (the property is about sparse inputs away from the border)
    ell, k, c_in, ncls = 4, 2, 2, 3
    rng = np.random.default_rng(20 + kshift)
    lo = 2 ** (kshift + 1)
    pts = rng.integers(lo, lo + 6, size=(25, 2))
    pts = np.unique(pts, axis=0)
    coords = np.concatenate([np.zeros((len(pts), 1), int), pts], 1)
    feats = rng.normal(size=(len(pts), c_in))
    Ws, bs = he_params(ell, k, c_in, ncls, 1)
    shifted = coords.copy()
    shifted[:, 1:] += 2 ** kshift
    outs = []
    for c in (coords, shifted):
        o = SparseDeepCNet(ell, k, c_in, ncls)
        o.build(c, 1)
        o.forward(feats, Ws, bs, [0])
        outs.append(o.layers[2 * kshift])  # layer after the k-th pooling stage
    a, b = outs
    assert a.n == b.n
    np.testing.assert_array_equal(a.sites[:, 1:] + 1, b.sites[:, 1:])
    np.testing.assert_allclose(a.X, b.X, rtol=1e-13, atol=1e-13)


def test_active_sets_match_library_dilation():
    rng = np.random.default_rng(30)
    for ell, p in [(2, 0.05), (3, 0.02), (4, 0.01)]:
        N = 3 * 2 ** ell
        coords, feats = _random_sites(rng, 3, N, p, 1, empty_samples=(1,))
        o = SparseDeepCNet(ell, 1, 1, 2)
        o.build(coords, 3)
        act = o.layers[0].P != 0
        for st, L in zip(o.stages, o.layers[1:]):
            act = dilate_reference(act, st.kind, st.F)
            np.testing.assert_array_equal(L.P != 0, act)


def _scipy_next(active, kind, F):
    out = []
    for a in active:
        v = scipy.signal.correlate2d(a.astype(np.int64), np.ones((F, F), np.int64), mode="valid") > 0
        out.append(v if kind == "conv" else v[::2, ::2])
    return np.stack(out)


def test_circle_fixture_active_counts():
    # Figure 2: a diameter-32 circle centred in the 96x96 input of DeepCNet(5, .)
    c = circle_sites(96, 32)
    o = SparseDeepCNet(5, 1, 1, 2)
    counts = o.build(c.coords, 1)
    act = o.layers[0].P != 0
    ref = [int(act.sum())]
    for st in o.stages:
        act = _scipy_next(act, st.kind, st.F)
        ref.append(int(act.sum()))
    assert counts == ref
    # sparsity is largest in the early layers (Figure 2 caption)
    frac = [n / (L.S * L.S) for n, L in zip(counts, o.layers)]
    assert frac[0] < 0.15 and frac[1] < 0.2 and frac[-1] == 1.0


def test_window_lists_point_at_the_right_sites():
    """R[o][f] is the row of location (step*Y + dy, step*X + dx) below, checked via the site lists."""
    rng = np.random.default_rng(31)
    coords, _ = _random_sites(rng, 2, 24, 0.05, 1)
    o = SparseDeepCNet(3, 1, 1, 2)
    o.build(coords, 2)
    for st, L, below in zip(o.stages, o.layers[1:], o.layers[:-1]):
        step = 1 if st.kind == "conv" else 2
        lookup = {tuple(s): i + 1 for i, s in enumerate(below.sites.tolist())}
        for row, (b, y, x) in enumerate(L.sites.tolist(), start=1):
            for dy in range(st.F):
                for dx in range(st.F):
                    want = lookup.get((b, step * y + dy, step * x + dx), 0)
                    assert L.R[row, dy * st.F + dx] == want


@pytest.mark.parametrize("arch", ["deepcnet", "deepcnin"])
def test_finite_differences(arch):
    ell, k, c_in, ncls, batch = 1, 2, 2, 3, 2
    rng = np.random.default_rng(40)
    coords, feats = _random_sites(rng, batch, 6, 0.3, c_in)
    Ws, bs = he_params(ell, k, c_in, ncls, 41, arch)
    labels = [1, 2]
    o = SparseDeepCNet(ell, k, c_in, ncls, "f64", arch)
    o.build(coords, batch)
    o.forward(feats, Ws, bs, labels)
    dW, db, dfeats = o.backward()

    def loss_at(Ws_, bs_, feats_):
        q = SparseDeepCNet(ell, k, c_in, ncls, "f64", arch)
        q.build(coords, batch)
        return q.forward(feats_, Ws_, bs_, labels)[1]

    h = 1e-6
    for li in range(len(Ws)):
        for _ in range(4):
            i = tuple(rng.integers(0, s) for s in Ws[li].shape)
            Wp = [w.copy() for w in Ws]
            Wm = [w.copy() for w in Ws]
            Wp[li][i] += h
            Wm[li][i] -= h
            fd = (loss_at(Wp, bs, feats) - loss_at(Wm, bs, feats)) / (2 * h)
            assert abs(fd - dW[li][i]) < 1e-6 * max(1.0, abs(fd))
        j = int(rng.integers(0, bs[li].size))
        bp = [b.copy() for b in bs]
        bm = [b.copy() for b in bs]
        bp[li][j] += h
        bm[li][j] -= h
        fd = (loss_at(Ws, bp, feats) - loss_at(Ws, bm, feats)) / (2 * h)
        assert abs(fd - db[li][j]) < 1e-6 * max(1.0, abs(fd))
    for _ in range(5):
        i = (int(rng.integers(0, feats.shape[0])), int(rng.integers(0, c_in)))
        fp, fm = feats.copy(), feats.copy()
        fp[i] += h
        fm[i] -= h
        fd = (loss_at(Ws, bs, fp) - loss_at(Ws, bs, fm)) / (2 * h)
        assert abs(fd - dfeats[i]) < 1e-6 * max(1.0, abs(fd))


def test_loss_is_textbook_cross_entropy():
    rng = np.random.default_rng(50)
    coords, feats = _random_sites(rng, 3, 12, 0.1, 1)
    Ws, bs = he_params(2, 2, 1, 7, 51)
    labels = [0, 6, 3]
    o = SparseDeepCNet(2, 2, 1, 7)
    o.build(coords, 3)
    logits, loss = o.forward(feats, Ws, bs, labels)
    ref = Fn.cross_entropy(torch.tensor(logits), torch.tensor(labels))
    assert abs(loss - float(ref)) < 1e-12
    o.backward()
    t = torch.tensor(logits, requires_grad=True)
    Fn.cross_entropy(t, torch.tensor(labels)).backward()
    np.testing.assert_allclose(o.dlogits, t.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_pool_argmax_takes_first_maximum():
    """Ties inside a pooling window go to the first position in (dy, dx) row-major order."""
    # ell = 1: conv3 (6 -> 4), pool (4 -> 2), conv2 (2 -> 1).  A centre-tap 3x3 filter with zero
    # bias copies input (y+1, x+1) to conv output (y, x), so the pool sees chosen values.
    vals = np.array([[1, 2, 2, 1],
                     [2, 1, 2, 2],
                     [3, 3, 4, 4],
                     [3, 3, 4, 4]], float)
    coords, feats = [], []
    for y in range(4):
        for x in range(4):
            coords.append((0, y + 1, x + 1))
            feats.append([vals[y, x]])
    W1 = np.zeros((9, 1))
    W1[4, 0] = 1.0
    Ws = [W1, np.ones((4, 2)), np.ones((2, 2))]
    bs = [np.zeros(1), np.zeros(2), np.zeros(2)]
    o = SparseDeepCNet(1, 1, 1, 2)
    o.build(np.array(coords), 1)
    o.forward(np.array(feats), Ws, bs, [0])
    L = o.layers[2]
    conv = o.layers[1]
    for row, (b, Y, X) in enumerate(L.sites.tolist(), start=1):
        window = [conv.X[conv.P[0, 2 * Y + dy, 2 * X + dx], 0] for dy in (0, 1) for dx in (0, 1)]
        best, first = -np.inf, -1
        for f, v in enumerate(window):
            if v > best:
                best, first = v, f
        assert L.argmax[row, 0] == first
    assert L.argmax[1:, 0].tolist() == [1, 0, 0, 0]


def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(60)
    x = np.concatenate([rng.normal(size=10000) * 10.0 ** rng.integers(-30, 30, size=10000),
                        [0.0, -0.0, 1.0, -1.0, 3.0e38, 1e-40]])
    # exact ties at the bfloat16 boundary: low 16 bits 0x8000 with kept LSB even and odd
    # (float32 values in [1, 2): exponent 0x3F8, the 7 kept mantissa bits random)
    base = (rng.integers(0, 128, size=200).astype(np.uint32) << 16) | np.uint32(0x3F800000)
    ties = ((base & ~np.uint32(0x10000)) | np.uint32(0x8000)).view(np.float32).astype(np.float64)
    ties_odd = (base | np.uint32(0x18000)).view(np.float32).astype(np.float64)
    for arr in (x, ties, ties_odd):
        ref = torch.tensor(arr.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
        np.testing.assert_array_equal(round_bf16(arr), ref)


def test_deepcnin_rectifier_is_leaky_x_over_3():
    # Section 2.2: f(x) = x for x >= 0 and x/3 for x < 0 on every hidden layer; the
    # 1x1 layers keep their input's active set (identity window lists)
    rng = np.random.default_rng(60)
    coords, feats = _random_sites(rng, 2, 12, 0.2, 1)
    Ws, bs = he_params(2, 3, 1, 4, 61, "deepcnin")
    o = SparseDeepCNet(2, 3, 1, 4, "f64", "deepcnin")
    o.build(coords, 2)
    o.forward(feats, Ws, bs, [0, 1])
    ci = 0
    neg = 0
    for si, st in enumerate(o.stages):
        L, below = o.layers[si + 1], o.layers[si]
        if st.kind != "conv":
            continue
        Z = below.X[L.R].reshape(L.R.shape[0], -1) @ Ws[ci] + bs[ci]
        np.testing.assert_allclose(L.X, np.where(Z >= 0, Z, Z / 3.0), rtol=0, atol=1e-12)
        neg += int((Z < 0).sum())
        if st.F == 1:
            assert L.n == below.n and np.array_equal(L.R[:, 0], np.arange(L.n + 1))
        ci += 1
    assert neg > 0  # the negative branch is exercised
