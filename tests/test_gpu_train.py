"""The training step on the GPU against the oracle: the 8-direction histogram input
encoding (Section 2.4) and the SGD update, then whole training steps.

Encoding: site lists bit-exact; features to the dtype's tolerance, and for float32
the move counts they imply exactly.  SGD: the update of the GPU's own gradients
against the oracle's update; the bfloat16 weight copy is exactly the rounded master.
"""

import math

import numpy as np
import pytest
import torch

from oracle import SparseDeepCNet as Oracle
from oracle.sgd import sgd_step
from oracle.sparse_deepcnet import round_bf16
from oracle.strokes import MOVE_LEN, encode_strokes
from tests.gpu_harness import TOL, log, rel_err, to_dtype
from workloads import get_config, he_params, make_paths, random_labels, stroke_paths

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1409_6070_amd import sscn
    sscn.load_library()


def _dev(p):
    d = torch.device("cuda")
    return (torch.tensor(p.points, dtype=torch.int32, device=d).contiguous(),
            torch.tensor(p.stroke_begin, dtype=torch.int32, device=d).contiguous(),
            torch.tensor(p.stroke_sample, dtype=torch.int32, device=d).contiguous())


def _check_encoding(p, dtype, max_sites=None):
    from paper_1409_6070_amd.sscn import StrokeEncoder
    want_c, want_f = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
    enc = StrokeEncoder(p.grid, p.batch, max_sites or max(want_c.shape[0], 1), dtype)
    c, f = enc.encode(*_dev(p), p.batch)
    torch.cuda.synchronize()
    c, f = c.cpu().numpy(), f.float().cpu().numpy()
    np.testing.assert_array_equal(c, want_c)
    e = rel_err(f, want_f)
    log(f"  sites {c.shape[0]}, feature rel err {e:.3g}")
    assert e <= TOL[dtype]
    if dtype == "f32":
        lens = np.array(MOVE_LEN)
        np.testing.assert_array_equal(np.rint(f[:, 1:] * 2 / lens), np.rint(want_f[:, 1:] * 2 / lens))
        np.testing.assert_array_equal(f[:, 0], want_f[:, 0])
    return c, f


ENC_CASES = [
    # name, batch, grid, strokes, points, box, sigma, seed
    ("g48_small", 6, 48, (1, 3), (1, 30), 32, 2.0, 1),
    ("g96_strokes", 40, 96, (1, 20), (1, 60), 64, 2.0, 2),
    ("g96_long_jumps", 8, 96, (1, 4), (2, 12), 90, 25.0, 3),
    ("g192_many", 16, 192, (1, 30), (1, 120), 128, 1.0, 4),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", ENC_CASES, ids=[c[0] for c in ENC_CASES])
def test_encoding_parity(case, dtype):
    name, batch, grid, strokes, points, box, sigma, seed = case
    p = stroke_paths(np.random.default_rng(seed), batch, grid, strokes, points, box, sigma)
    log(f"[encode] {name} {dtype} points={p.n_points} strokes={p.n_strokes}")
    _check_encoding(p, dtype)


def test_encoding_full_workload():
    cfg = get_config("deepcnet4_20_paths_m9_b100")
    for i in range(2):
        p = make_paths(cfg, i)
        log(f"[encode] {cfg.name} batch {i} points={p.n_points}")
        _check_encoding(p, "bf16")


def test_encoding_edge_cases():
    from paper_1409_6070_amd import sscn
    from workloads import Paths
    log("[encode] edge cases")
    # single-point strokes, an empty stroke, repeated points, grid corners, an empty sample
    pts = np.array([[0, 0], [11, 11], [11, 11], [11, 0], [5, 5], [0, 11], [0, 11]], np.int32)
    p = Paths(points=pts, stroke_begin=np.array([0, 1, 1, 4, 5, 7], np.int32),
              stroke_sample=np.array([0, 0, 2, 2, 0], np.int32), batch=4, grid=12)
    c, f = _check_encoding(p, "f32")
    assert 1 not in c[:, 0] and 3 not in c[:, 0]
    # nothing at all
    empty = Paths(points=np.zeros((0, 2), np.int32), stroke_begin=np.zeros(1, np.int32),
                  stroke_sample=np.zeros(0, np.int32), batch=3, grid=12)
    c, f = _check_encoding(empty, "bf16")
    assert c.shape[0] == 0
    # more sites than the buffers hold: the count comes back with the error
    big = stroke_paths(np.random.default_rng(9), 4, 48, (2, 3), (10, 20), 32, 2.0)
    n = encode_strokes(big.points, big.stroke_begin, big.stroke_sample, 4, 48)[0].shape[0]
    enc = sscn.StrokeEncoder(48, 4, n - 1, "f32")
    with pytest.raises(sscn.SSCNError) as e:
        enc.encode(*_dev(big), 4)
    assert e.value.name == "SSCN_ERR_CAPACITY" and e.value.count == n
    # a point outside the grid, a sample outside the batch, offsets that do not cover the points
    for bad in ("point", "sample", "offsets"):
        q = stroke_paths(np.random.default_rng(10), 2, 24, (1, 2), (3, 6), 16, 2.0)
        pts, beg, smp = q.points.copy(), q.stroke_begin.copy(), q.stroke_sample.copy()
        if bad == "point":
            pts[2] = (24, 3)
        elif bad == "sample":
            smp[0] = 2
        else:
            beg[-1] -= 1
        d = torch.device("cuda")
        enc = sscn.StrokeEncoder(24, 2, 500, "f32")
        with pytest.raises(sscn.SSCNError) as e:
            enc.encode(torch.tensor(pts, device=d), torch.tensor(beg, device=d), torch.tensor(smp, device=d), 2)
        assert e.value.name == {"point": "SSCN_ERR_OUT_OF_RANGE", "sample": "SSCN_ERR_OUT_OF_RANGE",
                                "offsets": "SSCN_ERR_INVALID_ARGUMENT"}[bad]


class Trainer:
    """GPU state of a training run: fp32 masters, storage copies, velocities."""

    def __init__(self, ell, k, ncls, batch, max_active, dtype, Ws, bs):
        from paper_1409_6070_amd.sscn import SparseDeepCNet
        d = torch.device("cuda")
        self.dtype = dtype
        self.net = SparseDeepCNet(ell, k, 9, ncls, batch_max=batch, max_active=max_active, dtype=dtype)
        self.W32 = [torch.tensor(np.asarray(W), dtype=torch.float32, device=d).contiguous() for W in Ws]
        self.W = [w.to(self.net.tdtype).contiguous() for w in self.W32] if dtype == "bf16" else self.W32
        self.b = [torch.tensor(np.asarray(x), dtype=torch.float32, device=d).contiguous() for x in bs]
        self.vW = [torch.zeros_like(w) for w in self.W32]
        self.vb = [torch.zeros_like(x) for x in self.b]

    def step(self, coords, feats, batch, labels_d, lr, mom, wd):
        net = self.net
        net.rulebook_build(coords, batch)
        _, loss = net.forward(feats, self.W, self.b, labels_d)
        loss = float(loss.cpu()[0])
        net.backward()
        net.sgd_step(self.W32, self.W if self.dtype == "bf16" else None, self.b, self.vW, self.vb, lr, mom, wd)
        return loss


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sgd_update_parity(dtype):
    """The update alone: the GPU's own gradients fed to the oracle's update."""
    log(f"[sgd] update {dtype}")
    from paper_1409_6070_amd.sscn import StrokeEncoder
    p = stroke_paths(np.random.default_rng(21), 6, 24, (1, 3), (3, 12), 16, 2.0)
    enc = StrokeEncoder(24, 6, 2000, dtype)
    coords, feats = enc.encode(*_dev(p), 6)
    Ws, bs = he_params(3, 8, 9, 5, 22)
    t = Trainer(3, 8, 5, 6, 2000, dtype, Ws, bs)
    rng = np.random.default_rng(23)
    for v in t.vW + t.vb:
        v.copy_(torch.tensor(rng.normal(0, 0.1, size=tuple(v.shape)), dtype=torch.float32))
    W0 = [w.cpu().double().numpy() for w in t.W32]
    b0 = [x.cpu().double().numpy() for x in t.b]
    v0 = [v.cpu().double().numpy() for v in t.vW]
    vb0 = [v.cpu().double().numpy() for v in t.vb]
    lab = torch.tensor(random_labels(6, 5, 24), dtype=torch.int32, device="cuda")
    t.step(coords, feats, 6, lab, 0.05, 0.9, 1e-3)
    torch.cuda.synchronize()
    dW = [g.cpu().double().numpy() for g in t.net.dW]
    db = [g.cpu().double().numpy() for g in t.net.db]
    Wn, Wst, bn, vWn, vbn = sgd_step(W0, b0, dW, db, v0, vb0, 0.05, 0.9, 1e-3, mode=dtype)
    for a, w in zip(t.W32, Wn):
        assert rel_err(a.cpu().numpy(), w) <= 1e-6
    for a, w in zip(t.b, bn):
        assert rel_err(a.cpu().numpy(), w) <= 1e-6
    for a, w in zip(t.vW + t.vb, vWn + vbn):
        assert rel_err(a.cpu().numpy(), w) <= 1e-6
    if dtype == "bf16":
        for a, m in zip(t.W, t.W32):  # the storage copy is exactly the rounded master
            np.testing.assert_array_equal(a.float().cpu().numpy(), round_bf16(m.cpu().double().numpy()))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_training_steps_match_oracle(dtype):
    """Three whole steps (encode, build, forward, backward, update) on both sides."""
    log(f"[train] 3 steps {dtype}")
    from paper_1409_6070_amd.sscn import StrokeEncoder
    ell, k, ncls, batch, N = 3, 8, 5, 6, 24
    paths = [stroke_paths(np.random.default_rng(30 + i), batch, N, (1, 3), (3, 12), 16, 2.0) for i in range(3)]
    Ws, bs = he_params(ell, k, 9, ncls, 31)
    labels = random_labels(batch, ncls, 32)
    lab_d = torch.tensor(labels, dtype=torch.int32, device="cuda")
    enc = StrokeEncoder(N, batch, 3000, dtype)
    t = Trainer(ell, k, ncls, batch, 3000, dtype, Ws, bs)
    # the oracle follows the same recipe in float64 (storage rounding of its mode)
    oW = [np.asarray(w, np.float64) for w in Ws]
    oWs = [np.asarray(round_bf16(w) if dtype == "bf16" else w, np.float64) for w in oW]
    ob = [np.asarray(x, np.float64) for x in bs]
    ovW = [np.zeros_like(w) for w in oW]
    ovb = [np.zeros_like(x) for x in ob]
    lr, mom, wd = 0.05, 0.9, 1e-3
    for i, p in enumerate(paths):
        coords, feats = enc.encode(*_dev(p), batch)
        loss = t.step(coords, feats, batch, lab_d, lr, mom, wd)
        c, f = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, batch, N)
        o = Oracle(ell, k, 9, ncls, dtype)
        o.build(c, batch)
        _, oloss = o.forward(to_dtype(f, dtype).double().numpy(), oWs, ob, labels)
        dW, db, _ = o.backward()
        oW, oWs, ob, ovW, ovb = sgd_step(oW, ob, dW, db, ovW, ovb, lr, mom, wd, mode=dtype)
        log(f"  step {i}: loss gpu {loss:.6f} oracle {oloss:.6f}")
        assert abs(loss - oloss) <= TOL[dtype] * max(1.0, abs(oloss))
    torch.cuda.synchronize()
    for a, w in zip(t.W32 + t.b, oW + ob):
        e = rel_err(a.cpu().numpy(), w)
        assert e <= TOL[dtype], e


def test_training_lowers_the_loss():
    """The loop closes on the GPU: the M = 9 DeepCNet(4,20) fits a fixed batch."""
    cfg = get_config("deepcnet4_20_paths_m9_b100")
    log(f"[train] {cfg.name}: 150 steps on one batch")
    from paper_1409_6070_amd.sscn import StrokeEncoder
    p = make_paths(cfg, 0)
    enc = StrokeEncoder(cfg.grid, cfg.batch, 20000, "bf16")
    coords, feats = enc.encode(*_dev(p), cfg.batch)
    Ws, bs = he_params(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.weight_seed)
    t = Trainer(cfg.ell, cfg.k, cfg.n_classes, cfg.batch, 20000, "bf16", Ws, bs)
    lab = torch.tensor(random_labels(cfg.batch, cfg.n_classes, cfg.label_seed), dtype=torch.int32, device="cuda")
    losses = [t.step(coords, feats, cfg.batch, lab, 0.05, 0.9, 1e-4) for _ in range(150)]
    log(f"  loss {losses[0]:.4f} -> {losses[49]:.4f} -> {losses[99]:.4f} -> {losses[-1]:.4f}")
    assert all(math.isfinite(x) for x in losses)
    assert np.mean(losses[-10:]) < 0.7 * np.mean(losses[:10])
