"""HIP path vs the CPU oracle, through the C interface, on the GPU.

Every case prints its name, seed and shape before touching the GPU.
"""

import numpy as np
import pytest
import torch

from oracle import SparseDeepCNet as Oracle
from tests.gpu_harness import Pair, TOL, check_structure, check_values, log, rel_err, to_dtype
from workloads import CONFIGS, circle_sites, get_config, he_params, make_batch, random_labels

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1409_6070_amd import sscn
    sscn.load_library()


def _sparse_case(seed, ell, batch, p, c_in, empty=(), full=()):
    rng = np.random.default_rng(seed)
    N = 3 * 2 ** ell
    coords = []
    for b in range(batch):
        if b in empty:
            continue
        m = np.ones((N, N), bool) if b in full else rng.random((N, N)) < p
        ys, xs = np.nonzero(m)
        coords.append(np.stack([np.full(ys.size, b), ys, xs], 1))
    coords = np.concatenate(coords) if coords else np.zeros((0, 3), np.int64)
    coords = coords[rng.permutation(len(coords))]
    feats = rng.normal(size=(len(coords), c_in))
    return coords, feats


SMALL = [
    # name, ell, k, c_in, classes, batch, p, empty, full, seed
    ("l1k3_m1_b2", 1, 3, 1, 4, 2, 0.3, (), (), 1),
    ("l2k5_m3_b3_empty", 2, 5, 3, 7, 3, 0.08, (1,), (), 2),
    ("l2k12_m1_b2_full", 2, 12, 1, 5, 2, 0.1, (), (0,), 3),
    ("l3k20_m2_b4", 3, 20, 2, 33, 4, 0.05, (), (), 4),
    ("l3k33_m9_b3", 3, 33, 9, 70, 3, 0.04, (2,), (), 5),
    ("l4k24_m1_b5", 4, 24, 1, 129, 5, 0.02, (), (), 6),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_networks(case, dtype):
    name, ell, k, c_in, ncls, batch, p, empty, full, seed = case
    coords, feats = _sparse_case(seed, ell, batch, p, c_in, empty, full)
    log(f"[small] {name} {dtype} n={len(coords)} seed={seed}")
    Ws, bs = he_params(ell, k, c_in, ncls, 100 + seed)
    labels = random_labels(batch, ncls, 200 + seed)
    pair = Pair(ell, k, c_in, ncls, batch, coords, feats, Ws, bs, labels, dtype).run_gpu()
    check_structure(pair)
    rep = check_values(pair)
    log(f"  worst rel err {max(v for k_, v in rep.items() if not k_.startswith(('argmax', 'relu'))):.3g}")


def _config_case(cfg, dtype, index=0):
    if cfg.generator == "paths":  # the parity of the net itself: inputs from the oracle's encoding
        from oracle.strokes import encode_strokes
        from workloads import Batch, make_paths
        p = make_paths(cfg, index)
        coords, feats = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
        b = Batch(coords=coords.astype(np.int32), feats=feats, batch=cfg.batch, grid=cfg.grid)
    else:
        b = make_batch(cfg, index)
    Ws, bs = he_params(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.weight_seed, cfg.arch)
    labels = random_labels(cfg.batch, cfg.n_classes, cfg.label_seed)
    return b, Ws, bs, labels


CFG_CASES = [(c.name, d) for c in CONFIGS for d in c.dtypes]


@pytest.mark.parametrize("name,dtype", CFG_CASES, ids=[f"{n}-{d}" for n, d in CFG_CASES])
def test_workload_parity_full_size(name, dtype):
    """The full workloads, every layer, every gradient, against the whole oracle."""
    cfg = get_config(name)
    b, Ws, bs, labels = _config_case(cfg, dtype)
    log(f"[workload] {name} {dtype} n={b.n} batch={cfg.batch}")
    pair = Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype,
                max_active=int(b.n * 1.25), arch=cfg.arch, rates=list(cfg.dropout) or None,
                dseed=cfg.dropout_seed).run_gpu()
    check_structure(pair)
    rep = check_values(pair)
    worst = {k_: v for k_, v in rep.items() if not k_.startswith(("argmax", "relu"))}
    log(f"  worst rel err {max(worst.values()):.3g} ({max(worst, key=worst.get)}); "
        f"near-tie flips: argmax {sum(v for k_, v in rep.items() if k_.startswith('argmax'))}, "
        f"relu {sum(v for k_, v in rep.items() if k_.startswith('relu'))}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pen_stroke_net_at_batch_400(dtype):
    """DeepCNet(5,50) on the pen-stroke generator at four times the measured batch (a point of
    the batch sweep): more output tiles than a launch's grid holds, so the GEMM, first-layer
    and weight-gradient kernels walk their tiles and row blocks in grid-stride loops, and
    the first layer's weight gradient reaches the split-K chunk limit."""
    import dataclasses
    base = get_config("deepcnet5_50_strokes_b100")
    cfg = dataclasses.replace(base, batch=400, name=f"{base.name}@400")
    b, Ws, bs, labels = _config_case(cfg, dtype)
    log(f"[batch-400] {dtype} n={b.n}")
    pair = Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype,
                max_active=b.n).run_gpu()
    check_structure(pair)
    rep = check_values(pair)
    worst = {k_: v for k_, v in rep.items() if not k_.startswith(("argmax", "relu"))}
    log(f"  worst rel err {max(worst.values()):.3g} ({max(worst, key=worst.get)})")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stage_kernels_on_oracle_inputs(dtype):
    """Each stage fed the oracle's exact input: pools bit-exact (values and argmax), convs to tolerance."""
    cfg = get_config("deepcnet4_20_strokes_b8")
    b, Ws, bs, labels = _config_case(cfg, dtype)
    log(f"[stage] {cfg.name} {dtype}")
    pair = Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype).run_gpu()
    o = pair.o
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    for s in range(1, len(o.layers)):
        below = pair.net.layer_view(s - 1, pair.counts[s - 1])
        C = below["channels"]
        inp = torch.zeros_like(below["features"])
        inp[:, :C] = torch.tensor(o.layers[s - 1].X, dtype=torch.float64).to(tdt).cuda()
        below["features"].copy_(inp)
        pair.net.forward_stage(s)
        torch.cuda.synchronize()
        v = pair.view(s)
        L = o.layers[s]
        if o.stages[s - 1].kind == "pool":
            np.testing.assert_array_equal(v["X"], L.X, err_msg=f"pool values stage {s}")
            np.testing.assert_array_equal(v["argmax"], L.argmax, err_msg=f"pool argmax stage {s}")
        else:
            e = rel_err(v["X"], L.X)
            assert e <= TOL[dtype] / 10, f"conv stage {s}: {e}"
    # backward, stage by stage from the oracle's gradients
    for s in range(len(o.layers) - 1, 0, -1):
        L = o.layers[s]
        v = pair.net.layer_view(s, pair.counts[s])
        C = v["channels"]
        g = torch.zeros_like(v["grad"])
        g[:, :C] = torch.tensor(L.grad, dtype=torch.float64).to(tdt).cuda()
        v["grad"].copy_(g)
        X = torch.zeros_like(v["features"])
        X[:, :C] = torch.tensor(L.X, dtype=torch.float64).to(tdt).cuda()
        v["features"].copy_(X)
        below = pair.net.layer_view(s - 1, pair.counts[s - 1])
        Xb = torch.zeros_like(below["features"])
        Xb[:, :below["channels"]] = torch.tensor(o.layers[s - 1].X, dtype=torch.float64).to(tdt).cuda()
        below["features"].copy_(Xb)
        pair.net.backward_stage(s)
        torch.cuda.synchronize()
        vb = pair.view(s - 1)
        e = rel_err(vb["G"], o.layers[s - 1].grad)
        if o.stages[s - 1].kind == "pool":
            # rows >= 1 are routed copies: exact; row 0 is a sum
            np.testing.assert_array_equal(vb["G"][1:], o.layers[s - 1].grad[1:], err_msg=f"pool bwd stage {s}")
        assert e <= TOL[dtype], f"backward stage {s}: {e}"


# every training workload's tile plans, both dtypes of the first two
PLAN_CASES = [("deepcnet4_20_strokes_b8", "f32"), ("deepcnet4_20_strokes_b8", "bf16"),
              ("deepcnet5_50_strokes_b100", "f32"), ("deepcnet5_50_strokes_b100", "bf16"),
              ("deepcnet5_50_strokes_m8_b100", "bf16"), ("deepcnet5_100_rgbpatch_b128", "bf16"),
              ("deepcnet6_100_strokes_b64", "bf16"), ("deepcnin5_50_strokes_b100", "bf16")]


@pytest.mark.parametrize("name,dtype", PLAN_CASES, ids=[f"{n}-{d}" for n, d in PLAN_CASES])
def test_fused_pool_forward_matches_stage_kernels(name, dtype):
    """The full forward pass runs each pooling layer in the epilogue of the convolution below it
    (GEMM rows in pooling-window order); the per-stage entry point runs the separate kernels.
    Both compute every row's dot products in the same order, so every layer's features and every
    argmax must agree bit for bit."""
    cfg = get_config(name)
    b, Ws, bs, labels = _config_case(cfg, dtype)
    log(f"[fused-pool] {name} {dtype}")
    pair = Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype,
                run_oracle=False, arch=cfg.arch).run_gpu()
    n = len(pair.counts)
    fused = [pair.view(s) for s in range(n)]
    fused = [(v["X"].copy(), None if "argmax" not in v else v["argmax"].copy()) for v in fused]
    for s in range(1, n):
        pair.net.forward_stage(s)
    torch.cuda.synchronize()
    for s in range(1, n):
        v = pair.view(s)
        np.testing.assert_array_equal(v["X"], fused[s][0], err_msg=f"features layer {s}")
        if fused[s][1] is not None:
            np.testing.assert_array_equal(v["argmax"], fused[s][1], err_msg=f"argmax layer {s}")


@pytest.mark.parametrize("c_in,narrow", [(1, True), (2, True), (3, True), (9, False)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_first_layer_kernel_choice(c_in, narrow, dtype):
    """A first layer with at most 32 products per output (3 x 3 window, c_in <= 3) runs on the
    vector-ALU kernel, a wider one as a gather GEMM; either way its output equals the oracle's
    (the per-stage entry point recomputes the layer in place, so it must reproduce the pass's bits)."""
    coords, feats = _sparse_case(40 + c_in, 2, 3, 0.15, c_in)
    Ws, bs = he_params(2, 6, c_in, 5, 140 + c_in)
    labels = random_labels(3, 5, 240 + c_in)
    log(f"[first-layer] c_in={c_in} {dtype} n={len(coords)}")
    pair = Pair(2, 6, c_in, 5, 3, coords, feats, Ws, bs, labels, dtype).run_gpu()
    before = pair.view(1)["X"].copy()
    pair.net.timing(["conv_narrow", "gather_gemm"])
    pair.net.forward_stage(1)
    torch.cuda.synchronize()
    n_narrow, _ = pair.net.timing_collect("conv_narrow")
    n_gemm, _ = pair.net.timing_collect("gather_gemm")
    pair.net.timing([])
    assert (n_narrow, n_gemm) == ((1, 0) if narrow else (0, 1))
    np.testing.assert_array_equal(pair.view(1)["X"], before)
    check_values(pair)


@pytest.mark.parametrize("batch", [1, 1024, 1100])
def test_rulebook_batch_sizes_around_offset_scan(batch):
    """Up to 1024 samples the window-list kernel scans the per-sample counts itself; above, a
    separate offsets launch does. Both must give the oracle's rows, windows and values."""
    coords, feats = _sparse_case(60 + batch % 7, 1, batch, 0.3, 1)
    log(f"[batch-scan] batch={batch} n={len(coords)}")
    Ws, bs = he_params(1, 3, 1, 4, 160)
    labels = random_labels(batch, 4, 260)
    pair = Pair(1, 3, 1, 4, batch, coords, feats, Ws, bs, labels, "f32").run_gpu()
    check_structure(pair)
    check_values(pair)


def test_rulebook_path_counts_full_grid():
    """Fully active 96x96 input of DeepCNet(5,.): routes through the GPU window lists (Section 2.6)."""
    ell, N = 5, 96
    ys, xs = np.meshgrid(np.arange(N), np.arange(N), indexing="ij")
    coords = np.stack([np.zeros(N * N, int), ys.ravel(), xs.ravel()], 1)
    log("[paths] ell=5 full grid")
    Ws, bs = he_params(ell, 1, 1, 2, 7)
    pair = Pair(ell, 1, 1, 2, 1, coords, np.ones((N * N, 1)), Ws, bs, [0], "f32", run_oracle=False).run_gpu()
    cnt = np.ones(pair.counts[-1] + 1)
    cnt[0] = 0
    for s in range(len(pair.counts) - 1, 0, -1):
        R = pair.view(s)["rules"]
        nxt = np.zeros(pair.counts[s - 1] + 1)
        np.add.at(nxt, R[1:].ravel(), np.repeat(cnt[1:], R.shape[1]))
        nxt[0] = 0
        cnt = nxt
    sites = pair.view(0)["sites"]
    grid = np.zeros((N, N))
    grid[sites // N, sites % N] = cnt[1:]
    assert grid[0, 0] == grid[0, N - 1] == grid[N - 1, 0] == grid[N - 1, N - 1] == 1
    assert np.all(grid[32:64, 32:64] == 9 * 4 ** (ell - 1)) and grid.max() == 9 * 4 ** (ell - 1)


def test_circle_fixture_counts():
    c = circle_sites(96, 32)
    log("[circle] diameter 32 in 96x96")
    Ws, bs = he_params(5, 4, 1, 3, 8)
    pair = Pair(5, 4, 1, 3, 1, c.coords, c.feats, Ws, bs, [1], "f32").run_gpu()
    check_structure(pair)
    check_values(pair)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_empty_inputs(dtype):
    """No active site at all: every layer is its ground row; gradients flow through row 0 only."""
    log(f"[empty] {dtype}")
    Ws, bs = he_params(3, 6, 2, 5, 9)
    pair = Pair(3, 6, 2, 5, 3, np.zeros((0, 3), np.int64), np.zeros((0, 2)), Ws, bs, [0, 4, 2], dtype,
                want_dfeats=False).run_gpu()
    assert pair.counts == [0] * 8
    check_values(pair)


@pytest.mark.parametrize("name,dtype", PLAN_CASES, ids=[f"{n}-{d}" for n, d in PLAN_CASES])
def test_repeat_runs_are_bitwise_identical(name, dtype):
    """No float atomics and fixed reduction orders: two runs of a step give the same bits in every
    layer's features and gradients, the logits, the loss and every parameter gradient."""
    cfg = get_config(name)
    b, Ws, bs, labels = _config_case(cfg, dtype, index=1)
    log(f"[determinism] {name} {dtype} batch 1")
    pair = Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype,
                run_oracle=False, arch=cfg.arch)
    outs = []
    for _ in range(2):
        pair.run_gpu()
        layers = [pair.view(s) for s in range(len(pair.counts))]
        outs.append([pair.logits.copy(), np.float64(pair.loss), *[w.copy() for w in pair.dW],
                     *[x.copy() for x in pair.db], pair.dfeats.copy(), *[v["X"].copy() for v in layers],
                     *[v["G"].copy() for v in layers]])
    for i, (a, c) in enumerate(zip(*outs)):
        np.testing.assert_array_equal(a, c, err_msg=f"output {i}")


@pytest.mark.parametrize("bad,status", [("dup", "SSCN_ERR_DUPLICATE_SITE"), ("range", "SSCN_ERR_OUT_OF_RANGE"),
                                        ("batch", "SSCN_ERR_OUT_OF_RANGE")])
def test_invalid_sites_are_reported(bad, status):
    from paper_1409_6070_amd import sscn
    log(f"[errors] {bad}")
    net = sscn.SparseDeepCNet(2, 3, 1, 4, batch_max=2, max_active=16, dtype="f32")
    coords = np.array([[0, 1, 1], [0, 2, 3], [1, 5, 5]], np.int32)
    if bad == "dup":
        coords[2] = coords[0]
    elif bad == "range":
        coords[1] = (0, 12, 0)
    else:
        coords[2] = (2, 0, 0)
    net.rulebook_build(torch.tensor(coords).cuda(), 2)
    with pytest.raises(sscn.SSCNError) as e:
        net.layer_sizes()
    assert e.value.name == status
    # a clean build afterwards succeeds
    ok = np.array([[0, 1, 1], [1, 2, 2]], np.int32)
    net.rulebook_build(torch.tensor(ok).cuda(), 2)
    assert net.layer_sizes()[0] == 2


def test_rebuilds_alternate_input_bitmaps():
    """Consecutive builds on one net.  Each build inserts into one of two input bitmaps (and error
    words) and clears the other for the next build, so every build must be bit-exact whatever the
    builds before it held: a larger batch after a smaller one, an empty batch, and a clean build
    right after one that reported a duplicate site."""
    from paper_1409_6070_amd import sscn
    from tests.gpu_harness import decode_sites
    ell, k, c_in, ncls, bmax = 3, 4, 1, 5, 5
    net = sscn.SparseDeepCNet(ell, k, c_in, ncls, batch_max=bmax, max_active=24 * 24 * bmax, dtype="f32")
    seq = [(5, 0.3, 11), (2, 0.05, 12), (0, 0.0, 13), (5, 0.15, 14), (4, 0.1, 15, "dup"), (3, 0.2, 16),
           (5, 0.02, 17), (1, 0.5, 18)]
    for step in seq:
        batch, p, seed = step[:3]
        coords, _ = _sparse_case(seed, ell, batch, p, c_in) if batch else (np.zeros((0, 3), np.int64), None)
        log(f"[rebuild] batch={batch} n={len(coords)} seed={seed} {'dup' if len(step) > 3 else ''}")
        if len(step) > 3:
            coords = np.concatenate([coords, coords[:1]])
            net.rulebook_build(torch.tensor(coords, dtype=torch.int32).cuda(), batch)
            with pytest.raises(sscn.SSCNError) as e:
                net.layer_sizes()
            assert e.value.name == "SSCN_ERR_DUPLICATE_SITE"
            continue
        net.rulebook_build(torch.tensor(coords, dtype=torch.int32).cuda().reshape(-1, 3), batch)
        counts = net.layer_sizes()
        o = Oracle(ell, k, c_in, ncls, "f32")
        o.build(np.asarray(coords).reshape(-1, 3), batch)
        assert counts == o.layer_sizes(), (counts, o.layer_sizes())
        for s_, L in enumerate(o.layers):
            v = net.layer_view(s_, counts[s_])
            np.testing.assert_array_equal(decode_sites(v["sites"].cpu().numpy(), L.S), L.sites,
                                          err_msg=f"sites layer {s_} batch {batch}")
            if s_:
                np.testing.assert_array_equal(v["rules"].cpu().numpy(), L.R, err_msg=f"rules layer {s_}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_inference_digits_full_size(dtype):
    """Forward-only classification (Section 3.2's timed workload, DeepCNet(5,10) on digit pictures
    in a 96 x 96 grid, batch 1000): no labels, logits against the oracle's forward; a backward
    after an inference forward is refused."""
    from paper_1409_6070_amd import sscn
    cfg = get_config("deepcnet5_10_digits_b1000")
    b, Ws, bs, labels = _config_case(cfg, dtype)
    log(f"[infer] {cfg.name} {dtype} n={b.n}")
    feats_t = to_dtype(b.feats, dtype)
    Ws_t = [to_dtype(W, dtype) for W in Ws]
    o = Oracle(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, dtype)
    o.build(b.coords, cfg.batch)
    o.forward(feats_t.double().numpy(), [w.double().numpy() for w in Ws_t], bs, labels)  # logits ignore labels
    net = sscn.SparseDeepCNet(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, batch_max=cfg.batch, max_active=b.n,
                              dtype=dtype)
    net.rulebook_build(torch.tensor(b.coords).cuda().contiguous(), cfg.batch)
    assert net.layer_sizes() == o.layer_sizes()
    logits, loss = net.forward(feats_t.cuda().contiguous(), [w.cuda().contiguous() for w in Ws_t],
                               [torch.tensor(np.asarray(x, np.float32)).cuda() for x in bs], None)
    torch.cuda.synchronize()
    assert loss is None
    e = rel_err(logits.cpu().numpy(), o.logits)
    log(f"  logits rel err {e:.3g}")
    assert e <= TOL[dtype]
    with pytest.raises(sscn.SSCNError) as err:
        net.backward()
    assert err.value.name == "SSCN_ERR_BAD_STATE"


SMALL_NIN = [
    # name, ell, k, c_in, classes, batch, p, empty, full, seed
    ("nin_l1k3_m1_b2", 1, 3, 1, 4, 2, 0.3, (), (), 31),
    ("nin_l2k5_m3_b3_empty", 2, 5, 3, 7, 3, 0.08, (1,), (), 32),
    ("nin_l2k12_m1_b2_full", 2, 12, 1, 5, 2, 0.1, (), (0,), 33),
    ("nin_l3k20_m2_b4", 3, 20, 2, 33, 4, 0.05, (), (), 34),
    ("nin_l4k24_m1_b5", 4, 24, 1, 129, 5, 0.02, (), (), 36),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", SMALL_NIN, ids=[c[0] for c in SMALL_NIN])
def test_small_deepcnin(case, dtype):
    """DeepCNiN (Section 2.2): 1x1 layers after every pool and the last convolution, leaky rectifier x/3."""
    name, ell, k, c_in, ncls, batch, p, empty, full, seed = case
    coords, feats = _sparse_case(seed, ell, batch, p, c_in, empty, full)
    log(f"[small-nin] {name} {dtype} n={len(coords)} seed={seed}")
    Ws, bs = he_params(ell, k, c_in, ncls, 100 + seed, "deepcnin")
    labels = random_labels(batch, ncls, 200 + seed)
    pair = Pair(ell, k, c_in, ncls, batch, coords, feats, Ws, bs, labels, dtype, arch="deepcnin").run_gpu()
    check_structure(pair)
    check_values(pair)


def test_out_of_range_label_is_reported():
    """A training forward with a label outside [0, n_classes) latches an error that the next
    sscn_layer_sizes reports once; the bad sample contributes nothing to the loss."""
    from paper_1409_6070_amd import sscn
    log("[errors] label out of range")
    coords, feats = _sparse_case(70, 2, 3, 0.2, 1)
    Ws, bs = he_params(2, 4, 1, 5, 170)
    good = random_labels(3, 5, 270)
    for bad_label in (5, -1):
        labels = good.copy()
        labels[1] = bad_label
        pair = Pair(2, 4, 1, 5, 3, coords, feats, Ws, bs, good, "f32")
        pair.labels_d = torch.tensor(labels, dtype=torch.int32).cuda()
        pair.run_gpu()
        # samples 0 and 2 as the oracle has them; sample 1 adds nothing to the mean
        o = pair.o
        z = o.logits - o.logits.max(axis=1, keepdims=True)
        terms = np.log(np.exp(z).sum(axis=1)) - z[np.arange(3), good]
        want = (terms[0] + terms[2]) / 3
        assert abs(pair.loss - want) <= 1e-5 * abs(want)
        net = pair.net
        net.rulebook_build(pair.coords_d, 3)
        with pytest.raises(sscn.SSCNError) as e:
            net.layer_sizes()
        assert e.value.name == "SSCN_ERR_OUT_OF_RANGE"
        assert net.layer_sizes() == o.layer_sizes()  # reported once
