"""The grouped rulebook build (sites grouped by sample, per-sample offsets given; the bitmap pass
inserts each sample's sites itself): the oracle's rows, window lists, transposes and values, the
ungrouped build's structures and pass outputs bit for bit, and the same device-side error reports."""
import numpy as np
import pytest
import torch

from tests.gpu_harness import Pair, check_structure, check_values, log
from tests.test_gpu_parity import _sparse_case
from workloads import get_config, he_params, make_batches, random_labels

pytestmark = pytest.mark.gpu


def grouped(coords, batch, seed):
    """The sites sorted by sample (shuffled within each sample) and the batch + 1 sample offsets."""
    c = np.asarray(coords, dtype=np.int64).reshape(-1, 3)
    c = c[np.random.default_rng(seed).permutation(len(c))]
    c = c[np.argsort(c[:, 0], kind="stable")]
    return c, np.searchsorted(c[:, 0], np.arange(batch + 1)).astype(np.int64)


def structures(net, counts):
    out = []
    for s, n in enumerate(counts):
        v = net.layer_view(s, n)
        item = [v["sites"].cpu().numpy()]
        if s > 0:
            item += [v["rules"].cpu().numpy(), net.rules_t(s, counts[s - 1]).cpu().numpy()]
            if "gmask" in v:
                item.append(v["gmask"].cpu().numpy())
        out.append(item)
    return out


# name, ell, k, c_in, classes, batch, density, empty samples, seed
CASES = [
    ("l2_b1", 2, 4, 1, 5, 1, 0.2, (), 70),
    ("l3_b7_empty", 3, 4, 2, 5, 7, 0.1, (0, 3, 6), 71),
    ("l1_b1024", 1, 3, 1, 4, 1024, 0.3, (5,), 72),
    ("l1_b1100", 1, 3, 1, 4, 1100, 0.3, (), 73),
    ("l4_b3_dense", 4, 3, 1, 6, 3, 0.6, (), 74),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_grouped_build_matches_oracle_and_ungrouped(case, dtype):
    name, ell, k, c_in, ncls, batch, p, empty, seed = case
    coords, feats = _sparse_case(seed, ell, batch, p, c_in, empty)
    c, begin = grouped(coords, batch, seed)
    # the features follow their sites through the reordering
    order = {tuple(r): i for i, r in enumerate(np.asarray(coords).reshape(-1, 3).tolist())}
    f = np.asarray(feats)[[order[tuple(r)] for r in c.tolist()]] if len(c) else feats
    log(f"[grouped] {name} {dtype} n={len(c)} batch={batch}")
    Ws, bs = he_params(ell, k, c_in, ncls, 100 + seed)
    labels = random_labels(batch, ncls, 200 + seed)
    pair = Pair(ell, k, c_in, ncls, batch, c, f, Ws, bs, labels, dtype)
    pair.run_gpu()
    ref = structures(pair.net, pair.counts)
    outs = [pair.logits.copy(), np.float64(pair.loss), *[w.copy() for w in pair.dW], *[x.copy() for x in pair.db],
            pair.dfeats.copy()]
    pair.run_gpu(sample_begin=begin)
    check_structure(pair)
    check_values(pair)
    got = structures(pair.net, pair.counts)
    for s, (a, b) in enumerate(zip(ref, got)):
        for i, (x, y) in enumerate(zip(a, b)):
            np.testing.assert_array_equal(x, y, err_msg=f"layer {s} structure {i}")
    for i, (x, y) in enumerate(zip(outs, [pair.logits, np.float64(pair.loss), *pair.dW, *pair.db, pair.dfeats])):
        np.testing.assert_array_equal(x, y, err_msg=f"output {i}")


def test_grouped_build_full_size_structures():
    """The bench workload's batch, grouped as generated: every structure equals the ungrouped build's."""
    from paper_1409_6070_amd import sscn
    cfg = get_config("deepcnet5_50_strokes_b100")
    b = make_batches(cfg, 1)[0]
    c, begin = grouped(b.coords, cfg.batch, 0)
    log(f"[grouped] full size n={len(c)}")
    net = sscn.SparseDeepCNet(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, batch_max=cfg.batch, max_active=len(c),
                              dtype="bf16")
    cd = torch.tensor(c, dtype=torch.int32).cuda().contiguous()
    net.rulebook_build(cd, cfg.batch)
    counts = net.layer_sizes()
    ref = structures(net, counts)
    net.rulebook_build(cd, cfg.batch, sample_begin=torch.tensor(begin, dtype=torch.int32).cuda())
    assert net.layer_sizes() == counts
    for s, (a, g) in enumerate(zip(ref, structures(net, counts))):
        for i, (x, y) in enumerate(zip(a, g)):
            np.testing.assert_array_equal(x, y, err_msg=f"layer {s} structure {i}")


@pytest.mark.parametrize("bad,status", [("dup", "SSCN_ERR_DUPLICATE_SITE"), ("range", "SSCN_ERR_OUT_OF_RANGE"),
                                        ("sample", "SSCN_ERR_OUT_OF_RANGE"), ("offsets", "SSCN_ERR_OUT_OF_RANGE"),
                                        ("past_n", "SSCN_ERR_OUT_OF_RANGE")])
def test_grouped_input_errors_are_reported(bad, status):
    """Errors latched on the device (offsets read clamped to 0..n, so no access leaves the arrays),
    and a clean grouped build afterwards succeeds."""
    from paper_1409_6070_amd import sscn
    log(f"[grouped errors] {bad}")
    net = sscn.SparseDeepCNet(2, 3, 1, 4, batch_max=2, max_active=16, dtype="f32")
    coords = np.array([[0, 1, 1], [0, 2, 3], [1, 5, 5]], np.int32)
    begin = np.array([0, 2, 3], np.int32)
    if bad == "dup":
        coords[1] = coords[0]
    elif bad == "range":
        coords[1] = (0, 12, 0)
    elif bad == "sample":
        coords[1] = (1, 2, 3)  # sample 1's site inside sample 0's range
    elif bad == "offsets":
        begin = np.array([0, 3, 2], np.int32)  # decreasing
    else:
        begin = np.array([0, 2, 7], np.int32)  # past n
    net.rulebook_build(torch.tensor(coords).cuda(), 2, sample_begin=torch.tensor(begin).cuda())
    with pytest.raises(sscn.SSCNError) as e:
        net.layer_sizes()
    assert e.value.name == status
    ok = np.array([[0, 1, 1], [1, 2, 2]], np.int32)
    net.rulebook_build(torch.tensor(ok).cuda(), 2, sample_begin=torch.tensor([0, 1, 2], dtype=torch.int32).cuda())
    assert net.layer_sizes()[0] == 2
