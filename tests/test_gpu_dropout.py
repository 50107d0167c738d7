"""Dropout per level (Section 2.1; none on DeepCNiN's 1x1 layers, Section 2.2) on the GPU
against the oracle, through the C interface.

Both sides draw the same masks from their own implementations of the counter-based
generator, so every kept/dropped decision must agree exactly: a single differing
element changes a feature by a full value and fails the normwise tolerance.
"""

import numpy as np
import pytest
import torch

from tests.gpu_harness import Pair, check_structure, check_values, log, to_dtype
from tests.test_gpu_parity import _sparse_case
from workloads import he_params, random_labels

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1409_6070_amd import sscn
    sscn.load_library()


DROP_CASES = [
    # name, arch, ell, k, c_in, classes, batch, density, empty, rates, seed
    ("cnet_l1k3_all", "deepcnet", 1, 3, 1, 4, 2, 0.3, (), [0.3, 0.5, 0.4], 41),
    ("cnet_l2k5_m3_empty", "deepcnet", 2, 5, 3, 7, 3, 0.08, (1,), [0.2, 0.0, 0.5, 0.25], 42),
    ("cnet_l3k20_upper", "deepcnet", 3, 20, 2, 33, 4, 0.05, (), [0.0, 0.0, 0.5, 0.5, 0.5], 43),
    ("cnet_l4k24_m1", "deepcnet", 4, 24, 1, 129, 5, 0.02, (), [0.1, 0.1, 0.2, 0.3, 0.4, 0.5], 44),
    ("nin_l2k5_m3_empty", "deepcnin", 2, 5, 3, 7, 3, 0.08, (1,), [0.5, 0.3, 0.2, 0.4], 45),
    ("nin_l3k20_m2", "deepcnin", 3, 20, 2, 33, 4, 0.05, (), [0.0, 0.25, 0.5, 0.5, 0.5], 46),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", DROP_CASES, ids=[c[0] for c in DROP_CASES])
def test_dropout_small(case, dtype):
    name, arch, ell, k, c_in, ncls, batch, density, empty, rates, seed = case
    coords, feats = _sparse_case(seed, ell, batch, density, c_in, empty)
    dseed = (seed << 40) | 0x5EED
    log(f"[dropout] {name} {dtype} n={len(coords)} seed={seed} rates={rates}")
    Ws, bs = he_params(ell, k, c_in, ncls, 100 + seed, arch)
    labels = random_labels(batch, ncls, 200 + seed)
    pair = Pair(ell, k, c_in, ncls, batch, coords, feats, Ws, bs, labels, dtype, arch=arch, rates=rates,
                dseed=dseed).run_gpu()
    check_structure(pair)
    check_values(pair)


def _plain_and_drop(dtype, rates, dseed=9, arch="deepcnet"):
    ell, k, c_in, ncls, batch = 3, 12, 2, 9, 3
    coords, feats = _sparse_case(50, ell, batch, 0.06, c_in)
    Ws, bs = he_params(ell, k, c_in, ncls, 150, arch)
    labels = random_labels(batch, ncls, 250)
    a = Pair(ell, k, c_in, ncls, batch, coords, feats, Ws, bs, labels, dtype, arch=arch, run_oracle=False)
    b = Pair(ell, k, c_in, ncls, batch, coords, feats, Ws, bs, labels, dtype, arch=arch, run_oracle=False,
             rates=rates, dseed=dseed)
    return a, b


def _outputs(p):
    return [p.logits, *p.dW, *p.db, p.dfeats] + [p.view(s)["G"] for s in range(len(p.counts))]


@pytest.mark.parametrize("arch", ["deepcnet", "deepcnin"])
def test_rate_zero_is_bitwise_plain(arch):
    """All rates 0 on a net with dropout workspace: the same launches' results as a net without."""
    log(f"[dropout] rate 0 {arch}")
    a, b = _plain_and_drop("bf16", [0.0] * 5, arch=arch)
    for x, y in zip(_outputs(a.run_gpu()), _outputs(b.run_gpu())):
        np.testing.assert_array_equal(x, y)


def test_inference_ignores_dropout_and_seed_changes_masks():
    from paper_1409_6070_amd import sscn
    log("[dropout] inference and seeds")
    a, b = _plain_and_drop("f32", [0.5] * 5)
    for p in (a, b):
        p.net.rulebook_build(p.coords_d, p.batch)
    la, _ = a.net.forward(a.feats_d, a.Ws_d, a.bs_d, None)
    la = la.clone()
    lb, _ = b.net.forward(b.feats_d, b.Ws_d, b.bs_d, None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(la.cpu().numpy(), lb.cpu().numpy())
    # a training pass applies the masks; the same seed repeats them, another seed does not
    b.run_gpu()
    first = [x.copy() for x in _outputs(b)]
    b.run_gpu()
    for x, y in zip(first, _outputs(b)):
        np.testing.assert_array_equal(x, y)
    b.net.set_dropout([0.5] * 5, 10)
    b.run_gpu()
    assert not np.array_equal(first[0], b.logits)
    # a new rate setting ends the pass: no backward until the next training forward
    b.net.set_dropout([0.5] * 5, 11)
    with pytest.raises(sscn.SSCNError) as e:
        b.net.backward()
    assert e.value.name == "SSCN_ERR_BAD_STATE"
