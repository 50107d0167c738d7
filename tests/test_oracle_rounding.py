"""Pins the oracle's storage-rounding modes ("f32", "bf16") to something other than itself.

The device path stores the input, the weights, every layer's output, the logits
(float32), the loss gradient at the logits, every convolution's dL/dZ and every
pooling layer's and the input's dL/dX in its storage type, and sums in float32;
the oracle rounds at the same points and sums in float64.  The independent
statement is the dense network (torch's conv2d / max_pool2d / rectifiers /
cross_entropy and autograd, float64) with torch's casts at those points
(``tests.dense_ref``, ``mode``).  Everything the sparse method computes for an
active site is then the same float64 arithmetic on the same rounded operands,
so it must agree bit for bit:

* every layer's features at active sites, and the ground row with the value
  of every inactive site (Section 2.3);
* logits; rows >= 1 of every gradient matrix (an active row's gradient only
  ever gathers from active rows of the layer above: every window holding an
  active site is active, and every active site's pooling parent is active).

Row 0 of a gradient (one rounding of a sum over inactive sites, where the dense
network rounds each site) and dW, db (which include row 0's contribution) agree
to a few storage ulps of the summed magnitudes.  Planted mistakes in the
oracle's rounding placement each fail this pin.
"""

import inspect
import sys
import types

import numpy as np
import pytest

import oracle.sparse_deepcnet as oracle_mod
from oracle import SparseDeepCNet
from tests.dense_ref import DenseDeepCNet
from workloads import he_params, random_labels

EPS = {"f32": 2.0 ** -24, "bf16": 2.0 ** -8}


def _sites(rng, batch, N, p, c_in, empty=(), full=()):
    coords = []
    for b in range(batch):
        if b in empty:
            continue
        mask = np.ones((N, N), bool) if b in full else rng.random((N, N)) < p
        ys, xs = np.nonzero(mask)
        coords.append(np.stack([np.full(ys.size, b), ys, xs], 1))
    coords = np.concatenate(coords) if coords else np.zeros((0, 3), np.int64)
    coords = coords[rng.permutation(coords.shape[0])]
    return coords.astype(np.int64), rng.normal(size=(coords.shape[0], c_in))


CASES = [
    # arch, ell, k, c_in, classes, batch, p, empty, full, seed
    ("deepcnet", 2, 3, 1, 5, 3, 0.1, (1,), (), 41),
    ("deepcnet", 3, 4, 2, 7, 2, 0.04, (), (), 42),
    ("deepcnet", 2, 5, 3, 4, 2, 0.15, (), (0,), 43),
    ("deepcnin", 2, 3, 1, 5, 3, 0.1, (2,), (), 44),
    ("deepcnin", 3, 3, 2, 6, 2, 0.05, (), (), 45),
]


def _pair(case, mode, cls=SparseDeepCNet):
    arch, ell, k, c_in, ncls, batch, p, empty, full, seed = case
    rng = np.random.default_rng(seed)
    coords, feats = _sites(rng, batch, 3 * 2 ** ell, p, c_in, empty, full)
    Ws, bs = he_params(ell, k, c_in, ncls, seed + 100, arch)
    labels = random_labels(batch, ncls, seed + 200)
    o = cls(ell, k, c_in, ncls, mode, arch)
    o.build(coords, batch)
    # both sides take the inputs as given; each rounds them to its storage type itself
    o.forward(feats, Ws, bs, labels)
    o.backward()
    d = DenseDeepCNet(ell, k, c_in, ncls, arch, mode).run(coords, feats, batch, Ws, bs, labels)
    return o, d


def _layer_grads(o, d):
    """(layer, dense gradient [B, S, S, C]) for every layer: dL/dZ for convolutions, dL/dX otherwise."""
    out = [(o.layers[0], d.x.grad.numpy().transpose(0, 2, 3, 1))]
    for s in range(1, len(o.layers)):
        st = o.stages[s - 1]
        g = d.Zs[s - 1].grad if st.kind == "conv" else d.Ys[s - 1].grad
        out.append((o.layers[s], g.numpy().transpose(0, 2, 3, 1)))
    return out


def check_rounding_pin(o, d, mode):
    eps = EPS[mode]
    # forward: bit for bit at active sites; the ground row is every inactive site's value
    for s in range(1, len(o.layers)):
        L = o.layers[s]
        dense = d.Ys[s - 1].detach().numpy().transpose(0, 2, 3, 1)
        act = L.P != 0
        np.testing.assert_array_equal(L.X[L.P[act]], dense[act], err_msg=f"features layer {s}")
        if (~act).any():
            np.testing.assert_array_equal(np.broadcast_to(L.X[0], dense[~act].shape), dense[~act],
                                          err_msg=f"ground row layer {s}")
    np.testing.assert_array_equal(o.logits, d.logits, err_msg="logits")
    assert abs(o.loss - d.loss) <= 1e-12 * max(1.0, abs(d.loss))
    # gradients: active rows bit for bit; row 0 within the rounding of its sum
    for i, (L, g) in enumerate(_layer_grads(o, d)):
        act = L.P != 0
        np.testing.assert_array_equal(L.grad[L.P[act]], g[act], err_msg=f"gradient rows >= 1, layer {i}")
        inact = g[~act]
        mag = np.abs(inact).sum(axis=0)
        assert np.all(np.abs(L.grad[0] - inact.sum(axis=0)) <= 4 * eps * (mag + np.abs(L.grad[0])) + 1e-300), \
            f"gradient row 0, layer {i}"
    # parameter gradients: within a few ulps of the summed magnitudes (they include row 0)
    for a, b in zip(o.dW + o.db, d.dW + d.db):
        assert np.abs(a - b).max() <= 8 * eps * max(np.abs(b).max(), 1e-300), "parameter gradient"


@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}_l{c[1]}k{c[2]}m{c[3]}" for c in CASES])
def test_oracle_rounding_equals_dense_network_with_casts(case, mode):
    o, d = _pair(case, mode)
    check_rounding_pin(o, d, mode)


def test_rounding_modes_differ_from_f64():
    """The pin has teeth only if the modes round at all: f32, bf16 and f64 results all differ."""
    case = CASES[0]
    grads = {m: _pair(case, m)[0].layers[1].grad for m in ("f64", "f32", "bf16")}
    assert not np.array_equal(grads["f64"], grads["f32"])
    assert not np.array_equal(grads["f32"], grads["bf16"])


def _mutant(old: str, new: str):
    """The oracle's class with one source line changed (a planted mistake, CPU only)."""
    src = inspect.getsource(oracle_mod)
    assert src.count(old) == 1, old
    name = "oracle._rounding_mutant"
    mod = types.ModuleType(name)
    mod.__package__ = "oracle"
    sys.modules[name] = mod
    try:
        exec(compile(src.replace(old, new), f"<{name}>", "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod.SparseDeepCNet


MUTANTS = [
    # the rectifier derivative applied after rounding dL/dY instead of before (below a convolution)
    ("below.grad = round_store(dX * self.act_grad(below), m)  # a convolution below: dL/dZ",
     "below.grad = round_store(dX, m) * self.act_grad(below)  # a convolution below: dL/dZ", "deepcnin"),
    # the same at the top layer
    ("top.grad = round_store(dY * self.act_grad(top), m)",
     "top.grad = round_store(dY, m) * self.act_grad(top)", "deepcnin"),
    # the same below a pooling layer
    ("below.grad = round_store(dX * self.act_grad(below), m)  # the convolution below: dL/dZ",
     "below.grad = round_store(dX, m) * self.act_grad(below)  # the convolution below: dL/dZ", "deepcnin"),
    # the loss gradient at the logits not rounded to the storage type
    ("dlogits = round_store((p - onehot) / max(B, 1), m)", "dlogits = (p - onehot) / max(B, 1)", "deepcnet"),
    # the logits not rounded to float32
    ("self.logits = logits if m == \"f064\" else round_f32(logits)".replace("f064", "f64"), "self.logits = logits",
     "deepcnet"),
    # a pooling layer's (or the input's) gradient not rounded
    ("below.grad = round_store(dX, m)  # pooling layer (or input): dL/dX",
     "below.grad = dX  # pooling layer (or input): dL/dX", "deepcnet"),
    # a convolution's output rounded before its rectifier and the bias added after
    ("Z = V.reshape(V.shape[0], -1) @ self.Ws[ci] + self.bs[ci]",
     "Z = round_store(V.reshape(V.shape[0], -1) @ self.Ws[ci], m) + self.bs[ci]", "deepcnet"),
]


@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("old,new,arch", MUTANTS, ids=[f"mutant{i}" for i in range(len(MUTANTS))])
def test_planted_rounding_mistakes_fail_the_pin(old, new, arch, mode):
    cls = _mutant(old, new)
    failed = 0
    for case in [c for c in CASES if c[0] == arch]:
        o, d = _pair(case, mode, cls)
        try:
            check_rounding_pin(o, d, mode)
        except AssertionError:
            failed += 1
    assert failed, "a planted rounding mistake passed the pin"
