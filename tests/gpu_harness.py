"""Runs the HIP path and the CPU oracle on the same seeded inputs and compares them.

Tolerances: float32 storage 1e-4, bfloat16 storage 2e-2, as the normwise
relative error max|gpu - ref| / max|ref| of each tensor.  Integer structures
(active counts, site lists, window lists and their transposes) must match
exactly.

Two discrete decisions are taken from floating-point values: the pool argmax
and the ReLU derivative [Z > 0].  Each must match the oracle's exactly except
at a near tie -- two window values within the tolerance of each other, or a
pre-activation within the tolerance of zero -- which a different (equally
valid) summation order can decide the other way.  Both decisions are then
correct, but they route a gradient differently, so gradients are compared with
the oracle's backward evaluated under the GPU's decision at those validated
near ties (and under its own decision everywhere else, which is everywhere
the two agree).  The oracle's arithmetic is unchanged; only which of two valid
answers it follows is aligned.
"""

import sys

import numpy as np
import torch

from oracle import SparseDeepCNet as Oracle
from paper_1409_6070_amd.sscn import SparseDeepCNet as GpuNet

TOL = {"f32": 1e-4, "bf16": 2e-2}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dtype(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.tensor(np.asarray(x, dtype=np.float64), dtype=torch.float32)
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref).max()
    diff = np.abs(got - ref).max()
    if scale == 0:
        return float(diff)
    return float(diff / scale)


class Pair:
    """One problem run through both paths."""

    def __init__(self, ell, k, c_in, n_classes, batch, coords, feats, Ws, bs, labels, dtype,
                 max_active=None, want_dfeats=True, run_oracle=True, arch="deepcnet", rates=None, dseed=0):
        self.dtype = dtype
        self.batch = batch
        dev = torch.device("cuda")
        feats_t = to_dtype(feats, dtype)
        Ws_t = [to_dtype(W, dtype) for W in Ws]
        bs_t = [torch.tensor(np.asarray(b, dtype=np.float32)) for b in bs]
        n = int(np.asarray(coords).shape[0])
        self.arch = arch
        self.net = GpuNet(ell, k, c_in, n_classes, batch_max=max(batch, 1), max_active=max_active or max(n, 1),
                          dtype=dtype, arch=arch, dropout=rates is not None)
        if rates is not None:
            self.net.set_dropout(rates, dseed)
        self.coords_d = torch.tensor(np.asarray(coords, dtype=np.int32).reshape(-1, 3)).to(dev).contiguous()
        self.feats_d = feats_t.to(dev).contiguous()
        self.Ws_d = [w.to(dev).contiguous() for w in Ws_t]
        self.bs_d = [b.to(dev).contiguous() for b in bs_t]
        self.labels_d = torch.tensor(np.asarray(labels, dtype=np.int32)).to(dev)
        self.want_dfeats = want_dfeats
        # the oracle receives exactly the values the GPU receives
        self.o = None
        if run_oracle:
            self.o = Oracle(ell, k, c_in, n_classes, dtype, arch)
            self.o.build(np.asarray(coords), batch)
            self.o.set_dropout(rates, dseed)
            self.o.forward(feats_t.double().numpy(), [w.double().numpy() for w in Ws_t],
                           [b.double().numpy() for b in bs_t], labels)
            self.o.backward()

    def run_gpu(self):
        net = self.net
        net.rulebook_build(self.coords_d, self.batch)
        self.counts = net.layer_sizes()
        logits, loss = net.forward(self.feats_d, self.Ws_d, self.bs_d, self.labels_d)
        dW, db, dfeats = net.backward(want_dfeats=self.want_dfeats)
        torch.cuda.synchronize()
        self.logits = logits.cpu().numpy()
        self.loss = float(loss.cpu()[0])
        self.dW = [t.cpu().numpy() for t in dW]
        self.db = [t.cpu().numpy() for t in db]
        self.dfeats = None if dfeats is None else dfeats.float().cpu().numpy()
        return self

    def view(self, layer):
        v = self.net.layer_view(layer, self.counts[layer])
        C = v["channels"]
        out = dict(v)
        out["X"] = v["features"].float().cpu().numpy()[:, :C]
        out["G"] = v["grad"].float().cpu().numpy()[:, :C]
        out["sites"] = v["sites"].cpu().numpy()
        if "rules" in v:
            out["rules"] = v["rules"].cpu().numpy()
        if "argmax" in v:
            out["argmax"] = v["argmax"].cpu().numpy()[:, :C]
        return out


def decode_sites(keys, S):
    keys = np.asarray(keys, dtype=np.int64)
    x = keys % S
    t = keys // S
    return np.stack([t // S, t % S, x], axis=1)


def expected_rules_t(R: np.ndarray, n_below: int, kind: str):
    """Transposed window lists from the oracle's window lists."""
    A = R.shape[1]
    n = R.shape[0] - 1
    if kind == "conv":
        Rt = -np.ones((n_below + 1, A), np.int64)
        o, f = np.nonzero(R[1:] > 0)
        Rt[R[1 + o, f], f] = 1 + o
        return Rt
    Pt = -np.ones(n_below + 1, np.int64)
    o, f = np.nonzero(R[1:] > 0)
    Pt[R[1 + o, f]] = (1 + o) * 4 + f
    return Pt


def check_structure(p: Pair):
    """Counts, site lists, window lists and transposes: bit-exact."""
    o = p.o
    assert p.counts == o.layer_sizes(), (p.counts, o.layer_sizes())
    for s, L in enumerate(o.layers):
        v = p.view(s)
        np.testing.assert_array_equal(decode_sites(v["sites"], L.S), L.sites, err_msg=f"sites layer {s}")
        if s == 0:
            continue
        np.testing.assert_array_equal(v["rules"], L.R, err_msg=f"rules layer {s}")
        st = o.stages[s - 1]
        Rt = p.net.rules_t(s, o.layers[s - 1].n).cpu().numpy()
        np.testing.assert_array_equal(Rt, expected_rules_t(L.R, o.layers[s - 1].n, st.kind),
                                      err_msg=f"transposed rules layer {s}")


def check_values(p: Pair, tol=None, check_grads=True):
    """Features, argmax, logits, loss, gradients: normwise within the dtype's tolerance.

    Every error is measured and printed before the first failing one is asserted."""
    try:
        return _check_values(p, tol, check_grads)
    finally:
        rep = getattr(p, "report", {})
        if rep:
            log("  " + " ".join(f"{k}={v:.2g}" if isinstance(v, float) else f"{k}={v}" for k, v in rep.items()))


def _check_values(p: Pair, tol=None, check_grads=True):
    o = p.o
    tol = tol if tol is not None else TOL[p.dtype]
    report = p.report = {}
    flipped = []
    relu_flips = []
    for s, L in enumerate(o.layers):
        v = p.view(s)
        e = rel_err(v["X"], L.X)
        report[f"X{s}"] = e
        assert e <= tol, f"features layer {s}: rel err {e:.3g} > {tol}"
        if "argmax" in v:
            below = o.layers[s - 1]
            V = below.X[L.R]  # [n+1, 4, C]
            bad = np.nonzero(v["argmax"] != L.argmax)
            if bad[0].size:
                rows, cols = bad
                gap = np.abs(V[rows, L.argmax[rows, cols], cols] - V[rows, v["argmax"][rows, cols].astype(np.int64), cols])
                scale = max(np.abs(below.X).max(), 1e-30)
                assert np.all(gap <= tol * scale), f"argmax layer {s}: {rows.size} mismatches, max gap {gap.max()}"
            report[f"argmax{s}_mismatch"] = int(bad[0].size)
            if bad[0].size:
                flipped.append((s, bad, v["argmax"][bad].astype(np.int64)))
        if L.relu_on is not None:
            # the GPU's rectifier branch from its stored output: ReLU y > 0; leaky x/3: sign bit clear
            gpu_on = v["X"] > 0 if o.slope == 0.0 else ~np.signbit(v["X"])
            bad = np.nonzero(gpu_on != L.relu_on)
            if bad[0].size:
                scale = max(np.abs(L.X).max(), 1e-30)
                near = np.maximum(np.abs(L.X[bad]), np.abs(v["X"][bad]))
                assert np.all(near <= tol * scale), f"rectifier decision layer {s}: {bad[0].size} flips, max |Z| {near.max()}"
                relu_flips.append((s, gpu_on))
            report[f"relu{s}_mismatch"] = int(bad[0].size)
    e = rel_err(p.logits, o.logits)
    report["logits"] = e
    assert e <= tol, f"logits rel err {e}"
    e = abs(p.loss - o.loss) / max(abs(o.loss), 1e-30)
    report["loss"] = e
    assert e <= tol, f"loss {p.loss} vs {o.loss}"
    if not check_grads:
        return report
    if flipped or relu_flips:
        # every differing decision was validated above as a near tie
        for s, idx, gpu_choice in flipped:
            o.layers[s].argmax[idx] = gpu_choice
        for s, gpu_on in relu_flips:
            o.layers[s].relu_on = gpu_on
        o.backward()
    for i, (a, b) in enumerate(zip(p.dW, o.dW)):
        e = rel_err(a, b)
        report[f"dW{i}"] = e
        assert e <= tol, f"dW[{i}] rel err {e:.3g}"
    for i, (a, b) in enumerate(zip(p.db, o.db)):
        e = rel_err(a, b)
        report[f"db{i}"] = e
        assert e <= tol, f"db[{i}] rel err {e:.3g}"
    for s, L in enumerate(o.layers):
        if s == 0 and not p.want_dfeats:
            continue
        v = p.view(s)
        e = rel_err(v["G"], L.grad)
        report[f"G{s}"] = e
        assert e <= tol, f"gradient layer {s}: rel err {e:.3g}"
    if p.want_dfeats:
        e = rel_err(p.dfeats, o.dfeats)
        report["dfeats"] = e
        assert e <= tol, f"dfeats rel err {e}"
    return report
