"""Oracle: sparse DeepCNet(ell, k) forward and backward on the CPU, NumPy float64.

TEST INFRASTRUCTURE ONLY -- the product path never imports this module.

What is computed (the paper's own description, restated):

* DeepCNet(ell, k) (Section 2.1): ell + 1 convolutional layers separated by ell
  layers of 2x2 max-pooling; the n-th convolution has n*k filters, 3x3 in the
  first layer and 2x2 afterwards; the input grid is N = 3 * 2**ell so that the
  last convolution leaves a 1x1 grid; ReLU on hidden layers and a softmax
  output layer (Section 2.1, activation paragraph).
* DeepCNiN(ell, k) (Section 2.2): the same with a network-in-network layer --
  a convolution with 1x1 filters, as many as the layer below has channels --
  after every pooling layer and after the last convolution, and the leaky
  rectifier f(x) = x for x >= 0, x/3 for x < 0 on every hidden layer.
* Spatial sparsity (Section 2.3): every hidden variable has a ground state,
  the value it takes when its input region holds no meaningful input; only
  sites whose value can differ from it are computed.  Each layer keeps a
  feature matrix (row 0 the ground state, then one row per active site) and a
  pointer matrix (one entry per spatial location of the layer, naming that
  location's feature-matrix row).  Backpropagation runs over the same
  structures in reverse (Section 2.3, last paragraph).
* Dropout (Section 2.1; Section 2.2 for DeepCNiN): one rate for the input of each
  convolution that is not 1x1 and one for the softmax layer's input; masks from
  the counter-based generator in ``philox``.

Readings where the paper is silent (each is also listed in the design notes):

* convolutions are "valid" with stride 1 and cross-correlation orientation;
  the weight row index is ``(dy*F + dx)*C_in + c`` (forced by N = 3*2**ell
  reaching exactly 1x1, Section 2.1);
* a site is active when any site of its receptive window in the layer below
  is active, whatever the values (Figure 2's caption); input sites are active
  exactly when listed;
* the input ground state is 0 (zero background, Sections 1 and 2.5);
* feature-matrix rows are in ascending (b, y, x) order;
* max-pool argmax is the first maximal window position in row-major order
  (dy, dx) = (0,0), (0,1), (1,0), (1,1);
* ReLU'(0) = 0; for the leaky rectifier f'(x) = 1 for x >= 0 and 1/3 for x < 0;
  the loss is softmax cross-entropy averaged over the batch;
* dropout is inverted (kept values times 1/(1 - p)) and touches only rows >= 1 of
  a layer: the ground row is never dropped, so inactive sites keep one shared
  ground state (``set_dropout``);
* the ground row takes part in backpropagation as one virtual site standing
  for all inactive sites together, so weight and bias gradients equal those
  of the dense network (derivation in ``backward``);
* storage rounding: in mode "f32" every stored matrix is rounded to float32;
  in mode "bf16" activations, gradients fed to products and the softmax
  layer's input/gradients are rounded to bfloat16 (round to nearest even)
  while sums stay in float64 here (float32 on the GPU); weight and bias
  gradients and logits are float32.  Mode "f64" rounds nothing and is what
  the pins against the dense network use.
"""

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .philox import drop_scale, dropout_keep


class OracleInputError(ValueError):
    """Raised for inputs the method does not define: duplicate or out-of-range sites."""

    def __init__(self, kind: str, msg: str):
        super().__init__(f"{kind}: {msg}")
        self.kind = kind


# ---------------------------------------------------------------------------
# storage rounding


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 through float32, nearest-even at each step.

    bfloat16 keeps the upper 16 bits of an IEEE float32.  Rounding adds 0x7FFF
    plus the lowest kept bit to the 32-bit pattern before truncation, which is
    round-to-nearest with ties to even.  (Finite inputs only.)
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32)
    lsb = u >> 16
    lsb &= 1
    u += np.uint32(0x7FFF)  # cannot overflow: finite patterns are <= 0xFF7FFFFF
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return f.astype(np.float64)


def round_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_store(x: np.ndarray, mode: str) -> np.ndarray:
    """Round to the storage type of ``mode`` ("f64": none, "f32", "bf16")."""
    if mode == "f64":
        return np.asarray(x, dtype=np.float64)
    if mode == "f32":
        return round_f32(x)
    if mode == "bf16":
        return round_bf16(x)
    raise ValueError(mode)


# ---------------------------------------------------------------------------
# architecture


@dataclass(frozen=True)
class Stage:
    kind: str  # "conv" or "pool"
    F: int  # window side: 3, 2 or 1 (network-in-network) for convolutions, 2 for pooling
    S_in: int  # spatial side of the layer below
    S: int  # spatial side of this layer
    c_in: int
    c_out: int

    @property
    def A(self) -> int:
        return self.F * self.F


ARCHS = ("deepcnet", "deepcnin")


def stage_plan(ell: int, k: int, c_in: int, arch: str = "deepcnet") -> List[Stage]:
    """The stages of DeepCNet(ell, k) (2*ell + 1 of them, Section 2.1) or DeepCNiN(ell, k)
    (Section 2.2: a 1x1 convolution added after every pooling layer and after the last
    convolution, 3*ell + 2 stages) on an N = 3*2**ell input.

    A valid FxF convolution shrinks the side by F - 1; a 2x2 stride-2 pool halves it.
    """
    if ell < 1 or k < 1 or c_in < 1:
        raise ValueError("ell, k and c_in must be positive")
    if arch not in ARCHS:
        raise ValueError(arch)
    nin = arch == "deepcnin"
    N = 3 * 2 ** ell
    stages = [Stage("conv", 3, N, N - 2, c_in, k)]
    S, C = N - 2, k
    for n in range(2, ell + 2):
        stages.append(Stage("pool", 2, S, S // 2, C, C))
        S //= 2
        if nin:
            stages.append(Stage("conv", 1, S, S, C, C))
        stages.append(Stage("conv", 2, S, S - 1, C, n * k))
        S, C = S - 1, n * k
    if nin:
        stages.append(Stage("conv", 1, S, S, C, C))
    assert S == 1
    return stages


# ---------------------------------------------------------------------------
# the sparse network


@dataclass
class Layer:
    """One layer's structures (Section 2.3).

    ``P``: pointer matrix [B, S, S]; 0 means "inactive, use the ground row".
    ``sites``: [n, 3] (b, y, x) of rows 1..n, in ascending order.
    ``R``: [n + 1, A] rows of the layer below read by each row's window (row 0 all 0).
    ``X``: feature matrix [n + 1, C], row 0 the ground state.
    """

    S: int
    P: np.ndarray
    sites: np.ndarray
    R: Optional[np.ndarray] = None
    X: Optional[np.ndarray] = None
    argmax: Optional[np.ndarray] = None  # pooling layers: [n + 1, C] window position of the max
    relu_on: Optional[np.ndarray] = None  # convolution layers: [n + 1, C] rectifier on its x >= 0 branch (ReLU: X > 0)
    grad: Optional[np.ndarray] = None  # conv: dL/dZ (pre-activation); pool and input: dL/dX
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.sites.shape[0])


def _pointer_from_active(active: np.ndarray):
    """Number the active locations 1..n in ascending (b, y, x) order."""
    b, y, x = np.nonzero(active)
    P = np.zeros(active.shape, dtype=np.int64)
    P[b, y, x] = np.arange(1, b.size + 1)
    return P, np.stack([b, y, x], axis=1).astype(np.int64)


class SparseDeepCNet:
    """Sparse DeepCNet(ell, k) or DeepCNiN(ell, k) with a softmax head; calls mirror the C interface.

    ``build`` makes every layer's pointer matrix and window lists, ``forward``
    fills the feature matrices and the loss, ``backward`` returns parameter
    gradients and, per layer, the gradient matrices.
    """

    def __init__(self, ell: int, k: int, c_in: int, n_classes: int, mode: str = "f64", arch: str = "deepcnet"):
        if mode not in ("f64", "f32", "bf16"):
            raise ValueError(mode)
        self.ell, self.k, self.c_in, self.n_classes, self.mode = ell, k, c_in, n_classes, mode
        self.arch = arch
        self.N = 3 * 2 ** ell
        self.stages = stage_plan(ell, k, c_in, arch)
        # negative-side slope of the hidden layers' rectifier: ReLU (Section 2.1) or
        # the leaky x/3 of DeepCNiN (Section 2.2)
        self.slope = 1.0 / 3.0 if arch == "deepcnin" else 0.0
        self.layers: List[Layer] = []
        self.rates = None
        self.seed = 0

    # -- dropout ------------------------------------------------------------
    def dropout_stages(self) -> List[int]:
        """Stage index of each convolution whose input takes dropout: every convolution
        except the 1x1 network-in-network layers (Section 2.2), in order; the softmax
        layer's input follows as dropout site ``len(...)`` (Section 2.1: ell + 2 rates)."""
        return [si for si, st in enumerate(self.stages) if st.kind == "conv" and st.F > 1]

    def set_dropout(self, rates, seed: int):
        """Dropout rates per level (ell + 1 convolution inputs, then the softmax layer's
        input) and the 64-bit seed of the masks; ``None`` switches dropout off.

        Reading: inverted dropout on the active rows of the layer feeding each of those
        convolutions; the ground row (row 0) is never dropped, so every inactive site
        keeps the shared ground state and the sparse structure of Section 2.3 is
        unchanged.  Masks come from ``philox.dropout_keep``; dropout only applies in a
        training pass (``forward`` with labels).
        """
        if rates is None:
            self.rates = None
            return
        rates = [float(r) for r in rates]
        if len(rates) != self.ell + 2:
            raise ValueError(f"need {self.ell + 2} dropout rates, got {len(rates)}")
        for r in rates:
            if not 0.0 <= r < 1.0:
                raise ValueError("dropout rates must be in [0, 1)")
        self.rates, self.seed = rates, int(seed) & 0xFFFFFFFFFFFFFFFF

    def _drop_factor(self, keys, channels: int, j: int):
        """[n, C] multiplier of dropout site j for rows with the given keys (None: rate 0)."""
        p = self.rates[j]
        if p == 0.0:
            return None
        return np.where(dropout_keep(keys, channels, j, p, self.seed), drop_scale(p), 0.0)

    def _apply_drop(self, X: np.ndarray, factor) -> np.ndarray:
        """X * factor, rounded first to float32 and then to the storage type (modes f32, bf16)."""
        Y = X * factor
        return Y if self.mode == "f64" else round_store(round_f32(Y), self.mode)

    # -- parameters ---------------------------------------------------------
    def param_shapes(self):
        """Weight shapes: convolutions ``[F*F*C_in, C_out]``, then the softmax layer ``[C_last, classes]``."""
        shapes = [(s.A * s.c_in, s.c_out) for s in self.stages if s.kind == "conv"]
        shapes.append((self.stages[-1].c_out, self.n_classes))
        return shapes

    # -- structure ----------------------------------------------------------
    def build(self, coords: np.ndarray, batch: int):
        """Pointer matrices and window lists for every layer (Section 2.3).

        Input layer: the listed sites are active, numbered in ascending order.
        Convolution layer: a location is active when some location of its FxF
        window in the layer below is active; its window list names the rows of
        those F*F locations (0 for the inactive ones).  Pooling layer: the same
        with the 2x2 stride-2 window.
        """
        coords = np.asarray(coords, dtype=np.int64).reshape(-1, 3)
        N = self.N
        if batch < 0:
            raise OracleInputError("invalid_argument", "negative batch")
        if coords.size:
            b, y, x = coords[:, 0], coords[:, 1], coords[:, 2]
            bad = (b < 0) | (b >= batch) | (y < 0) | (y >= N) | (x < 0) | (x >= N)
            if bad.any():
                raise OracleInputError("out_of_range", f"site {coords[np.argmax(bad)].tolist()} outside batch/grid")
            keys = (b * N + y) * N + x
            if np.unique(keys).size != keys.size:
                raise OracleInputError("duplicate", "a site is listed twice")
        self.batch = batch
        n_in = coords.shape[0]
        P0 = np.zeros((batch, N, N), dtype=np.int64)
        if n_in:
            keys = (coords[:, 0] * N + coords[:, 1]) * N + coords[:, 2]
            order = np.argsort(keys, kind="stable")  # row r+1 holds caller site order[r]
            P0[coords[order, 0], coords[order, 1], coords[order, 2]] = np.arange(1, n_in + 1)
        else:
            order = np.zeros(0, dtype=np.int64)
        self.input_order = order
        self.layers = [Layer(S=N, P=P0, sites=coords[order] if n_in else np.zeros((0, 3), np.int64))]

        for st in self.stages:
            below = self.layers[-1]
            step = 1 if st.kind == "conv" else 2
            # window location (dy, dx) of output (Y, X) is (step*Y + dy, step*X + dx) below
            win = np.zeros((batch, st.S, st.S, st.A), dtype=np.int64)
            for dy in range(st.F):
                for dx in range(st.F):
                    win[..., dy * st.F + dx] = below.P[:, dy: dy + step * st.S: step, dx: dx + step * st.S: step]
            active = (win != 0).any(axis=-1)
            P, sites = _pointer_from_active(active)
            R = np.zeros((sites.shape[0] + 1, st.A), dtype=np.int64)
            R[1:] = win[sites[:, 0], sites[:, 1], sites[:, 2]]
            self.layers.append(Layer(S=st.S, P=P, sites=sites, R=R))
        return self.layer_sizes()

    def layer_sizes(self):
        """Active-site counts n_0 .. n_{2 ell + 1} (ground rows not counted)."""
        return [L.n for L in self.layers]

    def head_rows(self) -> np.ndarray:
        """Row of each sample's single top-layer site (0, the ground row, for an empty sample)."""
        return self.layers[-1].P[:, 0, 0].copy()

    # -- forward ------------------------------------------------------------
    def forward(self, feats, Ws, bs, labels):
        """Feature matrices of every layer, logits and mean softmax cross-entropy.

        ``labels=None`` is an inference pass: logits only (loss None), no dropout.
        With dropout set (``set_dropout``) a training pass multiplies rows >= 1 of
        each dropout site's input by its mask factor before use; the convolution
        (and its weight gradient) reads the dropped matrix.

        Convolution: row o of the output is ReLU(b + sum_f W_f^T x_{R[o][f]}),
        row 0 included -- its window is all ground rows, which makes it the
        layer's ground state.  Pooling: channel-wise max over the window's rows
        (row 0 passes the ground state through).  Head: each sample's top-layer
        row (the ground row if the sample is empty) feeds the softmax layer.
        """
        m = self.mode
        L0 = self.layers[0]
        feats = np.asarray(feats, dtype=np.float64).reshape(-1, self.c_in)
        X = np.zeros((L0.n + 1, self.c_in))
        X[1:] = feats[self.input_order]
        L0.X = round_store(X, m)
        self.Ws = [round_store(np.asarray(W, dtype=np.float64), m) for W in Ws]
        self.bs = [np.asarray(b, dtype=np.float64) for b in bs]
        train = labels is not None
        drop = train and self.rates is not None
        dsite = {si: j for j, si in enumerate(self.dropout_stages())}
        ci = 0
        for si, st in enumerate(self.stages):
            L, below = self.layers[si + 1], self.layers[si]
            Xin = below.X
            L.extra.pop("drop", None)
            if drop and si in dsite:
                keys = (below.sites[:, 0] * below.S + below.sites[:, 1]) * below.S + below.sites[:, 2]
                fac = self._drop_factor(keys, st.c_in, dsite[si])
                if fac is not None:
                    Xin = below.X.copy()
                    Xin[1:] = self._apply_drop(below.X[1:], fac)
                    L.extra["drop"] = fac  # [n_below, C_in] factor on rows 1.. of the layer below
            L.extra["Xin"] = Xin
            V = Xin[L.R]  # [n + 1, A, C_in]: the gathered windows
            if st.kind == "conv":
                Z = V.reshape(V.shape[0], -1) @ self.Ws[ci] + self.bs[ci]
                if self.slope == 0.0:
                    L.X = round_store(np.maximum(Z, 0.0), m)
                    L.relu_on = L.X > 0  # ReLU'(Z): 1 where the stored output is positive, 0 at Z <= 0
                else:
                    L.relu_on = Z >= 0.0  # f'(Z) = 1 on the x >= 0 branch, 1/3 below
                    L.X = round_store(np.where(L.relu_on, Z, Z / 3.0), m)
                ci += 1
            else:
                L.argmax = np.argmax(V, axis=1)  # first maximal window position
                L.X = V.max(axis=1)
        rows = self.head_rows()
        self.h = self.layers[-1].X[rows]
        self.h_drop = None
        if drop:
            self.h_drop = self._drop_factor(np.arange(self.batch), self.h.shape[1], len(dsite))
            if self.h_drop is not None:
                self.h = self._apply_drop(self.h, self.h_drop)
        logits = self.h @ self.Ws[-1] + self.bs[-1]
        self.logits = logits if m == "f64" else round_f32(logits)
        self.trained = train
        if not train:
            self.labels, self.loss = None, None
            return self.logits, None
        labels = np.asarray(labels, dtype=np.int64)
        self.labels = labels
        z = self.logits - self.logits.max(axis=1, keepdims=True)
        lse = np.log(np.exp(z).sum(axis=1))
        self.loss = float(np.mean(lse - z[np.arange(self.batch), labels])) if self.batch else 0.0
        return self.logits, self.loss

    # -- backward -----------------------------------------------------------
    def backward(self):
        """Gradients of the mean loss with respect to every parameter and layer.

        Each layer's gradient matrix has the feature matrix's rows; row 0 holds
        the sum of the dense network's gradients over all of that layer's
        inactive sites.  Because an inactive output's window is entirely
        inactive, its contribution to a weight gradient is (ground row) x
        (its gradient), so summing those gradients into row 0 first and then
        treating row 0 as one more site gives the dense weight and bias
        gradients exactly; the same argument gives row 0 of the layer below.
        """
        if not getattr(self, "trained", False):
            raise RuntimeError("backward needs a training forward pass (with labels)")
        m = self.mode
        B = self.batch
        p = np.exp(self.logits - self.logits.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        onehot = np.zeros_like(p)
        onehot[np.arange(B), self.labels] = 1.0
        dlogits = round_store((p - onehot) / max(B, 1), m)
        self.dlogits = dlogits
        dW = [None] * len(self.Ws)
        db = [None] * len(self.Ws)
        dW[-1] = self.h.T @ dlogits
        db[-1] = dlogits.sum(axis=0)
        dh = dlogits @ self.Ws[-1].T
        if self.h_drop is not None:
            dh = dh * self.h_drop  # through the softmax layer's dropout
        top = self.layers[-1]
        dY = np.zeros_like(top.X)
        np.add.at(dY, self.head_rows(), dh)
        top.grad = round_store(dY * self.act_grad(top), m)  # dL/dZ of the last convolution

        ci = len(self.Ws) - 2
        for si in range(len(self.stages) - 1, -1, -1):
            st, L, below = self.stages[si], self.layers[si + 1], self.layers[si]
            if st.kind == "conv":
                delta = L.grad  # [n + 1, C_out]
                V = L.extra["Xin"][L.R].reshape(L.R.shape[0], -1)
                dW[ci] = V.T @ delta
                db[ci] = delta.sum(axis=0)
                dV = (delta @ self.Ws[ci].T).reshape(L.R.shape[0], st.A, st.c_in)
                dX = np.zeros((below.n + 1, st.c_in))
                np.add.at(dX, L.R.ravel(), dV.reshape(-1, st.c_in))
                if "drop" in L.extra:
                    dX[1:] *= L.extra["drop"]  # through this convolution's input dropout
                if si > 0 and self.stages[si - 1].kind == "conv":
                    below.grad = round_store(dX * self.act_grad(below), m)  # a convolution below: dL/dZ
                else:
                    below.grad = round_store(dX, m)  # pooling layer (or input): dL/dX
                ci -= 1
            else:
                dYp = L.grad  # dL/dY of the pooling layer
                rows = L.R[np.arange(L.R.shape[0])[:, None], L.argmax]  # [n + 1, C] row of each max
                dX = np.zeros((below.n + 1, st.c_in))
                np.add.at(dX, (rows, np.broadcast_to(np.arange(st.c_in), rows.shape)), dYp)
                below.grad = round_store(dX * self.act_grad(below), m)  # the convolution below: dL/dZ
        self.dW, self.db = dW, db
        dfeats = np.zeros((self.layers[0].n, self.c_in))
        dfeats[self.input_order] = self.layers[0].grad[1:]
        self.dfeats = dfeats
        return dW, db, dfeats

    def act_grad(self, L: Layer) -> np.ndarray:
        """Derivative of the hidden layers' rectifier at each of L's pre-activations."""
        return np.where(L.relu_on, 1.0, self.slope)

    # -- inspection ---------------------------------------------------------
    def layer_view(self, i: int) -> Layer:
        """Layer i: 0 is the input, 1 .. 2 ell + 1 follow the stages."""
        return self.layers[i]
