"""Dense brute force for pinning the oracle: the ordinary (non-sparse) DeepCNet.

The sparse method is an exact memoisation of the dense network evaluated on a
zero-filled N x N input grid (Section 2.3), so the dense network computed with
library routines -- torch's conv2d / max_pool2d / relu / cross_entropy and
autograd, on the CPU in float64 -- is an independent statement of the result.
It shares nothing with the oracle beyond the weight layout convention
(row ``(dy*F + dx)*C_in + c`` of a ``[F*F*C_in, C_out]`` matrix).
"""

import numpy as np
import torch
import torch.nn.functional as Fn


def conv_weight(W: np.ndarray, F: int, c_in: int) -> torch.Tensor:
    """[F*F*C_in, C_out] -> torch's [C_out, C_in, F, F] (cross-correlation)."""
    c_out = W.shape[1]
    w = torch.tensor(W, dtype=torch.float64).reshape(F, F, c_in, c_out)
    return w.permute(3, 2, 0, 1).contiguous()


def cast_storage(t: torch.Tensor, mode: str) -> torch.Tensor:
    """Value of a float64 tensor after storing it in the mode's type: float32, or bfloat16 through
    float32 (the device accumulates in float32 and rounds that to bfloat16), by torch's casts."""
    if mode == "f64":
        return t
    t32 = t.to(torch.float32)
    return (t32 if mode == "f32" else t32.to(torch.bfloat16)).to(torch.float64)


class StoreValue(torch.autograd.Function):
    """Rounds a value to the storage type; the gradient passes unchanged."""

    @staticmethod
    def forward(ctx, x, mode):
        return cast_storage(x, mode)

    @staticmethod
    def backward(ctx, g):
        return g, None


class StoreGrad(torch.autograd.Function):
    """Leaves a value unchanged; rounds the gradient flowing back through it to the storage type."""

    @staticmethod
    def forward(ctx, x, mode):
        ctx.mode = mode
        return x.view_as(x)

    @staticmethod
    def backward(ctx, g):
        return cast_storage(g, ctx.mode), None


def dense_grid(coords, feats, batch, N, c_in):
    x = torch.zeros(batch, c_in, N, N, dtype=torch.float64)
    coords = np.asarray(coords).reshape(-1, 3)
    if coords.shape[0]:
        x[coords[:, 0], :, coords[:, 1], coords[:, 2]] = torch.tensor(np.asarray(feats), dtype=torch.float64)
    return x


class DenseDeepCNet:
    """Dense DeepCNet(ell, k): 3x3 conv, then (2x2/2 max-pool, 2x2 conv) x ell, ReLU, softmax head.

    arch="deepcnin": DeepCNiN(ell, k) (Section 2.2), a 1x1 convolution after every
    pool and after the last convolution, and the leaky rectifier x/3 for x < 0
    (torch's leaky_relu with negative slope 1/3) on every hidden layer.
    """

    def __init__(self, ell, k, c_in, n_classes, arch="deepcnet", mode="f64"):
        self.ell, self.k, self.c_in, self.n_classes = ell, k, c_in, n_classes
        self.arch = arch
        self.N = 3 * 2 ** ell
        # "f64": no rounding.  "f32" / "bf16": every stored quantity of the device path rounded to
        # that type where it is stored -- the input, the weights, every layer's output, the
        # logits (float32), the loss gradient at the logits, every convolution's dL/dZ and every
        # pooling layer's and the input's dL/dX -- with all products and sums in float64.
        self.mode = mode

    def run(self, coords, feats, batch, Ws, bs, labels, masks=None):
        """Forward and autograd backward.  ``masks``: optional per-level dropout multipliers,
        one per convolution that is not 1x1 ([B, C_in, S, S], multiplying that convolution's
        input) and one for the softmax layer's input ([B, C]); None entries mean no dropout."""
        masks = masks or [None] * (self.ell + 2)
        m = self.mode
        sv = (lambda t: t) if m == "f64" else (lambda t: StoreValue.apply(t, m))
        sg = (lambda t: t) if m == "f64" else (lambda t: StoreGrad.apply(t, m))
        x = cast_storage(dense_grid(coords, feats, batch, self.N, self.c_in), m).requires_grad_(True)
        params = []
        for W, b in zip(Ws, bs):
            w = cast_storage(torch.tensor(np.asarray(W), dtype=torch.float64), m)
            params.append(w.requires_grad_(True))
            params.append(torch.tensor(np.asarray(b), dtype=torch.float64, requires_grad=True))
        nin = self.arch == "deepcnin"
        act = (lambda z: Fn.leaky_relu(z, 1.0 / 3.0)) if nin else torch.relu
        Zs, Ys = [], []  # per stage: pre-activation (conv) and output
        h = sg(x)  # the input's gradient is stored
        c = self.c_in
        pi = 0
        di = 0

        def conv(h, F, c):
            nonlocal pi, di
            W, b = params[2 * pi], params[2 * pi + 1]
            pi += 1
            if F > 1:
                if masks[di] is not None:
                    # the dropped copy is stored: rounded to float32, then to the storage type
                    h = h * torch.as_tensor(masks[di], dtype=torch.float64)
                    if m != "f64":
                        h = sv(StoreValue.apply(h, "f32"))
                di += 1
            wt = W.reshape(F, F, c, W.shape[1]).permute(3, 2, 0, 1)
            z = Fn.conv2d(h, wt) + b.view(1, -1, 1, 1)
            z.retain_grad()
            y = sv(act(sg(z)))  # dL/dZ and the output are stored
            Zs.append(z)
            Ys.append(y)
            return y, W.shape[1]

        for li in range(self.ell + 1):
            if li > 0:
                pooled = Fn.max_pool2d(h, 2)
                pooled.retain_grad()
                Zs.append(None)
                Ys.append(pooled)
                h = sg(pooled)  # the pooling layer's dL/dX is stored
                if nin:
                    h, c = conv(h, 1, c)
            h, c = conv(h, 3 if li == 0 else 2, c)
        if nin:
            h, c = conv(h, 1, c)
        assert h.shape[-1] == 1 and h.shape[-2] == 1
        feat = h[:, :, 0, 0]
        if masks[-1] is not None:
            feat = feat * torch.as_tensor(masks[-1], dtype=torch.float64)
            if m != "f64":
                feat = sv(StoreValue.apply(feat, "f32"))
        logits = feat @ params[-2] + params[-1]
        if m != "f64":  # logits are float32; the loss gradient at them is stored
            logits = sg(StoreValue.apply(logits, "f32"))
        loss = Fn.cross_entropy(logits, torch.tensor(np.asarray(labels), dtype=torch.int64))
        loss.backward()
        self.x, self.params, self.Zs, self.Ys = x, params, Zs, Ys
        self.logits, self.loss = logits.detach().numpy(), float(loss)
        self.dW = [p.grad.numpy() for p in params[0::2]]
        self.db = [p.grad.numpy() for p in params[1::2]]
        return self


def dilate_reference(active: np.ndarray, kind: str, F: int) -> np.ndarray:
    """Active set of the next layer from a boolean [B, S, S] grid, via library routines.

    Convolution: conv2d of the indicator with an all-ones FxF kernel is non-zero.
    Pooling: max_pool2d(2) of the indicator.
    """
    t = torch.tensor(active.astype(np.float64))[:, None]
    if kind == "conv":
        out = Fn.conv2d(t, torch.ones(1, 1, F, F, dtype=torch.float64)) > 0
    else:
        out = Fn.max_pool2d(t, 2) > 0
    return out[:, 0].numpy()
