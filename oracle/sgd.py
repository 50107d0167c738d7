"""One stochastic-gradient-descent update of the network's parameters (test infrastructure only).

The paper trains its networks by backpropagation (Sections 2.3 and 3) without
stating the optimiser's form.  Reading (listed in the design notes): SGD with
classical momentum and L2 weight decay on the weight matrices (not the biases),
in the convention of the common library optimiser:

    g = dL/dw + weight_decay * w        (weights; biases: g = dL/db)
    v = momentum * v + g
    w = w - lr * v

with float32 master weights and velocities on the GPU (float64 here); after the
update the storage copy of each weight matrix (what the next forward pass reads)
is the master rounded to float32 and then to the storage type.
"""

from typing import List, Sequence, Tuple

import numpy as np

from .sparse_deepcnet import round_store


def sgd_step(W32: Sequence[np.ndarray], b: Sequence[np.ndarray], dW: Sequence[np.ndarray], db: Sequence[np.ndarray],
             vW: Sequence[np.ndarray], vb: Sequence[np.ndarray], lr: float, momentum: float, weight_decay: float,
             mode: str = "f32") -> Tuple[List[np.ndarray], ...]:
    """Returns (W32, W_storage, b, vW, vb) after one update, all in float64 arrays.

    ``mode`` names the storage type of the weight copy ("f32" or "bf16").
    """
    W_new, Ws_new, b_new, vW_new, vb_new = [], [], [], [], []
    for w, g, v in zip(W32, dW, vW):
        w = np.asarray(w, np.float64)
        vn = momentum * np.asarray(v, np.float64) + (np.asarray(g, np.float64) + weight_decay * w)
        wn = w - lr * vn
        W_new.append(wn)
        vW_new.append(vn)
        Ws_new.append(round_store(wn.astype(np.float32).astype(np.float64), mode))
    for c, g, v in zip(b, db, vb):
        vn = momentum * np.asarray(v, np.float64) + np.asarray(g, np.float64)
        b_new.append(np.asarray(c, np.float64) - lr * vn)
        vb_new.append(vn)
    return W_new, Ws_new, b_new, vW_new, vb_new
