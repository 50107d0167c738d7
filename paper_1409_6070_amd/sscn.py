"""ctypes binding of libsscn (include/sscn.h): argument marshalling only.

The functions ``sscn_*`` below carry the C names and signatures one to one.
``SparseDeepCNet`` is a convenience wrapper that allocates the caller-owned
device buffers with torch (workspace, gradients, logits) and passes raw
pointers plus torch's current HIP stream; every step of the computation runs
in the HIP kernels of the library.  If the library is not built, loading
fails with an error -- there is no fallback path.
"""

import ctypes
import os
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsscn.so")

SSCN_F32, SSCN_BF16 = 0, 1
ARCHS = ("deepcnet", "deepcnin")  # sscn_arch values 0, 1
STATUS = {
    0: "SSCN_OK",
    1: "SSCN_ERR_INVALID_ARGUMENT",
    2: "SSCN_ERR_OUT_OF_RANGE",
    3: "SSCN_ERR_DUPLICATE_SITE",
    4: "SSCN_ERR_CAPACITY",
    5: "SSCN_ERR_BAD_STATE",
    6: "SSCN_ERR_HIP",
    7: "SSCN_ERR_WORKSPACE",
}
EXPORTED = [
    "sscn_net_create", "sscn_net_destroy", "sscn_status_string", "sscn_net_num_params", "sscn_net_param_shape",
    "sscn_net_workspace_bytes", "sscn_rulebook_build", "sscn_rulebook_build_grouped", "sscn_layer_sizes", "sscn_forward", "sscn_backward",
    "sscn_forward_stage", "sscn_backward_stage", "sscn_layer_view_get", "sscn_timing_enable", "sscn_timing_collect",
    "sscn_timing_launches",
    "sscn_set_dropout", "sscn_philox4x32_10", "sscn_sgd_step", "sscn_encode_workspace_bytes", "sscn_encode_strokes",
    "sscn_encode_strokes_static",
]
KERNEL_CLASSES = ["rulebook", "gather_gemm", "wgrad", "wgrad_reduce", "pool_fwd", "pool_bwd", "head", "ground",
                  "dropout", "sgd", "conv_narrow"]


class SSCNError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.name}")


class NetDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32)
                for n in ("ell", "k", "c_in", "n_classes", "batch_max", "max_active", "dtype", "arch", "dropout")]


class LayerView(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("side", ctypes.c_int32), ("channels", ctypes.c_int32),
        ("row_stride", ctypes.c_int32), ("window", ctypes.c_int32), ("capacity", ctypes.c_int32),
        ("count", ctypes.c_void_p), ("sites", ctypes.c_void_p), ("rules", ctypes.c_void_p),
        ("rules_t", ctypes.c_void_p), ("features", ctypes.c_void_p), ("grad", ctypes.c_void_p),
        ("argmax", ctypes.c_void_p), ("gmask", ctypes.c_void_p),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libsscn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_1409_6070_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, VP, SZ = ctypes.POINTER, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
    sig = {
        "sscn_net_create": (I32, [P(NetDesc), P(VP)]),
        "sscn_net_destroy": (None, [VP]),
        "sscn_status_string": (ctypes.c_char_p, [I32]),
        "sscn_net_num_params": (I32, [VP]),
        "sscn_net_param_shape": (I32, [VP, I32, P(ctypes.c_int64), P(ctypes.c_int64)]),
        "sscn_net_workspace_bytes": (I32, [VP, P(SZ)]),
        "sscn_rulebook_build": (I32, [VP, VP, I32, I32, VP, SZ, VP]),
        "sscn_rulebook_build_grouped": (I32, [VP, VP, VP, I32, I32, VP, SZ, VP]),
        "sscn_layer_sizes": (I32, [VP, P(I32), VP]),
        "sscn_forward": (I32, [VP, VP, P(VP), P(VP), VP, VP, VP, VP]),
        "sscn_backward": (I32, [VP, P(VP), P(VP), VP, VP]),
        "sscn_forward_stage": (I32, [VP, I32, VP]),
        "sscn_backward_stage": (I32, [VP, I32, VP]),
        "sscn_layer_view_get": (I32, [VP, I32, P(LayerView)]),
        "sscn_timing_enable": (I32, [VP, ctypes.c_uint32]),
        "sscn_timing_collect": (I32, [VP, I32, P(I32), P(ctypes.c_float), VP]),
        "sscn_timing_launches": (I32, [VP, I32, P(I32), P(ctypes.c_float), I32, P(I32), VP]),
        "sscn_set_dropout": (I32, [VP, P(ctypes.c_double), I32, ctypes.c_uint64]),
        "sscn_philox4x32_10": (None, [P(ctypes.c_uint32), P(ctypes.c_uint32), P(ctypes.c_uint32)]),
        "sscn_sgd_step": (I32, [VP, P(VP), P(VP), P(VP), P(VP), P(VP), ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                VP]),
        "sscn_encode_workspace_bytes": (I32, [I32, I32, I32, P(SZ)]),
        "sscn_encode_strokes": (I32, [I32, I32, VP, I32, VP, VP, I32, I32, VP, VP, I32, P(I32), VP, SZ, VP]),
        "sscn_encode_strokes_static": (I32, [I32, I32, VP, I32, VP, VP, I32, I32, VP, VP, I32, P(I32), VP]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != 0:
        raise SSCNError(status, where)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


# ---------------------------------------------------------------------------
# the C calls, same names


def sscn_net_create(desc: NetDesc) -> int:
    h = ctypes.c_void_p()
    _check(load_library().sscn_net_create(ctypes.byref(desc), ctypes.byref(h)), "sscn_net_create")
    return h.value


def sscn_net_destroy(net: int) -> None:
    load_library().sscn_net_destroy(net)


def sscn_status_string(status: int) -> str:
    return load_library().sscn_status_string(status).decode()


def sscn_net_num_params(net: int) -> int:
    return load_library().sscn_net_num_params(net)


def sscn_net_param_shape(net: int, layer: int):
    r, c = ctypes.c_int64(), ctypes.c_int64()
    _check(load_library().sscn_net_param_shape(net, layer, ctypes.byref(r), ctypes.byref(c)), "sscn_net_param_shape")
    return r.value, c.value


def sscn_net_workspace_bytes(net: int) -> int:
    b = ctypes.c_size_t()
    _check(load_library().sscn_net_workspace_bytes(net, ctypes.byref(b)), "sscn_net_workspace_bytes")
    return b.value


def sscn_rulebook_build(net: int, d_coords: int, n: int, batch: int, d_ws: int, ws_bytes: int, stream: int) -> None:
    _check(load_library().sscn_rulebook_build(net, d_coords, n, batch, d_ws, ws_bytes, stream), "sscn_rulebook_build")


def sscn_rulebook_build_grouped(net: int, d_coords: int, d_sample_begin: int, n: int, batch: int, d_ws: int,
                                ws_bytes: int, stream: int) -> None:
    _check(load_library().sscn_rulebook_build_grouped(net, d_coords, d_sample_begin, n, batch, d_ws, ws_bytes, stream),
           "sscn_rulebook_build_grouped")


def sscn_layer_sizes(net: int, nlayers: int, stream: int) -> List[int]:
    arr = (ctypes.c_int32 * nlayers)()
    _check(load_library().sscn_layer_sizes(net, arr, stream), "sscn_layer_sizes")
    return list(arr)


def _ptr_array(ptrs: Sequence[int]):
    return (ctypes.c_void_p * len(ptrs))(*ptrs)


def sscn_forward(net, d_feats, W_ptrs, b_ptrs, d_labels, d_logits, d_loss, stream) -> None:
    _check(load_library().sscn_forward(net, d_feats, _ptr_array(W_ptrs), _ptr_array(b_ptrs), d_labels, d_logits,
                                       d_loss, stream), "sscn_forward")


def sscn_backward(net, dW_ptrs, db_ptrs, d_dfeats, stream) -> None:
    _check(load_library().sscn_backward(net, _ptr_array(dW_ptrs), _ptr_array(db_ptrs), d_dfeats, stream),
           "sscn_backward")


def sscn_forward_stage(net, stage, stream) -> None:
    _check(load_library().sscn_forward_stage(net, stage, stream), "sscn_forward_stage")


def sscn_backward_stage(net, stage, stream) -> None:
    _check(load_library().sscn_backward_stage(net, stage, stream), "sscn_backward_stage")


def sscn_layer_view_get(net, layer) -> LayerView:
    v = LayerView()
    _check(load_library().sscn_layer_view_get(net, layer, ctypes.byref(v)), "sscn_layer_view_get")
    return v


def sscn_set_dropout(net, rates: Optional[Sequence[float]], seed: int) -> None:
    rates = list(rates or [])
    arr = (ctypes.c_double * max(len(rates), 1))(*rates)
    _check(load_library().sscn_set_dropout(net, arr if rates else None, len(rates), seed & (2 ** 64 - 1)),
           "sscn_set_dropout")


def sscn_philox4x32_10(counter: Sequence[int], key: Sequence[int]) -> List[int]:
    c = (ctypes.c_uint32 * 4)(*counter)
    k = (ctypes.c_uint32 * 2)(*key)
    out = (ctypes.c_uint32 * 4)()
    load_library().sscn_philox4x32_10(c, k, out)
    return list(out)


def sscn_sgd_step(net, W32_ptrs, W_ptrs, b_ptrs, vW_ptrs, vb_ptrs, lr, momentum, weight_decay, stream) -> None:
    _check(load_library().sscn_sgd_step(net, _ptr_array(W32_ptrs), _ptr_array(W_ptrs) if W_ptrs is not None else None,
                                        _ptr_array(b_ptrs), _ptr_array(vW_ptrs), _ptr_array(vb_ptrs), lr, momentum,
                                        weight_decay, stream), "sscn_sgd_step")


def sscn_encode_workspace_bytes(N: int, batch_max: int, max_sites: int) -> int:
    out = ctypes.c_size_t()
    _check(load_library().sscn_encode_workspace_bytes(N, batch_max, max_sites, ctypes.byref(out)),
           "sscn_encode_workspace_bytes")
    return out.value


def sscn_encode_strokes(N, dtype, d_points, n_points, d_begin, d_sample, n_strokes, batch, d_coords, d_feats,
                        max_sites, d_ws, ws_bytes, stream) -> int:
    """Returns the site count; raises SSCNError (the count is in .count) on failure."""
    cnt = ctypes.c_int32(0)
    st = load_library().sscn_encode_strokes(N, dtype, d_points, n_points, d_begin, d_sample, n_strokes, batch,
                                            d_coords, d_feats, max_sites, ctypes.byref(cnt), d_ws, ws_bytes, stream)
    if st != 0:
        err = SSCNError(st, "sscn_encode_strokes")
        err.count = cnt.value
        raise err
    return cnt.value


ENCODE_STATIC_SCRATCH_BYTES = 16 << 20  # SSCN_ENCODE_STATIC_SCRATCH_BYTES


def sscn_encode_strokes_static(N, dtype, d_points, n_points, d_begin, d_sample, n_strokes, batch, d_coords,
                               d_feats, max_sites, stream) -> int:
    """sscn_encode_strokes without a workspace (the library's fixed per-GPU scratch); returns the site count."""
    cnt = ctypes.c_int32(0)
    st = load_library().sscn_encode_strokes_static(N, dtype, d_points, n_points, d_begin, d_sample, n_strokes,
                                                   batch, d_coords, d_feats, max_sites, ctypes.byref(cnt), stream)
    if st != 0:
        err = SSCNError(st, "sscn_encode_strokes_static")
        err.count = cnt.value
        raise err
    return cnt.value


def sscn_timing_enable(net, class_mask: int) -> None:
    _check(load_library().sscn_timing_enable(net, class_mask), "sscn_timing_enable")


def sscn_timing_collect(net, kernel_class: int, stream):
    n, ms = ctypes.c_int32(), ctypes.c_float()
    _check(load_library().sscn_timing_collect(net, kernel_class, ctypes.byref(n), ctypes.byref(ms), stream),
           "sscn_timing_collect")
    return n.value, ms.value


def sscn_timing_launches(net, kernel_class: int, capacity: int, stream):
    tags = (ctypes.c_int32 * max(capacity, 1))()
    ms = (ctypes.c_float * max(capacity, 1))()
    n = ctypes.c_int32()
    _check(load_library().sscn_timing_launches(net, kernel_class, tags, ms, capacity, ctypes.byref(n), stream),
           "sscn_timing_launches")
    k = min(n.value, capacity)
    return list(tags[:k]), list(ms[:k]), n.value


# ---------------------------------------------------------------------------
# convenience wrapper


class SparseDeepCNet:
    """DeepCNet(ell, k) or DeepCNiN(ell, k) on the GPU through libsscn; torch supplies memory and the stream."""

    def __init__(self, ell: int, k: int, c_in: int, n_classes: int, batch_max: int, max_active: int,
                 dtype: str = "bf16", device: str = "cuda", arch: str = "deepcnet", dropout: bool = False):
        if dtype not in ("f32", "bf16"):
            raise ValueError(dtype)
        if arch not in ARCHS:
            raise ValueError(arch)
        self.ell, self.k, self.c_in, self.n_classes = ell, k, c_in, n_classes
        self.dtype = dtype
        self.arch = arch
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.device = torch.device(device)
        self.nlayers = (3 * ell + 3) if arch == "deepcnin" else (2 * ell + 2)
        desc = NetDesc(ell, k, c_in, n_classes, batch_max, max_active, SSCN_BF16 if dtype == "bf16" else SSCN_F32,
                       ARCHS.index(arch), int(bool(dropout)))
        self.handle = sscn_net_create(desc)
        self.ws_bytes = sscn_net_workspace_bytes(self.handle)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.param_shapes = [sscn_net_param_shape(self.handle, i) for i in range(sscn_net_num_params(self.handle))]
        self.dW = [torch.empty(r, c, dtype=torch.float32, device=self.device) for r, c in self.param_shapes]
        self.db = [torch.empty(c, dtype=torch.float32, device=self.device) for _, c in self.param_shapes]
        self.loss = torch.empty(1, dtype=torch.float32, device=self.device)
        self.logits = None
        self._keep = []

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                sscn_net_destroy(h)
            except Exception:
                pass
            self.handle = None

    # -- calls ---------------------------------------------------------------
    def rulebook_build(self, coords: torch.Tensor, batch: int, sample_begin: Optional[torch.Tensor] = None) -> None:
        """coords [n][3] int32 (b, y, x); with sample_begin (int32 [batch + 1] on the device) the sites are
        grouped by sample and the grouped build is used."""
        assert coords.dtype == torch.int32 and coords.is_contiguous() and coords.device.type == "cuda"
        self.batch = batch
        self.n = int(coords.shape[0])
        self._coords = coords
        if sample_begin is None:
            sscn_rulebook_build(self.handle, coords.data_ptr() if self.n else None, self.n, batch, self.ws.data_ptr(),
                                self.ws_bytes, _stream())
        else:
            assert sample_begin.dtype == torch.int32 and sample_begin.is_contiguous()
            assert sample_begin.device.type == "cuda" and int(sample_begin.numel()) == batch + 1
            self._sample_begin = sample_begin
            sscn_rulebook_build_grouped(self.handle, coords.data_ptr() if self.n else None, sample_begin.data_ptr(),
                                        self.n, batch, self.ws.data_ptr(), self.ws_bytes, _stream())

    def set_dropout(self, rates: Optional[Sequence[float]], seed: int = 0) -> None:
        """Dropout rates per level (ell + 2: each convolution that is not 1x1, then the softmax
        input) for the following training passes; None switches it off."""
        sscn_set_dropout(self.handle, rates, seed)

    def layer_sizes(self) -> List[int]:
        return sscn_layer_sizes(self.handle, self.nlayers, _stream())

    def forward(self, feats: torch.Tensor, Ws: Sequence[torch.Tensor], bs: Sequence[torch.Tensor],
                labels: Optional[torch.Tensor]):
        """Forward pass; ``labels=None`` is inference (logits only, no loss, no backward)."""
        assert feats.dtype == self.tdtype and feats.is_contiguous()
        assert labels is None or labels.dtype == torch.int32
        for W in Ws:
            assert W.dtype == self.tdtype and W.is_contiguous()
        for b in bs:
            assert b.dtype == torch.float32 and b.is_contiguous()
        if self.logits is None or self.logits.shape[0] != self.batch:
            self.logits = torch.empty(self.batch, self.n_classes, dtype=torch.float32, device=self.device)
        self._keep = [feats, list(Ws), list(bs), labels]
        sscn_forward(self.handle, feats.data_ptr() if feats.numel() else None, [W.data_ptr() for W in Ws],
                     [b.data_ptr() for b in bs], labels.data_ptr() if labels is not None else None,
                     self.logits.data_ptr(), self.loss.data_ptr() if labels is not None else None, _stream())
        return self.logits, (self.loss if labels is not None else None)

    def backward(self, want_dfeats: bool = False):
        dfeats = None
        if want_dfeats:
            dfeats = torch.empty(self.n, self.c_in, dtype=self.tdtype, device=self.device)
        sscn_backward(self.handle, [t.data_ptr() for t in self.dW], [t.data_ptr() for t in self.db],
                      dfeats.data_ptr() if (dfeats is not None and self.n) else None, _stream())
        return self.dW, self.db, dfeats

    def sgd_step(self, W32: Sequence[torch.Tensor], W: Optional[Sequence[torch.Tensor]], bs: Sequence[torch.Tensor],
                 vW: Sequence[torch.Tensor], vb: Sequence[torch.Tensor], lr: float, momentum: float = 0.0,
                 weight_decay: float = 0.0) -> None:
        """SGD update from the last backward's gradients: fp32 masters W32 (and biases, velocities)
        in place, then the storage copies W the next forward reads."""
        for t in list(W32) + list(bs) + list(vW) + list(vb):
            assert t.dtype == torch.float32 and t.is_contiguous()
        if W is not None:
            for t in W:
                assert t.dtype == self.tdtype and t.is_contiguous()
        sscn_sgd_step(self.handle, [t.data_ptr() for t in W32], [t.data_ptr() for t in W] if W is not None else None,
                      [t.data_ptr() for t in bs], [t.data_ptr() for t in vW], [t.data_ptr() for t in vb], lr,
                      momentum, weight_decay, _stream())

    def timing(self, classes: Sequence[str]) -> None:
        """Bracket launches of the named kernel classes with HIP events (empty: off)."""
        mask = 0
        for c in classes:
            mask |= 1 << KERNEL_CLASSES.index(c)
        sscn_timing_enable(self.handle, mask)

    def timing_collect(self, kernel_class: str):
        """(launches, total milliseconds) of a class since the last collect."""
        return sscn_timing_collect(self.handle, KERNEL_CLASSES.index(kernel_class), _stream())

    def timing_launches(self, kernel_class: str, capacity: int = 65536):
        """Per-launch records of a class since the last collect: [(tag, milliseconds)], launch order."""
        tags, ms, _ = sscn_timing_launches(self.handle, KERNEL_CLASSES.index(kernel_class), capacity, _stream())
        return list(zip(tags, ms))

    def forward_stage(self, stage: int) -> None:
        sscn_forward_stage(self.handle, stage, _stream())

    def backward_stage(self, stage: int) -> None:
        sscn_backward_stage(self.handle, stage, _stream())

    # -- inspection ----------------------------------------------------------
    def _slice(self, ptr: int, nbytes: int, dtype) -> torch.Tensor:
        off = ptr - self.ws.data_ptr()
        assert 0 <= off and off + nbytes <= self.ws_bytes
        return self.ws[off: off + nbytes].view(dtype)

    def layer_view(self, layer: int, n: Optional[int] = None) -> dict:
        """Tensors viewing layer `layer` in the workspace, trimmed to n active rows (+ the ground row)."""
        v = sscn_layer_view_get(self.handle, layer)
        if n is None:
            n = self.layer_sizes()[layer]
        es = 2 if self.dtype == "bf16" else 4
        out = dict(kind=v.kind, side=v.side, channels=v.channels, row_stride=v.row_stride, window=v.window,
                   capacity=v.capacity, n=n)
        rs = v.row_stride
        out["features"] = self._slice(v.features, (n + 1) * rs * es, self.tdtype).view(n + 1, rs)
        out["grad"] = self._slice(v.grad, (n + 1) * rs * es, self.tdtype).view(n + 1, rs)
        out["sites"] = self._slice(v.sites, max(n, 0) * 4, torch.int32) if n else torch.zeros(0, dtype=torch.int32)
        if layer > 0:
            A = v.window
            out["rules"] = self._slice(v.rules, (n + 1) * A * 4, torch.int32).view(n + 1, A)
            if v.argmax:
                out["argmax"] = self._slice(v.argmax, (n + 1) * rs, torch.uint8).view(n + 1, rs)
            if v.gmask:
                out["gmask"] = self._slice(v.gmask, (n + 1) * 2, torch.int16)
        return out

    def rules_t(self, layer: int, n_below: int) -> torch.Tensor:
        v = sscn_layer_view_get(self.handle, layer)
        if v.kind == 1:
            return self._slice(v.rules_t, (n_below + 1) * v.window * 4, torch.int32).view(n_below + 1, v.window)
        return self._slice(v.rules_t, (n_below + 1) * 4, torch.int32)


class StrokeEncoder:
    """Pen paths -> sparse input with 9 features per site (Section 2.4) on the GPU, through
    sscn_encode_strokes; holds the scratch and output buffers for batches within its limits."""

    def __init__(self, N: int, batch_max: int, max_sites: int, dtype: str = "bf16", device: str = "cuda"):
        if dtype not in ("f32", "bf16"):
            raise ValueError(dtype)
        self.N, self.batch_max, self.max_sites, self.dtype = N, batch_max, max_sites, dtype
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.device = torch.device(device)
        self.ws_bytes = sscn_encode_workspace_bytes(N, batch_max, max_sites)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.coords = torch.empty(max(max_sites, 1), 3, dtype=torch.int32, device=self.device)
        self.feats = torch.empty(max(max_sites, 1), 9, dtype=self.tdtype, device=self.device)

    def encode(self, points: torch.Tensor, stroke_begin: torch.Tensor, stroke_sample: torch.Tensor, batch: int):
        """(coords [n, 3], feats [n, 9]) views of the encoder's buffers (valid until the next call)."""
        for t in (points, stroke_begin, stroke_sample):
            assert t.dtype == torch.int32 and t.is_contiguous() and t.device.type == "cuda"
        if batch > self.batch_max:
            raise SSCNError(4, "StrokeEncoder.encode")
        n_strokes = int(stroke_sample.shape[0])
        n = sscn_encode_strokes(self.N, SSCN_BF16 if self.dtype == "bf16" else SSCN_F32,
                                points.data_ptr() if points.numel() else None, int(points.shape[0]),
                                stroke_begin.data_ptr(), stroke_sample.data_ptr() if n_strokes else None, n_strokes,
                                batch, self.coords.data_ptr(), self.feats.data_ptr(), self.max_sites,
                                self.ws.data_ptr(), self.ws_bytes, _stream())
        return self.coords[:n], self.feats[:n]
