"""The synthetic workloads the hot path is tested and measured on.

Each names a DeepCNet(ell, k) (Section 2.1), an input feature count M, a batch,
a class count for the softmax head, a storage dtype, and an input generator
with its parameters.  The generators stand in for the paper's datasets:

* pen strokes on a centred box stand in for the online-handwriting sets of
  Sections 2.4 and 3.1 (Pendigits, UJIpenchars, Assamese, CASIA; the 3755-class
  heads follow CASIA-OLHWDB1.1 in Section 3.1.3);
* a dense RGB patch centred in a 96 x 96 grid stands in for CIFAR (Section 2.5,
  Section 3.3);
* the DeepCNet(5,50) pen strokes also feed a DeepCNiN(5,50) (Section 2.2);
* grey-level digit strokes of about 150 pixels in the middle of a 96 x 96 grid
  stand in for MNIST (Section 2.5), on the small network the paper times at test
  time (DeepCNet(5,10), Section 3.2): a forward-only ("infer") workload;
* the DeepCNet(5,50) pen strokes once more with dropout per level (Section 2.1);
* raw pen paths for DeepCNet(4,20), encoded by the method itself into 9 features
  per site (picture plus 8-direction histograms, Section 2.4), for a whole
  training step with the SGD update.
"""

from dataclasses import dataclass, field
from typing import Dict, Tuple


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    ell: int
    k: int
    c_in: int
    batch: int
    n_classes: int
    dtypes: Tuple[str, ...]
    generator: str  # "strokes", "patch", "digits" or "paths" (raw pen paths, encoded by the method)
    gen_args: Dict = field(default_factory=dict)
    seed: int = 0  # input seed; weights use 100 + seed, labels 200 + seed
    mode: str = "train"  # "train": build + forward + backward; "infer": build + forward (logits)
    arch: str = "deepcnet"  # or "deepcnin" (Section 2.2)
    dropout: Tuple[float, ...] = ()  # rates per level (ell + 2, Section 2.1); () for none
    sgd: Tuple[float, ...] = ()  # (lr, momentum, weight decay): a training step ends with the update

    @property
    def dropout_seed(self) -> int:
        return 300 + self.seed

    @property
    def grid(self) -> int:
        return 3 * 2 ** self.ell

    @property
    def weight_seed(self) -> int:
        return 100 + self.seed

    @property
    def label_seed(self) -> int:
        return 200 + self.seed


CONFIGS = [
    # DeepCNet(4,20), 48x48 grid, 1-3 strokes of 10-30 points, step sd 2 px,
    # 32x32 drawing box, binary pen feature.
    WorkloadConfig(
        name="deepcnet4_20_strokes_b8",
        ell=4, k=20, c_in=1, batch=8, n_classes=10, dtypes=("f32",),
        generator="strokes",
        gen_args=dict(strokes=(1, 3), points=(10, 30), box=32, sigma=2.0, features="ones"),
        seed=0,
    ),
    # DeepCNet(5,50), 96x96 grid, 1-20 strokes of 10-60 points in a 64x64 box.
    WorkloadConfig(
        name="deepcnet5_50_strokes_b100",
        ell=5, k=50, c_in=1, batch=100, n_classes=3755, dtypes=("f32", "bf16"),
        generator="strokes",
        gen_args=dict(strokes=(1, 20), points=(10, 60), box=64, sigma=2.0, features="ones"),
        seed=1,
    ),
    # As above with 8 N(0,1) features per pen pixel.
    WorkloadConfig(
        name="deepcnet5_50_strokes_m8_b100",
        ell=5, k=50, c_in=8, batch=100, n_classes=3755, dtypes=("bf16",),
        generator="strokes",
        gen_args=dict(strokes=(1, 20), points=(10, 60), box=64, sigma=2.0, features="normal"),
        seed=2,
    ),
    # DeepCNet(5,100), 96x96 grid, a dense 32x32 RGB patch (U[0,1)) at a random
    # offset inside the centred 40x40 region.
    WorkloadConfig(
        name="deepcnet5_100_rgbpatch_b128",
        ell=5, k=100, c_in=3, batch=128, n_classes=10, dtypes=("bf16",),
        generator="patch",
        gen_args=dict(patch=32, region=40),
        seed=3,
    ),
    # DeepCNet(6,100), 192x192 grid, 1-30 strokes of 10-120 points, step sd 1 px,
    # 128x128 box.
    WorkloadConfig(
        name="deepcnet6_100_strokes_b64",
        ell=6, k=100, c_in=1, batch=64, n_classes=3755, dtypes=("bf16",),
        generator="strokes",
        gen_args=dict(strokes=(1, 30), points=(10, 120), box=128, sigma=1.0, features="ones"),
        seed=4,
    ),
    # DeepCNet(5,10) classifying digit pictures: 28x28 frame (about 150 grey-level
    # pixels) in the middle of the 96x96 grid, 10 classes, forward only.
    WorkloadConfig(
        name="deepcnet5_10_digits_b1000",
        ell=5, k=10, c_in=1, batch=1000, n_classes=10, dtypes=("f32", "bf16"),
        generator="digits",
        gen_args=dict(strokes=(2, 4), points=(10, 18), box=20, sigma=2.5, brush=2),
        seed=5, mode="infer",
    ),
    # DeepCNiN(5,50) (1x1 layers after every pool and the last convolution, leaky
    # rectifier) on the DeepCNet(5,50) pen-stroke inputs.
    WorkloadConfig(
        name="deepcnin5_50_strokes_b100",
        ell=5, k=50, c_in=1, batch=100, n_classes=3755, dtypes=("bf16",),
        generator="strokes",
        gen_args=dict(strokes=(1, 20), points=(10, 60), box=64, sigma=2.0, features="ones"),
        seed=6, arch="deepcnin",
    ),
    # DeepCNet(5,50) pen strokes trained with dropout per level (Section 2.1): none
    # on the three lowest convolutions, one half on the three above them and on the
    # softmax layer's input -- the profile of the paper's dropout DeepCNet(5,60)
    # (Section 3.2).
    WorkloadConfig(
        name="deepcnet5_50_strokes_dropout_b100",
        ell=5, k=50, c_in=1, batch=100, n_classes=3755, dtypes=("bf16",),
        generator="strokes",
        gen_args=dict(strokes=(1, 20), points=(10, 60), box=64, sigma=2.0, features="ones"),
        seed=7, dropout=(0.0, 0.0, 0.0, 0.5, 0.5, 0.5, 0.5),
    ),
    # A whole training step on DeepCNet(4,20) (the network of Section 3.1.2's M = 1 / M = 9
    # comparison): raw pen paths (1-3 strokes of 10-30 points, step sd 2 px, 32x32 box in
    # 48x48), encoded on the device into the picture plus 8-direction histograms (M = 9,
    # Section 2.4), then build + forward + backward + SGD update.
    WorkloadConfig(
        name="deepcnet4_20_paths_m9_b100",
        ell=4, k=20, c_in=9, batch=100, n_classes=10, dtypes=("f32", "bf16"),
        generator="paths",
        gen_args=dict(strokes=(1, 3), points=(10, 30), box=32, sigma=2.0),
        seed=8, sgd=(0.01, 0.9, 1e-4),
    ),
]

_BY_NAME = {c.name: c for c in CONFIGS}


def get_config(name: str) -> WorkloadConfig:
    return _BY_NAME[name]
