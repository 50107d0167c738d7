"""Seeded synthetic inputs for the sparse DeepCNet hot path.

This module only draws random numbers and rasterises pen strokes for the picture
inputs (the histogram encoding of raw pen paths is a method step and lives on
both sides, not here): it holds none of the network's arithmetic, so the CPU
oracle and the HIP path can both take their inputs from it without sharing any
of the method.

The paper's workloads (online handwriting, MNIST, CIFAR; Sections 2.4, 2.5 and
3) are datasets that are not available here.  The generators below stand in for
them with the same input representation: a sparse set of active sites on an
N x N grid, N = 3 * 2**ell (Section 2.1), each carrying M features, with zero
background (Sections 1 and 2.5).
"""

from .configs import CONFIGS, WorkloadConfig, get_config
from .synth import (
    Batch,
    circle_sites,
    he_params,
    make_batch,
    make_batches,
    make_paths,
    patch_batch,
    Paths,
    random_labels,
    stroke_batch,
    stroke_paths,
)

__all__ = [
    "CONFIGS",
    "WorkloadConfig",
    "get_config",
    "Batch",
    "circle_sites",
    "he_params",
    "make_batch",
    "make_batches",
    "make_paths",
    "patch_batch",
    "Paths",
    "stroke_paths",
    "random_labels",
    "stroke_batch",
]
