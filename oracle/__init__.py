"""CPU oracle for the spatially-sparse DeepCNet forward and backward pass.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything under ``oracle/``; only
the tests, the smoke check and the benchmark's CPU-baseline leg use it.

The oracle is plain NumPy in float64.  It follows the paper's own data
structures (Section 2.3): for every layer a feature matrix (row 0 the ground
state, one row per active site) and a pointer matrix over the layer's spatial
grid.  See ``sparse_deepcnet`` for the per-function citations.
"""

from .sparse_deepcnet import (
    OracleInputError,
    SparseDeepCNet,
    round_bf16,
    round_store,
    stage_plan,
)

__all__ = ["OracleInputError", "SparseDeepCNet", "round_bf16", "round_store", "stage_plan"]
