"""Seeded synthetic inputs for the sparse DNN forward pass.

This package only draws random matrices.  It holds none of the method's
arithmetic (no products, no bias, no nonlinearity), so both the CPU oracle and
the GPU path may use it without sharing any computation.
"""

from .gen import (  # noqa: F401
    Layer,
    Problem,
    SEED_ROOT,
    CONFIG_NAMES,
    make_config,
    paper_grid,
    PAPER_GRID_SIZES,
    PAPER_GRID_INV_SPARSITY,
    tiny_random,
    integer_shadow,
    dense_to_csr,
    csr_rows,
)
