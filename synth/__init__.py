"""Seeded synthetic inputs shared by the CPU oracle, the tests and the benchmark.

This package holds *inputs only*: the fixed pseudo-random tables of the RSLM
codec (256 signs, a 128-element permutation, the Lloyd-Max codebooks stored
as data) and generators of synthetic embedding collections.  It contains none
of the codec's arithmetic (no rotation, quantisation, scaling or scoring), so
both the oracle under ``oracle/`` and the HIP library consume the very same
bytes without sharing any computation.
"""

from .tables import sign_table, permutation_table, codebook, codebook_shape
from .data import (
    gmix_means, gmix, aniso_params, aniso, aniso_torch, aniso_torch_block, TORCH_BLOCK,
    queries_like, random_rows,
)

__all__ = [
    "sign_table", "permutation_table", "codebook", "codebook_shape",
    "gmix_means", "gmix", "aniso_params", "aniso", "aniso_torch", "aniso_torch_block",
    "TORCH_BLOCK", "queries_like", "random_rows",
]
