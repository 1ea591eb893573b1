"""Seeded synthetic inputs for the outlier-aware W4A16 decode matmul.

This package only draws random inputs and writes them in the storage layout
the library consumes (bf16/fp16 bit patterns, INT4 codes packed into 32-bit
words).  It contains none of the method's arithmetic: no dequantisation, no
matrix product and no Tile-COO encoding.  Both the CPU oracle and the GPU
path read the arrays it returns.
"""

from .gen import (  # noqa: F401
    Problem,
    WORKLOADS,
    bf16_bits_from_f32,
    make_activations,
    make_dense_weight,
    make_exact_problem,
    make_problem,
    seed_for,
)
