"""Seeded synthetic sparse matrices shaped like the paper's SpGEMM workloads.

This package only produces inputs. It holds none of the product's
arithmetic, so both the CPU oracle and the GPU library can be fed from it
without sharing any code with each other.
"""
from .csr import CSR
from .generators import (
    CONFIGS,
    MATRICES,
    config,
    matrix,
    er,
    er_rect,
    laplacian2d,
    rmat,
    arrowhead,
    identity,
    permutation,
    diagonal,
    random_sparse,
    shuffled_copy,
    sparse_vector,
    transpose,
)

__all__ = [
    "CSR",
    "CONFIGS",
    "MATRICES",
    "config",
    "matrix",
    "er",
    "er_rect",
    "laplacian2d",
    "rmat",
    "arrowhead",
    "identity",
    "permutation",
    "diagonal",
    "random_sparse",
    "shuffled_copy",
    "sparse_vector",
    "transpose",
]
