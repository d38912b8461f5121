"""fp64 oracle of the sparse input layer of section 2.2 -- TEST INFRASTRUCTURE ONLY.

A K-sparse input x (indices u, values v; index -1 marks an empty slot, repeated
indices add their values) is the dense D_in-vector it represents; the layer's
forward pass is a = W1^T x and its update W1 <- W1 - eta x grad_a^T, both written
here with the dense matrix X (one row per example) from the definition.  Shares
nothing with the HIP path.
"""
from __future__ import annotations

import numpy as np

from .dense import dense_targets

F64 = np.float64


def input_matrix(D_in: int, idx, val) -> np.ndarray:
    """The m x D_in dense inputs (the transpose of the dense targets' construction)."""
    return dense_targets(D_in, idx, val).T


def input_forward(W1, idx, val) -> np.ndarray:
    """A = X W1 (m x d): row j is W1^T x_j."""
    W1 = np.asarray(W1, dtype=F64)
    return input_matrix(W1.shape[0], idx, val) @ W1


def input_update(W1, idx, val, grad_A, lr) -> np.ndarray:
    """W1 - eta X^T grad_A: the sum over the minibatch of the rank-one updates x grad_a^T."""
    W1 = np.asarray(W1, dtype=F64)
    X = input_matrix(W1.shape[0], idx, val)
    return W1 - F64(lr) * (X.T @ np.asarray(grad_A, dtype=F64))
