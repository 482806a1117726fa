"""Oracle for the TCU Johnson-Lindenstrauss transform -- TEST INFRASTRUCTURE ONLY.

Section 3 (Lemma 3) of Ahle & Silvestri defines the dimensionality reduction
as one matrix, the product of Kronecker factors

    M = (I_{r_l} (x) A_l) ... (I_{r_2} (x) A_2) (I_{r_1} (x) A_1),

where A_i is k_i x c_i, I_r the r x r identity, and the sizes chain as
d = r_1 c_1,  r_i k_i = r_{i+1} c_{i+1},  r_l k_l = k (the reduced dimension).
The oracle is that definition written out in float64: it builds M densely
with numpy's Kronecker product and matrix product and returns X M^T for a
batch of rows X (n x d).  No blocking, no reshaping: a reader can check it
against the lemma by eye.
"""
from __future__ import annotations

import numpy as np


def check_chain(d: int, shapes) -> int:
    """Validates the size chain of Lemma 3 for (k_i, c_i, r_i) per level and
    returns the output dimension r_l k_l."""
    shapes = [tuple(int(v) for v in s) for s in shapes]
    if not shapes:
        raise ValueError("at least one level")
    length = d
    for (k, c, r) in shapes:
        if k < 1 or c < 1 or r < 1:
            raise ValueError(f"level sizes must be positive: {(k, c, r)}")
        if r * c != length:
            raise ValueError(f"r * c = {r * c} does not match the input length {length}")
        length = r * k
    return length


def dense_matrix(d: int, shapes, As) -> np.ndarray:
    """M = (I_{r_l} (x) A_l) ... (I_{r_1} (x) A_1) as a dense float64 matrix."""
    check_chain(d, shapes)
    M = np.eye(d)
    for (k, c, r), A in zip(shapes, As):
        A = np.asarray(A, dtype=np.float64)
        if A.shape != (k, c):
            raise ValueError(f"A has shape {A.shape}, expected {(k, c)}")
        M = np.kron(np.eye(r), A) @ M
    return M


def transform(X: np.ndarray, shapes, As) -> np.ndarray:
    """The reduced rows: (M x)^T for every row x of X (n x d, float64 values)."""
    X = np.asarray(X, dtype=np.float64)
    M = dense_matrix(X.shape[1], shapes, As)
    return X @ M.T


def abs_bound(X: np.ndarray, shapes, As) -> np.ndarray:
    """|M| |x| per row with every factor replaced by its absolute value (the
    scale of the rounding-error bound of any evaluation order)."""
    X = np.abs(np.asarray(X, dtype=np.float64))
    M = dense_matrix(X.shape[1], shapes, [np.abs(np.asarray(A, np.float64)) for A in As])
    return X @ M.T
