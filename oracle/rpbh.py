"""RPBH transform (test infrastructure only).

Sec. 4.4, Eq. (9): Pi_d = blkdiag(H_h D_1, ..., H_h D_{d/h}) P_pi.  The
permutation acts first (gather), then the Rademacher signs, then a
Walsh-Hadamard transform on each block of h consecutive positions.  The
supplement's proof setup fixes the normalisation (H_h)_{li} = +-1/sqrt(h), so
Pi_d is orthogonal.  Reading taken for the ordering of H_h: the Sylvester
(natural) order, H[r][c] = (-1)^popcount(r & c) / sqrt(h).

Rows are transformed independently (Sec. 4.3: applied row-wise as x Pi^T).
"""

import numpy as np

from .plan import Plan


def sylvester_hadamard(h: int) -> np.ndarray:
    """Unnormalised Sylvester matrix of order h as a Kronecker power of [[1,1],[1,-1]] (int64)."""
    if h < 1 or (h & (h - 1)) != 0:
        raise ValueError("h must be a power of two")
    H = np.ones((1, 1), dtype=np.int64)
    base = np.array([[1, 1], [1, -1]], dtype=np.int64)
    while H.shape[0] < h:
        H = np.kron(base, H)
    return H


def fwht_blocks(Y: np.ndarray, h: int) -> np.ndarray:
    """Unnormalised Walsh-Hadamard transform of every length-h block of each row.

    log2(h) butterfly passes: at stride s, positions i and i+s of each 2s-group
    become (a + b, a - b).  This equals multiplication by sylvester_hadamard(h).
    """
    M, d = Y.shape
    k = d // h
    Z = np.array(Y, dtype=np.float64).reshape(M, k, h)
    s = 1
    while s < h:
        Z = Z.reshape(M, k, h // (2 * s), 2, s)
        a = Z[:, :, :, 0, :]
        b = Z[:, :, :, 1, :]
        Z = np.stack([a + b, a - b], axis=3)
        s *= 2
    return Z.reshape(M, d)


def rpbh_forward(X: np.ndarray, plan: Plan) -> np.ndarray:
    """x' = Pi_d x for every row of X (rows are tokens), fp64."""
    X = np.asarray(X, dtype=np.float64)
    Y = X[:, plan.perm] * plan.sign[None, :]       # gather by pi, then D
    return fwht_blocks(Y, plan.h) / np.sqrt(plan.h)  # H_h / sqrt(h) per block


def rpbh_inverse(Z: np.ndarray, plan: Plan) -> np.ndarray:
    """x = Pi_d^T x': the normalised Sylvester matrix is its own inverse, then D, then scatter."""
    Z = np.asarray(Z, dtype=np.float64)
    Y = fwht_blocks(Z, plan.h) / np.sqrt(plan.h)
    Y = Y * plan.sign[None, :]
    X = np.empty_like(Y)
    X[:, plan.perm] = Y
    return X
