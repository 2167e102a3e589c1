"""Quantized linear layer on codes (test infrastructure only).

Sec. 4.3: weights absorb Pi_d^T and activations apply Pi_d, so
W' x' = W Pi^T Pi x = W x and the layer computes W^' x^' with no inverse
rotation.  With x^'_n = s_n * L_a[code_x[n]] (Eq. (8)) and
w^'_i = r'_i * L_w[code_w[i]] (Eq. (6)), and the tokens as rows of X:

    Y[n, i] = s_n * r'_i * sum_k L_a[code_x[n, k]] * L_w[code_w[i, k]]

computed here in fp64 with one library matmul.
"""

import numpy as np


def qlinear(codes_x, s, levels_a, codes_w, r, levels_w) -> np.ndarray:
    """Y = diag(s) (L_a[codes_x]) (L_w[codes_w])^T diag(r'), fp64."""
    A = np.asarray(levels_a, dtype=np.float64)[np.asarray(codes_x)]
    B = np.asarray(levels_w, dtype=np.float64)[np.asarray(codes_w)]
    return (np.asarray(s, dtype=np.float64)[:, None] * (A @ B.T)) * np.asarray(r, dtype=np.float64)[None, :]


def qlinear_dense_reference(X, W) -> np.ndarray:
    """The unquantized layer Y = X W^T (Eq. (1), tokens as rows), fp64."""
    return np.asarray(X, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def layer_epilogue(Y, bias=None, gelu: bool = False, out_bf16: bool = False) -> np.ndarray:
    """The rest of a DiT linear after the contraction: + bias, then GELU x*Phi(x) with the exact
    error function, then (optionally) rounding to BF16 as the next layer's input, all in fp64."""
    from scipy.special import erf
    from .quantize import bf16_round
    Y = np.asarray(Y, dtype=np.float64)
    if bias is not None:
        Y = Y + np.asarray(bias, dtype=np.float64)[None, :]
    if gelu:
        Y = 0.5 * Y * (1.0 + erf(Y / np.sqrt(2.0)))
    return bf16_round(Y) if out_bf16 else Y
