"""Normalize, encode and pack (test infrastructure only).

Activations, Sec. 4.3, Eqs. (7)-(8) and Alg. 1 online stage:
    x' = Pi_d x,  s = ||x'||_2,  x~' = x' / (s + eps),  x^' = s * Q_b(x~')
Weights, Sec. 4.2, Eqs. (4)-(6) and Alg. 1 offline stage:
    w'_i = Pi_d w_i,  r'_i = ||w'_i||_2,  w~'_i = w'_i / r'_i,  W^' = diag(r') Q_b(W~'),
    with r' stored in BF16.
Nearest-centroid map, Eq. (3), applied coordinate-wise.

Readings taken where the paper is silent:
  * eps = 1e-10 divides (s + eps) and the rescale uses s; the weight rows use
    the same guard (Eq. (5) has none), so a zero row gives r' = 0.
  * s is kept in fp32 by the kernels, r' is rounded to BF16 round-to-nearest-even.
  * At an exact tie between two levels the upper code is taken:
    code = #{j : tau_j <= u}.  Codes index the ascending levels (0 = most negative).
  * Packing is an LSB-first bit stream per row: code k occupies bits
    [k*b, k*b + b) of the row, so a row of K codes is K*b/8 bytes.
  * Stored codes are sign-magnitude labels of the level index (the paper fixes no
    storage labels): index c >= 2^(b-1) (a positive level) is stored as c - 2^(b-1),
    index c < 2^(b-1) as 2^b - 1 - c.  The label's top bit is the sign of the level and
    its low bits rank |level|; to_labels / from_labels convert.
"""

import numpy as np

from .rpbh import rpbh_forward


def bf16_round(x) -> np.ndarray:
    """Round fp64 values to the nearest BF16 value (8 significant bits), ties to even."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                 # x = m * 2^e, |m| in [0.5, 1)
    return np.ldexp(np.round(m * 256.0), e - 8)


def bf16_bits(x) -> np.ndarray:
    """BF16 bit pattern (uint16) of values that are already BF16-representable."""
    return (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def fp16_round(x) -> np.ndarray:
    """Round to IEEE half precision (library conversion, round-to-nearest-even), back to fp64."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def normalize_rows(Z: np.ndarray, eps: float):
    """s = ||z||_2 per row and u = z / (s + eps)  (Eq. (7))."""
    s = np.sqrt(np.sum(Z * Z, axis=1))
    return s, Z / (s + eps)[:, None]


def encode(U: np.ndarray, thresholds: np.ndarray) -> np.ndarray:
    """Nearest centroid of Eq. (3) through the midpoint thresholds: code = #{j : tau_j <= u}."""
    return np.searchsorted(thresholds, U, side="right").astype(np.int64)


def near_tie_mask(U: np.ndarray, thresholds: np.ndarray, band: float) -> np.ndarray:
    """True where a coordinate lies within `band` of some decision threshold.

    The thresholds are sorted, so the nearest one is a neighbour of the insertion point."""
    U = np.asarray(U, dtype=np.float64)
    t = np.asarray(thresholds, dtype=np.float64)
    idx = np.searchsorted(t, U)
    lo = np.abs(U - t[np.clip(idx - 1, 0, len(t) - 1)])
    hi = np.abs(U - t[np.clip(idx, 0, len(t) - 1)])
    return np.minimum(lo, hi) <= band


def nearest_threshold(U: np.ndarray, thresholds: np.ndarray) -> np.ndarray:
    """Index j of the decision threshold nearest to each coordinate.

    Threshold tau_j is the midpoint of levels j and j+1 (Eq. (3) with the midpoint condition of
    Lloyd-Max), so at u = tau_j exactly the argmin of Eq. (3) is the pair {j, j+1}: those are the
    only two codes a nearest-centroid map may return for a coordinate within rounding of tau_j."""
    U = np.asarray(U, dtype=np.float64)
    t = np.asarray(thresholds, dtype=np.float64)
    idx = np.searchsorted(t, U)
    lo = np.clip(idx - 1, 0, len(t) - 1)
    hi = np.clip(idx, 0, len(t) - 1)
    return np.where(np.abs(U - t[lo]) <= np.abs(U - t[hi]), lo, hi)


def to_labels(codes, bits: int) -> np.ndarray:
    """Level indices (0 = most negative level) -> stored sign-magnitude labels."""
    c = np.asarray(codes, dtype=np.int64)
    half = 1 << (bits - 1)
    return np.where(c >= half, c - half, (2 * half - 1) - c)


def from_labels(labels, bits: int) -> np.ndarray:
    """Stored sign-magnitude labels -> level indices (the inverse of to_labels)."""
    lab = np.asarray(labels, dtype=np.int64)
    half = 1 << (bits - 1)
    return np.where(lab < half, lab + half, (2 * half - 1) - lab)


def decode_levels(codes: np.ndarray, levels: np.ndarray) -> np.ndarray:
    return np.asarray(levels)[codes]


def pack_codes(codes: np.ndarray, bits: int) -> np.ndarray:
    """LSB-first bit stream per row: bit t of code k goes to stream bit k*bits + t."""
    codes = np.asarray(codes, dtype=np.int64)
    M, K = codes.shape
    if (K * bits) % 8:
        raise ValueError("K*bits must be a whole number of bytes")
    stream = ((codes[:, :, None] >> np.arange(bits)[None, None, :]) & 1).astype(np.uint8)
    return np.packbits(stream.reshape(M, K * bits), axis=1, bitorder="little")


def unpack_codes(packed: np.ndarray, bits: int, K: int) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.uint8)
    M = packed.shape[0]
    stream = np.unpackbits(packed, axis=1, bitorder="little")[:, :K * bits].reshape(M, K, bits)
    return np.sum(stream.astype(np.int64) << np.arange(bits)[None, None, :], axis=2)


def quantize_act(X: np.ndarray, plan, cb, eps: float = 1e-10):
    """Online activation quantization (Alg. 1 online stage; Eqs. (7)-(8)).

    Returns (codes int64 [M,K], s fp64 [M], u fp64 [M,K]) where u is the
    normalized rotated coordinate the thresholds are compared against.
    """
    Z = rpbh_forward(X, plan)
    s, U = normalize_rows(Z, eps)
    return encode(U, cb.thresholds), s, U


def quantize_weights(W: np.ndarray, plan, cb, eps: float = 1e-10):
    """Offline weight quantization (Alg. 1 offline stage; Eqs. (4)-(6)).

    Returns (codes int64 [N,K], r' as BF16 values in fp64 [N], u fp64 [N,K]).
    Codes use the unrounded norm; only the stored magnitude is rounded to BF16.
    """
    Z = rpbh_forward(W, plan)
    r, U = normalize_rows(Z, eps)
    return encode(U, cb.thresholds), bf16_round(r), U
