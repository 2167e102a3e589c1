"""Lloyd-Max codebook on f_d (test infrastructure only).

Sec. 3.2 (Eq. (3) and the text around it) and Sec. 4.5: for every input
dimension d and bit-width b the codebook C^(d,b) is the set of 2^b MSE-optimal
centroids for the density f_d of Eq. (2); it carries no scale or zero-point.
Lloyd (1982) and Max (1960), both cited by the paper, characterise the
optimum by two conditions, which this module iterates to a fixed point:

  * midpoint condition: each decision threshold is the midpoint of its two
    neighbouring levels;
  * centroid condition: each level is the conditional mean of f_d over its cell.

Reading taken (the paper says "tightly approximated by N(0, 1/d)" but also
"run Lloyd-Max on f_d"): the codebook is fitted to the exact f_d, not to the
Gaussian approximation.  f_d is log-concave for d >= 3, so the fixed point is
unique and does not depend on the start.
"""

from dataclasses import dataclass

import numpy as np

from .marginal import marginal_mass, marginal_partial_moment


@dataclass(frozen=True)
class Codebook:
    """C^(d,b): ascending levels (2^b) and midpoint thresholds (2^b - 1), fp64."""
    bits: int
    d: int
    levels: np.ndarray
    thresholds: np.ndarray
    iterations: int


def _centroids(thresholds: np.ndarray, d: int) -> np.ndarray:
    """Centroid condition: c_j = int_cell t f_d / int_cell f_d, cells bounded by -1, tau, +1."""
    edges = np.concatenate(([-1.0], thresholds, [1.0]))
    lo, hi = edges[:-1], edges[1:]
    return marginal_partial_moment(lo, hi, d) / marginal_mass(lo, hi, d)


def lloydmax_codebook(bits: int, d: int, start=None, tol: float = 1e-15, max_iter: int = 100000) -> Codebook:
    """Fixed-point Lloyd-Max iteration on f_d (Sec. 3.2; Alg. 1, offline stage).

    start: optional initial levels (ascending); the default spreads 2^b levels
    evenly over +-3 standard deviations of f_d (variance 1/d), kept inside (-1, 1).

    The iteration contracts linearly with some rate rho < 1 (about 0.96 for
    4 bits), so the distance to the fixed point after a step of size delta is
    about delta * rho / (1 - rho); iteration stops when that estimate, in units
    of 1/sqrt(d), is below tol, or when the step stops shrinking for 200
    iterations (the fp64 rounding floor has been reached).
    """
    if bits < 1 or d < 3:
        raise ValueError("need bits >= 1 and d >= 3")
    n = 1 << bits
    sd = 1.0 / np.sqrt(d)
    if start is None:
        c = (np.arange(n) - (n - 1) / 2.0) * (2.0 / n) * min(3.0 * sd, 0.9)
    else:
        c = np.array(start, dtype=np.float64)
    prev, best, since_best = np.inf, np.inf, 0
    it = 0
    for it in range(1, max_iter + 1):
        tau = 0.5 * (c[:-1] + c[1:])            # midpoint condition
        c_new = _centroids(tau, d)               # centroid condition
        delta = np.max(np.abs(c_new - c)) / sd
        c = c_new
        rho = delta / prev if np.isfinite(prev) and prev > 0 else 1.0
        prev = delta
        if delta == 0.0 or (rho < 1.0 and delta * rho / (1.0 - rho) < tol):
            break
        if delta < best:
            best, since_best = delta, 0
        else:
            since_best += 1
            if since_best >= 200:
                break
    tau = 0.5 * (c[:-1] + c[1:])
    return Codebook(bits=bits, d=d, levels=c, thresholds=tau, iterations=it)
