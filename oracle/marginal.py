"""The rotated-coordinate marginal f_d (test infrastructure only).

Sec. 3.2, Eq. (2): after a Haar-random rotation of a unit vector in R^d, each
coordinate t has density

    f_d(t) = Gamma(d/2) / (sqrt(pi) Gamma((d-1)/2)) * (1 - t^2)^((d-3)/2),  t in [-1, 1].

Facts used below, derived from Eq. (2) by elementary calculus:
  * t^2 ~ Beta(1/2, (d-1)/2), so F_d(t) = 1/2 + sgn(t)/2 * I_{t^2}(1/2, (d-1)/2)
    with I the regularized incomplete beta function (a library primitive here).
  * d/dt (1-t^2)^((d-1)/2) = -(d-1) t (1-t^2)^((d-3)/2), hence
    int_a^b t f_d(t) dt = C_d/(d-1) * [(1-a^2)^((d-1)/2) - (1-b^2)^((d-1)/2)].
"""

from functools import lru_cache

import mpmath
import numpy as np
from scipy import special


@lru_cache(maxsize=None)
def log_norm_const(d: int) -> float:
    """log C_d with C_d = Gamma(d/2) / (sqrt(pi) Gamma((d-1)/2))  (Eq. (2)).

    Evaluated with 40-digit log-gamma: the difference of two fp64 log-gammas
    near d/2 ~ 10^4 would lose about 1e-12 of relative precision."""
    with mpmath.workdps(40):
        dd = mpmath.mpf(int(d))
        v = mpmath.loggamma(dd / 2) - mpmath.loggamma((dd - 1) / 2) - mpmath.log(mpmath.pi) / 2
    return float(v)


def marginal_pdf(t, d: int):
    """f_d(t) of Eq. (2); zero outside [-1, 1]."""
    t = np.asarray(t, dtype=np.float64)
    inside = np.abs(t) < 1.0
    out = np.zeros_like(t)
    ti = t[inside]
    out[inside] = np.exp(log_norm_const(d) + 0.5 * (d - 3.0) * np.log1p(-ti * ti))
    return out


def marginal_cdf(t, d: int):
    """F_d(t) = 1/2 + sgn(t)/2 * I_{t^2}(1/2, (d-1)/2), from t^2 ~ Beta(1/2, (d-1)/2)."""
    t = np.clip(np.asarray(t, dtype=np.float64), -1.0, 1.0)
    return 0.5 + 0.5 * np.sign(t) * special.betainc(0.5, 0.5 * (d - 1.0), t * t)


def marginal_mass(a, b, d: int):
    """P(a < t <= b) under f_d.

    For a cell on one side of zero the difference of two CDF values is taken in
    the tail form (via the complementary incomplete beta) so that the outer
    cells keep their relative precision.
    """
    a = np.clip(np.asarray(a, dtype=np.float64), -1.0, 1.0)
    b = np.clip(np.asarray(b, dtype=np.float64), -1.0, 1.0)
    beta_b = 0.5 * (d - 1.0)
    # upper tail Q(x) = P(t > x) for x >= 0 is 1/2 * I^c_{x^2}(1/2, (d-1)/2)
    def upper(x):
        return 0.5 * special.betaincc(0.5, beta_b, x * x)
    a_, b_ = np.broadcast_arrays(a, b)
    out = np.empty(a_.shape, dtype=np.float64)
    pos = a_ >= 0.0
    neg = b_ <= 0.0
    mid = ~(pos | neg)
    out[pos] = upper(a_[pos]) - upper(b_[pos])
    out[neg] = upper(-b_[neg]) - upper(-a_[neg])
    out[mid] = 1.0 - upper(-a_[mid]) - upper(b_[mid])
    return out


def marginal_partial_moment(a, b, d: int):
    """int_a^b t f_d(t) dt in closed form (antiderivative of t f_d derived from Eq. (2))."""
    a = np.clip(np.asarray(a, dtype=np.float64), -1.0, 1.0)
    b = np.clip(np.asarray(b, dtype=np.float64), -1.0, 1.0)
    lc = log_norm_const(d)
    e = 0.5 * (d - 1.0)

    def g(x):
        # (1 - x^2)^((d-1)/2), exactly 0 at |x| = 1
        with np.errstate(divide="ignore"):
            return np.where(np.abs(x) < 1.0, np.exp(e * np.log1p(-x * x)), 0.0)

    return np.exp(lc) / (d - 1.0) * (g(a) - g(b))
