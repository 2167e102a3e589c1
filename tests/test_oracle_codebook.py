"""Pins for the oracle's marginal f_d and Lloyd-Max codebook (CPU only).

What fixes the right answer here is not the oracle itself:
  * an independent quadrature of Eq. (2) (Gauss-Legendre after t = sin(theta),
    written in this file) for the CDF, the cell masses and the first moments;
  * closed forms derived from Eq. (2): the d = 3 marginal is uniform, whose
    Lloyd-Max quantizer is the uniform midpoint quantizer; the 1-bit level is
    E|t| = Gamma(d/2) / (sqrt(pi) Gamma((d+1)/2)); the 1-bit Gaussian MSE is 1 - 2/pi;
  * the Gaussian limit of f_d (Sec. 3.2) against Max's 1960 table (golden file);
  * the two optimality conditions, symmetry and uniqueness of the fixed point.
A dropped term, a wrong exponent or a wrong normalising constant in the oracle
fails at least one of these.
"""

import math

import numpy as np
import pytest
from scipy import special

import oracle
from oracle.marginal import marginal_cdf, marginal_mass, marginal_partial_moment, marginal_pdf
from tests.conftest import read_golden

DIMS = [3, 4, 5, 16, 64, 3072, 5120, 12288, 13824]


def norm_const_by_recurrence(d):
    """C_d = Gamma(d/2) / (sqrt(pi) Gamma((d-1)/2)) from Gamma(z+1) = z Gamma(z):
    R(d) = Gamma(d/2)/Gamma((d-1)/2) has R(2) = 1/sqrt(pi), R(3) = sqrt(pi)/2, R(d+2) = R(d) d/(d-1)."""
    j = np.arange(5 if d % 2 else 4, d + 1, 2, dtype=np.float64)      # R(j) = R(j-2) (j-2)/(j-3)
    log_r = (math.log(math.sqrt(math.pi) / 2) if d % 2 else -0.5 * math.log(math.pi)) + math.fsum(np.log1p(1.0 / (j - 3.0)))
    return log_r - 0.5 * math.log(math.pi)


def quad_theta(fun_t, a, b, d, panels=None, nodes=24):
    """int_a^b fun_t(t) * (1 - t^2)^((d-3)/2) dt * C_d via t = sin(theta), composite Gauss-Legendre.

    Independent of the oracle: C_d by the Gamma recurrence, the integrand written out here."""
    logc = norm_const_by_recurrence(d)
    ta, tb = math.asin(max(-1.0, min(1.0, a))), math.asin(max(-1.0, min(1.0, b)))
    if panels is None:
        width = 0.15 / math.sqrt(d)
        panels = max(8, min(4000, int(math.ceil((tb - ta) / width))))
    x, w = np.polynomial.legendre.leggauss(nodes)
    edges = np.linspace(ta, tb, panels + 1)
    total = 0.0
    for lo, hi in zip(edges[:-1], edges[1:]):
        th = 0.5 * (hi - lo) * x + 0.5 * (hi + lo)
        c = np.cos(th)
        with np.errstate(divide="ignore"):
            val = np.where(c > 0, np.exp(logc + (d - 2) * np.log(np.maximum(c, 1e-300))), 0.0)
        total += 0.5 * (hi - lo) * np.sum(w * fun_t(np.sin(th)) * val)
    return total


@pytest.mark.parametrize("d", DIMS + [20001, 20002])
def test_norm_const_against_gamma_recurrence(d):
    assert abs(oracle.log_norm_const(d) - norm_const_by_recurrence(d)) < 2e-15 * max(1.0, abs(norm_const_by_recurrence(d)))
    if d < 300:
        c = math.gamma(d / 2) / (math.sqrt(math.pi) * math.gamma((d - 1) / 2))
        assert abs(math.exp(oracle.log_norm_const(d)) / c - 1) < 1e-14


@pytest.mark.parametrize("d", DIMS)
def test_marginal_normalised_and_variance(d):
    # int f_d = 1 and E[t^2] = 1/d (a unit vector's coordinates have mean square 1/d)
    T = min(1.0, 60.0 / math.sqrt(d))
    assert abs(quad_theta(lambda t: np.ones_like(t), -T, T, d) - 1.0) < 1e-12
    assert abs(quad_theta(lambda t: t * t, -T, T, d) * d - 1.0) < 1e-11


@pytest.mark.parametrize("d", DIMS)
def test_marginal_cdf_mass_moment_against_quadrature(d):
    sd = 1.0 / math.sqrt(d)
    pts = [x * sd for x in (-3.1, -1.2, -0.3, 0.0, 0.4, 1.7, 2.6)]
    pts = [max(-0.999, min(0.999, p)) for p in pts]
    for p in pts:
        q = quad_theta(lambda t: np.ones_like(t), -1.0, p, d)
        assert abs(float(marginal_cdf(p, d)) - q) < 1e-13
    for a, b in zip(pts[:-1], pts[1:]):
        m = quad_theta(lambda t: np.ones_like(t), a, b, d)
        assert abs(float(marginal_mass(a, b, d)) - m) <= 1e-13 + 1e-12 * m
        pm = quad_theta(lambda t: t, a, b, d)
        assert abs(float(marginal_partial_moment(a, b, d)) - pm) <= 1e-16 + 1e-11 * abs(pm)
    # the pdf itself at a few points, against the formula written out with math.gamma
    if d < 100:
        c = math.gamma(d / 2) / (math.sqrt(math.pi) * math.gamma((d - 1) / 2))
        for p in (-0.7, 0.0, 0.33):
            assert abs(float(marginal_pdf(p, d)) - c * (1 - p * p) ** ((d - 3) / 2)) < 1e-13


def test_d3_is_uniform_closed_form():
    # d = 3: f_3(t) = 1/2 on [-1, 1]; CDF (t+1)/2; Lloyd-Max = uniform midpoint quantizer
    for t in (-0.9, -0.25, 0.0, 0.6):
        assert abs(float(marginal_cdf(t, 3)) - (t + 1) / 2) < 1e-15
        assert abs(float(marginal_pdf(t, 3)) - 0.5) < 1e-15
    for b in (1, 2, 3, 4):
        n = 1 << b
        cb = oracle.lloydmax_codebook(b, 3)
        want = -1.0 + (2.0 * np.arange(n) + 1.0) / n
        assert np.max(np.abs(cb.levels - want)) < 1e-13


@pytest.mark.parametrize("d", [3072, 5120, 12288, 13824, 64])
def test_one_bit_closed_form(d):
    # 1 bit: the positive level is E[t | t > 0] = 2 int_0^1 t f_d = Gamma(d/2)/(sqrt(pi) Gamma((d+1)/2))
    cb = oracle.lloydmax_codebook(1, d)
    # Gamma(d/2)/Gamma((d+1)/2) = 1/R(d+1) with R from the Gamma recurrence above
    want = math.exp(-norm_const_by_recurrence(d + 1) - math.log(math.pi))
    assert abs(cb.levels[1] - want) < 1e-14 * want
    assert cb.levels[0] == -cb.levels[1]
    assert cb.thresholds[0] == 0.0


def _gaussian_table():
    rows = {}
    for bits, lv, th, mse in read_golden("max1960_gaussian_lloydmax.txt"):
        rows[int(bits)] = ([float(v) for v in lv.split()], [float(v) for v in th.split()], float(mse))
    return rows


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_gaussian_limit_matches_max_1960(bits):
    levels, thr, mse = _gaussian_table()[bits]
    d = 10 ** 6
    cb = oracle.lloydmax_codebook(bits, d)
    n = 1 << bits
    pos_levels = cb.levels[n // 2:] * math.sqrt(d)
    pos_thr = cb.thresholds[n // 2 - 1:] * math.sqrt(d)
    assert np.max(np.abs(pos_levels - np.array(levels))) < 6e-4
    assert np.max(np.abs(pos_thr - np.array(thr))) < 6e-4
    # distortion of the limit quantizer for N(0, 1): sum over cells of int (t - c)^2 phi
    edges = np.concatenate(([-np.inf], cb.thresholds * math.sqrt(d), [np.inf]))
    c = cb.levels * math.sqrt(d)
    phi = lambda x: np.exp(-0.5 * x * x) / math.sqrt(2 * math.pi)
    Phi = lambda x: 0.5 * special.erfc(-x / math.sqrt(2))
    a, b = edges[:-1], edges[1:]
    # closed forms for the Gaussian: int t^2 phi = Phi - t phi ; int t phi = -phi
    def m2(x):
        return np.where(np.isfinite(x), Phi(x) - np.where(np.isfinite(x), x, 0) * phi(x), Phi(x))
    mass = Phi(b) - Phi(a)
    m1 = phi(a) - phi(b)
    dist = np.sum(m2(b) - m2(a) - 2 * c * m1 + c * c * mass)
    assert abs(dist - mse) < 1e-4
    if bits == 1:
        assert abs(dist - (1 - 2 / math.pi)) < 1e-6


@pytest.mark.parametrize("bits", [2, 3, 4])
@pytest.mark.parametrize("d", [64, 3072, 13824])
def test_optimality_conditions_by_independent_quadrature(bits, d):
    cb = oracle.lloydmax_codebook(bits, d)
    n = 1 << bits
    sd = 1.0 / math.sqrt(d)
    # midpoint condition
    assert np.max(np.abs(cb.thresholds - 0.5 * (cb.levels[:-1] + cb.levels[1:]))) < 1e-16
    # centroid condition, each cell integrated independently
    edges = np.concatenate(([-1.0], cb.thresholds, [1.0]))
    for j in range(n):
        lo, hi = max(edges[j], -60 * sd), min(edges[j + 1], 60 * sd)
        mass = quad_theta(lambda t: np.ones_like(t), lo, hi, d)
        mom = quad_theta(lambda t: t, lo, hi, d)
        assert abs(mom / mass - cb.levels[j]) < 1e-12 * sd
    # symmetry about zero
    assert np.max(np.abs(cb.levels + cb.levels[::-1])) < 1e-15 * 10
    assert cb.thresholds[n // 2 - 1] == pytest.approx(0.0, abs=1e-18)


@pytest.mark.parametrize("bits", [2, 4])
def test_fixed_point_unique_from_three_starts(bits):
    d = 3072
    n = 1 << bits
    sd = 1 / math.sqrt(d)
    base = oracle.lloydmax_codebook(bits, d)
    starts = [np.linspace(-2.5, 2.5, n) * sd,
              np.sort(np.random.default_rng(0).normal(size=n)) * sd,
              (np.arange(n) - n / 2 + 0.5) * 0.01 * sd]
    for s in starts:
        cb = oracle.lloydmax_codebook(bits, d, start=s)
        assert np.max(np.abs(cb.levels - base.levels)) < 1e-13 * sd


def test_finite_d_approaches_gaussian_at_rate_one_over_d():
    # sqrt(d) c^(d,b) -> g^(b) with an error that scales like 1/d (Eq. (2) -> N(0,1/d))
    g = oracle.lloydmax_codebook(2, 10 ** 6).levels * math.sqrt(10 ** 6)
    e1 = np.max(np.abs(oracle.lloydmax_codebook(2, 3072).levels * math.sqrt(3072) - g))
    e4 = np.max(np.abs(oracle.lloydmax_codebook(2, 12288).levels * math.sqrt(12288) - g))
    assert 3.6 < e1 / e4 < 4.4


def test_exact_marginal_differs_from_gaussian_beyond_tie_band():
    # the reading "fit the exact f_d" matters: at d=3072, b=4 the outer thresholds
    # move by more than the 1e-5 near-tie band relative to the N(0,1/d) fit
    d = 3072
    exact = oracle.lloydmax_codebook(4, d).thresholds
    gauss = oracle.lloydmax_codebook(4, 10 ** 6).thresholds * math.sqrt(10 ** 6) / math.sqrt(d)
    assert np.max(np.abs(exact - gauss)) > 1e-5


def test_bf16_lut_rounding_error_within_half_ulp():
    # the GEMM's bf16 images of the levels: each within half an ulp at 8 significant bits
    # (2^-8 of the value at most), and the levels are not bf16 values, so the rounding is real
    worst = 0.0
    for d in (3072, 5120, 12288, 13824):
        for b in (2, 3, 4, 6):
            lv = oracle.lloydmax_codebook(b, d).levels
            r = oracle.bf16_round(lv)
            assert np.array_equal(r, -r[::-1])          # rounding keeps the antisymmetry
            worst = max(worst, np.max(np.abs(r - lv) / np.abs(lv)))
    assert 1e-3 < worst <= 2.0 ** -8
