"""Pins for the oracle's RPBH plan and transform (CPU only).

Fixed independently of the oracle by: the SplitMix64 known-answer values
(golden file), exact integer identities of the Sylvester matrix, the explicit
dense matrix blkdiag(H_h D_1, ..., H_h D_k) P_pi assembled here from the
definition in Eq. (9), orthogonality, the supplement's exact per-coordinate
variance M_j / h (enumerated over all sign patterns), and the rotation
cancellation of Sec. 4.3.
"""

import itertools
import math

import numpy as np
import pytest
import scipy.linalg

import oracle
from oracle.plan import SplitMix64
from tests.conftest import read_golden


def test_splitmix64_known_answers():
    for seed, outs in read_golden("splitmix64_kat.txt"):
        g = SplitMix64(int(seed))
        assert [g.next() for _ in range(5)] == [int(v) for v in outs.split()]


def test_bounded_draw_is_uniform():
    g = SplitMix64(7)
    counts = np.bincount([g.below(6) for _ in range(60000)], minlength=6)
    chi2 = np.sum((counts - 10000.0) ** 2 / 10000.0)
    assert chi2 < 25.0   # 5 dof, p ~ 1e-4


def test_plan_is_permutation_with_signs_and_deterministic():
    for d, h in ((3072, 128), (128, 128), (24, 8), (5, 1)):
        p = oracle.rpbh_plan(d, h, seed=3)
        assert sorted(p.perm.tolist()) == list(range(d))
        assert set(np.unique(p.sign).tolist()) <= {-1.0, 1.0}
        q = oracle.rpbh_plan(d, h, seed=3)
        assert np.array_equal(p.perm, q.perm) and np.array_equal(p.sign, q.sign)
    a, b = oracle.rpbh_plan(3072, 128, 0), oracle.rpbh_plan(3072, 128, 1)
    assert not np.array_equal(a.perm, b.perm)
    assert abs(np.mean(a.sign)) < 0.1


def test_fisher_yates_uniform_over_small_perms():
    counts = {}
    for seed in range(6000):
        key = tuple(oracle.rpbh_plan(3, 1, seed).perm.tolist())
        counts[key] = counts.get(key, 0) + 1
    assert len(counts) == 6
    chi2 = sum((c - 1000.0) ** 2 / 1000.0 for c in counts.values())
    assert chi2 < 25.0


def test_plan_rejects_bad_block():
    for d, h in ((100, 3), (96, 64), (0, 1)):
        with pytest.raises(ValueError):
            oracle.rpbh_plan(d, h, 0)


@pytest.mark.parametrize("h", [1, 2, 4, 8, 16, 32, 64, 128, 256])
def test_sylvester_integer_identities(h):
    H = oracle.sylvester_hadamard(h)
    assert np.array_equal(H @ H.T, h * np.eye(h, dtype=np.int64))
    # natural (Sylvester) order: H[r, c] = (-1)^popcount(r & c)
    r, c = np.meshgrid(np.arange(h), np.arange(h), indexing="ij")
    pop = np.vectorize(lambda v: bin(int(v)).count("1"))(r & c)
    assert np.array_equal(H, np.where(pop % 2 == 0, 1, -1))


@pytest.mark.parametrize("h", [2, 8, 64, 256])
def test_fwht_equals_explicit_matrix(h):
    rng = np.random.default_rng(h)
    Y = rng.normal(size=(5, 3 * h))
    Z = oracle.fwht_blocks(Y, h)
    H = oracle.sylvester_hadamard(h).astype(np.float64)
    want = np.concatenate([Y[:, j * h:(j + 1) * h] @ H.T for j in range(3)], axis=1)
    assert np.max(np.abs(Z - want)) < 1e-12 * h


def _dense_pi(plan):
    """blkdiag(H_h D_1, ..., H_h D_k) P_pi assembled from Eq. (9)."""
    d, h = plan.d, plan.h
    H = oracle.sylvester_hadamard(h).astype(np.float64) / math.sqrt(h)
    blocks = [H @ np.diag(plan.sign[j * h:(j + 1) * h]) for j in range(d // h)]
    P = np.zeros((d, d))
    P[np.arange(d), plan.perm] = 1.0          # (P x)_j = x[perm[j]]
    return scipy.linalg.block_diag(*blocks) @ P


@pytest.mark.parametrize("d,h", [(24, 8), (64, 16), (384, 128), (10, 2), (7, 1)])
def test_forward_is_eq9_and_orthogonal(d, h):
    plan = oracle.rpbh_plan(d, h, seed=11)
    Pi = _dense_pi(plan)
    rng = np.random.default_rng(d)
    X = rng.normal(size=(6, d))
    assert np.max(np.abs(oracle.rpbh_forward(X, plan) - X @ Pi.T)) < 1e-13
    assert np.max(np.abs(Pi @ Pi.T - np.eye(d))) < 1e-13
    Z = oracle.rpbh_forward(X, plan)
    assert np.max(np.abs(oracle.rpbh_inverse(Z, plan) - X)) < 1e-13
    assert np.max(np.abs(np.linalg.norm(Z, axis=1) - np.linalg.norm(X, axis=1))) < 1e-12


def test_block_size_one_is_signed_permutation():
    plan = oracle.rpbh_plan(9, 1, seed=5)
    X = np.arange(1.0, 10.0)[None, :]
    assert np.array_equal(oracle.rpbh_forward(X, plan)[0], X[0, plan.perm] * plan.sign)


def test_exact_conditional_variance_by_sign_enumeration():
    # Suppl. A (Lemma 1 proof): given pi, z_l in block j is a Rademacher sum with variance M_j / h
    d, h = 16, 8
    rng = np.random.default_rng(2)
    x = rng.normal(size=d)
    x /= np.linalg.norm(x)
    plan = oracle.rpbh_plan(d, h, seed=4)
    y = x[plan.perm]
    masses = [np.sum(y[j * h:(j + 1) * h] ** 2) for j in range(d // h)]
    acc = np.zeros(d)
    accm = np.zeros(d)
    n = 0
    for s in itertools.product((-1.0, 1.0), repeat=d):
        p = oracle.Plan(d=d, h=h, perm=plan.perm, sign=np.array(s))
        z = oracle.rpbh_forward(x[None, :], p)[0]
        acc += z * z
        accm += z
        n += 1
    var = acc / n
    assert np.max(np.abs(accm / n)) < 1e-14
    for j in range(d // h):
        assert np.max(np.abs(var[j * h:(j + 1) * h] - masses[j] / h)) < 1e-13


def test_rotation_cancels_in_the_product():
    # Sec. 4.3: (W Pi^T)(Pi x) = W x for the orthogonal RPBH
    rng = np.random.default_rng(9)
    d = 384
    plan = oracle.rpbh_plan(d, 128, seed=2)
    X = rng.normal(size=(7, d))
    W = rng.normal(size=(5, d))
    Wr = oracle.rpbh_forward(W, plan)          # rows w'_i = Pi w_i, i.e. W Pi^T
    Xr = oracle.rpbh_forward(X, plan)
    assert np.max(np.abs(Xr @ Wr.T - X @ W.T)) < 1e-12


def test_permutation_spreads_a_clustered_outlier():
    # Sec. 4.4 / Lemma 2: with pi the block masses are balanced; without pi an
    # outlier confined to one block stays there
    d, h = 3072, 128
    k = d // h
    x = np.full(d, 1e-3)
    x[:64] = 1.0                                   # all outlier mass inside block 0
    x /= np.linalg.norm(x)
    ident = oracle.Plan(d=d, h=h, perm=np.arange(d), sign=np.ones(d))
    mass_id = [np.sum(x[j * h:(j + 1) * h] ** 2) for j in range(k)]
    assert max(mass_id) > 0.99
    plan = oracle.rpbh_plan(d, h, seed=0)
    y = x[plan.perm]
    mass = np.array([np.sum(y[j * h:(j + 1) * h] ** 2) for j in range(k)])
    mu_inf = np.max(x ** 2)
    delta = 0.01
    bound = mu_inf * math.sqrt(0.5 * h * math.log(4 * k / delta))   # Eq. (12)
    assert np.max(np.abs(mass - 1.0 / k)) <= bound
    assert max(mass) < 0.2
    z_id = oracle.rpbh_forward(x[None, :], ident)[0]
    assert np.max(np.abs(z_id[h:])) < 1e-2       # blocks 1.. saw no outlier energy


def _violations(values, bound):
    return int(np.sum(np.asarray(values) > bound))


def test_lemma1_per_block_incoherence():
    # Suppl. proof sketch, Lemma 1: for any partition, over the signs, ||z||_inf <= sqrt(2 log(4d/delta)/h)
    # with probability >= 1 - delta/2.  The test vector is the worst case for a missing sign: a flat
    # block holding all the mass (without D, H maps it to a single spike of size 1)
    d, h, delta, trials = 3072, 128, 0.05, 300
    x = np.zeros(d)
    x[:h] = 1.0 / np.sqrt(h)
    bound = math.sqrt(2 * math.log(4 * d / delta) / h)
    rng = np.random.default_rng(11)
    norms = []
    for _ in range(trials):
        p = oracle.Plan(d=d, h=h, perm=np.arange(d), sign=rng.choice([-1.0, 1.0], size=d))
        norms.append(np.max(np.abs(oracle.rpbh_forward(x[None, :], p))))
    assert _violations(norms, bound) <= delta / 2 * trials
    no_sign = oracle.Plan(d=d, h=h, perm=np.arange(d), sign=np.ones(d))
    assert np.max(np.abs(oracle.rpbh_forward(x[None, :], no_sign))) > 0.99 > bound


def test_lemma2_mass_balancing():
    # Lemma 2: over pi, |M_j - 1/k| <= mu_inf sqrt((h/2) log(4k/delta)) for all j, w.p. >= 1 - delta/2
    d, h, delta, trials = 3072, 128, 0.05, 300
    k = d // h
    rng = np.random.default_rng(12)
    x = 1.0 + 0.1 * rng.random(d)
    x[:h] *= 1.5                                    # block 0 of the channels is heavier
    x /= np.linalg.norm(x)
    mu = np.max(x * x)
    bound = mu * math.sqrt(h / 2 * math.log(4 * k / delta))
    devs = []
    for t in range(trials):
        p = oracle.rpbh_plan(d, h, seed=1000 + t)
        y = x[p.perm]
        M = np.sum(y.reshape(k, h) ** 2, axis=1)
        devs.append(np.max(np.abs(M - 1.0 / k)))
    assert _violations(devs, bound) <= delta / 2 * trials
    # without pi the heavier channels stay together in block 0, beyond the bound
    M0 = np.sum(x[:h] ** 2)
    assert abs(M0 - 1.0 / k) > bound


def test_proposition_sup_norm_bound():
    # Proposition (restated in the supplement): ||Pi_d x||_inf <= sqrt((2/d)(1 + rho) log(4d/delta)),
    # rho = d mu_inf sqrt(log(4k/delta) / (2h)), w.p. >= 1 - delta over the plan
    d, h, delta, trials = 3072, 128, 0.05, 200
    k = d // h
    rng = np.random.default_rng(13)
    x = rng.standard_normal(d)
    x /= np.linalg.norm(x)
    mu = np.max(x * x)
    rho = d * mu * math.sqrt(math.log(4 * k / delta) / (2 * h))
    bound = math.sqrt(2.0 / d * (1 + rho) * math.log(4 * d / delta))
    norms = [np.max(np.abs(oracle.rpbh_forward(x[None, :], oracle.rpbh_plan(d, h, seed=2000 + t))))
             for t in range(trials)]
    assert _violations(norms, bound) <= delta * trials
    assert max(norms) > 0.3 * bound                 # the bound is not vacuous at this size
