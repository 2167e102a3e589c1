"""The rotation classes compared in the paper's rotation ablation (Sec. 6.1, Table 4), on the
oracle: RPBH, Block-RHT (RPBH without the permutation), Full RHT (one Hadamard block over the
whole power-of-two dimension) and a dense Haar rotation.  Codebook compatibility needs the
rotated, normalized coordinates to follow f_d (Sec. 4.4; Fig. 3); with outlier channels
clustered inside one 128-block, the permutation is what spreads them (Prop. 1), so Block-RHT
leaves a marginal far from f_d while RPBH stays close, and larger blocks get closer still."""

import numpy as np
import scipy.stats as st

import oracle
from oracle.plan import Plan


def _clustered(M, K, seed):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((M, K))
    X[:, 5:37] *= 30.0   # 32 outlier channels, all inside the first 128-block
    return X, rng


def _ks(X, plan):
    U = oracle.normalize_rows(oracle.rpbh_forward(X, plan), 1e-10)[1]
    return st.kstest(U.ravel(), lambda t: oracle.marginal_cdf(t, X.shape[1])).statistic


def _block_rht(plan):
    return Plan(plan.d, plan.h, np.arange(plan.d), plan.sign.copy())


def test_permutation_spreads_clustered_outliers():
    X, _ = _clustered(64, 3072, 0)
    for h in (128, 1024):
        p = oracle.rpbh_plan(3072, h, 0)
        k_rpbh, k_block = _ks(X, p), _ks(X, _block_rht(p))
        assert k_rpbh < 0.5 * k_block, (h, k_rpbh, k_block)
    # without any rotation the marginal is far from f_d; Block-RHT barely helps
    U0 = oracle.normalize_rows(X, 1e-10)[1]
    k_none = st.kstest(U0.ravel(), lambda t: oracle.marginal_cdf(t, 3072)).statistic
    assert k_none > 0.2
    # the paper's larger block (1024 for d = 3072) mixes more: closer to f_d than h = 128
    assert _ks(X, oracle.rpbh_plan(3072, 1024, 0)) < _ks(X, oracle.rpbh_plan(3072, 128, 0))


def test_dense_and_full_rotations_match_the_marginal():
    X, rng = _clustered(64, 4096, 1)
    Q, _ = np.linalg.qr(rng.standard_normal((4096, 4096)))
    Zh = X @ Q.T
    k_haar = st.kstest(oracle.normalize_rows(Zh, 1e-10)[1].ravel(),
                       lambda t: oracle.marginal_cdf(t, 4096)).statistic
    full = _block_rht(oracle.rpbh_plan(4096, 4096, 0))   # Full RHT: one block, no permutation needed
    k_full = _ks(X, full)
    assert k_haar < 0.01 and k_full < 0.02
    assert k_full < _ks(X, oracle.rpbh_plan(4096, 128, 0))
