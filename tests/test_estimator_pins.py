"""Pins of the estimator oracle (online least squares, Sec. 3.3.1) against
what the mathematics fixes, independently of the oracle's own formulas:
exact recovery of noiseless linear data, the closed form of simple linear
regression, the normal equations evaluated directly on the samples, agreement
with an SVD least-squares routine, invariance to sample order and batching,
rank handling, and the integer rounding rule."""
import math

import numpy as np
import pytest

from oracle import estimator as est


def well_conditioned(rng, S, F):
    x = rng.uniform(-1.0, 1.0, (S, F))
    x[:, -1] = 1.0  # constant term, as in the paper's models
    return x


def fit(x, y, n_est=1, ids=None):
    E = est.EstimatorSet(n_est, x.shape[1])
    E.add(np.zeros(len(y), np.int64) if ids is None else ids, x, y)
    return E.solve()


def test_exact_recovery_of_noiseless_models():
    rng = np.random.default_rng(1)
    for F in (1, 2, 3, 5, 8):
        x = well_conditioned(rng, 40, F)
        beta = rng.uniform(-3, 3, F)
        coef, status = fit(x, x @ beta)
        assert status[0] == est.FITTED
        assert np.allclose(coef[0], beta, rtol=1e-10, atol=1e-10)


def test_simple_regression_closed_form():
    """t = alpha * size + c: alpha = cov(size, t) / var(size), c = mean(t) - alpha mean(size)."""
    rng = np.random.default_rng(2)
    size = rng.uniform(1e3, 1e7, 200)
    t = 3.0 + size / 50_000.0 + rng.normal(0, 2.0, 200)
    coef, status = fit(np.stack([size, np.ones_like(size)], 1), t)
    sm, tm = size.mean(), t.mean()
    alpha = ((size - sm) * (t - tm)).sum() / ((size - sm) ** 2).sum()
    c = tm - alpha * sm
    assert status[0] == est.FITTED
    assert math.isclose(coef[0][0], alpha, rel_tol=1e-8) and math.isclose(coef[0][1], c, rel_tol=1e-6)


def test_transfer_estimator_recovers_bandwidth_and_latency():
    """Noiseless transfers t = lat + bytes / bw give alpha = 1 / bw and c = lat."""
    size = np.array([0.0, 64.0, 1 << 20, 1 << 26, 12_345_678.0])
    bw, lat = 12_500.0, 7.0
    coef, status = fit(np.stack([size, np.ones_like(size)], 1), lat + size / bw)
    assert status[0] == est.FITTED
    assert math.isclose(coef[0][0], 1 / bw, rel_tol=1e-9) and math.isclose(coef[0][1], lat, rel_tol=1e-9)


def test_residual_satisfies_the_normal_equations():
    """The least-squares residual is orthogonal to every feature column,
    evaluated from the raw samples (not from the stored sums)."""
    rng = np.random.default_rng(3)
    x = well_conditioned(rng, 300, 5)
    y = x @ rng.uniform(-2, 2, 5) + rng.normal(0, 0.1, 300)
    coef, _ = fit(x, y)
    r = y - x @ coef[0]
    assert np.abs(x.T @ r).max() < 1e-9 * np.abs(x.T @ y).max()


def test_agrees_with_svd_least_squares():
    rng = np.random.default_rng(4)
    for F in (2, 4, 6):
        x = well_conditioned(rng, 120, F)
        y = x @ rng.uniform(-5, 5, F) + rng.normal(0, 0.5, 120)
        coef, _ = fit(x, y)
        ref = np.linalg.lstsq(x, y, rcond=None)[0]
        assert np.allclose(coef[0], ref, rtol=1e-9, atol=1e-9)


def test_operator_model_with_shape_features():
    """A batched matrix multiply model t = b1 bmnk + b2 bmk + b3 bkn + b4 bmn + b5
    over varied shapes, features scaled to comparable magnitudes."""
    rng = np.random.default_rng(5)
    shapes = rng.integers(1, 64, (80, 4)).astype(np.float64)
    b, m, n, k = shapes.T
    phi = np.stack([b * m * n * k / 1e5, b * m * k / 1e3, b * k * n / 1e3, b * m * n / 1e3, np.ones(80)], 1)
    beta = np.array([2.0, 0.5, 0.25, 0.75, 11.0])
    coef, status = fit(phi, phi @ beta)
    assert status[0] == est.FITTED and np.allclose(coef[0], beta, rtol=1e-9)


def test_sample_order_and_batching_do_not_matter():
    rng = np.random.default_rng(6)
    n_est, F, S = 7, 3, 500
    ids = rng.integers(0, n_est, S)
    x = well_conditioned(rng, S, F)
    y = rng.normal(0, 1, S)
    one = est.EstimatorSet(n_est, F)
    one.add(ids, x, y)
    perm = rng.permutation(S)
    two = est.EstimatorSet(n_est, F)
    two.add(ids[perm[:200]], x[perm[:200]], y[perm[:200]])
    two.add(ids[perm[200:]], x[perm[200:]], y[perm[200:]])
    c1, s1 = one.solve()
    c2, s2 = two.solve()
    assert np.array_equal(s1, s2) and np.allclose(c1, c2, rtol=1e-10, atol=1e-12)
    assert np.array_equal(one.count, np.bincount(ids, minlength=n_est))


def test_estimators_are_independent():
    """Each estimator fits only its own samples."""
    rng = np.random.default_rng(7)
    x = well_conditioned(rng, 60, 2)
    ids = np.repeat([0, 1, 2], 20)
    betas = np.array([[1.0, 2.0], [-3.0, 0.5], [0.0, 9.0]])
    y = np.einsum("sf,sf->s", x, betas[ids])
    coef, status = fit(x, y, n_est=4, ids=ids)
    assert list(status) == [est.FITTED] * 3 + [est.UNDERDETERMINED]
    assert np.allclose(coef[:3], betas, rtol=1e-10) and not coef[3].any()


def test_rank_handling():
    rng = np.random.default_rng(8)
    x = well_conditioned(rng, 3, 5)  # fewer samples than features
    assert fit(x, np.ones(3))[1][0] == est.UNDERDETERMINED
    x = well_conditioned(rng, 30, 3)
    dup = np.concatenate([x, x[:, :1]], 1)  # a repeated column
    coef, status = fit(dup, np.ones(30))
    assert status[0] == est.SINGULAR and not coef[0].any()
    zero = x.copy()
    zero[:, 0] = 0.0  # a feature that never varies from zero
    assert fit(zero, np.ones(30))[1][0] == est.SINGULAR


@pytest.mark.parametrize("t,expect", [(2.0, 2), (2.000001, 3), (0.3, 1), (-5.0, 1), (1e6 + 0.5, 1_000_001),
                                      (0.0, 1)])
def test_integer_times_round_up_with_a_floor_of_one(t, expect):
    coef = np.array([[t]])
    assert est.predict_us(coef, [0], [[1.0]])[0] == expect


def test_invalid_queries_give_zero():
    coef = np.array([[2.0], [1e300]])
    assert list(est.predict_us(coef, [0, 1, 2, -1], [[1.5], [10.0], [1.0], [1.0]])) == [3, 0, 0, 0]
    assert est.predict_us(np.array([[float("nan")]]), [0], [[1.0]])[0] == 0
