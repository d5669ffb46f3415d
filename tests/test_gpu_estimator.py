"""Parity of the online estimators on the GPU (ss_est_*, Sec. 3.3.1) with the
estimator oracle.

Coefficients are float64 results of the same normal equations summed in a
different order, so they are compared within a tolerance derived from the
arithmetic (rtol 1e-9 on well-conditioned fits, see the design notes); fit
statuses and the integer times of ss_est_predict are compared exactly (the
prediction rounds each product and sum in feature order on both sides, so the
ceiling sees the same float64 value).
"""
import numpy as np
import pytest

from oracle import estimator as est
from paper_2608_15762_amd import ss

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
RTOL, ATOL = 1e-9, 1e-9


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ss.lib()
    return torch.device("cuda:0")


def grouped(rng, n_est, F, counts, noise=0.1, scale=1.0):
    """Samples grouped by estimator: ptr, x, y, ids and the true coefficients."""
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    S = int(ptr[-1])
    ids = np.repeat(np.arange(n_est), counts)
    x = rng.uniform(-1.0, 1.0, (S, F)) * scale
    x[:, -1] = 1.0
    beta = rng.uniform(-3, 3, (n_est, F))
    y = np.einsum("sf,sf->s", x, beta[ids]) + rng.normal(0, noise, S)
    return ptr, x, y, ids, beta


def to_dev(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def gpu_fit(dev, n_est, F, batches):
    E = ss.Estimators(n_est, F)
    for ptr, x, y in batches:
        E.add(to_dev(ptr, dev), to_dev(x, dev), to_dev(y, dev))
    coef, status = E.solve()
    torch.cuda.synchronize()
    out = coef.cpu().numpy(), status.cpu().numpy()
    E.free()
    return out


@pytest.mark.parametrize("F", range(1, 9))
def test_fit_parity_every_feature_count(dev, F):
    rng = np.random.default_rng(100 + F)
    n_est = 37
    counts = rng.integers(0, 90, n_est)
    counts[:3] = [0, max(F - 1, 0), F]  # empty, underdetermined, just determined
    ptr, x, y, ids, _ = grouped(rng, n_est, F, counts)
    ref = est.EstimatorSet(n_est, F)
    ref.add(ids, x, y)
    rc, rs = ref.solve()
    gc, gs = gpu_fit(dev, n_est, F, [(ptr, x, y)])
    assert np.array_equal(gs, rs)
    assert np.allclose(gc, rc, rtol=RTOL, atol=ATOL), np.abs(gc - rc).max()


def test_online_batches_accumulate(dev):
    rng = np.random.default_rng(7)
    n_est, F = 50, 4
    batches, ref = [], est.EstimatorSet(n_est, F)
    for b in range(3):
        ptr, x, y, ids, _ = grouped(rng, n_est, F, rng.integers(0, 30, n_est))
        batches.append((ptr, x, y))
        ref.add(ids, x, y)
    rc, rs = ref.solve()
    gc, gs = gpu_fit(dev, n_est, F, batches)
    assert np.array_equal(gs, rs) and np.allclose(gc, rc, rtol=RTOL, atol=ATOL)


def test_rank_handling_on_gpu(dev):
    rng = np.random.default_rng(8)
    F = 4
    x = rng.uniform(-1, 1, (60, F))
    x[:, -1] = 1.0
    x[:30, 1] = x[:30, 0]  # estimator 0: a repeated column
    x[30:, 2] = 0.0        # estimator 1: a column that is always zero
    y = rng.normal(0, 1, 60)
    ptr = np.array([0, 30, 60, 60], np.int64)
    gc, gs = gpu_fit(dev, 3, F, [(ptr, x, y)])
    assert list(gs) == [est.SINGULAR, est.SINGULAR, est.UNDERDETERMINED] and not gc.any()


def test_sample_ranges_are_clamped(dev):
    """Offsets past the sample count are clamped to it: the last estimator
    sees only the samples that exist."""
    rng = np.random.default_rng(9)
    F = 2
    x = rng.uniform(-1, 1, (40, F))
    x[:, -1] = 1.0
    y = rng.normal(0, 1, 40)
    ptr = np.array([0, 25, 1000], np.int64)
    ref = est.EstimatorSet(2, F)
    ref.add(np.repeat([0, 1], [25, 15]), x, y)
    rc, rs = ref.solve()
    gc, gs = gpu_fit(dev, 2, F, [(ptr, x, y)])
    assert np.array_equal(gs, rs) and np.allclose(gc, rc, rtol=RTOL, atol=ATOL)


def test_operator_model_recovery_on_gpu(dev):
    """Batched matrix multiply features (bmnk, bmk, bkn, bmn, 1), one model per
    (device class, operator): noiseless times give the coefficients back."""
    rng = np.random.default_rng(10)
    n_est, per = 12, 40
    shapes = rng.integers(1, 64, (n_est * per, 4)).astype(np.float64)
    b, m, n, k = shapes.T
    phi = np.stack([b * m * n * k / 1e5, b * m * k / 1e3, b * k * n / 1e3, b * m * n / 1e3, np.ones(len(b))], 1)
    beta = rng.uniform(0.1, 5.0, (n_est, 5))
    ids = np.repeat(np.arange(n_est), per)
    y = np.einsum("sf,sf->s", phi, beta[ids])
    gc, gs = gpu_fit(dev, n_est, 5, [(np.arange(0, n_est * per + 1, per, dtype=np.int64), phi, y)])
    assert (gs == est.FITTED).all() and np.allclose(gc, beta, rtol=1e-8)


def test_predict_parity_exact(dev):
    """Integer times from the oracle's coefficients: bit-exact, including the
    floor of 1, values exactly on an integer, unknown estimators and overflow."""
    rng = np.random.default_rng(11)
    n_est, F, M = 20, 3, 4000
    coef = rng.uniform(-50, 500, (n_est, F))
    coef[0] = [2.0, 0.0, 0.0]
    coef[1] = [1e300, 0.0, 0.0]
    est_of = rng.integers(-2, n_est + 2, M).astype(np.int32)
    x = rng.uniform(0, 10, (M, F))
    x[:50] = [[1.5, 0.0, 0.0]]  # 3.0 exactly with estimator 0
    est_of[:50] = 0
    ref = est.predict_us(coef, est_of, x)
    got = ss.est_predict(to_dev(coef, dev), to_dev(est_of, dev), to_dev(x, dev)).cpu().numpy()
    assert np.array_equal(got, ref)
    assert (ref[:50] == 3).all() and (ref == 0).any() and (ref == 1).any()


def test_large_set_sampled(dev):
    """The size the benchmark times: 65,536 estimators of 5 features, 16
    samples each on average, checked on a sample of estimators."""
    rng = np.random.default_rng(12)
    n_est, F = 65536, 5
    counts = rng.integers(0, 33, n_est)
    ptr, x, y, ids, _ = grouped(rng, n_est, F, counts)
    gc, gs = gpu_fit(dev, n_est, F, [(ptr, x, y)])
    pick = np.unique(np.concatenate([[0, n_est - 1], rng.choice(n_est, 300, replace=False)]))
    ref = est.EstimatorSet(len(pick), F)
    for i, e in enumerate(pick):
        s0, s1 = ptr[e], ptr[e + 1]
        ref.add(np.full(s1 - s0, i), x[s0:s1], y[s0:s1])
    rc, rs = ref.solve()
    assert np.array_equal(gs[pick], rs) and np.allclose(gc[pick], rc, rtol=RTOL, atol=ATOL)


@pytest.mark.parametrize("n_est,hi", [(1000, 6), (300, 20), (40, 400), (3, 1)])
def test_lane_groups_for_every_batch_density(dev, n_est, hi):
    """Batches with about 3, 10, 200 and under 1 samples per estimator take
    different lane-group sizes (and estimator counts not divisible by them)."""
    rng = np.random.default_rng(n_est + hi)
    F = 3
    ptr, x, y, ids, _ = grouped(rng, n_est, F, rng.integers(0, hi + 1, n_est))
    ref = est.EstimatorSet(n_est, F)
    ref.add(ids, x, y)
    rc, rs = ref.solve()
    gc, gs = gpu_fit(dev, n_est, F, [(ptr, x, y)])
    assert np.array_equal(gs, rs) and np.allclose(gc, rc, rtol=RTOL, atol=ATOL)
