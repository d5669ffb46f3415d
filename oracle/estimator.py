"""Oracle for the online linear estimators -- TEST INFRASTRUCTURE ONLY.

Written from the paper (SliceScheduler, arXiv 2608.15762), Sec. 3.3.1:
  - transfer estimator, one per accelerator pair: t = alpha * size + c;
  - operator estimator, one per (accelerator type, operator of a template):
    t = sum_j beta_j * phi_j(shape), shape-derived features such as
    (bmnk, bmk, bkn, bmn, 1) for a batched matrix multiply;
  - both are refined online as the executor feeds back measured times.
Each estimator is an ordinary least-squares fit of its samples.  Online
refinement keeps the sufficient statistics of that fit: the Gram matrix
X^T X, the moment vector X^T y and the sample count, summed over every batch
of samples fed back so far; a solve turns them into coefficients.

Readings where the paper is silent (each is listed in the design notes):
  - an estimator with fewer samples than features is not fitted (status 1);
  - a Gram matrix that is not positive definite (collinear features) is not
    fitted (status 2); the relative pivot threshold is 1e-12;
  - unfitted estimators report zero coefficients;
  - an integer time for the simulator is max(1, ceil(x . beta)) microseconds
    (the simulator takes integer durations >= 1); a query naming an unknown
    estimator, or whose prediction is not finite or reaches 2^62, gets 0 (a
    value no valid prediction takes).

Everything is float64, plain numpy; nothing here is shared with the library.
Pinned by tests/test_estimator_pins.py (exact recovery, the closed form of
simple regression, the normal equations as an invariant, agreement with an
SVD least-squares routine, order and batching invariance, rank handling).
"""
from __future__ import annotations

import math

import numpy as np

FITTED, UNDERDETERMINED, SINGULAR = 0, 1, 2
PIVOT_RTOL = 1e-12


class EstimatorSet:
    """Sufficient statistics of n_est least-squares fits with n_feat features."""

    def __init__(self, n_est: int, n_feat: int):
        self.n_est, self.n_feat = n_est, n_feat
        self.gram = np.zeros((n_est, n_feat, n_feat), np.float64)  # sum of x x^T
        self.mom = np.zeros((n_est, n_feat), np.float64)           # sum of x y
        self.count = np.zeros(n_est, np.int64)

    def add(self, est, x, y):
        """Feed back samples: est[S] estimator ids, x[S][n_feat] features, y[S] times."""
        est = np.asarray(est, np.int64)
        x = np.asarray(x, np.float64).reshape(len(est), self.n_feat)
        y = np.asarray(y, np.float64)
        for s in range(len(est)):
            e = est[s]
            self.gram[e] += np.outer(x[s], x[s])
            self.mom[e] += x[s] * y[s]
            self.count[e] += 1

    def solve(self):
        """(coef[n_est][n_feat], status[n_est]): the normal equations
        gram . beta = mom solved by a Cholesky factorisation."""
        F = self.n_feat
        coef = np.zeros((self.n_est, F), np.float64)
        status = np.zeros(self.n_est, np.int32)
        for e in range(self.n_est):
            if self.count[e] < F:
                status[e] = UNDERDETERMINED
                continue
            L = cholesky(self.gram[e])
            if L is None:
                status[e] = SINGULAR
                continue
            # L L^T beta = mom: forward, then back substitution
            z = np.zeros(F)
            for i in range(F):
                z[i] = (self.mom[e][i] - sum(L[i][k] * z[k] for k in range(i))) / L[i][i]
            beta = np.zeros(F)
            for i in reversed(range(F)):
                beta[i] = (z[i] - sum(L[k][i] * beta[k] for k in range(i + 1, F))) / L[i][i]
            coef[e] = beta
        return coef, status


def cholesky(a):
    """Lower-triangular L with L L^T = a, or None when a pivot falls to
    PIVOT_RTOL times its diagonal entry or below (not positive definite)."""
    n = len(a)
    L = np.zeros((n, n))
    for j in range(n):
        d = a[j][j] - sum(L[j][k] ** 2 for k in range(j))
        if not (d > PIVOT_RTOL * abs(a[j][j])) or a[j][j] <= 0:
            return None
        L[j][j] = math.sqrt(d)
        for i in range(j + 1, n):
            L[i][j] = (a[i][j] - sum(L[i][k] * L[j][k] for k in range(j))) / L[j][j]
    return L


def predict(coef, est, x):
    """Predicted times x . coef[est] (float64)."""
    coef = np.asarray(coef, np.float64)
    x = np.asarray(x, np.float64)
    return np.array([float(np.dot(x[i], coef[e])) for i, e in enumerate(np.asarray(est, np.int64))])


def predict_us(coef, est, x):
    """Integer times for the simulator: max(1, ceil(x . coef[est])), or 0 for a
    query naming an unknown estimator or predicting a non-finite time or one
    of 2^62 or more."""
    coef = np.asarray(coef, np.float64)
    x = np.asarray(x, np.float64)
    out = []
    for i, e in enumerate(np.asarray(est, np.int64)):
        if not 0 <= e < len(coef):
            out.append(0)
            continue
        t = 0.0
        for j in range(coef.shape[1]):  # the sum in feature order
            t += x[i][j] * coef[e][j]
        out.append(0 if not (math.isfinite(t) and math.ceil(t) < 2 ** 62) else max(1, math.ceil(t)))
    return np.array(out, np.int64)
