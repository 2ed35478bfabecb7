"""Pins of the oracle's per-round metrics (CPU only).

Appendix A states the problem as minimising (1/n) sum_i f_i at one common
point and measures consensus by ||W - 1 w_bar^T||; every expected value below
is worked out by hand from those definitions.
"""
import math

import numpy as np
import pytest

from oracle import metrics


def test_mean_model_hand_built():
    W = np.array([[1.0, 2.0, -3.0],
                  [3.0, 6.0, 3.0]])
    assert metrics.mean_model(W).tolist() == [2.0, 4.0, 0.0]      # column means, not row means
    assert metrics.mean_model(W[::-1]).tolist() == [2.0, 4.0, 0.0]
    assert metrics.mean_model(np.array([[5.0, -1.0]])).tolist() == [5.0, -1.0]


def test_consensus_distance_hand_built():
    a = np.array([1.0, 2.0, 3.0])
    assert metrics.consensus_distance(np.stack([a, a, a])) == 0.0
    b = np.array([4.0, 6.0, 3.0])
    # two rows: each is (a - b)/2 away from the mean, ||.||_F = ||a - b|| / sqrt 2 = 5 / sqrt 2
    assert metrics.consensus_distance(np.stack([a, b])) == pytest.approx(5.0 / math.sqrt(2.0), rel=1e-15)
    # three rows (0), (3), (6) in one column: deviations -3, 0, 3
    assert metrics.consensus_distance(np.array([[0.0], [3.0], [6.0]])) == pytest.approx(math.sqrt(18.0), rel=1e-15)


def test_consensus_bound_is_geometric():
    assert metrics.consensus_bound(2.0, 0.5, 3) == 0.25


def _shard_dense():
    X = np.array([[1.0, 0.0], [0.0, 2.0]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    return ("dense", X, y)


def test_mean_objective_hand_computed():
    # w = (1, 0.5): margins m = (1, 1), y m = (1, -1)
    w = np.array([1.0, 0.5])
    sh = _shard_dense()
    logistic = (math.log1p(math.exp(-1.0)) + math.log1p(math.exp(1.0))) / 2
    assert metrics.mean_objective(w, [sh], "logistic", 0.0) == pytest.approx(logistic, rel=1e-14)
    # hinge: max(0, 1 - 1) = 0 and max(0, 1 + 1) = 2, mean 1; l2/2 ||w||^2 = 0.1 * 1.25
    assert metrics.mean_objective(w, [sh], "hinge", 0.2) == pytest.approx(1.0 + 0.125, rel=1e-14)
    # the same shard in CSR form gives the same value
    csr = ("csr", np.array([0, 1, 2]), np.array([0, 1], np.int32), np.array([1.0, 2.0], np.float32), sh[2])
    assert metrics.mean_objective(w, [csr], "hinge", 0.2) == pytest.approx(1.125, rel=1e-14)


def test_mean_objective_averages_workers():
    # one worker: F = f_1; two shards: the mean of the two private objectives
    w = np.array([0.3, -0.2])
    a = _shard_dense()
    b = ("dense", np.array([[2.0, 1.0]], np.float32), np.array([-1.0], np.float32))
    fa = metrics.mean_objective(w, [a], "logistic", 0.0)
    fb = math.log1p(math.exp(2.0 * 0.3 - 0.2))           # y m = -(0.6 - 0.2) = -0.4
    assert metrics.mean_objective(w, [b], "logistic", 0.0) == pytest.approx(fb, rel=1e-14)
    assert metrics.mean_objective(w, [a, b], "logistic", 0.0) == pytest.approx((fa + fb) / 2, rel=1e-14)
    assert metrics.mean_objective(w, [a, a, a], "logistic", 0.0) == pytest.approx(fa, rel=1e-14)
