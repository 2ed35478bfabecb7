"""Per-round metrics (oracle, fp64).

Appendix A states the problem as minimising the sum over nodes of the private
objectives f_i at a common point, and bounds the distance of P^t x from the
uniform vector by sigma_2(P)^t.  The metrics follow those two statements:

* F(w_bar) = (1/n) sum_i f_i(w_bar) at the mean model w_bar (the paper's sum
  up to the constant 1/n);
* mean_i f_i(w_i), each worker at its own model;
* the consensus distance ||W - 1 w_bar^T||_F;
* the mean model itself (preserved by a doubly-stochastic reduce).

Pins (tests/test_oracle_metrics.py): the mean and the consensus distance of
hand-built matrices whose values are worked out by hand (identical rows give
distance 0; two rows a, b give ||a - b|| / sqrt 2); F(w_bar) of one worker is
f_1 at its own model; F of identical shards is the shared f; hand-computed
logistic and hinge values of a two-sample shard.
"""
from __future__ import annotations

import numpy as np

from . import sgd


def mean_model(W) -> np.ndarray:
    return np.asarray(W, np.float64).mean(axis=0)


def consensus_distance(W) -> float:
    W = np.asarray(W, np.float64)
    return float(np.linalg.norm(W - W.mean(axis=0, keepdims=True)))


def consensus_bound(dev0: float, sigma2: float, t: int) -> float:
    """||W_t - 1 w_bar^T||_F <= sigma_2(P)^t ||W_0 - 1 w_bar^T||_F."""
    return dev0 * sigma2 ** t


def mean_objective(wbar, shards, loss: str, l2: float) -> float:
    """F(w) = (1/n) sum_i f_i(w) over the workers' shards, each
    ("dense", X, y) or ("csr", row_ptr, col, val, y) with local offsets."""
    tot = 0.0
    for sh in shards:
        if sh[0] == "dense":
            tot += sgd.objective_dense(wbar, sh[1], sh[2], loss, l2)
        else:
            tot += sgd.objective_csr(wbar, sh[1], sh[2], sh[3], sh[4], loss, l2)
    return tot / len(shards)
