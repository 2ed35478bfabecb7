"""Per-round metrics (oracle, fp64).

Appendix A states the problem as minimising the sum over nodes of the private
objectives f_i at a common point, and bounds the distance of P^t x from the
uniform vector by sigma_2(P)^t.  The metrics follow those two statements:

* F(w_bar) = (1/n) sum_i f_i(w_bar) at the mean model w_bar (the paper's sum
  up to the constant 1/n);
* mean_i f_i(w_i), each worker at its own model;
* the consensus distance ||W - 1 w_bar^T||_F;
* the mean model itself (preserved by a doubly-stochastic reduce).

Pins: consensus distance of identical rows is 0; F(w_bar) of a single worker
is f_1; both checked in the oracle tests.
"""
from __future__ import annotations

import numpy as np


def mean_model(W) -> np.ndarray:
    return np.asarray(W, np.float64).mean(axis=0)


def consensus_distance(W) -> float:
    W = np.asarray(W, np.float64)
    return float(np.linalg.norm(W - W.mean(axis=0, keepdims=True)))


def consensus_bound(dev0: float, sigma2: float, t: int) -> float:
    """||W_t - 1 w_bar^T||_F <= sigma_2(P)^t ||W_0 - 1 w_bar^T||_F."""
    return dev0 * sigma2 ** t
