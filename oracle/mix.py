"""Stochastic reduce (oracle, fp64).

Appendix A, update equation (A.2), second line: after its half-step every node
replaces its model by the average of the half-step models of its in-neighbours
(itself included).  With the weights of the mixing matrix P this is
W'[i] = sum_{j in N_in(i)} P_ij W[j]; Section 5 describes the same operation as
each replica averaging the models it received with its own.

Pins: dense P @ W through BLAS, the complete graph (every row becomes the exact
column mean, i.e. all-reduce averaging), identity P, preservation of the mean
of all models when P is doubly stochastic, and consensus decay at the rate set
by sigma_2(P) (the bound of the "Spectral Gap" paragraph).
"""
from __future__ import annotations

import numpy as np


def stochastic_reduce(W, ptr, idx, w) -> np.ndarray:
    """W' = P W over the CSR rows of P; W [n, D] any float dtype, result fp64."""
    W = np.asarray(W, np.float64)
    n = len(ptr) - 1
    out = np.zeros((n, W.shape[1]))
    for i in range(n):
        for p in range(ptr[i], ptr[i + 1]):
            out[i] += float(w[p]) * W[idx[p]]
    return out


def stochastic_reduce_rows(W_rows_of, ptr, idx, w, rows):
    """Only the listed output rows; W_rows_of(j) returns row j (any dtype)."""
    res = []
    for i in rows:
        acc = None
        for p in range(ptr[i], ptr[i + 1]):
            term = float(w[p]) * np.asarray(W_rows_of(int(idx[p])), np.float64)
            acc = term if acc is None else acc + term
        res.append(acc)
    return np.stack(res)
