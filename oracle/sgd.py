"""Local minibatch SGD half-step of every worker (oracle, fp64).

Appendix A, update equation (A.2), first line: each node takes a gradient step
on its private objective f_i from its current model.  Section 5 runs that step
as SGD over a few examples of the node's own data partition before it
communicates; Section 6 uses an SVM trained with Bottou's SVM-SGD.

Reading used here (the paper fixes no minibatch rule, no logistic loss and no
step-size schedule; these come from the workload definitions):

* f_i(w) = mean over the shard of loss(y <x, w>) + (l2 / 2) ||w||^2;
* logistic loss = softplus(-y m), derivative c = -y sigmoid(-y m);
  hinge loss = max(0, 1 - y m), subgradient c = -y if y m < 1 else 0
  (zero at the kink);
* minibatch k of round r is positions [kB, min((k+1)B, S)) of the round's
  schedule; all margins use the pre-step model; the gradient is the batch mean
  (1/B') sum_b c_b x_b + l2 w; the update is w <- w - eta_t g with
  t = r * ceil(S / B) + k + 1 counted from 1 per worker across rounds, and
  eta_t = lr0 (constant) or lr0 / sqrt(t);
* one round = one full pass over the shard (local_steps = 0), or L
  minibatch steps of the sequence of passes (local_steps = L, L dividing the
  number of steps K of a pass; L = 1 is (A.2) as printed, one gradient step
  per mix): round r takes steps k0 .. k0 + L - 1 of pass q, with
  q = (r L) div K and k0 = (r L) mod K (`round_steps`), and t counts
  q K + k + 1.

With l2 > 0 the update multiplies every entry of w by (1 - eta_t l2) each
step.  `sgd_pass_csr_scaled` writes w = s v (Bottou's trick for SVM-SGD, which
Section 6 uses) so a step touches only the minibatch's columns: s <- s (1 -
eta_t l2), v_j <- v_j - (eta_t / s) g_j over the batch's columns.  It is the
same update up to fp64 rounding and exists to make full-size oracle runs fast.

Pins: closed forms at m = 0, central finite differences of the loss on tiny
inputs, a hand-computed step, the dense-vs-CSR agreement on the same data, the
scale form against the plain dense decay (1e-12).
"""
from __future__ import annotations

import math

import numpy as np

LOGISTIC = "logistic"
HINGE = "hinge"


def loss_value(margin_y: np.ndarray, loss: str) -> np.ndarray:
    """Per-sample loss as a function of y*m (fp64)."""
    if loss == LOGISTIC:
        return np.logaddexp(0.0, -margin_y)
    if loss == HINGE:
        return np.maximum(0.0, 1.0 - margin_y)
    raise ValueError(loss)


def loss_coef(m: np.ndarray, y: np.ndarray, loss: str) -> np.ndarray:
    """d loss(y m) / d m for each sample (hinge: zero at and beyond the kink)."""
    ym = y * m
    if loss == LOGISTIC:
        # -y * sigmoid(-y m), written without overflow for either sign of ym.
        e = np.exp(-np.abs(ym))
        sig_neg = np.where(ym >= 0, e / (1.0 + e), 1.0 / (1.0 + e))
        return -y * sig_neg
    if loss == HINGE:
        return np.where(ym < 1.0, -y, 0.0)
    raise ValueError(loss)


def step_size(lr_kind: str, lr0: float, t: int) -> float:
    if lr_kind == "const":
        return float(lr0)
    if lr_kind == "inv_sqrt":
        return float(lr0) / math.sqrt(t)
    raise ValueError(lr_kind)


def n_steps(S: int, B: int) -> int:
    return -(-S // B)


def round_steps(rnd: int, local_steps: int, K: int):
    """(pass q, first step k0, end step k1) of round rnd: the whole pass
    when local_steps == 0, else local_steps steps (which must divide K)."""
    if local_steps == 0:
        return rnd, 0, K
    if local_steps < 0 or K % local_steps:
        raise ValueError("local_steps must divide the steps of a pass")
    g = rnd * local_steps
    return g // K, g % K, g % K + local_steps


def sgd_pass_dense(w0, X, y, sched, *, batch, loss, lr_kind, lr0, l2, rnd, steps=None):
    """One local pass of one worker on dense data; returns the new model (fp64).

    w0 [D], X [S, D], y [S], sched = permutation of [0, S) (of pass rnd);
    steps = (k0, k1) runs only steps k0 .. k1 - 1 of the pass.
    """
    w = np.asarray(w0, np.float64).copy()
    y = np.asarray(y, np.float64)
    S = X.shape[0]
    K = n_steps(S, batch)
    k0, k1 = (0, K) if steps is None else steps
    for k in range(k0, k1):
        rows = sched[k * batch:min((k + 1) * batch, S)]
        xb, yb = np.asarray(X[rows], np.float64), y[rows]
        m = xb @ w
        c = loss_coef(m, yb, loss)
        g = (c @ xb) / len(rows) + l2 * w
        w = w - step_size(lr_kind, lr0, rnd * K + k + 1) * g
    return w


def sgd_pass_csr(w0, row_ptr, col, val, y, sched, *, batch, loss, lr_kind, lr0, l2, rnd,
                 ambiguous=None, steps=None):
    """One local pass of one worker on CSR data (local row offsets); fp64.

    The L2 term is applied densely every step, exactly as the update states.
    If `ambiguous` is a list, rows whose hinge decision y m < 1 lies within
    fp32 rounding of the kink (|y m - 1| <= 1e-5 (1 + sum_j |w_j x_j|)) at
    the step that uses them are appended to it.
    """
    w = np.asarray(w0, np.float64).copy()
    row_ptr = np.asarray(row_ptr, np.int64)
    S = len(row_ptr) - 1
    K = n_steps(S, batch)
    k0, k1 = (0, K) if steps is None else steps
    for k in range(k0, k1):
        rows = np.asarray(sched[k * batch:min((k + 1) * batch, S)], np.int64)
        lo, lens = row_ptr[rows], row_ptr[rows + 1] - row_ptr[rows]
        seg = np.repeat(np.arange(len(rows)), lens)               # pair -> position in batch
        pos = np.arange(lens.sum()) - np.repeat(np.cumsum(lens) - lens, lens) + np.repeat(lo, lens)
        cols, vals = col[pos], val[pos].astype(np.float64)
        prod = vals * w[cols]
        m = np.bincount(seg, weights=prod, minlength=len(rows))   # margins, pre-step w
        yb = y[rows].astype(np.float64)
        if ambiguous is not None and loss == HINGE:
            absum = np.bincount(seg, weights=np.abs(prod), minlength=len(rows))
            hit = np.abs(yb * m - 1.0) <= 1e-5 * (1.0 + absum)
            ambiguous.extend(int(r) for r in rows[hit])
        c = loss_coef(m, yb, loss)
        g = l2 * w
        np.add.at(g, cols, c[seg] * vals / len(rows))
        w = w - step_size(lr_kind, lr0, rnd * K + k + 1) * g
    return w


def sgd_pass_csr_scaled(w0, row_ptr, col, val, y, sched, *, batch, loss, lr_kind, lr0, l2, rnd,
                        ambiguous=None, steps=None):
    """`sgd_pass_csr` with w kept as s * v, so that the L2 decay of a step is
    one multiplication of s; returns the new model s * v (fp64).  The margins,
    the hinge ambiguity test and the data gradient are those of `sgd_pass_csr`
    evaluated at w = s v."""
    v = np.asarray(w0, np.float64).copy()
    s = 1.0
    row_ptr = np.asarray(row_ptr, np.int64)
    S = len(row_ptr) - 1
    K = n_steps(S, batch)
    k0, k1 = (0, K) if steps is None else steps
    for k in range(k0, k1):
        rows = np.asarray(sched[k * batch:min((k + 1) * batch, S)], np.int64)
        lo, lens = row_ptr[rows], row_ptr[rows + 1] - row_ptr[rows]
        seg = np.repeat(np.arange(len(rows)), lens)
        pos = np.arange(lens.sum()) - np.repeat(np.cumsum(lens) - lens, lens) + np.repeat(lo, lens)
        cols, vals = col[pos], val[pos].astype(np.float64)
        prod = vals * (s * v[cols])
        m = np.bincount(seg, weights=prod, minlength=len(rows))
        yb = y[rows].astype(np.float64)
        if ambiguous is not None and loss == HINGE:
            absum = np.bincount(seg, weights=np.abs(prod), minlength=len(rows))
            hit = np.abs(yb * m - 1.0) <= 1e-5 * (1.0 + absum)
            ambiguous.extend(int(r) for r in rows[hit])
        c = loss_coef(m, yb, loss)
        eta = step_size(lr_kind, lr0, rnd * K + k + 1)
        s = s * (1.0 - eta * l2)
        np.add.at(v, cols, -(eta / s) * (c[seg] * vals / len(rows)))
    return s * v


def objective_dense(w, X, y, loss, l2) -> float:
    """f_i(w) on a dense shard (fp64; the margins are formed 4096 rows at a
    time so that a large fp32 shard is never copied to fp64 whole)."""
    w = np.asarray(w, np.float64)
    m = np.empty(X.shape[0])
    for r0 in range(0, X.shape[0], 4096):
        m[r0:r0 + 4096] = np.asarray(X[r0:r0 + 4096], np.float64) @ w
    return float(np.mean(loss_value(np.asarray(y, np.float64) * m, loss))
                 + 0.5 * l2 * np.dot(w, w))


def margins_csr(w, row_ptr, col, val) -> np.ndarray:
    """<x_s, w> for every row of a CSR shard (fp64, library sparse product)."""
    import scipy.sparse as sp
    S = len(row_ptr) - 1
    A = sp.csr_matrix((np.asarray(val, np.float64), np.asarray(col, np.int64),
                       np.asarray(row_ptr, np.int64) - int(row_ptr[0])),
                      shape=(S, len(w)))
    return A @ np.asarray(w, np.float64)


def objective_csr(w, row_ptr, col, val, y, loss, l2) -> float:
    """f_i(w) on a CSR shard (fp64)."""
    w = np.asarray(w, np.float64)
    m = margins_csr(w, row_ptr, col, val)
    return float(np.mean(loss_value(np.asarray(y, np.float64) * m, loss))
                 + 0.5 * l2 * np.dot(w, w))
