"""One ASAP round as Appendix A's update equation (A.2) states it (oracle).

Every worker first takes its local half-step (line one of (A.2): here a full
local SGD pass over its shard, Section 5), then every worker mixes the
half-step models of its in-neighbours (line two of (A.2), weights P).  The
half-step of one worker never reads another worker's model, so the order of
workers inside the half-step is immaterial; the reduce reads only half-step
models, which is what the NOTIFY-ACK protocol of Section 4 guarantees (no model
is overwritten before all of its readers consumed it).

The composition is generic over the half-step so that a test can force the
gradients (the unrolled form (A.3) with frozen g_t).
"""
from __future__ import annotations

import numpy as np

from . import prng, sgd
from .mix import stochastic_reduce


def half_step_then_reduce(W, half_step, ptr, idx, w):
    """(A.2): W_half[i] = half_step(i, W[i]); return (P W_half, W_half)."""
    W = np.asarray(W, np.float64)
    half = np.stack([half_step(i, W[i]) for i in range(W.shape[0])])
    return stochastic_reduce(half, ptr, idx, w), half


def local_pass(i, wi, shard, *, S, seed, rnd, batch, loss, lr_kind, lr0, l2):
    """Worker i's SGD pass of round rnd on its own shard (dense or CSR)."""
    sched = prng.schedule(S, seed, i, rnd)
    kw = dict(batch=batch, loss=loss, lr_kind=lr_kind, lr0=lr0, l2=l2, rnd=rnd)
    if shard[0] == "dense":
        _, X, y = shard
        return sgd.sgd_pass_dense(wi, X, y, sched, **kw)
    _, row_ptr, col, val, y = shard
    return sgd.sgd_pass_csr(wi, row_ptr, col, val, y, sched, **kw)


def asap_round(W, shards, ptr, idx, w, *, seed, rnd, batch, loss, lr_kind, lr0, l2):
    """One round over all workers; shards[i] = ("dense", X, y) or ("csr", rp, col, val, y)."""
    def hs(i, wi):
        S = shards[i][1].shape[0] if shards[i][0] == "dense" else len(shards[i][1]) - 1
        return local_pass(i, wi, shards[i], S=S, seed=seed, rnd=rnd, batch=batch,
                          loss=loss, lr_kind=lr_kind, lr0=lr0, l2=l2)
    return half_step_then_reduce(W, hs, ptr, idx, w)
