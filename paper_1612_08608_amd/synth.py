"""Seeded synthetic inputs for the ASAP hot path.

This module only *draws data*: feature shards, labels, planted models and the
initial model matrix of the mixing stress test.  It holds none of the method's
arithmetic (no SGD step, no loss derivative, no mixing, no graph, no sample
schedule), so both sides of every parity check -- the CPU oracle and the HIP
library -- can take their inputs from it without sharing any of the method.

The shapes follow the paper's linear workloads (Section 6: SVM-SGD on large
sparse text data such as RCV1, webspam and splice-site).  Those datasets are not
available here; the synthetic shards below stand in for them:

* dense shards: x ~ N(0, I) (optionally a fixed subset of columns scaled x10),
  labels y = sign(<x, w*>) with sign(0) = +1 and i.i.d. label flips;
* CSR shards: per row k = min(max(Poisson(lambda), 1), D) nonzeros, so that a
  row's nonzero count follows Poisson(lambda); the columns are the first k
  distinct ones of the row's stream of draws, ranks from a Zipf(s) law
  truncated to [1, D], mapped to columns by the bijection
  col = ((rank - 1) * 2654435761) mod D, then sorted; values are
  lognormal(0, 1) per column or 1 (binary); each row is L2-normalised;
  labels from a planted w* ~ N(0, I) as above.

Every worker's shard is a pure function of (seed, worker), so any worker can be
regenerated alone (the 32-worker dense workload holds 32 GiB of features).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

# Multiplier of the rank -> column scramble; an odd prime, so it is a bijection
# modulo any D it does not divide (in particular every power of two).
RANK_SCRAMBLE = 2654435761

# Stream tags of numpy SeedSequence entropy; keep data streams apart.
_TAG_DENSE = 0xD0
_TAG_CSR = 0xC5
_TAG_MODELS = 0x30


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: worker count, model size, data shape, SGD knobs."""

    name: str
    n_workers: int
    dim: int
    samples: int            # samples per worker
    batch: int
    loss: str               # "logistic" | "hinge" | "none" (mixing only)
    lr_kind: str            # "const" | "inv_sqrt"
    lr0: float
    l2: float
    rounds: int
    graph: str              # "ring" | "random_regular" | "complete"
    degree: int = 2
    features: str = "dense"  # "dense" | "csr" | "none"
    flip: float = 0.05
    scaled_frac: float = 0.0  # dense: fraction of columns scaled x10
    nnz_mean: float = 0.0     # csr: Poisson mean of nonzeros per row
    zipf_s: float = 1.0       # csr: Zipf exponent of column ranks
    values: str = "lognormal"  # csr: "lognormal" | "binary"
    seed: int = 0

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


RING8_DENSE_LR = Workload(
    name="ring8_dense_lr", n_workers=8, dim=64, samples=1024, batch=16,
    loss="logistic", lr_kind="const", lr0=0.1, l2=0.0, rounds=20,
    graph="ring", degree=2, features="dense", flip=0.05)

SPARSE_LR_64W = Workload(
    name="sparse_lr_64w", n_workers=64, dim=1 << 20, samples=20480, batch=64,
    loss="logistic", lr_kind="inv_sqrt", lr0=0.5, l2=0.0, rounds=50,
    graph="random_regular", degree=4, features="csr", flip=0.05,
    nnz_mean=80.0, zipf_s=1.1, values="lognormal")

SPARSE_SVM_256W = Workload(
    name="sparse_svm_256w", n_workers=256, dim=1 << 18, samples=8192, batch=32,
    loss="hinge", lr_kind="inv_sqrt", lr0=0.5, l2=1e-5, rounds=50,
    graph="random_regular", degree=8, features="csr", flip=0.05,
    nnz_mean=40.0, zipf_s=1.2, values="binary")

DENSE_LR_32W = Workload(
    name="dense_lr_32w", n_workers=32, dim=4096, samples=65536, batch=256,
    loss="logistic", lr_kind="const", lr0=0.05, l2=0.0, rounds=30,
    graph="random_regular", degree=6, features="dense", flip=0.02,
    scaled_frac=0.1)

MIX_STRESS_1024W = Workload(
    name="mix_stress_1024w", n_workers=1024, dim=1 << 20, samples=0, batch=1,
    loss="none", lr_kind="const", lr0=0.0, l2=0.0, rounds=100,
    graph="random_regular", degree=4, features="none")

WORKLOADS = {w.name: w for w in (RING8_DENSE_LR, SPARSE_LR_64W, SPARSE_SVM_256W,
                                 DENSE_LR_32W, MIX_STRESS_1024W)}


def _pool_size() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return max(1, min(16, os.cpu_count() or 1))


def _signed_labels(margin: np.ndarray, flips: np.ndarray) -> np.ndarray:
    y = np.where(margin >= 0.0, 1.0, -1.0)
    y[flips] = -y[flips]
    return y.astype(np.float32)


# ----------------------------------------------------------------------------
# dense shards
# ----------------------------------------------------------------------------
def dense_planted(wl: Workload):
    """Planted model w* (fp64) and the indices of the x10 columns."""
    rng = np.random.default_rng([wl.seed, _TAG_DENSE, 0])
    wstar = rng.standard_normal(wl.dim)
    n_scaled = int(round(wl.scaled_frac * wl.dim))
    scaled = np.sort(rng.permutation(wl.dim)[:n_scaled]) if n_scaled else np.zeros(0, np.int64)
    return wstar, scaled


def dense_shard(wl: Workload, worker: int, planted=None):
    """Worker's dense shard: X [S, D] fp32 row-major, y [S] fp32 in {-1, +1}."""
    wstar, scaled = planted if planted is not None else dense_planted(wl)
    rng = np.random.default_rng([wl.seed, _TAG_DENSE, 1, worker])
    X = rng.standard_normal((wl.samples, wl.dim), dtype=np.float32)
    if scaled.size:
        X[:, scaled] *= np.float32(10.0)
    margin = X.astype(np.float64) @ wstar
    flips = rng.random(wl.samples) < wl.flip
    return X, _signed_labels(margin, flips)


def dense_data(wl: Workload, workers=None):
    """Stacked shards X [n, S, D], y [n, S] for the listed workers (default all)."""
    workers = range(wl.n_workers) if workers is None else list(workers)
    planted = dense_planted(wl)
    X = np.empty((len(workers), wl.samples, wl.dim), np.float32)
    y = np.empty((len(workers), wl.samples), np.float32)

    def fill(k_w):
        k, w = k_w
        X[k], y[k] = dense_shard(wl, w, planted)

    with ThreadPoolExecutor(_pool_size()) as ex:
        list(ex.map(fill, enumerate(workers)))
    return X, y


# ----------------------------------------------------------------------------
# CSR shards
# ----------------------------------------------------------------------------
def zipf_cdf(dim: int, s: float) -> np.ndarray:
    """CDF of Zipf(s) truncated to ranks 1..dim (fp64)."""
    w = np.arange(1, dim + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def csr_planted(wl: Workload) -> np.ndarray:
    rng = np.random.default_rng([wl.seed, _TAG_CSR, 0])
    return rng.standard_normal(wl.dim)


def csr_shard(wl: Workload, worker: int, cdf=None, wstar=None):
    """Worker's CSR shard with local offsets.

    Returns (row_ptr int64 [S+1], col int32 [nnz], val fp32 [nnz], y fp32 [S]).
    Columns are unique and ascending within each row.
    """
    D, S = wl.dim, wl.samples
    cdf = zipf_cdf(D, wl.zipf_s) if cdf is None else cdf
    wstar = csr_planted(wl) if wstar is None else wstar
    rng = np.random.default_rng([wl.seed, _TAG_CSR, 1, worker])
    k = np.minimum(np.maximum(rng.poisson(wl.nnz_mean, S), 1), D)

    def draw(m):
        rank = np.minimum(np.searchsorted(cdf, rng.random(m), side="right"), D - 1)  # rank - 1
        return (rank.astype(np.int64) * RANK_SCRAMBLE) % D

    # first pass: 2k + 32 draws per row; keep each row's first k distinct
    # columns in draw order
    pool = 2 * k + 32
    rows = np.repeat(np.arange(S, dtype=np.int64), pool)
    keys, first = np.unique(rows * D + draw(int(pool.sum())), return_index=True)
    urow = keys // D
    order = np.lexsort((first, urow))
    urow_o = urow[order]
    have = np.bincount(urow, minlength=S)
    start = np.concatenate([[0], np.cumsum(have)[:-1]])
    within = np.arange(keys.size) - start[urow_o]
    keep = order[within < k[urow_o]]
    keys = np.sort(keys[keep])
    # rows whose pool held fewer than k distinct columns draw on, one by one
    short = np.nonzero(have < k)[0]
    if short.size:
        extra = []
        for r in short:
            seen = list(dict.fromkeys(int(c) for c in np.sort(keys[keys // D == r]) - r * D))
            seen_set = set(seen)
            while len(seen) < k[r]:
                for c in draw(2 * int(k[r] - len(seen)) + 32):
                    if int(c) not in seen_set and len(seen) < k[r]:
                        seen_set.add(int(c))
                        seen.append(int(c))
            extra.append(np.int64(r) * D + np.array(seen, np.int64))
        keys = np.sort(np.concatenate([keys[~np.isin(keys // D, short)], *extra]))
    urow = keys // D
    col = (keys - urow * D).astype(np.int32)
    counts = np.bincount(urow, minlength=S)
    row_ptr = np.zeros(S + 1, np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    if wl.values == "lognormal":
        v = rng.lognormal(0.0, 1.0, col.size)
    else:
        v = np.ones(col.size)
    norm = np.sqrt(np.add.reduceat(v * v, row_ptr[:-1]))
    v = v / np.repeat(norm, counts)
    val = v.astype(np.float32)
    margin = np.add.reduceat(val.astype(np.float64) * wstar[col], row_ptr[:-1])
    flips = rng.random(S) < wl.flip
    return row_ptr, col, val, _signed_labels(margin, flips)


def csr_data(wl: Workload, workers=None):
    """Concatenated shards of the listed workers (default all), global offsets.

    Returns (row_ptr int64 [m*S+1], col int32, val fp32, y fp32 [m*S]) where
    worker k's rows are [k*S, (k+1)*S).
    """
    workers = range(wl.n_workers) if workers is None else list(workers)
    cdf = zipf_cdf(wl.dim, wl.zipf_s)
    wstar = csr_planted(wl)
    with ThreadPoolExecutor(_pool_size()) as ex:
        shards = list(ex.map(lambda w: csr_shard(wl, w, cdf, wstar), workers))
    nnz = np.array([s[1].size for s in shards], np.int64)
    base = np.concatenate([[0], np.cumsum(nnz)])
    S = wl.samples
    row_ptr = np.empty(len(shards) * S + 1, np.int64)
    for k, s in enumerate(shards):
        row_ptr[k * S:(k + 1) * S] = s[0][:-1] + base[k]
    row_ptr[-1] = base[-1]
    col = np.concatenate([s[1] for s in shards])
    val = np.concatenate([s[2] for s in shards])
    y = np.concatenate([s[3] for s in shards])
    return row_ptr, col, val, y


# ----------------------------------------------------------------------------
# initial models
# ----------------------------------------------------------------------------
def initial_models(wl: Workload, rows=None, cols=None) -> np.ndarray:
    """W0 ~ N(0, 1) fp32 [len(rows), D] (or only the listed columns).

    Row i is drawn from its own stream, so any row or column sample of the
    1024 x 2^20 stress matrix can be regenerated without the rest.
    """
    rows = range(wl.n_workers) if rows is None else list(rows)
    ncol = wl.dim if cols is None else len(cols)
    out = np.empty((len(rows), ncol), np.float32)

    def fill(k_i):
        k, i = k_i
        r = np.random.default_rng([wl.seed, _TAG_MODELS, i]).standard_normal(wl.dim, dtype=np.float32)
        out[k] = r if cols is None else r[cols]

    with ThreadPoolExecutor(_pool_size()) as ex:
        list(ex.map(fill, enumerate(rows)))
    return out
