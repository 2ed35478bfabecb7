#!/usr/bin/env python3
"""Write the full-size oracle trajectories the GPU parity tests compare with.

For each workload below this runs every round of the method on the CPU oracle
alone -- each worker's local pass (update (A.2), first line), then the
stochastic reduce (second line) -- from zero models, for the workload's full
data and rounds, and stores what a test can compare cheaply:

* ``loss[r]``      F(w_bar) after round r (Appendix A's objective at the mean
                   model), fp64;
* ``cons[r]``      the consensus distance ||W - 1 w_bar^T||_F after round r;
* ``mean[r]``      the mean of all model entries after round r;
* ``norms[r, i]``  ||w_i||_2 of every worker after round r;
* ``sample[r]``    W[rows][:, cols] after round r (4 rows x 256 columns);
* ``amb``          (round, worker, row) of every hinge decision within fp32
                   rounding of the kink (|y m - 1| <= 1e-5 (1 + sum |w_j x_j|)),
                   where a GPU run may legitimately decide the other way.

Only `oracle/` and the seeded generators of `paper_1612_08608_amd.synth` are
used; nothing here reads a GPU result.  The local passes and the reduce rows
run in worker processes (fork), the model matrices live in /dev/shm.

    python tests/golden/make_fullsize.py [NAME ...] [--procs 8]

NAME is one of sparse_lr_64w, sparse_svm_256w, sparse_svm_256w_complete,
dense_lr_32w (default: all).  Output: tests/golden/fullsize_<NAME>.npz.
"""
from __future__ import annotations

import os

for _v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_v] = "1"

import argparse  # noqa: E402
import multiprocessing as mp  # noqa: E402
import sys  # noqa: E402
import tempfile  # noqa: E402
import time  # noqa: E402

import numpy as np  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_1612_08608_amd import synth  # noqa: E402

N_ROWS, N_COLS = 4, 256

# (workload, graph kind, rounds)
CONFIGS = {
    "sparse_lr_64w": (synth.SPARSE_LR_64W, "random", 50),
    "sparse_svm_256w": (synth.SPARSE_SVM_256W, "random", 50),
    "sparse_svm_256w_complete": (synth.SPARSE_SVM_256W, "complete", 50),
    "dense_lr_32w": (synth.DENSE_LR_32W, "random", 30),
}

# state shared with the forked worker processes
G = {}


def _kw(wl):
    return dict(batch=wl.batch, loss=wl.loss, lr_kind=wl.lr_kind, lr0=float(np.float32(wl.lr0)),
                l2=float(np.float32(wl.l2)))


def _shard(k):
    wl = G["wl"]
    if wl.features == "dense":
        return ("dense", G["X"][k], G["y"][k])
    rp, col, val, y = G["data"]
    S = wl.samples
    lo, hi = rp[k * S], rp[(k + 1) * S]
    return ("csr", rp[k * S:(k + 1) * S + 1] - lo, col[lo:hi], val[lo:hi], y[k * S:(k + 1) * S])


def _pass(args):
    """Worker k's local pass of round r from W[k] into H[k]; returns its
    ambiguous hinge rows."""
    k, r = args
    wl = G["wl"]
    sh = _shard(k)
    sched = oracle.prng.schedule(wl.samples, wl.seed, k, r)
    W, H = G["W"], G["H"]
    if sh[0] == "dense":
        H[k] = oracle.sgd.sgd_pass_dense(W[k], sh[1], sh[2], sched, rnd=r, **_kw(wl))
        return k, []
    amb = []
    H[k] = oracle.sgd.sgd_pass_csr_scaled(W[k], sh[1], sh[2], sh[3], sh[4], sched, rnd=r, ambiguous=amb,
                                          **_kw(wl))
    return k, amb


def _reduce(rows):
    """Rows of the stochastic reduce W = P H."""
    p, i, w = G["graph"]
    H = G["H"]
    G["W"][rows] = oracle.mix.stochastic_reduce_rows(lambda j: H[j], p, i, w, rows)
    return len(rows)


def _objective(k):
    """f_k at the mean model (held in G['wbar'])."""
    wl = G["wl"]
    return k, oracle.metrics.mean_objective(np.asarray(G["wbar"]), [_shard(k)], wl.loss, float(np.float32(wl.l2)))


def sample_columns(wl, rng):
    if wl.features == "dense":
        return np.sort(rng.choice(wl.dim, N_COLS, replace=False))
    col = G["data"][1]
    picked = []
    while len(picked) < N_COLS:                          # nonzero-weighted: hot and rare columns
        for c in col[rng.integers(0, col.size, 4 * N_COLS)]:
            if int(c) not in picked:
                picked.append(int(c))
            if len(picked) == N_COLS:
                break
    return np.sort(np.asarray(picked, np.int64))


def run(name, procs):
    wl, kind, R = CONFIGS[name]
    t0 = time.time()
    n, D = wl.n_workers, wl.dim
    if kind == "complete":
        p, i = oracle.graphs.complete(n)
    else:
        p, i = oracle.graphs.random_regular(n, wl.degree, wl.seed)
    w = oracle.graphs.metropolis_weights(p, i)
    G.clear()
    G["wl"], G["graph"] = wl, (p, i, w)
    if wl.features == "dense":
        G["X"], G["y"] = synth.dense_data(wl)
    else:
        G["data"] = synth.csr_data(wl)
    print(f"[{name}] data ready in {time.time() - t0:.0f} s", flush=True)
    rng = np.random.default_rng(20240601)
    rows = np.linspace(0, n - 1, N_ROWS).round().astype(np.int64)
    cols = sample_columns(wl, rng)
    tmp = tempfile.mkdtemp(prefix="fullsize_", dir="/dev/shm")
    try:
        G["W"] = np.memmap(os.path.join(tmp, "W"), np.float64, "w+", shape=(n, D))
        G["H"] = np.memmap(os.path.join(tmp, "H"), np.float64, "w+", shape=(n, D))
        G["wbar"] = np.memmap(os.path.join(tmp, "wbar"), np.float64, "w+", shape=(D,))
        G["W"][:] = 0.0
        out = {k: [] for k in ("loss", "cons", "mean", "norms", "sample")}
        amb_all = []
        chunks = np.array_split(np.arange(n), min(n, 8 * procs))
        with mp.get_context("fork").Pool(procs) as pool:
            for r in range(R):
                t1 = time.time()
                for k, amb in pool.imap_unordered(_pass, [(k, r) for k in range(n)]):
                    amb_all += [(r, k, q) for q in amb]
                list(pool.imap_unordered(_reduce, [c.tolist() for c in chunks]))
                W = G["W"]
                G["wbar"][:] = oracle.metrics.mean_model(W)
                fk = dict(pool.imap_unordered(_objective, range(n)))
                tot = 0.0
                for k in range(n):                       # the sum of mean_objective, in worker order
                    tot += fk[k]
                out["loss"].append(tot / n)
                out["cons"].append(oracle.metrics.consensus_distance(W))
                out["mean"].append(float(np.asarray(W).mean()))
                out["norms"].append(np.linalg.norm(W, axis=1))
                out["sample"].append(np.asarray(W)[rows][:, cols])
                n_amb = sum(1 for a in amb_all if a[0] == r)
                print(f"[{name}] round {r}: F(w_bar) {out['loss'][-1]:.6f} consensus {out['cons'][-1]:.4e} "
                      f"ambiguous {n_amb} ({time.time() - t1:.1f} s)", flush=True)
    finally:
        for f in ("W", "H", "wbar"):
            try:
                os.remove(os.path.join(tmp, f))
            except FileNotFoundError:
                pass
        os.rmdir(tmp)
    path = os.path.join(HERE, f"fullsize_{name}.npz")
    np.savez_compressed(path, workload=wl.name, graph=kind, rounds=R, rows=rows, cols=cols,
                        loss=np.asarray(out["loss"]), cons=np.asarray(out["cons"]), mean=np.asarray(out["mean"]),
                        norms=np.stack(out["norms"]), sample=np.stack(out["sample"]),
                        amb=np.asarray(amb_all, np.int64).reshape(-1, 3))
    print(f"[{name}] wrote {path} ({os.path.getsize(path) / 1024:.0f} KiB) in {time.time() - t0:.0f} s", flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("names", nargs="*", default=list(CONFIGS))
    ap.add_argument("--procs", type=int, default=min(8, len(os.sched_getaffinity(0))))
    args = ap.parse_args()
    for name in args.names:
        run(name, args.procs)


if __name__ == "__main__":
    main()
