#!/usr/bin/env python3
"""Throughput of the ASAP round on one MI355X.

A step is one round of the hot path over the whole synthetic workload: the
sample schedule, every worker's local SGD pass and the stochastic reduce
(Appendix A, update equation (A.2)).  Inputs are resident in HBM before the
timed region; K steps are bracketed by device synchronisation and timed with
the host clock, and each phase of each step is timed with HIP events on the
stream it runs on (medians are reported).  One JSON line is printed.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--degree D]

Default: every workload is measured.  The headline (`value`, `config`,
`roofline`, `cpu_baseline`) is the largest single-GPU workload with SGD,
`dense_lr_32w` (32 workers, dense logistic regression, D = 4096, 65536
samples each, 34.6 GB of rows per round); every workload, the headline
included, also has its own entry under `configs` (samples/s, or GB/s for the
mixing stress, with its roofline and the oracle's CPU rate).
`--workload NAME` measures one workload only.

Other modes: `--copy-probe GIB` runs a plain device copy of known size and
`--gather-probe GIB` a random 4-byte gather of known size (HBM counter
calibration); `--run-rounds` times the multi-round NOTIFY-ACK launch
beside stream-ordered rounds; `--converge R` runs the convergence-versus-
network-cost comparison of Section 6 on three graphs.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "worker-SGD samples/s; stochastic-reduce HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD public spec
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
CSRC = os.path.join(ROOT, "paper_1612_08608_amd", "csrc")
HEADLINE = "dense_lr_32w"
CSR_MEMBERS = 0  # --csr-members
# (entry name, workload, graph override, degree override)
ALL_CONFIGS = [
    ("ring8_dense_lr", "ring8_dense_lr", None, None),
    ("sparse_lr_64w", "sparse_lr_64w", None, None),
    ("sparse_svm_256w", "sparse_svm_256w", None, None),
    ("sparse_svm_256w_complete", "sparse_svm_256w", "complete", None),
    ("dense_lr_32w", "dense_lr_32w", None, None),
    ("mix_stress_1024w_d2", "mix_stress_1024w", None, 2),
    ("mix_stress_1024w_d4", "mix_stress_1024w", None, 4),
    ("mix_stress_1024w_d8", "mix_stress_1024w", None, 8),
    ("mix_stress_1024w_d16", "mix_stress_1024w", None, 16),
]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def sha256(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def host_cores():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def copy_probe(gib: int):
    import torch
    n = gib << 28  # floats
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(3):
        b.copy_(a)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / 3
    print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n, "launches": 3,
                      "ms_per_copy": ms, "GB/s": 8 * n / ms / 1e6}))


def gather_probe(gib: int):
    """A random 4-byte gather of known traffic (torch.index_select over a
    `gib` GiB fp32 array at 2^24 random positions): reads the int64 indices
    (8 B each, in order), one random 4-byte element per index, and writes 4 B
    per index.  Calibrates what the HBM byte counters report for random
    4-byte reads (the model gathers of the CSR pass)."""
    import torch
    n_src, n_idx = gib << 28, 1 << 24
    src = torch.ones(n_src, dtype=torch.float32, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    idx = torch.randint(0, n_src, (n_idx,), device="cuda", generator=g, dtype=torch.int64)
    out = torch.empty(n_idx, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(3):
        torch.index_select(src, 0, idx, out=out)
    t1.record()
    torch.cuda.synchronize()
    lines = torch.unique(idx // 32).numel()  # distinct 128-byte lines touched
    print(json.dumps({"gather_probe_indices": n_idx, "index_bytes": 8 * n_idx, "output_bytes": 4 * n_idx,
                      "distinct_128B_lines": lines, "launches": 3, "ms_per_gather": t0.elapsed_time(t1) / 3}))


def graph_for(wl):
    from paper_1612_08608_amd import asap
    if wl.graph == "ring":
        p, i = asap.asap_graph_ring(wl.n_workers)
    elif wl.graph == "complete":
        p, i = asap.asap_graph_complete(wl.n_workers)
    elif wl.graph == "root_expander":
        p, i = asap.asap_graph_root_expander(wl.n_workers)
    elif wl.graph == "chain":
        p, i = asap.asap_graph_chain(wl.n_workers)
    else:
        p, i = asap.asap_graph_random_regular(wl.n_workers, wl.degree, wl.seed)
    return p, i, asap.asap_metropolis_weights(p, i)


# ----------------------------------------------------------------------------
# algorithmic bytes
# ----------------------------------------------------------------------------
def dense_bytes(wl):
    """One SGD launch (a whole pass of every worker): each sample row and
    label once, plus the model read and written once per minibatch step;
    second figure adds a 4-byte schedule entry per sample."""
    n, S, B, D = wl.n_workers, wl.samples, wl.batch, wl.dim
    K = -(-S // B)
    alg = n * (S * (4 * D + 4) + K * 8 * D)
    return alg, alg + 4 * n * S


def csr_bytes(wl, rp, col, sample_workers=4):
    """One SGD launch: per nonzero its column, value and the model entry it
    reads (12 B), per sample its row offset and label (8 B).  Second figure
    adds a schedule entry and row descriptor per sample (8 B) and one 4-byte
    model write per distinct column per step (counted on a few workers for
    round 0 and scaled)."""
    from paper_1612_08608_amd import asap
    nnz_total = int(rp[-1])
    n, S, B, D = wl.n_workers, wl.samples, wl.batch, wl.dim
    alg = 12 * nnz_total + 8 * n * S
    uniq = 0
    for k in range(sample_workers):
        sched = asap.asap_schedule(S, wl.seed, k, 0)
        rows = k * S + sched.astype(np.int64)
        lens = rp[rows + 1] - rp[rows]
        step = np.repeat(np.arange(S) // B, lens)
        pos = np.arange(lens.sum()) - np.repeat(np.cumsum(lens) - lens, lens) + np.repeat(rp[rows], lens)
        uniq += np.unique(step.astype(np.int64) * D + col[pos]).size
    return alg, alg + 8 * n * S + 4 * uniq * n / sample_workers


SYNTH = os.path.join(ROOT, "paper_1612_08608_amd", "synth.py")


def traffic_for(kernel_key, source):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source or different data
    (the generator of the synthetic inputs)."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        tab = json.load(f)
    ent = tab.get(kernel_key)
    if not ent or ent.get("source_sha256") != sha256(source) or ent.get("data_sha256") != sha256(SYNTH):
        return None
    return ent["fetch_bytes"] + ent["write_bytes"]


def roofline(kernel, source, key, ms, alg, alg_wide):
    ach = alg / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBPS,
            "traffic": traffic_for(key, source), "kernel": kernel, "algorithmic_bytes": alg,
            "launch_ms_median": ms, "bytes_incl_schedule_and_writes": alg_wide,
            "frac_incl_schedule_and_writes": alg_wide / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}


# ----------------------------------------------------------------------------
# the oracle on the host cores (a reported baseline, never the target)
# ----------------------------------------------------------------------------
def _oracle_kw(wl):
    return dict(batch=wl.batch, loss=wl.loss, lr_kind=wl.lr_kind, lr0=float(np.float32(wl.lr0)),
                l2=float(np.float32(wl.l2)), rnd=0)


def _baseline(value, unit, sample):
    return {"value": value, "unit": unit, "cores": 1, "kind": "oracle", "sample": sample,
            "cpu_model": cpu_model(), "host_cores_available": host_cores()}


def cpu_baseline_csr(wl, shards, p, i, w, budget_s):
    """Round-0 SGD passes of the first workers until ~budget_s, plus their
    reduce rows (the oracle, NumPy fp64, one thread)."""
    import oracle
    t0 = time.perf_counter()
    halves = {}
    while len(halves) < len(shards) and time.perf_counter() - t0 < budget_s:
        k = len(halves)
        _, rpk, ck, vk, yk = shards[k]
        halves[k] = oracle.sgd.sgd_pass_csr(np.zeros(wl.dim), rpk, ck, vk, yk,
                                            oracle.prng.schedule(wl.samples, wl.seed, k, 0), **_oracle_kw(wl))
    t_sgd = time.perf_counter() - t0
    done = len(halves)
    t1 = time.perf_counter()
    oracle.mix.stochastic_reduce_rows(lambda j: halves.get(j, halves[0]), p, i, w, list(range(done)))
    dt = t_sgd + time.perf_counter() - t1
    return _baseline(done * wl.samples / dt, "samples/s",
                     f"{done} of {wl.n_workers} workers' round-0 SGD passes ({done * wl.samples} samples) and "
                     f"their {done} reduced rows (rows of workers not run stand in for their inputs), "
                     f"single-threaded NumPy fp64, {dt:.1f} s")


def cpu_baseline_dense(wl, budget_s, rounds_per_shard=16):
    """SGD passes of the first workers until ~budget_s: each worker's passes
    of rounds 0, 1, ... (chained from a zero model, up to rounds_per_shard),
    then the next worker.  A shard is generated before its passes, outside
    the timing (generating a shard takes longer than a pass on it)."""
    import oracle
    from paper_1612_08608_amd import synth
    planted = synth.dense_planted(wl)
    dt = 0.0
    workers = passes = 0
    wall0 = time.perf_counter()
    while workers < wl.n_workers and dt < budget_s and time.perf_counter() - wall0 < 3 * budget_s:
        X, y = synth.dense_shard(wl, workers, planted)
        w = np.zeros(wl.dim)
        for r in range(rounds_per_shard):
            if dt >= budget_s:
                break
            t0 = time.perf_counter()
            kw = dict(_oracle_kw(wl), rnd=r)
            w = oracle.sgd.sgd_pass_dense(w, X, y, oracle.prng.schedule(wl.samples, wl.seed, workers, r), **kw)
            dt += time.perf_counter() - t0
            passes += 1
        workers += 1
    return _baseline(passes * wl.samples / dt, "samples/s",
                     f"{passes} SGD passes ({passes * wl.samples} samples): rounds 0.. of the first {workers} of "
                     f"{wl.n_workers} workers, each chained from a zero model without the reduce, NumPy fp64 with "
                     f"BLAS limited to one thread, {dt:.1f} s")


def cpu_baseline_mix(wl, p, i, w, budget_s):
    import oracle
    from paper_1612_08608_amd import synth
    cols = np.arange(1 << 14)
    W = synth.initial_models(wl, cols=cols).astype(np.float64)
    t0 = time.perf_counter()
    rounds = 0
    while rounds == 0 or time.perf_counter() - t0 < budget_s:
        W = oracle.mix.stochastic_reduce(W, p, i, w)
        rounds += 1
    dt = time.perf_counter() - t0
    return _baseline(rounds * 2 * wl.n_workers * cols.size * 4 / dt / 1e9, "GB/s",
                     f"{rounds} reduce rounds of all {wl.n_workers} workers on a {cols.size}-column slice of the "
                     f"{wl.dim}-column models (fp32-equivalent compulsory bytes), single-threaded NumPy fp64, "
                     f"{dt:.1f} s")


# ----------------------------------------------------------------------------
# one workload
# ----------------------------------------------------------------------------
def workload(name, graph=None, degree=None):
    from paper_1612_08608_amd import synth
    wl = synth.WORKLOADS[name]
    if graph:
        wl = wl.with_(graph=graph)
    if degree:
        wl = wl.with_(degree=degree)
    return wl


def measure(entry, wl, steps, warmup, cpu_budget, torch):
    """Set up `wl` resident in HBM, run `warmup` rounds, time `steps` rounds.
    Returns the entry's result dict."""
    from threadpoolctl import threadpool_limits
    from paper_1612_08608_amd import asap, synth
    p, i, w = graph_for(wl)
    log(f"[bench] {entry}: n={wl.n_workers} D={wl.dim} S={wl.samples} B={wl.batch} graph={wl.graph} "
        f"d={wl.degree}")
    t0 = time.perf_counter()
    sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
    cpu_in = None
    if wl.features == "csr":
        rp, col, val, y = synth.csr_data(wl)
        sess.bind_csr(rp, col, val, y, wl.samples)
        if CSR_MEMBERS:
            sess.set_csr_members(CSR_MEMBERS)
        members = sess.csr_members()
        alg, alg_wide = csr_bytes(wl, rp, col)
        S = wl.samples
        cpu_in = [("csr", rp[k * S:(k + 1) * S + 1] - rp[k * S], col[rp[k * S]:rp[(k + 1) * S]],
                   val[rp[k * S]:rp[(k + 1) * S]], y[k * S:(k + 1) * S]) for k in range(min(8, wl.n_workers))]
        max_row = int(np.diff(rp).max())
        del rp, col, val, y
    elif wl.features == "dense":
        X, y = synth.dense_data(wl)
        sess.bind_dense(X, y)
        alg, alg_wide = dense_bytes(wl)
        del X, y
    else:
        sess.set_models(synth.initial_models(wl))
        alg = alg_wide = 2 * wl.n_workers * wl.dim * 4
    sess.ready()
    torch.cuda.synchronize()
    log(f"[bench] {entry}: inputs resident in HBM after {time.perf_counter() - t0:.1f} s")

    prm = asap.sgd_params(wl.loss, wl.lr_kind, wl.lr0, wl.l2, wl.batch, wl.seed) if wl.features != "none" else None
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if prm is not None:
            # the round's schedule and plan first (or the wait for the plan
            # made during the previous round), so that the event pair
            # brackets the SGD kernels alone
            sess.prepare_sgd(prm)
            if ev:
                ev[0].record(stream)
            sess.local_sgd(prm)
        if ev:
            ev[1].record(stream)
        sess.stochastic_reduce()
        if ev:
            ev[2].record(stream)

    for _ in range(warmup):
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    st, bad = sess.check()
    if st != asap.OK:
        raise RuntimeError(f"{entry}: epoch-tag check failed during the benchmark (worker {bad})")
    sess.close()
    del sess
    torch.cuda.empty_cache()
    sgd_ms = float(np.median([e[0].elapsed_time(e[1]) for e in evs])) if prm is not None else 0.0
    mix_ms = float(np.median([e[1].elapsed_time(e[2]) for e in evs]))
    log(f"[bench] {entry}: {steps} steps in {wall:.3f} s; median SGD phase {sgd_ms:.3f} ms, "
        f"reduce {mix_ms:.3f} ms per step")

    n, D = wl.n_workers, wl.dim
    mix_bytes = 2 * n * D * 4
    mix_gbps = mix_bytes / (mix_ms * 1e-3) / 1e9
    reduce_key = "mix_slab_kernel" if wl.graph != "complete" else "mean_kernel"
    res = {"ms_per_step": wall / steps * 1e3, "steps": steps, "warmup": warmup}
    res["reduce"] = {"GB/s": mix_gbps, "frac_of_hbm_peak": mix_gbps / HBM_PEAK_GBPS, "ms_median": mix_ms,
                     "algorithmic_bytes": mix_bytes}
    cfg = {"workload": wl.name, "workers": n, "dim": D, "graph": wl.graph}
    if wl.graph == "random_regular":
        cfg["degree"] = wl.degree
    with threadpool_limits(1):
        if wl.features == "none":
            res.update(value=mix_gbps, unit="GB/s", higher_is_better=True)
            res["roofline"] = roofline(reduce_key, os.path.join(CSRC, "kernels_mix.hip"),
                                       f"mix_kernel@{wl.name}_d{wl.degree}", mix_ms, mix_bytes, mix_bytes)
            if cpu_budget > 0:
                res["cpu_baseline"] = cpu_baseline_mix(wl, p, i, w, cpu_budget)
        else:
            samples = n * wl.samples
            res.update(value=samples * steps / wall, unit="samples/s", higher_is_better=True)
            res["sgd_samples_per_s"] = samples / (sgd_ms * 1e-3)
            cfg.update(samples_per_worker=wl.samples, batch=wl.batch, loss=wl.loss, features=wl.features)
            if wl.features == "csr":
                # the planned pass takes minibatches of up to 64 rows of up to
                # 128 nonzeros; anything else runs the general kernel
                if wl.batch <= 64 and max_row <= 128:
                    kernel, src = "sgd_csr_fast_kernel", os.path.join(CSRC, "kernels_csr_plan.hip")
                else:
                    kernel, src = "sgd_csr_kernel", os.path.join(CSRC, "kernels_csr.hip")
                cfg["mean_nnz_per_row"] = (alg - 8 * samples) / 12 / samples
                cfg["pass_workgroups_per_worker"] = members
            elif 1024 < D <= 8192:
                kernel, src = "sgd_dense_wide_kernel", os.path.join(CSRC, "kernels_dense.hip")
            else:
                kernel, src = "sgd_dense_kernel", os.path.join(CSRC, "kernels_sgd.hip")
            key = f"{kernel}@{wl.name}" + ("_complete" if wl.graph == "complete" else "")
            res["roofline"] = roofline(kernel, src, key, sgd_ms, alg, alg_wide)
            if cpu_budget > 0:
                if wl.features == "csr":
                    res["cpu_baseline"] = cpu_baseline_csr(wl, cpu_in, p, i, w, cpu_budget)
                else:
                    res["cpu_baseline"] = cpu_baseline_dense(wl, cpu_budget)
    res["config"] = cfg
    return res


# ----------------------------------------------------------------------------
# other modes
# ----------------------------------------------------------------------------
def converge(wl, rounds, scale):
    """Loss F(w_bar) and consensus distance after every round on three graphs
    of Figure 2 (all-reduce, root expander, chain), and the bytes a worker
    sends per round (its out-degree times the model), as in the convergence-
    versus-network-cost comparisons of Section 6.  `scale` > 1 divides the
    workload's samples and dimension."""
    from paper_1612_08608_amd import asap, synth
    if scale > 1:
        wl = wl.with_(samples=max(wl.samples // scale, wl.batch), dim=max(wl.dim // scale, 64))
    out = {"metric": "loss F(w_bar) per round and bytes sent per worker", "workload": wl.name,
           "workers": wl.n_workers, "dim": wl.dim, "samples_per_worker": wl.samples, "graphs": {}}
    data = synth.csr_data(wl) if wl.features == "csr" else synth.dense_data(wl)
    for g in ("complete", "root_expander", "chain"):
        gw = wl.with_(graph=g)
        p, i, w = graph_for(gw)
        sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
        if wl.features == "csr":
            sess.bind_csr(*data, wl.samples)
            if CSR_MEMBERS:
                sess.set_csr_members(CSR_MEMBERS)
        else:
            sess.bind_dense(*data)
        prm = asap.sgd_params(wl.loss, wl.lr_kind, wl.lr0, wl.l2, wl.batch, wl.seed)
        losses, local, spread = [], [], []
        for _ in range(rounds):
            sess.round(prm)
            m = sess.metrics(wl.loss, wl.l2)
            local.append(float(m[0]))
            losses.append(float(m[1]))
            spread.append(float(m[2]))
        st, _ = sess.check()
        sess.close()
        if st != asap.OK:
            raise RuntimeError(f"epoch-tag check failed on {g}")
        out_degree = int(p[1] - p[0]) - 1  # every builder here is regular
        P = np.zeros((wl.n_workers, wl.n_workers))
        for r in range(wl.n_workers):
            P[r, i[p[r]:p[r + 1]]] = w[p[r]:p[r + 1]]
        sv = np.linalg.svd(P, compute_uv=False)
        # consensus decay per round against the bound sigma_2 of the mixing
        # alone (the local passes push the models apart again every round)
        decay = [spread[r] / spread[r - 1] if spread[r - 1] > 0 else None for r in range(1, rounds)]
        out["graphs"][g] = {"spectral_gap": 1.0 - float(sv[1]), "sigma2": float(sv[1]), "out_degree": out_degree,
                            "bytes_per_worker_per_round": out_degree * wl.dim * 4, "loss": losses,
                            "mean_local_loss": local, "consensus_distance": spread, "consensus_ratio": decay}
        log(f"[converge] {g}: gap {1.0 - float(sv[1]):.4f}, F(w_bar) after {rounds} rounds {losses[-1]:.6f}, "
            f"mean f_i(w_i) {local[-1]:.6f}, consensus distance {spread[-1]:.4e}")
    # rounds and bytes each worker sends before a loss first reaches a
    # target: the complete graph's value after a quarter of the rounds
    for key, name in (("loss", "F(w_bar)"), ("mean_local_loss", "mean_i f_i(w_i)")):
        target = out["graphs"]["complete"][key][max(0, rounds // 4 - 1)]
        out.setdefault("targets", {})[name] = target
        for g, rec in out["graphs"].items():
            hit = next((r for r, f in enumerate(rec[key]) if f <= target), None)
            rec.setdefault("rounds_to_target", {})[name] = None if hit is None else hit + 1
            rec.setdefault("bytes_per_worker_to_target", {})[name] = (
                None if hit is None else (hit + 1) * rec["bytes_per_worker_per_round"])
    print(json.dumps(out), flush=True)


def run_rounds_bench(name, wl, args, torch):
    """K rounds stream-ordered (asap_prepare_sgd / asap_local_sgd /
    asap_stochastic_reduce per round), then K rounds as one multi-round
    launch from the state they left; both timed by the host clock between
    device synchronisations."""
    from paper_1612_08608_amd import asap, synth
    p, i, w = graph_for(wl)
    sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
    if wl.features == "csr":
        sess.bind_csr(*synth.csr_data(wl), wl.samples)
        if CSR_MEMBERS:
            sess.set_csr_members(CSR_MEMBERS)
    else:
        sess.bind_dense(*synth.dense_data(wl))
    prm = asap.sgd_params(wl.loss, wl.lr_kind, wl.lr0, wl.l2, wl.batch, wl.seed)
    K = args.steps
    planned = wl.features == "csr" and wl.batch <= 64
    if planned:
        # plans for every pass of the launches below, so that the launch runs
        # the planned pass as the stream-ordered rounds do
        sess.bind_rounds_plan(K)

    def step():
        sess.prepare_sgd(prm)
        sess.local_sgd(prm)
        sess.stochastic_reduce()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    stream_s = time.perf_counter() - t0
    sess.run_rounds(prm, 1)  # first launch of the kernel (code object load) outside the timing
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sess.run_rounds(prm, K)
    torch.cuda.synchronize()
    launch_s = time.perf_counter() - t0
    st, bad = sess.check()
    sess.close()
    if st != asap.OK:
        raise RuntimeError(f"multi-round launch reported a stale neighbour (worker {bad})")
    samples = wl.n_workers * wl.samples
    out = {"metric": "rounds/s, one multi-round launch vs stream-ordered rounds", "mode": "notify_ack",
           "n_gpus": 1, "steps": K, "warmup": args.warmup, "dtype": "f32", "data": "synthetic",
           "higher_is_better": True,
           "config": {"workload": name, "workers": wl.n_workers, "dim": wl.dim, "samples_per_worker": wl.samples,
                      "batch": wl.batch, "graph": wl.graph, "degree": wl.degree},
           "stream_ms_per_round": stream_s / K * 1e3, "launch_ms_per_round": launch_s / K * 1e3,
           "stream_samples_per_s": samples * K / stream_s, "launch_samples_per_s": samples * K / launch_s,
           "speedup": stream_s / launch_s,
           "sgd_code": "planned CSR pass (plan ring bound)" if planned else
                       ("general CSR pass" if wl.features == "csr" else "dense pass")}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="all",
                    choices=["all", "sparse_lr_64w", "ring8_dense_lr", "sparse_svm_256w", "sparse_svm_256w_complete",
                             "dense_lr_32w", "mix_stress_1024w"])
    ap.add_argument("--degree", type=int, default=None, help="graph degree override (mixing stress: 2, 4, 8, 16)")
    ap.add_argument("--graph", default=None, choices=["ring", "complete", "random_regular", "root_expander", "chain"],
                    help="communication graph override")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="budget of each workload's oracle CPU leg (0: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--converge", type=int, default=0, metavar="ROUNDS",
                    help="instead of timing: loss and consensus distance per round on the complete, root-expander "
                         "and chain graphs, and the bytes each worker sends to reach a target loss")
    ap.add_argument("--converge-scale", type=int, default=1,
                    help="divide the workload's samples and dimension by this for --converge")
    ap.add_argument("--run-rounds", action="store_true",
                    help="instead of the headline line: time the rounds as one multi-round launch "
                         "(asap_run_rounds, per-worker NOTIFY-ACK) beside the same rounds stream-ordered")
    ap.add_argument("--csr-members", type=int, default=0, choices=[0, 1, 2, 4],
                    help="workgroups per worker of the planned CSR pass (0: the library's choice)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="GIB")
    ap.add_argument("--gather-probe", type=int, default=0, metavar="GIB")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: every logical worker runs on a single MI355X "
              "and there is no multi-GPU path (--gpus 1 only)", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gather_probe:
        gather_probe(args.gather_probe)
        return

    import torch
    from paper_1612_08608_amd import asap

    global CSR_MEMBERS
    CSR_MEMBERS = args.csr_members
    asap.lib()  # fail loudly without the HIP library
    cpu_budget = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    if args.workload == "all":
        if args.converge or args.run_rounds or args.graph or args.degree:
            raise SystemExit("--converge, --run-rounds, --graph and --degree need --workload")
        todo = ALL_CONFIGS
    else:
        base = "sparse_svm_256w" if args.workload == "sparse_svm_256w_complete" else args.workload
        g = "complete" if args.workload == "sparse_svm_256w_complete" else args.graph
        wl = workload(base, g, args.degree)
        if args.converge:
            converge(wl, args.converge, args.converge_scale)
            return
        if args.run_rounds:
            run_rounds_bench(args.workload, wl, args, torch)
            return
        entry = args.workload + (f"_d{args.degree}" if args.degree else "") + (f"_{args.graph}" if args.graph else "")
        todo = [(entry, base, g, args.degree)]

    results, failed = {}, []
    for entry, base, g, d in todo:
        try:
            results[entry] = measure(entry, workload(base, g, d), args.steps, args.warmup, cpu_budget, torch)
        except Exception as e:  # noqa: BLE001 -- recorded in the line, and the exit status says so
            log(f"[bench] {entry} FAILED: {e!r}")
            results[entry] = {"error": repr(e)}
            failed.append(entry)
    head_name = HEADLINE if args.workload == "all" else todo[0][0]
    head = results[head_name]
    out = {"metric": METRIC, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": head.get("ms_per_step"), "value": head.get("value"), "unit": head.get("unit"),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (seeded; shaped like the paper's linear workloads)",
           "config": head.get("config"), "roofline": head.get("roofline")}
    if "cpu_baseline" in head:
        out["cpu_baseline"] = head["cpu_baseline"]
    if "sgd_samples_per_s" in head:
        out["sgd_samples_per_s"] = head["sgd_samples_per_s"]
    if "reduce" in head:
        out["reduce"] = head["reduce"]
    out["configs"] = results
    print(json.dumps(out), flush=True)
    if failed:
        sys.exit(1)


if __name__ == "__main__":
    main()
