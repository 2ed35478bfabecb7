#!/usr/bin/env python3
"""Throughput of the ASAP round on one MI355X.

A step is one round of the hot path over the whole synthetic workload: the
sample schedule, every worker's local SGD pass and the stochastic reduce
(Appendix A, update equation (A.2)).  Inputs are resident in HBM before the
timed region; K steps are bracketed by device synchronisation and timed with
the host clock, and each kernel phase is timed with HIP events on the stream
it runs on.  One JSON line is printed.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

Default workload: 64 workers, CSR logistic regression, D = 2^20, 20480
samples per worker, minibatch 64, lr 0.5/sqrt(t), random 4-regular graph.
`--copy-probe GIB` instead runs a plain device copy of known size (used to
calibrate the HBM byte counters of rocprofv3).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "worker-SGD samples/s; stochastic-reduce HBM GB/s (% of MI355X peak)"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD public spec
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def sha256(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


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


def graph_for(wl, d=None):
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
        p, i = asap.asap_graph_random_regular(wl.n_workers, wl.degree if d is None else d, wl.seed)
    return p, i, asap.asap_metropolis_weights(p, i)


def csr_algorithmic_bytes(wl, rp, col, sample_workers=4):
    """Bytes one SGD launch must move: per nonzero col + val + the model
    entry it reads (12 B), per sample row offset + label + schedule entry
    (16 B), and one 4-byte write per distinct column per minibatch step
    (measured on a few workers for round 0 and scaled)."""
    from paper_1612_08608_amd import asap
    nnz_total = int(rp[-1])
    n, S, B, D = wl.n_workers, wl.samples, wl.batch, wl.dim
    reads = 12 * nnz_total + 16 * n * S
    uniq = 0
    for k in range(sample_workers):
        sched = asap.asap_schedule(S, wl.seed, k, 0)
        rows = k * S + sched.astype(np.int64)
        lens = rp[rows + 1] - rp[rows]
        step = np.repeat(np.arange(S) // B, lens)
        pos = np.arange(lens.sum()) - np.repeat(np.cumsum(lens) - lens, lens) + np.repeat(rp[rows], lens)
        uniq += np.unique(step.astype(np.int64) * D + col[pos]).size
    writes = 4 * uniq * n / sample_workers
    return reads + writes, reads, writes


def cpu_baseline_csr(wl, rp, col, val, y, p, i, w, budget_s=15.0):
    """The oracle (NumPy fp64, one thread) on a bounded sample of the round:
    SGD passes of the first workers until ~budget_s, plus their reduce rows."""
    import oracle
    S = wl.samples
    kw = dict(batch=wl.batch, loss=wl.loss, lr_kind=wl.lr_kind, lr0=float(np.float32(wl.lr0)),
              l2=float(np.float32(wl.l2)), rnd=0)
    t0 = time.perf_counter()
    halves = {}
    done = 0
    while done < wl.n_workers and time.perf_counter() - t0 < budget_s:
        k = done
        lo = rp[k * S]
        halves[k] = oracle.sgd.sgd_pass_csr(np.zeros(wl.dim), rp[k * S:(k + 1) * S + 1] - lo,
                                            col[lo:rp[(k + 1) * S]], val[lo:rp[(k + 1) * S]],
                                            y[k * S:(k + 1) * S], oracle.prng.schedule(S, wl.seed, k, 0), **kw)
        done += 1
    t_sgd = time.perf_counter() - t0
    # reduce of `done` rows (neighbour rows stand in for unavailable half-steps)
    src = lambda j: halves.get(j, halves[0])
    t1 = time.perf_counter()
    oracle.mix.stochastic_reduce_rows(src, p, i, w, list(range(done)))
    t_mix = time.perf_counter() - t1
    return {"value": done * S / (t_sgd + t_mix), "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {wl.n_workers} workers' round-0 SGD passes ({done * S} samples) "
                      f"and their {done} reduced rows, single-threaded NumPy fp64; "
                      f"{t_sgd + t_mix:.1f} s on {platform.processor() or platform.machine()}"}


def cpu_baseline_dense(wl, X, y, budget_s=15.0):
    """The oracle (NumPy fp64) on the first workers' round-0 passes."""
    import oracle
    kw = dict(batch=wl.batch, loss=wl.loss, lr_kind=wl.lr_kind, lr0=float(np.float32(wl.lr0)),
              l2=float(np.float32(wl.l2)), rnd=0)
    t0 = time.perf_counter()
    done = 0
    while done < wl.n_workers and time.perf_counter() - t0 < budget_s:
        oracle.sgd.sgd_pass_dense(np.zeros(wl.dim), X[done], y[done],
                                  oracle.prng.schedule(wl.samples, wl.seed, done, 0), **kw)
        done += 1
    dt = time.perf_counter() - t0
    return {"value": done * wl.samples / dt, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {wl.n_workers} workers' round-0 SGD passes, NumPy fp64 "
                      f"(BLAS limited to one thread)"}


def cpu_baseline_mix(wl, p, i, w, budget_s=15.0):
    import oracle
    from paper_1612_08608_amd import synth
    cols = np.arange(1 << 14)
    W = synth.initial_models(wl, cols=cols).astype(np.float64)
    t0 = time.perf_counter()
    rounds = 0
    while time.perf_counter() - t0 < budget_s:
        W = oracle.mix.stochastic_reduce(W, p, i, w)
        rounds += 1
    dt = time.perf_counter() - t0
    gbps = rounds * 2 * wl.n_workers * cols.size * 4 / dt / 1e9
    return {"value": gbps, "unit": "GB/s (fp32-equivalent compulsory bytes)", "cores": 1, "kind": "oracle",
            "sample": f"{rounds} reduce rounds of all {wl.n_workers} workers on a {cols.size}-column slice "
                      f"(of {wl.dim}), single-threaded NumPy fp64"}


def traffic_for(kernel_key, source):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        tab = json.load(f)
    ent = tab.get(kernel_key)
    if not ent or ent.get("source_sha256") != sha256(source):
        return None
    return ent["fetch_bytes"] + ent["write_bytes"]


def converge(wl, rounds):
    """Loss F(w_bar) after every round on three graphs of Figure 2 (all-reduce,
    root expander, chain), and the bytes a worker sends per round (its
    out-degree times the model), as in the convergence-versus-network-cost
    comparisons of Section 6.  Synthetic data shaped like the workload, at
    1/16 of its samples and dimension so that each graph runs in seconds."""
    import torch
    from paper_1612_08608_amd import asap, synth
    wl = wl.with_(samples=max(wl.samples // 16, wl.batch), dim=max(wl.dim // 16, 64))
    out = {"metric": "loss F(w_bar) per round and bytes sent per worker", "workload": wl.name,
           "workers": wl.n_workers, "dim": wl.dim, "samples_per_worker": wl.samples, "graphs": {}}
    if wl.features == "csr":
        data = synth.csr_data(wl)
    else:
        data = synth.dense_data(wl)
    for g in ("complete", "root_expander", "chain"):
        gw = wl.with_(graph=g)
        p, i, w = graph_for(gw)
        sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
        if wl.features == "csr":
            sess.bind_csr(*data, wl.samples)
        else:
            sess.bind_dense(*data)
        prm = asap.sgd_params(wl.loss, wl.lr_kind, wl.lr0, wl.l2, wl.batch, wl.seed)
        losses, spread = [], []
        for _ in range(rounds):
            sess.round(prm)
            m = sess.metrics(wl.loss, wl.l2)
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
        gap = 1.0 - float(np.linalg.svd(P, compute_uv=False)[1])
        out["graphs"][g] = {"spectral_gap": gap, "out_degree": out_degree,
                            "bytes_per_worker_per_round": out_degree * wl.dim * 4, "loss": losses,
                            "consensus_distance": spread}
    print(json.dumps(out), flush=True)


def run_rounds_bench(sess, prm, step, args, wl, name, torch):
    """K rounds stream-ordered (asap_prepare_sgd / asap_local_sgd /
    asap_stochastic_reduce per round), then K rounds as one multi-round
    launch from the state they left; both timed by the host clock between
    device synchronisations.  The same models at the end are not expected:
    the two runs cover different rounds (the launch continues the first)."""
    from paper_1612_08608_amd import asap
    K = args.steps
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
    if st != asap.OK:
        raise RuntimeError(f"multi-round launch reported a stale neighbour (worker {bad})")
    samples = wl.n_workers * wl.samples
    planned = wl.features == "csr" and wl.batch <= 64
    out = {"metric": "rounds/s, one multi-round launch vs stream-ordered rounds", "mode": "notify_ack",
           "n_gpus": 1, "steps": K, "warmup": args.warmup, "dtype": "f32", "data": "synthetic",
           "higher_is_better": True,
           "config": {"workload": name, "workers": wl.n_workers, "dim": wl.dim, "samples_per_worker": wl.samples,
                      "batch": wl.batch, "graph": wl.graph, "degree": wl.degree},
           "stream_ms_per_round": stream_s / K * 1e3, "launch_ms_per_round": launch_s / K * 1e3,
           "stream_samples_per_s": samples * K / stream_s, "launch_samples_per_s": samples * K / launch_s,
           "speedup": stream_s / launch_s,
           "stream_sgd_kernel": "planned CSR pass" if planned else "the launch's half-step code",
           "launch_sgd_kernel": "general CSR pass" if wl.features == "csr" else "dense pass"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="sparse_lr_64w",
                    choices=["sparse_lr_64w", "ring8_dense_lr", "sparse_svm_256w", "sparse_svm_256w_complete",
                             "dense_lr_32w", "mix_stress_1024w"])
    ap.add_argument("--degree", type=int, default=None, help="graph degree override (mixing stress)")
    ap.add_argument("--graph", default=None, choices=["ring", "complete", "random_regular", "root_expander", "chain"],
                    help="communication graph override")
    ap.add_argument("--converge", type=int, default=0, metavar="ROUNDS",
                    help="instead of timing: loss per round on the complete, root-expander and chain graphs "
                         "(the workload at 1/16 of its samples and dimension), and the bytes each worker sends")
    ap.add_argument("--run-rounds", action="store_true",
                    help="instead of the headline line: time the rounds as one multi-round launch "
                         "(asap_run_rounds, per-worker NOTIFY-ACK) beside the same rounds stream-ordered")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="GIB")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: every logical worker runs on a single MI355X "
              "and there is no multi-GPU path (--gpus 1 only)", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import torch
    from paper_1612_08608_amd import asap, synth

    asap.lib()  # fail loudly without the HIP library
    name = args.workload
    wl = synth.WORKLOADS["sparse_svm_256w" if name == "sparse_svm_256w_complete" else name]
    if name == "sparse_svm_256w_complete":
        wl = wl.with_(graph="complete")
    if args.degree:
        wl = wl.with_(degree=args.degree)
    if args.graph:
        wl = wl.with_(graph=args.graph)
    if args.converge:
        converge(wl, args.converge)
        return
    p, i, w = graph_for(wl)
    log(f"[bench] workload {name}: n={wl.n_workers} D={wl.dim} S={wl.samples} B={wl.batch} "
        f"graph={wl.graph} d={wl.degree}")

    t0 = time.perf_counter()
    sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
    rp = col = val = y = None
    if wl.features == "csr":
        rp, col, val, y = synth.csr_data(wl)
        sess.bind_csr(rp, col, val, y, wl.samples)
    elif wl.features == "dense":
        X, y = synth.dense_data(wl)
        sess.bind_dense(X, y)
    else:
        sess.set_models(synth.initial_models(wl))
    sess.ready()
    torch.cuda.synchronize()
    log(f"[bench] inputs resident in HBM after {time.perf_counter() - t0:.1f} s")

    prm = asap.sgd_params(wl.loss, wl.lr_kind, wl.lr0, wl.l2, wl.batch, wl.seed) if wl.features != "none" else None
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if prm is not None:
            # the round's schedule and plan first (waits for the plan made
            # during the previous round), so that the event pair brackets the
            # SGD kernels alone
            sess.prepare_sgd(prm)
            if ev:
                ev[0].record(stream)
            sess.local_sgd(prm)
        if ev:
            ev[1].record(stream)
        sess.stochastic_reduce()
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.run_rounds:
        if prm is None:
            raise SystemExit("--run-rounds needs a workload with SGD")
        run_rounds_bench(sess, prm, step, args, wl, name, torch)
        sess.close()
        return
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    st, bad = sess.check()
    if st != asap.OK:
        raise RuntimeError(f"epoch-tag check failed during the benchmark (worker {bad})")
    sgd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) if prm is not None else 0.0
    mix_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    log(f"[bench] {args.steps} steps in {wall:.3f} s; SGD phase {sgd_ms:.3f} ms, reduce {mix_ms:.3f} ms per step")

    n, D = wl.n_workers, wl.dim
    mix_bytes = 2 * n * D * 4
    mix_gbps = mix_bytes / (mix_ms * 1e-3) / 1e9
    out = {"metric": METRIC, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic"}
    csrc = os.path.join(ROOT, "paper_1612_08608_amd", "csrc")
    reduce_info = {"GB/s": mix_gbps, "frac_of_hbm_peak": mix_gbps / HBM_PEAK_GBPS, "ms": mix_ms,
                   "algorithmic_bytes": mix_bytes}
    if wl.features == "none":
        out.update(value=mix_gbps, unit="GB/s")
        out["config"] = {"workload": name, "workers": n, "dim": D, "graph": f"random {wl.degree}-regular",
                         "rounds_timed": args.steps}
        key = f"mix_kernel@{name}" + (f"_d{wl.degree}" if args.degree else "")
        out["roofline"] = {"bound": "hbm", "achieved": mix_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                           "frac": mix_gbps / HBM_PEAK_GBPS,
                           "traffic": traffic_for(key, os.path.join(csrc, "kernels_mix.hip"))}
        if not args.no_cpu_baseline:
            log("[bench] oracle CPU baseline ...")
            out["cpu_baseline"] = cpu_baseline_mix(wl, p, i, w)
    else:
        samples = n * wl.samples
        out.update(value=samples * args.steps / wall, unit="samples/s")
        out["config"] = {"workload": name, "workers": n, "dim": D, "samples_per_worker": wl.samples,
                         "batch": wl.batch, "loss": wl.loss, "features": wl.features, "graph": wl.graph,
                         "degree": wl.degree}
        out["sgd_samples_per_s"] = samples / (sgd_ms * 1e-3)
        out["reduce"] = reduce_info
        if wl.features == "csr":
            alg, reads, writes = csr_algorithmic_bytes(wl, rp, col)
            # the planned pass takes minibatches of up to 64 rows of up to 128
            # nonzeros; anything else runs the general kernel
            if wl.batch <= 64 and int(np.diff(rp).max()) <= 128:
                kernel, src = "sgd_csr_fast_kernel", os.path.join(csrc, "kernels_csr_plan.hip")
            else:
                kernel, src = "sgd_csr_kernel", os.path.join(csrc, "kernels_csr.hip")
        else:
            S, B = wl.samples, wl.batch
            steps_per_pass = -(-S // B)
            alg = n * (S * (4 * D + 4 + 4) + steps_per_pass * 8 * D)
            if 1024 < D <= 8192:
                kernel, src = "sgd_dense_wide_kernel", os.path.join(csrc, "kernels_dense.hip")
            else:
                kernel, src = "sgd_dense_kernel", os.path.join(csrc, "kernels_sgd.hip")
        ach = alg / (sgd_ms * 1e-3) / 1e9
        out["roofline"] = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                           "frac": ach / HBM_PEAK_GBPS, "kernel": kernel, "algorithmic_bytes": alg,
                           "traffic": traffic_for(f"{kernel}@{name}", src)}
        if not args.no_cpu_baseline:
            log("[bench] oracle CPU baseline ...")
            if wl.features == "csr":
                out["cpu_baseline"] = cpu_baseline_csr(wl, rp, col, val, y, p, i, w)
            else:
                out["cpu_baseline"] = cpu_baseline_dense(wl, X, y)
    sess.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
