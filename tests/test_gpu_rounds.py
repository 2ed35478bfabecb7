"""Multi-round launch with per-worker NOTIFY-ACK (Section 4), through the C ABI.

asap_run_rounds runs R rounds in one persistent launch, each worker waiting
only for its own neighbours.  The data dependencies are those of R calls of
asap_round, so the result must be the same bits (same half-step code, same
reduce arithmetic); both paths are also checked against the oracle, and the
stream-ordered path continues from the state the launch leaves.
"""
import numpy as np
import pytest

from conftest import assert_models_close
from paper_1612_08608_amd import asap, synth
import oracle
from test_gpu_parity import graph, params, oracle_kw, csr_shards, ambiguity_mask

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "GPU tests need a GPU"
    asap.lib()
    return _t


@pytest.fixture(autouse=True)
def _announce(request):
    print(f"\n[gpu] {request.node.nodeid}", flush=True)
    yield


def _session(wl, kind, d, W0=None, members=0):
    p, i, w = graph(kind, wl.n_workers, d)
    sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
    if W0 is not None:
        sess.set_models(W0)
    if wl.features == "dense":
        X, y = synth.dense_data(wl)
        sess.bind_dense(X, y)
    else:
        rp, col, val, yy = synth.csr_data(wl)
        sess.bind_csr(rp, col, val, yy, wl.samples)
        if members:
            sess.set_csr_members(members)
    return sess, (p, i, w)


def _bits(sess):
    return sess.models().cpu().numpy().view(np.uint32).copy()


# (workload, graph kind, degree, rounds, local steps); the reduce runs the
# slab kernel's arithmetic (n a power of two, short rows), the tile kernel's
# (other n) or the mean kernel's (complete uniform graph)
CASES = {
    "dense_ring8": (synth.RING8_DENSE_LR.with_(samples=256), "ring", 2, 5, 0),
    "dense_random12_ragged": (synth.RING8_DENSE_LR.with_(n_workers=12, dim=101, samples=203, batch=16),
                              "random", 4, 4, 0),
    "dense_complete6": (synth.RING8_DENSE_LR.with_(n_workers=6, samples=160), "complete", 0, 4, 0),
    "dense_chain16": (synth.RING8_DENSE_LR.with_(n_workers=16, samples=128), "chain", 0, 4, 0),
    "dense_root10": (synth.RING8_DENSE_LR.with_(n_workers=10, samples=128), "root", 0, 4, 0),
    "dense_one_step_per_mix": (synth.RING8_DENSE_LR.with_(samples=128, batch=16), "ring", 2, 19, 1),
    "wide_8w": (synth.DENSE_LR_32W.with_(n_workers=8, dim=2048, samples=192, batch=32), "random", 4, 3, 0),
    "wide_32w_4096": (synth.DENSE_LR_32W.with_(samples=1024, batch=256), "random", 6, 3, 0),
    "wide_3w_L3": (synth.DENSE_LR_32W.with_(n_workers=3, dim=2048, samples=72, batch=8, lr_kind="inv_sqrt",
                                            lr0=0.2), "complete", 0, 7, 3),
    "csr_general": (synth.SPARSE_LR_64W.with_(n_workers=16, dim=1 << 14, samples=600, batch=100), "random", 4, 3, 0),
    "csr_hinge_l2": (synth.SPARSE_SVM_256W.with_(n_workers=32, dim=1 << 12, samples=560, batch=80, l2=1e-3),
                     "random", 8, 3, 0),
    "csr_long_rows_ring": (synth.SPARSE_LR_64W.with_(n_workers=4, dim=1 << 13, samples=240, batch=40,
                                                     nnz_mean=200.0, zipf_s=0.9), "ring", 2, 3, 0),
    "csr_local_steps": (synth.SPARSE_LR_64W.with_(n_workers=8, dim=1 << 13, samples=400, batch=100), "chain", 0,
                        9, 2),
}


@pytest.mark.parametrize("case", list(CASES))
def test_run_rounds_is_bitwise_the_stream_path(torch, case):
    wl, kind, d, R, L = CASES[case]
    prm = params(wl, L)
    # rows of ~200 nonzeros: one member per worker keeps them on the general
    # kernel (a member's share of them would fit the planned pass)
    members = 1 if case == "csr_long_rows_ring" else 0
    a, _ = _session(wl, kind, d, members=members)
    b, _ = _session(wl, kind, d, members=members)
    for _ in range(R):
        a.round(prm)
    b.run_rounds(prm, R, wait_ms=3000)
    assert b.check()[0] == asap.OK
    assert b.current() == a.current()
    assert np.array_equal(_bits(b), _bits(a)), case
    # the stream-ordered path continues from the launch's state (tags included)
    for s in (a, b):
        s.round(prm)
    assert a.check()[0] == asap.OK and b.check()[0] == asap.OK
    assert np.array_equal(_bits(b), _bits(a)), case
    # and a launch continues from a stream-ordered round
    a.round(prm)
    a.round(prm)
    b.run_rounds(prm, 2, wait_ms=3000)
    assert b.check()[0] == asap.OK
    assert b.current() == a.current()
    assert np.array_equal(_bits(b), _bits(a)), case
    a.close()
    b.close()


@pytest.mark.parametrize("case", ["c2_shape", "c3_shape"])
def test_run_rounds_against_the_oracle(torch, case):
    # minibatches of at most 64 rows: the stream-ordered path would plan the
    # pass; the launch runs the general CSR code, checked against the oracle
    if case == "c2_shape":
        wl, kind, d = synth.SPARSE_LR_64W.with_(n_workers=16, dim=1 << 14, samples=512), "random", 4
    else:
        wl, kind, d = synth.SPARSE_SVM_256W.with_(n_workers=16, dim=1 << 12, samples=256), "random", 8
    # the oracle first: if a round has hinge decisions within rounding of the
    # kink, the launch covers the rounds up to and including it and that
    # round is compared outside the entries those decisions can change
    R = 3
    p, i, w = graph(kind, wl.n_workers, d)
    rp, col, val, yy = synth.csr_data(wl)
    shards = csr_shards(wl, rp, col, val, yy)
    W = np.zeros((wl.n_workers, wl.dim))
    mask = None
    for r in range(R):
        halves, amb = [], []
        for k in range(wl.n_workers):
            sched = oracle.prng.schedule(wl.samples, wl.seed, k, r)
            _, rpk, ck, vk, yk = shards[k]
            a = []
            halves.append(oracle.sgd.sgd_pass_csr(W[k], rpk, ck, vk, yk, sched, rnd=r, ambiguous=a, **oracle_kw(wl)))
            amb += [(k, q) for q in a]
        W = oracle.mix.stochastic_reduce(np.stack(halves), p, i, w)
        if amb:
            mask = ambiguity_mask(amb, shards, p, i, W.shape)
            print(f"round {r}: {len(amb)} ambiguous hinge rows; the launch runs {r + 1} rounds", flush=True)
            R = r + 1
            break
    sess, _ = _session(wl, kind, d)
    sess.run_rounds(params(wl), R, wait_ms=3000)
    assert sess.check()[0] == asap.OK
    assert sess.current()[1] == R
    assert_models_close(sess.models().cpu().numpy(), W, what=f"{case} after {R} rounds", mask=mask)
    sess.close()


def test_run_rounds_stale_start_tag_stops_and_reports(torch):
    wl = synth.RING8_DENSE_LR.with_(samples=128)
    prm = params(wl)
    sess, _ = _session(wl, "ring", 2)
    sess.round(prm)
    buf, rnd, _ = sess.current()
    asap.asap_debug_set_tag(sess.ctx, buf, 3, 2 * rnd - 2)  # worker 3 looks a round behind
    sess.run_rounds(prm, 3, wait_ms=50)  # neighbours give up after 50 ms
    st, bad = sess.check()
    assert st == asap.E_EPOCH and 0 <= bad < wl.n_workers
    # a restart from a known state runs again
    sess.set_models(np.zeros((wl.n_workers, wl.dim), np.float32))
    ref, _ = _session(wl, "ring", 2)
    sess.run_rounds(prm, 2, wait_ms=3000)
    ref.round(prm)
    ref.round(prm)
    assert sess.check()[0] == asap.OK
    assert np.array_equal(_bits(sess), _bits(ref))
    sess.close()
    ref.close()


def test_run_rounds_rejects_hubs_and_bad_arguments(torch):
    wl = synth.RING8_DENSE_LR.with_(n_workers=70, samples=16)
    sess, _ = _session(wl, "complete", 0)  # 70 in- and out-neighbours per worker
    with pytest.raises(asap.AsapError) as e:
        sess.run_rounds(params(wl), 2)
    assert e.value.status == asap.E_STATE
    sess.close()
    wl = synth.RING8_DENSE_LR.with_(samples=16)
    sess, _ = _session(wl, "ring", 2)
    for R, ms in ((0, 0), (2, -1)):
        with pytest.raises(asap.AsapError) as e:
            sess.run_rounds(params(wl), R, wait_ms=ms)
        assert e.value.status == asap.E_INVALID_ARG
    sess.local_sgd(params(wl))
    with pytest.raises(asap.AsapError) as e:  # a half-step is pending
        sess.run_rounds(params(wl), 1)
    assert e.value.status == asap.E_STATE
    sess.close()


def _empty_row_csr(wl):
    """The workload's shards with every 7th row emptied and worker 1's shard
    empty altogether."""
    rp, col, val, yy = synth.csr_data(wl)
    S = wl.samples
    keep_row = np.ones(wl.n_workers * S, bool)
    keep_row[::7] = False
    keep_row[S:2 * S] = False
    lens = np.diff(rp) * keep_row
    rp2 = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    keep_nz = np.repeat(keep_row, np.diff(rp))
    return rp2, col[keep_nz], val[keep_nz], yy


@pytest.mark.parametrize("case", ["empty_rows", "single_worker"])
def test_run_rounds_edge_cases_match_the_stream_path(torch, case):
    if case == "empty_rows":
        wl = synth.SPARSE_LR_64W.with_(n_workers=4, dim=1 << 12, samples=150, batch=100, nnz_mean=20.0)
        data = _empty_row_csr(wl)
        p, i, w = graph("ring", wl.n_workers, 2)
    else:
        wl = synth.SPARSE_SVM_256W.with_(n_workers=1, dim=1 << 11, samples=160, batch=40, l2=1e-3)
        data = synth.csr_data(wl)
        p, i, w = np.array([0, 1], np.int32), np.array([0], np.int32), np.array([1.0], np.float32)
    prm = params(wl)
    runs = []
    for launch in (False, True):
        sess = asap.Session(wl.n_workers, wl.dim, p, i, w)
        sess.bind_csr(*data, wl.samples)
        if launch:
            sess.run_rounds(prm, 3, wait_ms=3000)
        else:
            for _ in range(3):
                sess.round(prm)
        assert sess.check()[0] == asap.OK
        runs.append(_bits(sess))
        sess.close()
    assert np.array_equal(runs[0], runs[1]), case


# Planned CSR passes inside the launch: with a plan ring bound, every pass of
# the launch runs the same planned-pass code as the stream-ordered rounds
# (or, where a step overflows the plan, the same general code), so the bits
# must be equal.  Small worker counts plan beside the launch on the library's
# look-ahead stream; 128 workers with their prefetch workgroups fill the
# device, so their plans are made before the launch.  The last field sets the
# workgroups per worker of the planned pass (0: the library's choice: 4 up
# to 32 workers, 2 up to 64, else 1); members of a worker exchange partial
# margins every step and publish the half-step only when all have finished.
PLANNED = {
    "c2_shape": (synth.SPARSE_LR_64W.with_(n_workers=16, dim=1 << 14, samples=512), "random", 4, 3, 0, 0),
    "c2_shape_64w": (synth.SPARSE_LR_64W.with_(n_workers=64, dim=1 << 14, samples=256), "random", 4, 3, 0, 0),
    "c2_shape_one_member": (synth.SPARSE_LR_64W.with_(n_workers=16, dim=1 << 14, samples=512), "random", 4, 3, 0, 1),
    "c3_shape_128w": (synth.SPARSE_SVM_256W.with_(n_workers=128, dim=1 << 13, samples=256), "random", 8, 3, 0, 0),
    "hinge_l2_2_members": (synth.SPARSE_SVM_256W.with_(n_workers=32, dim=1 << 13, samples=256, l2=1e-3), "random",
                           8, 3, 0, 2),
    # 12 workers: members of a worker on different XCDs
    "members_several_xcds": (synth.SPARSE_LR_64W.with_(n_workers=12, dim=1 << 13, samples=256), "random", 4, 3, 0,
                             2),
    "local_steps": (synth.SPARSE_LR_64W.with_(n_workers=8, dim=1 << 13, samples=512, batch=64), "chain", 0, 7, 2, 0),
    # ~3800 distinct rarely used columns per step: every plan overflows and
    # every pass runs the general code, on both paths
    "overflow": (synth.SPARSE_LR_64W.with_(n_workers=4, samples=256, nnz_mean=60.0, zipf_s=0.3), "ring", 2, 2, 0,
                 0),
}


@pytest.mark.parametrize("case", list(PLANNED))
def test_run_rounds_planned_pass_is_bitwise_the_stream_path(torch, case):
    wl, kind, d, R, L, members = PLANNED[case]
    prm = params(wl, L)
    a, _ = _session(wl, kind, d, members=members)
    b, _ = _session(wl, kind, d, members=members)
    for _ in range(R):
        a.round(prm)
    K = -(-wl.samples // wl.batch)
    passes = R if L == 0 else (R * L) // K + 2
    b.bind_rounds_plan(passes)
    b.run_rounds(prm, R, wait_ms=3000)
    assert b.check()[0] == asap.OK
    assert b.current() == a.current()
    assert np.array_equal(_bits(b), _bits(a)), case
    # the stream-ordered path continues from the launch, and a second launch
    # (the ring reused, its plans remade) from the stream-ordered path
    for s in (a, b):
        s.round(prm)
    assert np.array_equal(_bits(b), _bits(a)), case
    for _ in range(2):
        a.round(prm)
    b.run_rounds(prm, 2, wait_ms=3000)
    assert a.check()[0] == asap.OK and b.check()[0] == asap.OK
    assert b.current() == a.current()
    assert np.array_equal(_bits(b), _bits(a)), case
    a.close()
    b.close()


def test_rounds_plan_ring_arguments(torch):
    wl = synth.SPARSE_LR_64W.with_(n_workers=8, dim=1 << 12, samples=128)
    sess, _ = _session(wl, "ring", 2)
    one = asap.asap_rounds_plan_size(sess.ready().ctx, 1)
    assert asap.asap_rounds_plan_size(sess.ctx, 3) > 2 * one
    for bad in (0, -1):
        with pytest.raises(asap.AsapError) as e:
            asap.asap_rounds_plan_size(sess.ctx, bad)
        assert e.value.status == asap.E_INVALID_ARG
    small = torch.empty(one // 2, dtype=torch.uint8, device="cuda")
    with pytest.raises(asap.AsapError) as e:
        asap.asap_bind_rounds_plan(sess.ctx, small, small.numel())
    assert e.value.status == asap.E_INVALID_ARG
    sess.close()
    dw = synth.RING8_DENSE_LR.with_(samples=64)
    dense, _ = _session(dw, "ring", 2)
    with pytest.raises(asap.AsapError) as e:
        asap.asap_rounds_plan_size(dense.ready().ctx, 1)
    assert e.value.status == asap.E_STATE
    dense.close()
