"""Pins of the oracle's stochastic reduce and round composition (CPU only)."""
import numpy as np
import pytest

from oracle import graphs, metrics, mix, rounds

RNG = np.random.default_rng(77)


def _graph(kind, n, d=4, seed=0):
    if kind == "ring":
        ptr, idx = graphs.ring(n)
    elif kind == "complete":
        ptr, idx = graphs.complete(n)
    else:
        ptr, idx = graphs.random_regular(n, d, seed)
    return ptr, idx, graphs.metropolis_weights(ptr, idx)


@pytest.mark.parametrize("kind,n,d", [("ring", 8, 2), ("random", 64, 4), ("random", 256, 8), ("complete", 16, 15)])
def test_reduce_equals_blas_dense_product(kind, n, d):
    ptr, idx, w = _graph(kind, n, d)
    W = RNG.standard_normal((n, 37)).astype(np.float32)
    P = graphs.dense_matrix(ptr, idx, w)
    assert np.allclose(mix.stochastic_reduce(W, ptr, idx, w), P @ W.astype(np.float64), rtol=1e-13, atol=1e-13)


def test_complete_graph_is_exact_allreduce_average():
    # Section 2/3: all-reduce = every node takes the average of all models.
    n = 256
    ptr, idx, w = _graph("complete", n)
    W = RNG.standard_normal((n, 19)).astype(np.float32)
    out = mix.stochastic_reduce(W, ptr, idx, w)
    mean = W.astype(np.float64).sum(axis=0) / n        # 1/256 is exact
    assert np.allclose(out, np.broadcast_to(mean, out.shape), rtol=0, atol=1e-13)


def test_identity_graph_is_noop():
    n = 5
    ptr = np.arange(n + 1, dtype=np.int32)
    idx = np.arange(n, dtype=np.int32)
    w = np.ones(n, np.float32)
    W = RNG.standard_normal((n, 7)).astype(np.float32)
    assert np.array_equal(mix.stochastic_reduce(W, ptr, idx, w), W.astype(np.float64))


def test_rows_helper_matches_full():
    ptr, idx, w = _graph("random", 32, 6)
    W = RNG.standard_normal((32, 11))
    full = mix.stochastic_reduce(W, ptr, idx, w)
    rows = [0, 7, 31]
    assert np.allclose(mix.stochastic_reduce_rows(lambda j: W[j], ptr, idx, w, rows), full[rows])


@pytest.mark.parametrize("d", [2, 4, 8, 16])
def test_mean_preserved_and_consensus_decays_at_sigma2(d):
    # "Network requirement": a doubly-stochastic P keeps every node's influence
    # equal, so 1^T P = 1^T and the mean model is invariant; "Spectral Gap":
    # the deviation from consensus shrinks at least like sigma_2(P)^t.
    n = 128
    ptr, idx, w = _graph("random", n, d, seed=3)
    P = graphs.dense_matrix(ptr, idx, w)
    s2 = graphs.sigma2(P)
    W = RNG.standard_normal((n, 64))
    mean0 = W.mean(axis=0)
    dev0 = metrics.consensus_distance(W)
    for t in range(1, 31):
        W = mix.stochastic_reduce(W, ptr, idx, w)
        # |1^T P - 1^T| <= (d+1) 2^-24 per column from fp32 weights
        assert np.allclose(W.mean(axis=0), mean0, atol=t * (d + 2) * 2 ** -24 * 6)
        assert metrics.consensus_distance(W) <= metrics.consensus_bound(dev0, s2, t) * (1 + 1e-9) + 1e-12


def test_consensus_decay_matches_eigen_prediction():
    # For symmetric P: ||dev_t||^2 = sum_k lambda_k^(2t) ||q_k^T dev_0||^2.
    n = 64
    ptr, idx, w = _graph("random", n, 4, seed=5)
    P = graphs.dense_matrix(ptr, idx, w)
    P = 0.5 * (P + P.T)          # symmetric to fp64 rounding already
    lam, Q = np.linalg.eigh(P)
    W = RNG.standard_normal((n, 32))
    dev0 = W - W.mean(axis=0)
    coef = (Q.T @ dev0) ** 2
    for t in range(1, 15):
        W = mix.stochastic_reduce(W, ptr, idx, w)
        pred = np.sqrt(np.sum((lam[:, None] ** (2 * t)) * coef))
        assert metrics.consensus_distance(W) == pytest.approx(pred, rel=1e-6)


def test_disconnected_components_keep_their_own_means():
    p5, i5 = graphs.ring(5)
    ptr = np.concatenate([p5, p5[1:] + 15]).astype(np.int32)
    idx = np.concatenate([i5, i5 + 5]).astype(np.int32)
    w = graphs.metropolis_weights(ptr, idx)
    W = np.concatenate([np.zeros((5, 3)), np.ones((5, 3))])
    for _ in range(50):
        W = mix.stochastic_reduce(W, ptr, idx, w)
    assert np.allclose(W[:5], 0) and np.allclose(W[5:], 1, atol=1e-6)


def test_unrolled_form_with_frozen_gradients():
    # Appendix A, (A.3): with d = 1, w_0 = 0 and forced gradients g_t,
    # w_t = - sum_{k<t} eta_k P^(t-k) g_k.
    n, T = 16, 9
    ptr, idx, w = _graph("random", n, 4, seed=2)
    P = graphs.dense_matrix(ptr, idx, w)
    g = RNG.standard_normal((T, n))
    eta = 0.5 / np.sqrt(np.arange(1, T + 1))
    W = np.zeros((n, 1))
    for t in range(T):
        W, _ = rounds.half_step_then_reduce(W, lambda i, wi: wi - eta[t] * g[t, i], ptr, idx, w)
        expect = -sum(eta[k] * np.linalg.matrix_power(P, t + 1 - k) @ g[k] for k in range(t + 1))
        assert np.allclose(W[:, 0], expect, rtol=1e-12, atol=1e-12)


def test_round_composes_local_pass_then_reduce():
    # Tiny dense round: the result equals P applied to the per-worker passes.
    from oracle import prng, sgd
    n, S, D, B = 4, 12, 3, 5
    ptr, idx = graphs.complete(n)
    w = graphs.metropolis_weights(ptr, idx)
    shards = [("dense", RNG.standard_normal((S, D)).astype(np.float32),
               np.where(RNG.random(S) < 0.5, -1.0, 1.0).astype(np.float32)) for _ in range(n)]
    W0 = RNG.standard_normal((n, D)).astype(np.float32)
    kw = dict(batch=B, loss="logistic", lr_kind="inv_sqrt", lr0=0.5, l2=0.0)
    out, half = rounds.asap_round(W0, shards, ptr, idx, w, seed=0, rnd=2, **kw)
    for i in range(n):
        ref = sgd.sgd_pass_dense(W0[i], shards[i][1], shards[i][2], prng.schedule(S, 0, i, 2), rnd=2, **kw)
        assert np.allclose(half[i], ref)
    assert np.allclose(out, np.broadcast_to(half.mean(axis=0), out.shape))
