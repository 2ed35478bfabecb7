"""Pins of the oracle's graph builders, mixing weights and spectral gap (CPU)."""
import math
import os

import numpy as np
import pytest

from oracle import graphs

F32_EPS = 2.0 ** -24


def _P(ptr, idx, w=None):
    w = graphs.metropolis_weights(ptr, idx) if w is None else w
    return graphs.dense_matrix(ptr, idx, w)


def test_ring8_sigma2_closed_form():
    # Circulant with (1/3, 1/3, 1/3): eigenvalues (1 + 2 cos(2 pi k / 8)) / 3,
    # sigma_2 = (1 + sqrt 2) / 3.
    ptr, idx = graphs.ring(8)
    assert ptr.tolist() == [0, 3, 6, 9, 12, 15, 18, 21, 24]
    assert idx[:3].tolist() == [0, 1, 7] and idx[3:6].tolist() == [0, 1, 2]
    w = graphs.metropolis_weights(ptr, idx)
    assert np.all(w == np.float32(1.0 / 3.0))
    assert abs(graphs.sigma2(_P(ptr, idx, w)) - (1 + math.sqrt(2)) / 3) < 8 * F32_EPS


def test_hamiltonian_cycle_sigma2():
    n = 1024
    ptr, idx = graphs.ring(n)
    s2 = graphs.sigma2(_P(ptr, idx))
    assert abs(s2 - (1 + 2 * math.cos(2 * math.pi / n)) / 3) < 8 * F32_EPS


def test_complete_graph_gap_is_figure2_allreduce(golden_dir):
    # Figure 2: all-reduce has spectral gap 1.00 for 6 and 25 nodes.
    rows = {}
    with open(os.path.join(golden_dir, "fig2_spectral_gaps.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, sg6, sg25, pinned = line.split()
                rows[name] = (float(sg6), float(sg25), pinned == "yes")
    sg6, sg25, pinned = rows["all-reduce"]
    assert pinned
    for n, want in ((6, sg6), (25, sg25)):
        ptr, idx = graphs.complete(n)
        assert abs(graphs.spectral_gap(_P(ptr, idx)) - want) < 1e-6
    # the other printed rows are unpinned by construction
    assert not any(r[2] for k, r in rows.items() if k != "all-reduce")


def _circulant_gap(n, offsets):
    # P = (1/m) sum_o Z^o with Z the cyclic shift: eigenvalues
    # (1/m) sum_o exp(2 pi i k o / n), P normal, so its singular values are
    # their moduli and the gap is 1 - max_{k != 0} |lambda_k|.
    k = np.arange(1, n)[:, None]
    lam = np.exp(2j * np.pi * k * np.asarray(offsets)[None, :] / n).sum(axis=1) / len(offsets)
    return 1.0 - float(np.abs(lam).max())


@pytest.mark.parametrize("n", [3, 4, 6, 25, 64, 100, 1024])
def test_root_expander_structure_and_spectrum(n):
    ptr, idx = graphs.root_expander(n)
    r = math.ceil(math.sqrt(n))
    assert ptr.tolist() == [3 * i for i in range(n + 1)]
    for i in range(n):
        assert idx[3 * i:3 * i + 3].tolist() == sorted({i, (i - 1) % n, (i - r) % n})
    # every worker is read by exactly three rows: out-degree 2 plus itself
    assert np.bincount(idx, minlength=n).tolist() == [3] * n
    w = graphs.metropolis_weights(ptr, idx)
    assert np.all(w == np.float32(1.0 / 3.0))
    P = _P(ptr, idx, w)
    assert np.allclose(P.sum(axis=0), 1.0, atol=4 * F32_EPS)
    assert abs(graphs.spectral_gap(P) - _circulant_gap(n, [0, 1, r])) < 16 * F32_EPS


@pytest.mark.parametrize("n", [2, 3, 6, 25, 64, 1000])
def test_chain_structure_and_closed_form_gap(n):
    ptr, idx = graphs.chain(n)
    assert ptr.tolist() == [2 * i for i in range(n + 1)]
    for i in range(n):
        assert idx[2 * i:2 * i + 2].tolist() == sorted({i, (i - 1) % n})
    w = graphs.metropolis_weights(ptr, idx)
    assert np.all(w == np.float32(0.5))
    # (I + Z)/2 has singular values |cos(pi k / n)|
    want = 1.0 - math.cos(math.pi / n) if n > 2 else 1.0
    assert abs(graphs.spectral_gap(_P(ptr, idx, w)) - want) < 16 * F32_EPS


def test_chain_gap_matches_section6(golden_dir):
    with open(os.path.join(golden_dir, "sec6_chain_gap.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    (name, nodes, gap), = rows
    assert name == "chain"
    ptr, idx = graphs.chain(int(nodes))
    got = graphs.spectral_gap(_P(ptr, idx))
    assert round(got, 3) == float(gap), got


def test_sparser_graphs_have_smaller_gaps():
    # Section 3: more edges, higher spectral gap (complete > root > chain)
    for n in (25, 64, 256):
        gaps = [graphs.spectral_gap(_P(*g(n))) for g in (graphs.complete, graphs.root_expander, graphs.chain)]
        assert gaps[0] > gaps[1] > gaps[2] > 0.0


def test_complete_graph_weights_uniform():
    for n in (1, 2, 4, 256):
        ptr, idx = graphs.complete(n)
        w = graphs.metropolis_weights(ptr, idx)
        assert idx.size == n * n
        assert np.all(w == np.float32(1.0 / n))


@pytest.mark.parametrize("n,d", [(64, 4), (256, 8), (32, 6), (1024, 2), (1024, 4), (1024, 8), (1024, 16), (10, 9)])
def test_random_regular_invariants(n, d):
    ptr, idx = graphs.random_regular(n, d, 0)
    assert ptr[0] == 0 and np.all(np.diff(ptr) == d + 1)
    rows = [idx[ptr[i]:ptr[i + 1]] for i in range(n)]
    A = np.zeros((n, n), bool)
    for i, r in enumerate(rows):
        assert np.all(np.diff(r) > 0), "ascending, unique"
        assert i in r, "self included"
        A[i, r] = True
    assert np.array_equal(A, A.T), "undirected"
    P = _P(ptr, idx)
    assert np.allclose(P.sum(axis=0), 1, atol=(d + 1) * F32_EPS)
    assert np.allclose(P.sum(axis=1), 1, atol=(d + 1) * F32_EPS)
    # connected <=> sigma_2 < 1 for a symmetric doubly-stochastic P with positive diagonal
    assert graphs.sigma2(P) < 1 - 1e-7
    # the paper's A/(d+1) on a d-regular graph
    assert np.all(graphs.metropolis_weights(ptr, idx) == np.float32(1.0 / (d + 1)))


def test_random_regular_deterministic_and_seeded():
    a = graphs.random_regular(64, 4, 0)
    b = graphs.random_regular(64, 4, 0)
    c = graphs.random_regular(64, 4, 1)
    assert np.array_equal(a[1], b[1])
    assert not np.array_equal(a[1], c[1])


def test_random_regular_rejects_bad_args():
    for n, d in ((5, 3), (4, 4), (4, 0), (6, 1)):
        with pytest.raises(ValueError):
            graphs.random_regular(n, d, 0)


def test_disconnected_graph_has_zero_gap():
    # Section 3: a disconnected graph has spectral gap zero.
    ptr_a, idx_a = graphs.ring(5)
    n = 10
    ptr = np.concatenate([ptr_a, ptr_a[1:] + ptr_a[-1]]).astype(np.int32)
    idx = np.concatenate([idx_a, idx_a + 5]).astype(np.int32)
    assert ptr[-1] == 30 and n == len(ptr) - 1
    assert abs(graphs.spectral_gap(_P(ptr, idx))) < 1e-7


def test_metropolis_on_irregular_graph_is_doubly_stochastic():
    # star plus a path: irregular degrees; Metropolis still gives a symmetric,
    # doubly-stochastic P (rows and columns sum to one).
    adj = {0: [1, 2, 3, 4], 1: [0], 2: [0], 3: [0, 4], 4: [0, 3]}
    ptr = [0]
    idx = []
    for i in range(5):
        r = sorted(set(adj[i]) | {i})
        idx += r
        ptr.append(len(idx))
    ptr, idx = np.array(ptr, np.int32), np.array(idx, np.int32)
    P = _P(ptr, idx)
    assert np.allclose(P, P.T)
    assert np.allclose(P.sum(0), 1, atol=1e-6) and np.allclose(P.sum(1), 1, atol=1e-6)
    assert P[1, 0] == np.float32(1 / 5) and P[1, 1] == np.float32(1 - 1 / 5)


def test_metropolis_requires_self():
    with pytest.raises(ValueError):
        graphs.metropolis_weights(np.array([0, 1, 2], np.int32), np.array([1, 0], np.int32))
