"""Communication graphs and the mixing matrix P (oracle).

Appendix A ("Network requirement") defines P from the adjacency matrix A of
in-edges (A_ij = 1 iff node i receives from node j, self-loop included, since a
node uses "its neighbours and itself") by scaling row i with 1 / in-degree, and
asks for P doubly stochastic so that every node has the same influence; the
"Spectral Gap" paragraph defines the gap as 1 - sigma_2(P).  Section 3 and the
Figure 2 caption name the all-reduce (complete graph), parameter-server,
expander and chain topologies.

Builders (the HIP library's host code implements the same rules on its own):

* ring(n): in-neighbours of i are {i-1, i, i+1} mod n (n >= 3);
* root_expander(n): i sends to i+1 and i+ceil(sqrt(n)) (Figure 2(c)), so its
  in-neighbours are {i-ceil(sqrt(n)), i-1, i} mod n (n >= 3);
* chain(n): i sends to i+1 with wrap-around (Figure 2(d) as a directed ring),
  in-neighbours {i-1, i} (n >= 2);
* complete(n): all j;
* random_regular(n, d, seed): stub pairing on a SplitMix64 stream keyed by
  K(seed, GRAPH, n, d, 0).  Stubs = [v repeated d times for v ascending].  Draw
  a = below(|S|), b = below(|S|); reject when a == b, the stubs share a vertex,
  or the edge exists; otherwise add the edge and delete index max(a, b), then
  min(a, b), each by swap-with-last-and-pop.  More than 100 * |S| consecutive
  rejections, or a disconnected result (BFS from 0), restarts with the stream
  continuing;
* every row lists its in-neighbours ascending, self included;
* weights: Metropolis-Hastings, P_ij = 1 / (1 + max(d_i, d_j)) for j != i and
  P_ii = 1 - sum_{j != i} P_ij (fp64, summed over ascending j), each rounded
  once to fp32; d_i is the row length minus one.  On a d-regular graph this is
  the paper's A / (d + 1).

Pins: closed-form spectra (ring-8, Hamiltonian cycle, complete graph gives the
Figure 2 all-reduce gap of 1.00), structural invariants (regular, symmetric,
simple, connected, doubly stochastic), and a disconnected graph with gap 0.
"""
from __future__ import annotations

import math
from collections import deque

import numpy as np

from .prng import TAG_GRAPH, SplitMix64, derive_key


def _csr_from_sets(adj):
    n = len(adj)
    ptr = np.zeros(n + 1, np.int32)
    idx = []
    for i in range(n):
        row = sorted(set(adj[i]) | {i})
        idx.extend(row)
        ptr[i + 1] = ptr[i] + len(row)
    return ptr, np.asarray(idx, np.int32)


def ring(n: int):
    if n < 3:
        raise ValueError("ring needs n >= 3")
    return _csr_from_sets([{(i - 1) % n, (i + 1) % n} for i in range(n)])


def root_expander(n: int):
    """Figure 2(c) / Section 3: i sends to i+1 and to i+r, r = ceil(sqrt(n)),
    mod n; as in-neighbours: {i-r, i-1, i}.  The rounding of sqrt(n) is not
    stated (reading: ceil)."""
    if n < 3:
        raise ValueError("root expander needs n >= 3")
    r = math.isqrt(n)
    if r * r < n:
        r += 1
    return _csr_from_sets([{(i - 1) % n, (i - r) % n} for i in range(n)])


def chain(n: int):
    """Figure 2(d): i sends to i+1 only; wrapped around (a directed ring) so
    that P = A/2 is doubly stochastic.  In-neighbours {i-1, i}."""
    if n < 2:
        raise ValueError("chain needs n >= 2")
    return _csr_from_sets([{(i - 1) % n} for i in range(n)])


def complete(n: int):
    if n < 1:
        raise ValueError("complete needs n >= 1")
    return _csr_from_sets([set(range(n)) for _ in range(n)])


def _connected(adj) -> bool:
    n = len(adj)
    seen = [False] * n
    seen[0] = True
    q = deque([0])
    while q:
        u = q.popleft()
        for v in adj[u]:
            if not seen[v]:
                seen[v] = True
                q.append(v)
    return all(seen)


def random_regular(n: int, d: int, seed: int):
    """Connected simple random d-regular graph as in-neighbour CSR (self included)."""
    if not (1 <= d < n) or (n * d) % 2 or (d == 1 and n > 2):
        # a 1-regular graph on more than two nodes is a matching: never connected
        raise ValueError("random_regular needs 1 <= d < n, n*d even, and d >= 2 unless n == 2")
    rng = SplitMix64(derive_key(seed, TAG_GRAPH, n, d, 0))
    while True:
        stubs = [v for v in range(n) for _ in range(d)]
        adj = [set() for _ in range(n)]
        stalls = 0
        complete_ok = True
        while stubs:
            m = len(stubs)
            a = rng.below(m)
            b = rng.below(m)
            u, v = stubs[a], stubs[b]
            if a == b or u == v or v in adj[u]:
                stalls += 1
                if stalls > 100 * m:
                    complete_ok = False
                    break
                continue
            stalls = 0
            adj[u].add(v)
            adj[v].add(u)
            for k in (max(a, b), min(a, b)):
                stubs[k] = stubs[-1]
                stubs.pop()
        if complete_ok and _connected(adj):
            return _csr_from_sets(adj)


def metropolis_weights(ptr, idx) -> np.ndarray:
    """Metropolis-Hastings weights of an in-neighbour CSR, fp64 then fp32."""
    n = len(ptr) - 1
    deg = [int(ptr[i + 1] - ptr[i]) - 1 for i in range(n)]
    w = np.zeros(len(idx), np.float32)
    for i in range(n):
        off = 0.0
        self_pos = -1
        for p in range(ptr[i], ptr[i + 1]):
            j = int(idx[p])
            if j == i:
                self_pos = p
                continue
            pij = 1.0 / (1.0 + max(deg[i], deg[j]))
            off += pij
            w[p] = np.float32(pij)
        if self_pos < 0:
            raise ValueError(f"row {i} lacks its self entry")
        w[self_pos] = np.float32(1.0 - off)
    return w


def dense_matrix(ptr, idx, w, n=None) -> np.ndarray:
    """P as a dense fp64 matrix (row i = weights on i's in-neighbours)."""
    n = len(ptr) - 1 if n is None else n
    P = np.zeros((n, n))
    for i in range(n):
        for p in range(ptr[i], ptr[i + 1]):
            P[i, idx[p]] += float(w[p])
    return P


def sigma2(P: np.ndarray) -> float:
    """Second-largest singular value of P."""
    s = np.linalg.svd(P, compute_uv=False)
    return float(s[1]) if s.size > 1 else 0.0


def spectral_gap(P: np.ndarray) -> float:
    """1 - sigma_2(P) (Appendix A, "Spectral Gap")."""
    return 1.0 - sigma2(P)
