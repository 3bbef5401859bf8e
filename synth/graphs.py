"""Graph structures, given weights and edge masks for the mixing topologies.

Every structure is returned in CSR form with an explicit diagonal entry per row
and column indices sorted ascending within each row:

    row_ptr : int32[M + 1]
    col_idx : int32[nnz]

Weights are only produced where the workload states them literally (ring with
1/3 on self and each neighbour, directed exponential graph with 1/5 on self and
each peer, complete graph with 1/M).  Metropolis-Hastings weights are *not*
computed here: callers pass the structure with the Metropolis reweighting mode
and each implementation derives the weights itself.

Random structures and masks use numpy's PCG64 generator with a fixed seed.
"""

from __future__ import annotations

import numpy as np


def _csr_from_rows(rows):
    """rows: list of sorted neighbour lists (each including the row itself)."""
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int32)
    for i, r in enumerate(rows):
        row_ptr[i + 1] = row_ptr[i] + len(r)
    col_idx = np.array([c for r in rows for c in r], dtype=np.int32)
    return row_ptr, col_idx


def ring(M: int):
    """Undirected ring: row i holds {i-1, i, i+1} mod M.  Needs M >= 3."""
    if M < 3:
        raise ValueError("a ring needs at least 3 workers")
    rows = [sorted({(i - 1) % M, i, (i + 1) % M}) for i in range(M)]
    return _csr_from_rows(rows)


def ring_weights(M: int):
    """Ring structure with the stated weights: 1/3 on self and each neighbour."""
    row_ptr, col_idx = ring(M)
    w = np.full(col_idx.shape[0], 1.0 / 3.0, dtype=np.float32)
    return row_ptr, col_idx, w


def exponential(M: int, hops=(1, 2, 4, 8)):
    """Directed exponential graph: row i pulls from {i} and {i + h mod M : h in hops}."""
    rows = []
    for i in range(M):
        r = {i}
        for h in hops:
            r.add((i + h) % M)
        rows.append(sorted(r))
    return _csr_from_rows(rows)


def exponential_weights(M: int, hops=(1, 2, 4, 8)):
    """Exponential graph with uniform stated weights 1/(len(hops)+1) including self.

    Only meaningful when the hops are distinct mod M (true for M=16 and hops
    1, 2, 4, 8), so every row has len(hops)+1 entries.
    """
    row_ptr, col_idx = exponential(M, hops)
    deg = np.diff(row_ptr)
    if not np.all(deg == len(hops) + 1):
        raise ValueError("hops collide modulo M")
    w = np.full(col_idx.shape[0], 1.0 / (len(hops) + 1), dtype=np.float32)
    return row_ptr, col_idx, w


def complete(M: int):
    """Complete graph including self loops: every row holds 0..M-1."""
    rows = [list(range(M)) for _ in range(M)]
    return _csr_from_rows(rows)


def complete_weights(M: int):
    row_ptr, col_idx = complete(M)
    w = np.full(col_idx.shape[0], 1.0 / M, dtype=np.float32)
    return row_ptr, col_idx, w


def identity(M: int):
    rows = [[i] for i in range(M)]
    row_ptr, col_idx = _csr_from_rows(rows)
    return row_ptr, col_idx, np.ones(M, dtype=np.float32)


def random_regular(M: int, d: int, seed: int, max_tries: int = 10000):
    """Seeded simple d-regular undirected graph by the configuration model.

    Stubs (d per node) are shuffled and paired; a pairing with a self loop or a
    repeated edge is rejected and redrawn.  Returns the CSR structure with the
    diagonal added.
    """
    if (M * d) % 2 != 0 or d >= M:
        raise ValueError("no simple d-regular graph for these M, d")
    rng = np.random.Generator(np.random.PCG64(seed))
    stubs = np.repeat(np.arange(M), d)
    for _ in range(max_tries):
        perm = rng.permutation(stubs)
        a, b = perm[0::2], perm[1::2]
        if np.any(a == b):
            continue
        edges = {(min(x, y), max(x, y)) for x, y in zip(a.tolist(), b.tolist())}
        if len(edges) != M * d // 2:
            continue
        nbr = [{i} for i in range(M)]
        for x, y in edges:
            nbr[x].add(y)
            nbr[y].add(x)
        return _csr_from_rows([sorted(s) for s in nbr])
    raise RuntimeError("configuration model did not produce a simple graph")


def undirected_edges(row_ptr, col_idx):
    """Off-diagonal undirected edges (i < j) present in the structure."""
    out = []
    for i in range(len(row_ptr) - 1):
        for e in range(row_ptr[i], row_ptr[i + 1]):
            j = int(col_idx[e])
            if i < j:
                out.append((i, j))
    return out


def masks_from_live_edges(row_ptr, col_idx, live_per_round):
    """Build uint8 masks[K][nnz]: diagonal always 1; entry (i,j) is 1 iff the
    undirected edge {i,j} is in that round's live set."""
    K = len(live_per_round)
    nnz = col_idx.shape[0]
    masks = np.zeros((K, nnz), dtype=np.uint8)
    for k, live in enumerate(live_per_round):
        live = {(min(a, b), max(a, b)) for a, b in live}
        for i in range(len(row_ptr) - 1):
            for e in range(row_ptr[i], row_ptr[i + 1]):
                j = int(col_idx[e])
                if i == j or (min(i, j), max(i, j)) in live:
                    masks[k, e] = 1
    return masks


def edge_drop_masks(row_ptr, col_idx, rounds: int, p_drop: float, seed: int):
    """Per round, drop each undirected edge independently with probability p_drop.

    The draw for round k uses PCG64 seeded with (seed, k); edges are visited in
    ascending (i, j) order, one uniform draw each.
    """
    edges = undirected_edges(row_ptr, col_idx)
    live_per_round = []
    for k in range(rounds):
        rng = np.random.Generator(np.random.PCG64([seed, k]))
        u = rng.random(len(edges))
        live_per_round.append([e for e, x in zip(edges, u) if x >= p_drop])
    return masks_from_live_edges(row_ptr, col_idx, live_per_round)


def random_matching_masks(M: int, rounds: int, seed: int):
    """Per round, a uniformly random maximal matching over the complete structure.

    Workers are shuffled and paired consecutively; with odd M the last one stays
    unmatched.  Returns (row_ptr, col_idx, masks[K][nnz]) on the complete graph.
    """
    row_ptr, col_idx = complete(M)
    live_per_round = []
    for k in range(rounds):
        rng = np.random.Generator(np.random.PCG64([seed, k]))
        perm = rng.permutation(M)
        live_per_round.append([(int(perm[2 * i]), int(perm[2 * i + 1])) for i in range(M // 2)])
    return row_ptr, col_idx, masks_from_live_edges(row_ptr, col_idx, live_per_round)


def all_perfect_matchings(M: int):
    """Every perfect matching of M (even) workers, as lists of pairs."""
    if M % 2:
        raise ValueError("M must be even")

    def rec(rest):
        if not rest:
            yield []
            return
        a = rest[0]
        for i in range(1, len(rest)):
            b = rest[i]
            for tail in rec(rest[1:i] + rest[i + 1:]):
                yield [(a, b)] + tail

    return list(rec(list(range(M))))


def random_symmetric_structure(M: int, p_edge: float, seed: int):
    """Erdos-Renyi undirected structure with diagonal, for property tests."""
    rng = np.random.Generator(np.random.PCG64(seed))
    nbr = [{i} for i in range(M)]
    for i in range(M):
        for j in range(i + 1, M):
            if rng.random() < p_edge:
                nbr[i].add(j)
                nbr[j].add(i)
    return _csr_from_rows([sorted(s) for s in nbr])
