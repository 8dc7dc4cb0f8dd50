"""Pins of the HPSA masks (Section 4.2, Fig. 2-3) and their counts (Section 5, Appendix A)."""
import os
from collections import deque

import numpy as np
import pytest

from workloads import CONFIGS
from workloads.configs import parity_check

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bfs_distances(H):
    """Tanner-graph distances by breadth-first search (independent of any matrix product)."""
    m, n = H.shape
    L = n + m
    adj = [[] for _ in range(L)]
    for j in range(m):
        for i in range(n):
            if H[j, i]:
                adj[i].append(n + j)
                adj[n + j].append(i)
    dist = np.full((L, L), -1, dtype=np.int64)
    for s in range(L):
        dist[s, s] = 0
        dq = deque([s])
        while dq:
            u = dq.popleft()
            if dist[s, u] >= 2:
                continue
            for v in adj[u]:
                if dist[s, v] < 0:
                    dist[s, v] = dist[s, u] + 1
                    dq.append(v)
    return dist


@pytest.mark.parametrize("c", [1, 2, 3])
def test_masks_are_distance_rings(oracle_mod, c):
    H = parity_check(CONFIGS[c])
    M1, M2 = oracle_mod.masks(H)
    dist = _bfs_distances(H)
    assert (M1 == (dist == 1)).all()                         # first ring: Tanner neighbours
    assert (M2 == ((dist == 0) | (dist == 2))).all()         # second ring: distance two (+ self)
    assert (M1 == M1.T).all() and (M2 == M2.T).all()
    assert not (M1 & M2).any()                               # bipartite: odd vs even distance
    ecct = (dist >= 0) & (dist <= 2)                          # ECCT mask g(H) of Section 3
    assert ((M1 | M2) == ecct).all()
    n = H.shape[1]
    assert not M1[:n, :n].any() and not M1[n:, n:].any()      # c->v / v->c blocks only
    assert not M2[:n, n:].any() and not M2[n:, :n].any()      # v->v / c->c blocks only


def test_hamming_counts_golden(oracle_mod):
    vals = {}
    for ln in open(os.path.join(GOLDEN, "hamming7_4_masks.txt")):
        if ln.strip() and not ln.startswith("#"):
            k, v = ln.split()
            vals[k] = int(v)
    H = parity_check(CONFIGS[1])
    M1, M2 = oracle_mod.masks(H)
    L = H.shape[0] + H.shape[1]
    assert H.sum() == vals["edges"]
    assert M1.sum() == vals["m1_pairs"] == 2 * vals["edges"]
    assert M2.sum() == vals["m2_pairs"]
    assert (M1 | M2).sum() == vals["casa_kept"]
    assert round(100 * (1 - (M1 | M2).sum() / L ** 2)) == vals["casa_sparsity_percent"]


@pytest.mark.parametrize("c", [1, 2, 3, 4])
def test_first_ring_count_and_hpsa_half_of_casa(oracle_mod, c):
    H = parity_check(CONFIGS[c])
    M1, M2 = oracle_mod.masks(H)
    E = int(H.sum())
    # Appendix A: the first-ring heads touch sum of all node degrees = 2|E| pairs
    assert M1.sum() == 2 * E
    # with h_f = h_s every head sees one of two disjoint masks whose union is CASA's, so the
    # total HPSA pair count over 8 heads is exactly half of CASA's (Section 5, Complexity)
    hpsa = 4 * M1.sum() + 4 * M2.sum()
    casa = 8 * (M1 | M2).sum()
    assert 2 * hpsa == casa


@pytest.mark.parametrize("c", [3, 4, 5])
def test_ldpc_closed_form_rows(oracle_mod, c):
    """(3,6)-regular, girth >= 6: v-row of M2 = 1 + 3*5 = 16, c-row = 1 + 6*2 = 13."""
    H = parity_check(CONFIGS[c])
    m, n = H.shape
    M1, M2 = oracle_mod.masks(H)
    r1 = M1.sum(1)
    r2 = M2.sum(1)
    assert (r1[:n] == 3).all() and (r1[n:] == 6).all()
    assert (r2[:n] == 16).all() and (r2[n:] == 13).all()
    assert M1.sum() == 6 * n and 2 * M2.sum() == 45 * n      # nnz 6n and 22.5n
