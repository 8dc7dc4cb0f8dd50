"""Parity-check matrices of the code families used for the synthetic workloads.

The problem setting (Section 3, "Problem Settings") defines a binary linear code by a
generator matrix G (k x n) and a parity-check matrix H ((n-k) x n) with G H^T = 0 over
GF(2); the Tanner graph of H has n variable nodes and n-k check nodes.  The paper takes
its matrices from a public database that is not available here, so this module builds
matrices of the same families from their textbook definitions.
"""
from __future__ import annotations

import numpy as np


# ----------------------------------------------------------------------------- GF(2) linear algebra

def gf2_rank(mat: np.ndarray) -> int:
    """Rank of a 0/1 matrix over GF(2) (row reduction)."""
    a = (np.asarray(mat, dtype=np.uint8) & 1).copy()
    rows, cols = a.shape
    r = 0
    for c in range(cols):
        piv = np.nonzero(a[r:, c])[0]
        if piv.size == 0:
            continue
        p = r + piv[0]
        if p != r:
            a[[r, p]] = a[[p, r]]
        hit = np.nonzero(a[:, c])[0]
        hit = hit[hit != r]
        a[hit] ^= a[r]
        r += 1
        if r == rows:
            break
    return r


def generator_from_parity(H: np.ndarray) -> np.ndarray:
    """A generator matrix G (k x n, k = n - rank H) with G H^T = 0 over GF(2).

    Gauss-Jordan elimination of H gives pivot columns P and free columns F; every
    codeword is fixed by its free bits, with each pivot bit equal to the GF(2) sum of
    the free bits its reduced row touches.  Row i of G sets free bit F[i] to one.
    """
    a = (np.asarray(H, dtype=np.uint8) & 1).copy()
    m, n = a.shape
    pivots = []
    r = 0
    for c in range(n):
        piv = np.nonzero(a[r:, c])[0]
        if piv.size == 0:
            continue
        p = r + piv[0]
        if p != r:
            a[[r, p]] = a[[p, r]]
        hit = np.nonzero(a[:, c])[0]
        hit = hit[hit != r]
        a[hit] ^= a[r]
        pivots.append(c)
        r += 1
        if r == m:
            break
    rank = r
    free = [c for c in range(n) if c not in set(pivots)]
    k = n - rank
    G = np.zeros((k, n), dtype=np.uint8)
    for i, f in enumerate(free):
        G[i, f] = 1
        for row, pc in enumerate(pivots):
            G[i, pc] = a[row, f]
    return G


# ----------------------------------------------------------------------------- Hamming(7,4)

def hamming_7_4() -> np.ndarray:
    """Systematic Hamming(7,4): H = [P^T | I_3] for P with rows 110, 101, 011, 111.

    The generator is G = [I_4 | P]; the parity part of H must then be P^T so that
    G H^T = P + P = 0.
    """
    P = np.array([[1, 1, 0], [1, 0, 1], [0, 1, 1], [1, 1, 1]], dtype=np.uint8)
    return np.concatenate([P.T, np.eye(3, dtype=np.uint8)], axis=1)


# ----------------------------------------------------------------------------- BCH(31,16), t = 3

def _gf32_tables(prim: int = 0b100101):
    """exp/log tables of GF(2^5) built from the primitive polynomial x^5 + x^2 + 1."""
    exp = np.zeros(62, dtype=np.int64)
    log = np.full(32, -1, dtype=np.int64)
    v = 1
    for i in range(31):
        exp[i] = v
        log[v] = i
        v <<= 1
        if v & 0b100000:
            v ^= prim
    exp[31:62] = exp[0:31]
    return exp, log


def _poly_mul_gf2(a: list[int], b: list[int]) -> list[int]:
    out = [0] * (len(a) + len(b) - 1)
    for i, x in enumerate(a):
        if x:
            for j, y in enumerate(b):
                out[i + j] ^= y
    return out


def _poly_divmod_gf2(num: list[int], den: list[int]):
    num = list(num)
    dd = len(den) - 1
    q = [0] * max(1, len(num) - dd)
    for i in range(len(num) - 1, dd - 1, -1):
        if num[i]:
            q[i - dd] = 1
            for j, c in enumerate(den):
                num[i - dd + j] ^= c
    return q, num[:dd]


def _minimal_polynomial(i: int, exp, log) -> list[int]:
    """Binary minimal polynomial of alpha^i (product over its cyclotomic coset)."""
    coset = []
    e = i % 31
    while e not in coset:
        coset.append(e)
        e = (2 * e) % 31
    # polynomial with GF(32) coefficients, low degree first
    poly = [1]
    for e in coset:
        root = int(exp[e])
        nxt = [0] * (len(poly) + 1)
        for d, c in enumerate(poly):
            nxt[d + 1] ^= c                       # c * x
            if c and root:                        # c * root
                nxt[d] ^= int(exp[(log[c] + log[root]) % 31])
        poly = nxt
    assert all(c in (0, 1) for c in poly), "minimal polynomial must be binary"
    return poly


def bch_generator_31() -> list[int]:
    """g(x) = lcm of the minimal polynomials of alpha, alpha^3, alpha^5 (designed distance 7)."""
    exp, log = _gf32_tables()
    g = [1]
    for i in (1, 3, 5):
        g = _poly_mul_gf2(g, _minimal_polynomial(i, exp, log))
    return g


def bch_31_16() -> np.ndarray:
    """Cyclic parity-check matrix of the binary BCH(31,16) code.

    h(x) = (x^31 - 1) / g(x) generates the dual code through its reciprocal
    h*(x) = x^16 h(1/x); the 15 rows of H are the shifts x^i h*(x), i = 0..14.
    """
    g = bch_generator_31()
    xn1 = [1] + [0] * 30 + [1]
    h, rem = _poly_divmod_gf2(xn1, g)
    assert not any(rem)
    hrec = h[::-1]
    n, m = 31, 15
    H = np.zeros((m, n), dtype=np.uint8)
    for i in range(m):
        H[i, i:i + len(hrec)] = hrec
    return H


def bch_31_16_generator() -> np.ndarray:
    """Cyclic generator matrix of BCH(31,16): rows x^i g(x), i = 0..15."""
    g = bch_generator_31()
    G = np.zeros((16, 31), dtype=np.uint8)
    for i in range(16):
        G[i, i:i + len(g)] = g
    return G


# ----------------------------------------------------------------------------- (3,6)-regular LDPC

def regular_ldpc_3_6(n: int, seed: int) -> np.ndarray:
    """Random (3,6)-regular LDPC parity-check matrix, n/2 x n, girth >= 6.

    Each variable node owns 3 edge sockets and each check node 6; a seeded
    permutation pairs them.  Repeated edges and 4-cycles (two checks sharing two or
    more variables) are then removed by seeded edge swaps that keep every degree.
    """
    assert n % 2 == 0
    m = n // 2
    rng = np.random.default_rng(seed)
    var_of_edge = np.repeat(np.arange(n), 3)
    chk_of_edge = np.repeat(np.arange(m), 6)[rng.permutation(3 * n)]
    n_edges = 3 * n
    for _sweep in range(10000):
        Hc = np.zeros((m, n), dtype=np.int64)
        np.add.at(Hc, (chk_of_edge, var_of_edge), 1)
        Hb = (Hc > 0).astype(np.float64)
        overlap = Hb @ Hb.T
        np.fill_diagonal(overlap, 0)
        bad_edges = set()
        rep = np.argwhere(Hc > 1)
        for c, v in rep:
            es = np.nonzero((chk_of_edge == c) & (var_of_edge == v))[0]
            bad_edges.update(es[1:].tolist())
        pairs = np.argwhere(np.triu(overlap) >= 2)
        for c1, c2 in pairs:
            shared = np.nonzero(Hb[c1] * Hb[c2])[0]
            v = shared[rng.integers(shared.size)]
            es = np.nonzero((chk_of_edge == c1) & (var_of_edge == v))[0]
            bad_edges.add(int(es[0]))
        if not bad_edges:
            break
        for e in sorted(bad_edges):
            f = int(rng.integers(n_edges))
            if f == e:
                continue
            ce, cf = chk_of_edge[e], chk_of_edge[f]
            ve, vf = var_of_edge[e], var_of_edge[f]
            if ce == cf or ve == vf:
                continue
            chk_of_edge[e], chk_of_edge[f] = cf, ce
    else:  # pragma: no cover - never hit for the sizes used here
        raise RuntimeError("4-cycle removal did not converge")
    H = np.zeros((m, n), dtype=np.uint8)
    H[chk_of_edge, var_of_edge] = 1
    return H
