"""Pins of the SPE oracle (Section 4.3) against closed forms, invariants and torch.

The Laplacian spectrum is pinned on graphs whose spectrum is known in closed form (the
complete bipartite graph, the cycle), the canonical eigenbasis on the cycle's explicit
cos/sin eigenvectors and on its invariance to the basis an eigensolver returns, and the
attention on torch's own multi-head attention in float64.
"""
import numpy as np
import pytest
import torch

from oracle import spe
from workloads import bch_31_16, hamming_7_4, random_spe_params, regular_ldpc_3_6


def cycle_code(n):
    """H whose Tanner graph is the cycle var0-chk0-var1-chk1-...-var(n-1)-chk(n-1)-var0."""
    H = np.zeros((n, n), np.uint8)
    for j in range(n):
        H[j, j] = 1
        H[j, (j + 1) % n] = 1
    return H


CODES = {"hamming": hamming_7_4(), "bch": bch_31_16(), "ldpc64": regular_ldpc_3_6(64, seed=7)}


@pytest.mark.parametrize("name", list(CODES))
def test_laplacian_structure(name):
    H = CODES[name].astype(np.int64)
    Lap = spe.tanner_laplacian(H)
    m, n = H.shape
    assert Lap.shape == (n + m, n + m)
    assert np.array_equal(Lap, Lap.T)
    assert np.all(Lap.sum(axis=1) == 0)
    assert np.trace(Lap) == 2 * H.sum()                      # sum of degrees = 2|E|
    assert np.array_equal(np.diag(Lap)[:n], H.sum(axis=0))   # variable degrees
    assert np.array_equal(np.diag(Lap)[n:], H.sum(axis=1))   # check degrees
    lam, V = spe.tanner_spectrum(H)
    assert abs(lam[0]) < 1e-10 and lam[1] > 1e-6             # connected: 0 is simple
    assert lam[-1] <= 2 * np.diag(Lap).max() + 1e-9
    # bipartite: D - A and D + A are similar, so the signless Laplacian has the same spectrum
    Qs = np.diag(np.diag(Lap)) + (np.diag(np.diag(Lap)) - Lap)
    assert np.allclose(np.linalg.eigvalsh(Qs.astype(float)), lam, atol=1e-9)


@pytest.mark.parametrize("a,b", [(3, 5), (4, 4), (2, 7)])
def test_complete_bipartite_spectrum(a, b):
    # K_{n,m}: Laplacian eigenvalues 0, m (n-1 times), n (m-1 times), n + m
    m, n = a, b
    lam, V = spe.tanner_spectrum(np.ones((m, n), np.uint8))
    want = np.sort(np.concatenate([[0.0], np.full(n - 1, m), np.full(m - 1, n), [n + m]]))
    assert np.allclose(lam, want, atol=1e-10)
    assert np.allclose(V.T @ V, np.eye(n + m), atol=1e-10)


@pytest.mark.parametrize("n", [5, 6, 8])
def test_cycle_closed_form(n):
    """The Tanner graph of cycle_code(n) is C_{2n}: eigenvalues 2 - 2 cos(pi k / n); each
    two-dimensional eigenspace is spanned by cos and sin of (pi k / n) times the position on
    the cycle, and the canonical basis is exactly those, scaled and signed as derived from
    the projector's columns taken in node order."""
    L = 2 * n
    pos = np.concatenate([2 * np.arange(n), 2 * np.arange(n) + 1])   # cycle position of node
    lam, V = spe.tanner_spectrum(cycle_code(n))
    k = np.arange(L)
    assert np.allclose(lam, np.sort(2 - 2 * np.cos(np.pi * k / n)), atol=1e-10)
    assert np.allclose(V[:, 0], np.full(L, 1 / np.sqrt(L)), atol=1e-10)
    assert np.allclose(V[:, -1], (-1.0) ** pos / np.sqrt(L), atol=1e-10)
    for kk in range(1, n):
        th = np.pi * kk / n
        i = 2 * kk - 1                                        # the pair for kk is at i, i + 1
        assert np.isclose(lam[i], 2 - 2 * np.cos(th)) and np.isclose(lam[i + 1], lam[i])
        u0 = np.cos(th * pos) / np.sqrt(n)
        s = np.sin(th * pos)
        c = next(c for c in range(L) if s[c] ** 2 / n > spe.ACCEPT_TOL)
        u1 = np.sign(s[c]) * s / np.sqrt(n)
        assert np.allclose(V[:, i], u0, atol=1e-10)
        assert np.allclose(V[:, i + 1], u1, atol=1e-10)


@pytest.mark.parametrize("name", list(CODES) + ["cycle6", "k35"])
def test_canonical_basis_invariant(name):
    H = {"cycle6": cycle_code(6), "k35": np.ones((3, 5), np.uint8)}.get(name, CODES.get(name))
    Lap = spe.tanner_laplacian(H).astype(float)
    lam0, vec0 = np.linalg.eigh(Lap)
    lam, V = spe.canonical_eigenbasis(lam0, vec0)
    assert np.allclose(V.T @ V, np.eye(len(lam)), atol=1e-10)
    assert np.allclose(V @ np.diag(lam) @ V.T, Lap, atol=1e-9)
    rng = np.random.default_rng(3)
    # another orthonormal basis of every eigenspace: random rotations and sign flips
    mixed = vec0.copy()
    tol = spe.CLUSTER_TOL * max(1.0, np.abs(lam0).max())
    s = 0
    while s < len(lam0):
        e = s + 1
        while e < len(lam0) and lam0[e] - lam0[e - 1] <= tol:
            e += 1
        R, _ = np.linalg.qr(rng.standard_normal((e - s, e - s)))
        mixed[:, s:e] = vec0[:, s:e] @ (R * rng.choice([-1.0, 1.0], e - s))
        s = e
    perm = rng.permutation(len(lam0))
    lam2, V2 = spe.canonical_eigenbasis(lam0[perm], mixed[:, perm])
    assert np.allclose(lam2, lam)
    assert np.allclose(V2, V, atol=1e-8)
    # simple eigenvalues: +-the solver's vector, first entry of size above the threshold positive
    for i in range(len(lam)):
        if (i == 0 or lam[i] - lam[i - 1] > tol) and (i == len(lam) - 1 or lam[i + 1] - lam[i] > tol):
            v = vec0[:, np.argsort(lam0, kind="stable")[i]]
            c = next(c for c in range(len(v)) if v[c] ** 2 > spe.ACCEPT_TOL)
            assert np.allclose(V[:, i], np.sign(v[c]) * v, atol=1e-10)


def torch_mhsa(Z, p):
    """torch's multi-head self-attention (float64) with the same parameters."""
    d_pe, heads = p["d_pe"], p["heads"]
    t = lambda a: torch.tensor(np.asarray(a, np.float64))
    in_w = torch.cat([t(p["w_" + k]).T for k in "qkv"], dim=0)
    in_b = torch.cat([t(p["b_" + k]) for k in "qkv"])
    x = t(Z)[:, None, :]
    out, _ = torch.nn.functional.multi_head_attention_forward(
        x, x, x, d_pe, heads, in_w, in_b, None, None, False, 0.0, t(p["w_o"]).T, t(p["b_o"]),
        training=False, need_weights=False)
    return out[:, 0, :].numpy()


@pytest.mark.parametrize("name,d_pe,heads", [("hamming", 8, 2), ("bch", 8, 1), ("bch", 16, 4),
                                             ("ldpc64", 12, 3)])
def test_attention_matches_torch(name, d_pe, heads):
    H = CODES[name]
    lam, V = spe.tanner_spectrum(H)
    L = len(lam)
    p = random_spe_params(L, d_pe, heads, seed=11)
    rng = np.random.default_rng(5)
    for j in rng.choice(L, size=min(L, 6), replace=False):
        Z = np.stack([lam, V[j]], 1) @ p["w_in"].astype(np.float64) + p["b_in"]
        U = spe.spe_node_attention(lam, V, j, p)
        assert np.allclose(U, torch_mhsa(Z, p), rtol=1e-12, atol=1e-12)
        # the reduction over the eigen-rows, against torch's mean pooling with w_red = 1/L
        q = dict(p, w_red=np.full(L, 1.0 / L), b_red=0.25)
        got = spe.spe_vectors(lam, V, q, nodes=[j])[0]
        assert np.allclose(got, torch_mhsa(Z, p).mean(axis=0) + 0.25, rtol=1e-12, atol=1e-12)


def test_zero_input_map_closed_form():
    # W_in = 0, b_in = 0: every eigen-row is the zero vector, the attention is uniform and
    # SPE_j = sum(w_red) (b_v W_o + b_o) + b_red for every node j
    H = CODES["bch"]
    lam, V = spe.tanner_spectrum(H)
    L = len(lam)
    p = random_spe_params(L, 8, 2, seed=4)
    p["w_in"] = np.zeros_like(p["w_in"])
    p["b_in"] = np.zeros_like(p["b_in"])
    want = p["w_red"].astype(np.float64).sum() * (p["b_v"].astype(np.float64) @ p["w_o"] + p["b_o"]) + p["b_red"]
    got = spe.spe_vectors(lam, V, p)
    assert np.allclose(got, want[None, :], rtol=1e-12, atol=1e-12)


def test_table_layout():
    H = CODES["hamming"]
    lam, V = spe.tanner_spectrum(H)
    p = random_spe_params(len(lam), 8, 2, seed=1)
    T = spe.spe_table_from_spectrum(lam, V, p, d=32)
    assert T.shape == (10, 32)
    assert np.all(T[:, :24] == 0)
    assert np.allclose(T[:, 24:], spe.spe_vectors(lam, V, p))
