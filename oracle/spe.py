"""Spectral positional encoding (SPE) of the Tanner graph -- TEST INFRASTRUCTURE ONLY.

Plain numpy, float64, one node at a time; the eigendecomposition is numpy's `eigh`
(a library primitive used as one step).  Only the test suite may use this module.

What is computed (Section 4.3, the SPE equations and Fig. 4):
  graph      the Tanner graph of H: L = n + m nodes, variable nodes 0..n-1 first, then
             the checks; node i and node n + j are joined where H[j, i] = 1;
  Laplacian  the combinatorial Laplacian D - A of that graph;
  spectrum   all L eigenvalues, ascending, with unit eigenvectors phi_1..phi_L in the
             canonical basis below (the paper leaves signs and bases within repeated
             eigenvalues unspecified);
  per node j Phi_j in R^{L x 2}: row i = (lambda_i, phi_i[j]);
             Z = Phi_j W_in + b_in (W_in = W_{2->d_PE});
             Q = K = V = Z, then textbook multi-head self-attention over the L rows:
               per head h, Q_h = Z W_q + b_q (its d_PE/heads columns), K_h, V_h alike,
               softmax(Q_h K_h^T / sqrt(d_PE/heads)) V_h, heads concatenated, then
               W_o + b_o, giving U in R^{L x d_PE};
             SPE_j = w_red^T U + b_red (W_{(2n-k)->1} as a linear map over the L rows);
  table      row j of the L x d positional table: zeros in columns 0..d-d_PE-1 and SPE_j
             in the last d_PE columns, so that with an embedding whose last d_PE
             columns are zero, t_j E_j + P_j is the concatenation [t_j E_j, SPE_j].

Canonical eigenbasis.  Eigenvalues are grouped into clusters of consecutive values that
differ by at most CLUSTER_TOL * max(1, max |lambda|).  Each cluster's eigenspace is given
by its orthogonal projector P (unique, whatever basis an eigensolver returns).  Its
basis is built by walking the columns P e_c in ascending c, removing from each the
components along the vectors already taken (twice, for orthogonality), and taking the
normalised remainder when its squared norm exceeds ACCEPT_TOL, until the cluster's
dimension is reached.  A vector so built has a positive entry at its column c, so this
also fixes signs: for a simple eigenvalue, the first entry of squared size above
ACCEPT_TOL is positive.
"""
from __future__ import annotations

import numpy as np

CLUSTER_TOL = 1e-8
ACCEPT_TOL = 1e-6


def tanner_laplacian(H) -> np.ndarray:
    """D - A of the Tanner graph (variable nodes first, then checks), int64."""
    H = np.asarray(H, dtype=np.int64)
    m, n = H.shape
    L = n + m
    A = np.zeros((L, L), np.int64)
    A[:n, n:] = H.T
    A[n:, :n] = H
    return np.diag(A.sum(axis=1)) - A


def canonical_eigenbasis(lam, vecs):
    """Ascending eigenvalues and the canonical basis of each eigenspace.

    lam: [L] eigenvalues; vecs: [L, L] with column i a unit eigenvector of lam[i] (any
    orthonormal basis).  Returns (lam sorted, V) with V[:, i] the canonical vector i.
    """
    lam = np.asarray(lam, np.float64)
    vecs = np.asarray(vecs, np.float64)
    order = np.argsort(lam, kind="stable")
    lam = lam[order]
    vecs = vecs[:, order]
    L = lam.size
    out = np.zeros_like(vecs)
    tol = CLUSTER_TOL * max(1.0, float(np.abs(lam).max()))
    start = 0
    while start < L:
        end = start + 1
        while end < L and lam[end] - lam[end - 1] <= tol:
            end += 1
        Vc = vecs[:, start:end]
        r = end - start
        basis = []
        for c in range(L):
            u = Vc @ Vc[c, :]                      # column c of the projector Vc Vc^T
            for _ in range(2):
                for b in basis:
                    u = u - (b @ u) * b
            nn = float(u @ u)
            if nn > ACCEPT_TOL:
                basis.append(u / np.sqrt(nn))
                if len(basis) == r:
                    break
        assert len(basis) == r, "eigenspace basis incomplete"
        out[:, start:end] = np.stack(basis, axis=1)
        start = end
    return lam, out


def tanner_spectrum(H):
    """(eigenvalues ascending [L], V [L, L] with column i the canonical eigenvector i)."""
    lam, vecs = np.linalg.eigh(tanner_laplacian(H).astype(np.float64))
    return canonical_eigenbasis(lam, vecs)


def _row(a, width):
    return np.zeros(width) if a is None else np.asarray(a, np.float64).reshape(width)


def spe_node_attention(lam, V, j, p):
    """U in R^{L x d_PE}: the multi-head self-attention output over node j's L eigen-rows."""
    d_pe, heads = p["d_pe"], p["heads"]
    dk = d_pe // heads
    Phi = np.stack([np.asarray(lam, np.float64), np.asarray(V, np.float64)[j, :]], axis=1)
    Z = Phi @ np.asarray(p["w_in"], np.float64).reshape(2, d_pe) + _row(p.get("b_in"), d_pe)
    proj = {}
    for name in ("q", "k", "v"):
        proj[name] = (Z @ np.asarray(p["w_" + name], np.float64).reshape(d_pe, d_pe)
                      + _row(p.get("b_" + name), d_pe))
    L = Z.shape[0]
    O = np.zeros((L, d_pe))
    for h in range(heads):
        cols = slice(h * dk, (h + 1) * dk)
        S = proj["q"][:, cols] @ proj["k"][:, cols].T / np.sqrt(dk)
        S = S - S.max(axis=1, keepdims=True)
        E = np.exp(S)
        O[:, cols] = (E / E.sum(axis=1, keepdims=True)) @ proj["v"][:, cols]
    return O @ np.asarray(p["w_o"], np.float64).reshape(d_pe, d_pe) + _row(p.get("b_o"), d_pe)


def spe_vectors(lam, V, p, nodes=None):
    """SPE_j for the given nodes (all by default), float64 [len(nodes), d_PE]."""
    L = len(lam)
    nodes = range(L) if nodes is None else nodes
    w_red = np.asarray(p["w_red"], np.float64).reshape(L)
    return np.stack([w_red @ spe_node_attention(lam, V, j, p) + float(p.get("b_red", 0.0))
                     for j in nodes])


def spe_table_from_spectrum(lam, V, p, d: int, nodes=None):
    """Positional table rows [len(nodes), d], float64: zeros, then SPE_j in the last d_PE columns."""
    s = spe_vectors(lam, V, p, nodes)
    t = np.zeros((s.shape[0], d))
    t[:, d - p["d_pe"]:] = s
    return t


def spe_table(H, p, d: int, nodes=None):
    """The whole Section 4.3 construction from H: spectrum, then the table."""
    lam, V = tanner_spectrum(H)
    return spe_table_from_spectrum(lam, V, p, d, nodes)
