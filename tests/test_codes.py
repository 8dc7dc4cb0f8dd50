"""Pins of the synthetic code constructions (Section 3, "Problem Settings": G H^T = 0, Hx = 0)."""
import itertools
import os

import numpy as np
import pytest

from workloads import hamming_7_4, bch_31_16, regular_ldpc_3_6, generator_from_parity, gf2_rank
from workloads.codes import bch_generator_31, bch_31_16_generator, _poly_divmod_gf2

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _codewords(G):
    k = G.shape[0]
    msgs = np.array(list(itertools.product([0, 1], repeat=k)), dtype=np.int64)
    return (msgs @ G.astype(np.int64)) & 1


def _dmin(G):
    cw = _codewords(G)
    w = cw.sum(1)
    return int(w[w > 0].min())


def test_hamming_matrix_and_distance():
    H = hamming_7_4()
    assert H.tolist() == [[1, 1, 0, 1, 1, 0, 0], [1, 0, 1, 1, 0, 1, 0], [0, 1, 1, 1, 0, 0, 1]]
    G = generator_from_parity(H)
    assert G.shape == (4, 7)
    assert not ((G.astype(int) @ H.T) % 2).any()
    assert _dmin(G) == 3


def test_bch_generator_matches_textbook_table():
    octal = [ln.split()[1] for ln in open(os.path.join(GOLDEN, "bch31_16_generator.txt"))
             if ln.startswith("octal")][0]
    bits = bin(int(octal, 8))[2:]                # highest degree first
    expected = [int(b) for b in bits[::-1]]      # low degree first
    g = bch_generator_31()
    assert g == expected
    assert len(g) - 1 == 15
    q, rem = _poly_divmod_gf2([1] + [0] * 30 + [1], g)
    assert not any(rem)


def test_bch_parity_check_and_distance():
    H = bch_31_16()
    assert H.shape == (15, 31)
    assert gf2_rank(H) == 15
    G = bch_31_16_generator()
    assert not ((G.astype(int) @ H.T) % 2).any()
    G2 = generator_from_parity(H)
    assert G2.shape == (16, 31)
    assert not ((G2.astype(int) @ H.T) % 2).any()
    assert _dmin(G) == 7                         # designed distance 2t+1 = 7, brute force over 2^16 words
    assert set(H.sum(1).tolist()) == {8}         # weight of h(x)


@pytest.mark.parametrize("n", [128, 256, 1024])
def test_ldpc_regular_girth6(n):
    H = regular_ldpc_3_6(n, seed=1000 + n)
    m = n // 2
    assert H.shape == (m, n)
    assert (H.sum(0) == 3).all() and (H.sum(1) == 6).all()
    Hf = H.astype(np.float64)
    ov = Hf @ Hf.T
    np.fill_diagonal(ov, 0)
    assert ov.max() <= 1                         # no two checks share two variables: no 4-cycle
    G = generator_from_parity(H)
    assert G.shape[0] == n - gf2_rank(H)
    assert not ((G.astype(np.int64) @ H.T) % 2).any()


def test_ldpc_seed_determinism():
    a = regular_ldpc_3_6(128, seed=7)
    b = regular_ldpc_3_6(128, seed=7)
    c = regular_ldpc_3_6(128, seed=8)
    assert (a == b).all() and (a != c).any()


def test_generator_from_parity_random():
    rng = np.random.default_rng(0)
    for _ in range(20):
        H = (rng.random((6, 12)) < 0.4).astype(np.uint8)
        G = generator_from_parity(H)
        assert G.shape[0] == 12 - gf2_rank(H)
        assert gf2_rank(G) == G.shape[0]
        assert not ((G.astype(int) @ H.T) % 2).any()
