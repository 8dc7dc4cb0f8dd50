"""BPSK over AWGN (Section 3, "Problem Settings"; SNR convention of Section 6).

A k-bit message m is encoded as x = m G (mod 2), modulated as x_s = 1 - 2x and sent
through y = x_s + eps with eps ~ N(0, sigma^2), where for a normalised SNR Eb/N0 (dB)
and rate R = k/n, sigma = (2 R 10^(Eb/N0 / 10))^(-1/2).
"""
from __future__ import annotations

import numpy as np


def awgn_words(G: np.ndarray, batch: int, ebn0_db, seed: int, *, zero_codeword: bool = False):
    """Return (y fp32 [B,n], x uint8 [B,n] codewords, ebn0 per word float64 [B])."""
    rng = np.random.default_rng(seed)
    k, n = G.shape
    rate = k / n
    if zero_codeword:
        x = np.zeros((batch, n), dtype=np.uint8)
    else:
        msg = rng.integers(0, 2, size=(batch, k), dtype=np.int64)
        x = ((msg @ G.astype(np.int64)) & 1).astype(np.uint8)
    levels = np.asarray(ebn0_db, dtype=np.float64)
    ebn0 = levels[rng.integers(0, levels.size, size=batch)]
    sigma = 1.0 / np.sqrt(2.0 * rate * 10.0 ** (ebn0 / 10.0))
    z = rng.standard_normal((batch, n))
    xs = 1.0 - 2.0 * x.astype(np.float64)
    y = (xs + sigma[:, None] * z).astype(np.float32)
    return y, x, ebn0
