"""The five synthetic workloads: codes, model sizes, batch and channel SNR sets.

Seeds: parity-check construction 1000+c, weights 2000+c, channel data 3000+c for
workload index c = 1..5.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .codes import hamming_7_4, bch_31_16, regular_ldpc_3_6, generator_from_parity
from .model import random_weights
from .channel import awgn_words


@dataclass(frozen=True)
class WorkloadConfig:
    index: int
    name: str
    code: str          # "hamming", "bch", "ldpc"
    n: int
    d: int
    n_layers: int
    heads: int
    p_zero: float
    ebn0: tuple
    batch: int

    @property
    def seeds(self):
        return 1000 + self.index, 2000 + self.index, 3000 + self.index


CONFIGS = {
    1: WorkloadConfig(1, "hamming7_4_d32_N2", "hamming", 7, 32, 2, 8, 0.5, (4.0, 5.0, 6.0), 1024),
    2: WorkloadConfig(2, "bch31_16_d32_N6", "bch", 31, 32, 6, 8, 0.5, (4.0, 5.0, 6.0, 7.0), 65536),
    3: WorkloadConfig(3, "ldpc128_64_d64_N6", "ldpc", 128, 64, 6, 8, 0.5, (2.0, 3.0, 4.0, 5.0), 32768),
    4: WorkloadConfig(4, "ldpc256_128_d128_N10", "ldpc", 256, 128, 10, 8, 0.6, (2.0, 3.0, 4.0, 5.0), 16384),
    5: WorkloadConfig(5, "ldpc1024_512_d128_N10", "ldpc", 1024, 128, 10, 8, 0.5, (1.5, 2.0, 2.5, 3.0), 4096),
}

_H_CACHE: dict = {}


def parity_check(cfg: WorkloadConfig) -> np.ndarray:
    key = cfg.index
    if key not in _H_CACHE:
        if cfg.code == "hamming":
            H = hamming_7_4()
        elif cfg.code == "bch":
            H = bch_31_16()
        else:
            H = regular_ldpc_3_6(cfg.n, seed=cfg.seeds[0])
        _H_CACHE[key] = H
    return _H_CACHE[key].copy()


def build_workload(index: int, batch: int | None = None, *, data_seed: int | None = None,
                   attention: str = "hpsa", first_ring_heads: int | None = None, act_scale: str = "token"):
    """(cfg, H, G, weights, y, x) for workload `index`; `batch` overrides the configured batch,
    `attention` picks the head-partitioned ("hpsa") or all-heads-ECCT-mask ("casa") model,
    `first_ring_heads` the number h_f of heads on the first-ring mask (default heads / 2),
    `act_scale` the Eq. 2 scale granularity ("token" or "word")."""
    cfg = CONFIGS[index]
    H = parity_check(cfg)
    G = generator_from_parity(H)
    m, n = H.shape
    w = random_weights(n, m, cfg.d, cfg.n_layers, cfg.heads, p_zero=cfg.p_zero, seed=cfg.seeds[1],
                       attention=attention, first_ring_heads=first_ring_heads, act_scale=act_scale)
    B = cfg.batch if batch is None else batch
    y, x, _ = awgn_words(G, B, cfg.ebn0, seed=cfg.seeds[2] if data_seed is None else data_seed)
    return cfg, H, G, w, y, x
