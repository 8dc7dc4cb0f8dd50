"""Seeded synthetic inputs for the AECCT inference path.

This package builds what a decoder is *given*: parity-check matrices of the
code families the paper evaluates (Hamming, BCH, regular LDPC), random ternary
model weights with the shapes of an AECCT encoder, and BPSK/AWGN channel words.
It holds none of the decoder's own arithmetic (no syndrome, no attention, no
quantisation), so that the CPU oracle and the GPU path can both be fed from it
without sharing any of the method's code.
"""
from .codes import hamming_7_4, bch_31_16, regular_ldpc_3_6, generator_from_parity, gf2_rank
from .model import random_weights, random_spe_params, random_qat_params, with_positional_table, ModelWeights
from .channel import awgn_words
from .configs import CONFIGS, WorkloadConfig, build_workload

__all__ = [
    "hamming_7_4", "bch_31_16", "regular_ldpc_3_6", "generator_from_parity", "gf2_rank",
    "random_weights", "random_spe_params", "random_qat_params", "with_positional_table", "ModelWeights", "awgn_words", "CONFIGS", "WorkloadConfig", "build_workload",
]
