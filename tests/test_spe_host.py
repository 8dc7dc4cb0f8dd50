"""The library's SPE host steps (no GPU): Tanner-graph spectrum and canonical eigenbasis
equal to the oracle's (numpy's eigh + the oracle's canonical basis), argument errors."""
import numpy as np
import pytest

import paper_2410_05911_amd as P
from oracle import spe
from workloads import CONFIGS, hamming_7_4, random_spe_params, regular_ldpc_3_6
from workloads.configs import parity_check


def cycle_code(n):
    H = np.zeros((n, n), np.uint8)
    for j in range(n):
        H[j, j] = 1
        H[j, (j + 1) % n] = 1
    return H


CODES = {
    **{f"workload{c}": (lambda c=c: parity_check(CONFIGS[c])) for c in CONFIGS},
    "ldpc64": lambda: regular_ldpc_3_6(64, seed=7),
    "cycle7": lambda: cycle_code(7),
    "k35": lambda: np.ones((3, 5), np.uint8),
    "k44": lambda: np.ones((4, 4), np.uint8),
}


@pytest.mark.parametrize("name", list(CODES))
def test_spectrum_matches_oracle(name):
    H = CODES[name]()
    lam, V = P.tanner_spectrum(H)            # rows are eigenvectors
    lam_o, V_o = spe.tanner_spectrum(H)      # columns are eigenvectors
    Lap = spe.tanner_laplacian(H).astype(np.float64)
    assert np.all(np.diff(lam) >= 0)
    assert np.allclose(lam, lam_o, atol=1e-10)
    assert np.allclose(V @ V.T, np.eye(lam.size), atol=1e-10)
    assert np.abs(V @ Lap - lam[:, None] * V).max() < 1e-9
    assert np.abs(V - V_o.T).max() < 1e-8


def test_disconnected_graph():
    # two copies of the Hamming graph side by side: eigenvalue 0 twice, each eigenspace
    # basis still canonical
    h = hamming_7_4()
    H = np.zeros((6, 14), np.uint8)
    H[:3, :7] = h
    H[3:, 7:] = h
    lam, V = P.tanner_spectrum(H)
    lam_o, V_o = spe.tanner_spectrum(H)
    assert abs(lam[0]) < 1e-12 and abs(lam[1]) < 1e-12 and lam[2] > 1e-3
    assert np.allclose(lam, lam_o, atol=1e-10)
    assert np.abs(V - V_o.T).max() < 1e-8


def test_spectrum_errors():
    with pytest.raises(P.AecctError) as e:
        P.tanner_spectrum(np.full((3, 7), 2, np.uint8))
    assert e.value.status == P.ERR_INVALID_ARG
    with pytest.raises(P.AecctError) as e:
        P.tanner_spectrum(np.ones((2048, 2049), np.uint8))   # L above 4096
    assert e.value.status == P.ERR_INVALID_ARG


@pytest.mark.parametrize("field,value", [("heads", 3), ("d_pe", 40), ("heads", 0), ("w_in", "nan"),
                                         ("w_q", None), ("w_red", None)])
def test_spe_table_argument_errors(field, value):
    # rejected before any GPU work, so these run on the host
    H = hamming_7_4()
    p = random_spe_params(10, 8, 2, seed=0)
    if value == "nan":
        p[field] = p[field].copy()
        p[field][0, 0] = np.nan
    else:
        p[field] = value
    with pytest.raises(P.AecctError) as e:
        P.spe_table(H, p, d=32)
    assert e.value.status == P.ERR_INVALID_ARG
