"""GPU parity of the spectral positional encoding (Section 4.3) against the float64 oracle.

The library runs the per-node attention on the GPU in fp32 (exp2 on the hardware unit)
after folding the projections into a 3 x 3 score form per head; the oracle runs the
textbook multi-head attention in float64.  Tolerance: the GPU's error is dominated by fp32
sums over the L eigen-rows (bounded by about L u times the sum of the absolute terms,
u = 2^-24), so the test allows 8 L u (1 + max |table|), and never less than
2e-5 (1 + max |table|) for the fp32 rounding of the scores and of 2^x.
A decode with the resulting table is then compared bit for bit with the oracle's decode
(the table is an ordinary fp32 input of the canonical path).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle import spe  # noqa: E402
from workloads import CONFIGS, build_workload, random_spe_params, with_positional_table  # noqa: E402
from workloads.configs import parity_check  # noqa: E402


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_05911_amd as P
    P.lib()
    return P


def _tol(L, ref):
    return max(8 * L * 2.0 ** -24, 2e-5) * (1.0 + float(np.abs(ref).max()))


def _cycle_code(n):
    H = np.zeros((n, n), np.uint8)
    for j in range(n):
        H[j, j] = 1
        H[j, (j + 1) % n] = 1
    return H


# (workload, d, d_pe, heads, nodes checked: None = all)
FROM_SPECTRUM = [(1, 32, 8, 2, None), (2, 32, 16, 4, None), (2, 32, 4, 4, None), (3, 64, 16, 4, None),
                 (4, 128, 32, 4, 48), (5, 128, 32, 8, 8)]


@pytest.mark.parametrize("c,d,d_pe,heads,n_nodes", FROM_SPECTRUM)
def test_spe_from_oracle_spectrum(P, c, d, d_pe, heads, n_nodes):
    """The library's table from the oracle's own spectrum: only the attention differs."""
    print(f"[spe] workload {c} d {d} d_pe {d_pe} heads {heads}", flush=True)
    H = parity_check(CONFIGS[c])
    lam, V = spe.tanner_spectrum(H)
    L = lam.size
    p = random_spe_params(L, d_pe, heads, seed=60 + c)
    got = P.spe_table_from_spectrum(lam, V.T, p, d)
    assert got.shape == (L, d) and got.dtype == np.float32
    assert np.all(got[:, :d - d_pe] == 0)
    nodes = None if n_nodes is None else np.random.default_rng(c).choice(L, n_nodes, replace=False)
    ref = spe.spe_table_from_spectrum(lam, V, p, d, nodes=nodes)
    g = got if nodes is None else got[nodes]
    err = np.abs(g.astype(np.float64) - ref).max()
    print(f"[spe] workload {c}: max |err| {err:.3g}, max |table| {np.abs(ref).max():.3g}", flush=True)
    assert err <= _tol(L, ref), err


@pytest.mark.parametrize("name", ["hamming", "bch", "ldpc128", "cycle9", "k35"])
def test_spe_table_end_to_end(P, name):
    """aecct_spe_table (library spectrum and canonical basis, then GPU attention) against the
    oracle's whole construction (numpy eigh, its own canonical basis, float64 attention)."""
    print(f"[spe-e2e] {name}", flush=True)
    H = {"hamming": lambda: parity_check(CONFIGS[1]), "bch": lambda: parity_check(CONFIGS[2]),
         "ldpc128": lambda: parity_check(CONFIGS[3]), "cycle9": lambda: _cycle_code(9),
         "k35": lambda: np.ones((3, 5), np.uint8)}[name]()
    m, n = H.shape
    p = random_spe_params(n + m, 8, 2, seed=77)
    got = P.spe_table(H, p, 32)
    ref = spe.spe_table(H, p, 32)
    err = np.abs(got.astype(np.float64) - ref).max()
    print(f"[spe-e2e] {name}: max |err| {err:.3g}", flush=True)
    assert err <= _tol(n + m, ref), err


def test_spe_largest_graph(P):
    """L = 4096, the largest accepted: the attention from an orthonormal DCT-II basis standing in
    for a spectrum (the table is defined for any orthonormal eigenvectors), 3 sampled nodes."""
    L, d = 4096, 128
    print("[spe-max] L 4096", flush=True)
    k = np.arange(L)[:, None]
    x = np.arange(L)[None, :]
    V_rows = np.sqrt(2.0 / L) * np.cos(np.pi * (x + 0.5) * k / L)
    V_rows[0] /= np.sqrt(2.0)
    lam = np.sort(np.random.default_rng(2).uniform(0.0, 12.0, L))
    p = random_spe_params(L, 32, 4, seed=8)
    got = P.spe_table_from_spectrum(lam, V_rows, p, d)
    nodes = [0, 1777, L - 1]
    ref = spe.spe_table_from_spectrum(lam, V_rows.T, p, d, nodes=nodes)
    err = np.abs(got[nodes].astype(np.float64) - ref).max()
    print(f"[spe-max] max |err| {err:.3g}", flush=True)
    assert err <= _tol(L, ref), err


def test_spe_zero_input_map(P):
    """W_in = 0, b_in = 0: uniform attention, every node's SPE = sum(w_red)(b_v W_o + b_o) + b_red."""
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    p = random_spe_params(n + m, 8, 2, seed=5)
    p["w_in"] = np.zeros_like(p["w_in"])
    p["b_in"] = np.zeros_like(p["b_in"])
    got = P.spe_table(H, p, 32)[:, 24:].astype(np.float64)
    want = p["w_red"].astype(np.float64).sum() * (p["b_v"].astype(np.float64) @ p["w_o"] + p["b_o"]) + p["b_red"]
    assert np.abs(got - want[None, :]).max() <= 1e-6 * (1 + np.abs(want).max())


@pytest.mark.parametrize("c,d_pe", [(2, 8), (3, 16)])
def test_decode_with_spe_table(P, oracle_mod, c, d_pe):
    """A model whose positional table is the library's SPE table (embedding's last d_pe
    columns zero): the GPU decode equals the oracle's decode bit for bit, on every path."""
    print(f"[spe-decode] workload {c}", flush=True)
    cfg, H, G, w, y, x = build_workload(c, batch=96)
    m, n = H.shape
    p = random_spe_params(n + m, d_pe, 4, seed=90 + c)
    table = P.spe_table(H, p, w.d)
    w2 = with_positional_table(w, table, d_pe)
    om = oracle_mod.OracleModel(H, w2)
    bo, fo = om.decode(y, n_threads=16)
    paths = (P.PATH_FUSED, P.PATH_LAYERED) if w.d == 32 else (P.PATH_LAYERED,)
    for path in paths:
        dec = P.Decoder(H, w2, path=path)
        yd = torch.from_numpy(np.ascontiguousarray(y)).cuda()
        bits, logits = dec.decode(yd)
        torch.cuda.synchronize()
        assert np.array_equal(logits.cpu().numpy(), fo)
        assert np.array_equal(bits.cpu().numpy(), bo)
