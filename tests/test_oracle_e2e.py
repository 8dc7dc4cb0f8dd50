"""End-to-end pins of the oracle's decode (Sections 3, 4, 6)."""
import math

import numpy as np
import pytest
import torch

from workloads import CONFIGS, build_workload, random_weights
from workloads.configs import parity_check
from workloads.channel import awgn_words
from workloads.codes import generator_from_parity


@pytest.mark.parametrize("c", [1, 2, 3])
def test_codeword_invariance(oracle_mod, c):
    """h(y) depends only on |y| and the syndrome (Section 3), so decoding x_s + e and 1 + x_s e
    gives the same noise estimate bit for bit and bits that differ exactly by the codeword."""
    cfg, H, G, w, y, x = build_workload(c, batch=64 if c < 3 else 4)
    om = oracle_mod.OracleModel(H, w)
    xs = (1 - 2 * x.astype(np.int8)).astype(np.float32)
    y0 = (xs * y).astype(np.float32)                    # exact: multiplying by +-1
    bits, f = om.decode(y, n_threads=8)
    bits0, f0 = om.decode(y0, n_threads=8)
    assert (f == f0).all()
    assert ((bits ^ x) == bits0).all()


def test_zero_weight_closed_form(oracle_mod):
    """All ternary weights zero: every linear layer returns its bias, attention rows average
    identical value rows, and the network reduces to X <- LN2(LN1(X + b_o) + b_ff2) per layer."""
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    w = random_weights(n, m, 32, 3, 8, seed=11, zero_linear=True)
    om = oracle_mod.OracleModel(H, w)
    G = generator_from_parity(H)
    y, x, _ = awgn_words(G, 8, (3.0,), seed=5)
    bits, f = om.decode(y)

    def ln(R, g, b):
        t = torch.tensor(R)
        return torch.nn.functional.layer_norm(t, (R.shape[1],), torch.tensor(g, dtype=torch.float64),
                                              torch.tensor(b, dtype=torch.float64), eps=w.ln_eps).numpy()
    L = n + m
    for bi in range(8):
        yb = y[bi].astype(np.float64)
        s = (H.astype(np.int64) @ (yb < 0).astype(np.int64)) % 2
        t = np.concatenate([np.abs(yb), 1 - 2 * s])
        X = t[:, None] * w.embed.astype(np.float64)
        for l in range(w.n_layers):
            X1 = ln(X + w.b["o"][l].astype(np.float64)[None], w.ln1_g[l], w.ln1_b[l])
            X = ln(X1 + w.b["ff2"][l].astype(np.float64)[None], w.ln2_g[l], w.ln2_b[l])
        z = X @ w.head_w1.astype(np.float64) + w.head_b1
        fr = z @ w.head_wo.astype(np.float64) + w.head_bo
        assert np.abs(f[bi] - fr).max() <= 2e-5


@pytest.mark.parametrize("attention", ["hpsa", "casa"])
def test_fp32_canonical_close_to_fp64_reference(oracle_mod, attention):
    """The canonical fp32 decode against the oracle's fp64 dense mode on Hamming(7,4), with the
    head-partitioned masks and with the ECCT mask on every head.  Differences come only from fp32
    rounding and the rare int8 code that sits on a rounding boundary; most words agree to ~1e-6."""
    cfg, H, G, w, y, x = build_workload(1, batch=1024, attention=attention)
    om = oracle_mod.OracleModel(H, w)
    bits, f = om.decode(y, n_threads=8)
    bits64, f64 = om.decode_ref64(y, n_threads=8)
    err = np.abs(f - f64).max(1)
    assert np.median(err) < 2e-6
    assert (err <= 1e-4).mean() >= 0.97
    assert err.max() < 0.05
    sure = np.abs(f64) > 0.05
    assert (bits[sure] == bits64[sure]).all()


def _q64(x):
    a = np.abs(x).max(1, keepdims=True)
    return np.clip(np.rint(x * (127.0 / np.where(a == 0, 1, a))), -127, 127), a[:, 0]


@pytest.mark.parametrize("c", [1, 2, 3])
def test_taps_stagewise_against_fp64(oracle_mod, c):
    """Every stage of the fp32 decode, fed the oracle's own int8 codes at each quantisation point,
    recomputed in fp64 with numpy/torch: QKV projections, HPSA attention, O projection + LN1,
    FFN + LN2 and the head all agree to fp32 rounding, and the int8 codes themselves differ from
    the fp64 rounding decision by at most one step on a rounding tie."""
    from test_oracle_units import _sdpa_reference
    cfg, H, G, w, y, x = build_workload(c, batch=2)
    om = oracle_mod.OracleModel(H, w)
    bits, f, t = om.decode_taps(y[1])
    d = w.d

    def lin(q, a, T, s, b):
        return (q.astype(np.int64) @ T.astype(np.int64)) * (float(s) * a[:, None] / 127.0) + b[None].astype(np.float64)

    def ln(R, g, b):
        return torch.nn.functional.layer_norm(torch.tensor(R), (d,), torch.tensor(g, dtype=torch.float64),
                                              torch.tensor(b, dtype=torch.float64), eps=w.ln_eps).numpy()

    def close(a, b, tol):
        assert np.abs(np.asarray(a, np.float64) - b).max() <= tol * max(1.0, np.abs(b).max())

    flips = 0
    for l in range(w.n_layers):
        sc = w.scale[l]
        q64, a64 = _q64(t["x_in"][l].astype(np.float64))
        flips += int((q64 != t["xq"][l]).sum())
        assert np.abs(q64 - t["xq"][l]).max() <= 1
        assert (a64 == t["ax"][l]).all()
        qkv = np.concatenate([lin(t["xq"][l], t["ax"][l], w.w[k][l], sc[i], w.b[k][l])
                              for i, k in enumerate(("q", "k", "v"))], 1)
        qkv[:, :d] *= math.log2(math.e) / math.sqrt(d // w.heads)      # scaled queries
        close(t["qkv"][l], qkv, 1e-6)
        close(t["o"][l], _sdpa_reference(H, w, t["qkv"][l]), 2e-6)
        q64, a64 = _q64(t["o"][l].astype(np.float64))
        flips += int((q64 != t["oq"][l]).sum())
        assert np.abs(q64 - t["oq"][l]).max() <= 1
        assert (t["acc_o"][l] == t["oq"][l].astype(np.int64) @ w.w["o"][l].astype(np.int64)).all()
        x1 = ln(t["x_in"][l].astype(np.float64) + lin(t["oq"][l], t["ao"][l], w.w["o"][l], sc[3], w.b["o"][l]),
                w.ln1_g[l], w.ln1_b[l])
        close(t["x1"][l], x1, 1e-5)
        F = np.maximum(lin(t["x1q"][l], t["a1"][l], w.w["ff1"][l], sc[4], w.b["ff1"][l]), 0)
        q64, a64 = _q64(F)
        flips += int((q64 != t["gq"][l]).sum())
        assert np.abs(q64 - t["gq"][l]).max() <= 1
        close(t["ag"][l], a64, 1e-6)
        xo = ln(t["x1"][l].astype(np.float64) + lin(t["gq"][l], t["ag"][l], w.w["ff2"][l], sc[5], w.b["ff2"][l]),
                w.ln2_g[l], w.ln2_b[l])
        close(t["x_out"][l], xo, 1e-5)
        if l + 1 < w.n_layers:
            assert (t["x_in"][l + 1] == t["x_out"][l]).all()
    z = t["x_out"][-1].astype(np.float64) @ w.head_w1.astype(np.float64) + w.head_b1
    close(t["z"], z, 1e-5)
    close(f, z @ w.head_wo.astype(np.float64) + w.head_bo, 1e-5)
    total = sum(t[k].size for k in ("xq", "oq", "gq"))
    assert flips <= max(3, total * 1e-4)
