"""Pins of the CPU oracle's building blocks against facts fixed outside it.

Each test checks an oracle function against mathematics or an independent library
routine (numpy int64 matmul, torch fp64 layer_norm / scaled-dot-product attention,
Python's math.exp), never against a retyped copy of the oracle's own formula.
"""
import math

import numpy as np
import pytest
import torch

from workloads import CONFIGS, build_workload, random_weights
from workloads.configs import parity_check


def _ulp(x):
    return np.spacing(np.float32(abs(x)))


# ------------------------------------------------------------------------ TREE order
def test_tree_sum_pairs_stride_halving(oracle_mod):
    # pairs (v0+v2), (v1+v3): the large terms cancel first, so the exact 2 survives;
    # a left-to-right sum would absorb the first 1 into 1e8 and give 1.
    assert oracle_mod.tree_sum([1e8, 1.0, -1e8, 1.0]) == np.float32(2.0)
    # w = 8: stride 4 pairs (0,4),(1,5),(2,6),(3,7)
    v = np.array([1e8, 0, 0, 1, -1e8, 0, 0, 1], np.float32)
    assert oracle_mod.tree_sum(v) == np.float32(2.0)
    rng = np.random.default_rng(0)
    for w in (1, 2, 4, 8, 16, 32, 64, 128, 512):
        ints = rng.integers(-1000, 1000, w).astype(np.float32)
        assert oracle_mod.tree_sum(ints) == np.float32(ints.astype(np.int64).sum())  # exact integer sums
        x = rng.standard_normal(w).astype(np.float32)
        exact = math.fsum(x.astype(np.float64))
        bound = (max(1, math.log2(w)) * 2 ** -24) * np.abs(x).astype(np.float64).sum() * 1.01
        assert abs(float(oracle_mod.tree_sum(x)) - exact) <= bound + 1e-30


# ------------------------------------------------------------------------ EXP2, RSQRT
def test_exp2_close_to_pow_and_exact_at_integers(oracle_mod):
    for k in range(0, 126):
        assert oracle_mod.exp2(-float(k)) == np.float32(2.0 ** -k)
    assert oracle_mod.exp2(-0.0) == np.float32(1.0)
    for k in range(1, 128):
        assert oracle_mod.exp2(float(k)) == np.float32(2.0 ** k)
    assert oracle_mod.exp2(-200.0) == np.float32(2.0 ** -125)      # clamped: stays a normal number
    for x in (128.0, 1e30):                                          # clamped at 128: 2^128 is +inf
        assert np.isinf(oracle_mod.exp2(x)) and oracle_mod.exp2(x) > 0
    for x in (np.float32(127.4), np.float32(127.75)):               # still finite below 2^128
        assert abs(float(oracle_mod.exp2(x)) - 2.0 ** float(x)) <= 3e-7 * 2.0 ** float(x)
    xs = np.concatenate([np.linspace(-125, 64, 50001, dtype=np.float32),
                         -np.random.default_rng(1).random(20000).astype(np.float32) * 125])
    worst = 0.0
    for x in xs:
        e = float(oracle_mod.exp2(x))
        ref = 2.0 ** float(x)
        worst = max(worst, abs(e - ref) / ref)
    assert worst <= 3e-7, worst


def test_rsqrt_close_to_exact(oracle_mod):
    rng = np.random.default_rng(2)
    vs = np.concatenate([np.exp(rng.uniform(math.log(1e-5), math.log(1e4), 20000)),
                         [1e-5, 0.25, 1.0, 2.0, 3.0, 4.0, 1e4]]).astype(np.float32)
    worst = 0.0
    for v in vs:
        ref = 1.0 / math.sqrt(float(v))
        worst = max(worst, abs(float(oracle_mod.rsqrt(v)) - ref) / float(_ulp(ref)))
    assert worst <= 2.0, worst


def test_query_scale(oracle_mod):
    for dh in (4, 8, 16):
        assert oracle_mod.query_scale(dh) == np.float32(1.0 / (math.log(2.0) * math.sqrt(dh)))


# ------------------------------------------------------------------------ pre-processing
def test_syndrome_of_codewords_is_zero(oracle_mod):
    for c in (1, 2, 3):
        cfg, H, G, w, y, x = build_workload(c, batch=64)
        m, n = H.shape
        xs = (1.0 - 2.0 * x).astype(np.float32)
        for b in range(16):
            t = oracle_mod.preprocess(H, xs[b])
            assert (t[:n] == 1.0).all()
            assert (t[n:] == 1.0).all()                       # s = 0  ->  1 - 2s = +1
            # magnitudes of a noisy word, and -0.0 counts as a positive sign (bit 0)
            t = oracle_mod.preprocess(H, y[b])
            assert (t[:n] == np.abs(y[b])).all()
        z = np.zeros(n, np.float32)
        z[0] = -0.0
        assert (oracle_mod.preprocess(H, z)[n:] == 1.0).all()


def test_single_error_syndrome_is_column(oracle_mod):
    H = parity_check(CONFIGS[2])
    m, n = H.shape
    for i in range(n):
        y = np.ones(n, np.float32)
        y[i] = -0.3
        t = oracle_mod.preprocess(H, y)
        s = (1 - t[n:]) / 2
        assert (s.astype(np.uint8) == H[:, i]).all()


# ------------------------------------------------------------------------ quantisation (Eq. 2)
def test_quant_invariants(oracle_mod):
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((400, 128)) * rng.exponential(1, (400, 1))).astype(np.float32)
    q, r = oracle_mod.quant_rows(x)
    assert (np.abs(q.astype(int)) <= 127).all()
    assert (r == np.abs(x).max(1)).all()
    am = np.abs(x).argmax(1)
    assert (np.abs(q[np.arange(400), am]) == 127).all()
    assert ((np.sign(q) == np.sign(x)) | (q == 0)).all()
    # monotone within a row
    for i in range(20):
        o = np.argsort(x[i], kind="stable")
        assert (np.diff(q[i][o].astype(int)) >= 0).all()
    err = np.abs(x.astype(np.float64) - q * r[:, None].astype(np.float64) / 127)
    assert (err <= r[:, None] / 254 * (1 + 2 ** -20)).all()


def test_quant_zero_row_and_half_even(oracle_mod):
    q, r = oracle_mod.quant_rows(np.zeros((2, 8), np.float32))
    assert (q == 0).all() and (r == 0).all()
    # alpha = 127 -> Q_b / alpha = 1 exactly: rounding ties go to even
    x = np.array([[127.0, 2.5, 3.5, -2.5, -0.5, 0.5, 1.5, -126.5]], np.float32)
    q, r = oracle_mod.quant_rows(x)
    assert q[0].tolist() == [127, 2, 4, -2, 0, 0, 2, -126]


def test_quant_word_alpha_and_invariants(oracle_mod):
    """Eq. 2 with one alpha per word (the reading of Section 4.1 that takes alpha = ||x||_inf over
    the whole layer input): alpha is the library maximum of |x| over every row, all rows share it,
    the codes keep the invariants of Eq. 2 with that alpha, and a one-row word or a word whose
    rows share one maximum is quantised exactly as the per-token form."""
    rng = np.random.default_rng(13)
    x = (rng.standard_normal((46, 128)) * rng.exponential(1, (46, 1))).astype(np.float32)
    q, r = oracle_mod.quant_word(x)
    a = np.abs(x).max()
    assert (r == a).all()
    assert (np.abs(q.astype(int)) <= 127).all()
    i, j = np.unravel_index(np.abs(x).argmax(), x.shape)
    assert abs(int(q[i, j])) == 127
    assert ((np.sign(q) == np.sign(x)) | (q == 0)).all()
    o = np.argsort(x.reshape(-1), kind="stable")
    assert (np.diff(q.reshape(-1)[o].astype(int)) >= 0).all()            # monotone over the word
    err = np.abs(x.astype(np.float64) - q * float(a) / 127)
    assert (err <= float(a) / 254 * (1 + 2 ** -20)).all()
    # rows of a smaller maximum use fewer code levels than their own per-token quantisation
    qt, rt = oracle_mod.quant_rows(x)
    small = rt < a
    assert (np.abs(q[small]).max(1) <= np.abs(qt[small]).max(1)).all()
    # special cases that reduce to the per-token form
    q1, r1 = oracle_mod.quant_word(x[:1])
    qt1, rt1 = oracle_mod.quant_rows(x[:1])
    assert (q1 == qt1).all() and (r1 == rt1).all()
    xs = x / np.abs(x).max(1, keepdims=True) * np.float32(3.0)             # every row's max is 3
    xs[np.arange(46), np.abs(xs).argmax(1)] = np.float32(3.0)
    qa, ra = oracle_mod.quant_word(xs)
    qb, rb = oracle_mod.quant_rows(xs)
    assert (qa == qb).all() and (ra == rb).all()
    qz, rz = oracle_mod.quant_word(np.zeros((3, 8), np.float32))
    assert (qz == 0).all() and (rz == 0).all()


# ------------------------------------------------------------------------ AAPLinear (Eq. 3)
def test_linear_accumulators_and_dequant(oracle_mod):
    rng = np.random.default_rng(4)
    for K, N in ((32, 96), (128, 32), (512, 128)):
        q = rng.integers(-127, 128, (50, K)).astype(np.int8)
        T = rng.choice(np.array([-1, 0, 1], np.int8), (K, N))
        r = (rng.random(50) * 3).astype(np.float32)
        b = rng.standard_normal(N).astype(np.float32)
        s = np.float32(1 / math.sqrt(K))
        out, acc = oracle_mod.linear_rows(q, r, T, s, b)
        assert (acc == q.astype(np.int64) @ T.astype(np.int64)).all()
        ref = acc.astype(np.float64) * (float(s) * r[:, None].astype(np.float64) / 127) + b.astype(np.float64)
        assert np.allclose(out, ref, rtol=4e-7, atol=4e-7)
        out0, acc0 = oracle_mod.linear_rows(q, r, np.zeros_like(T), s, b)
        assert (acc0 == 0).all() and (out0 == b[None, :]).all()      # zero weights: output = bias


# ------------------------------------------------------------------------ LayerNorm
def test_layernorm_against_torch_fp64(oracle_mod):
    rng = np.random.default_rng(5)
    for d in (32, 64, 128):
        R = (rng.standard_normal((300, d)) * 3 + rng.standard_normal((300, 1))).astype(np.float32)
        g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
        b = (0.1 * rng.standard_normal(d)).astype(np.float32)
        out = oracle_mod.layernorm_rows(R, g, b, 1e-5)
        ref = torch.nn.functional.layer_norm(torch.tensor(R, dtype=torch.float64), (d,),
                                             torch.tensor(g, dtype=torch.float64),
                                             torch.tensor(b, dtype=torch.float64), eps=1e-5).numpy()
        assert np.abs(out - ref).max() <= 1e-5


# ------------------------------------------------------------------------ HPSA attention
def _sdpa_reference(H, w, qkv, scale=math.log(2.0)):
    """torch fp64 scaled-dot-product attention per head with boolean masks from H.  The oracle's
    query rows carry log2(e)/sqrt(d_h), so softmax(ln2 * q'.k) is the base-e softmax of q.k/sqrt(d_h)."""
    m, n = H.shape
    L = n + m
    A = np.zeros((L, L), np.int64)
    A[:n, n:] = H.T
    A[n:, :n] = H
    M1 = torch.tensor(A != 0)
    Af = A.astype(np.float64)                   # exact small integers; BLAS instead of an int64 loop
    M2 = torch.tensor((Af @ Af) != 0)
    d, h = w.d, w.heads
    dh = d // h
    t = torch.tensor(qkv, dtype=torch.float64)
    Q, K, V = t[:, :d], t[:, d:2 * d], t[:, 2 * d:]
    out = torch.zeros(L, d, dtype=torch.float64)
    for hh in range(h):
        sl = slice(hh * dh, (hh + 1) * dh)
        if getattr(w, "attention", "hpsa") == "casa":
            mask = M1 | M2                          # the ECCT mask for every head
        else:
            mask = M1 if hh < w.first_ring_heads else M2
        out[:, sl] = torch.nn.functional.scaled_dot_product_attention(
            Q[None, None, :, sl], K[None, None, :, sl].contiguous(), V[None, None, :, sl], attn_mask=mask,
            scale=scale)[0, 0]
    return out.numpy()


@pytest.mark.parametrize("attention", ["hpsa", "casa"])
@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_attention_against_fp64_sdpa(oracle_mod, c, attention):
    """Every workload's head width: d_h = 4 (Hamming, BCH), 8 (LDPC(128,64)) and 16 (the two
    d = 128 LDPC codes, whose dot products the canonical order splits into two 8-term halves)."""
    cfg, H, G, w, y, x = build_workload(c, batch=1, attention=attention)
    om = oracle_mod.OracleModel(H, w)
    rng = np.random.default_rng(6)
    qkv = rng.standard_normal((om.L, 3 * w.d)) * 2
    qkv[:, :w.d] *= math.sqrt(4 / (w.d // w.heads))    # the same score spread for every head width
    qkv = qkv.astype(np.float32)
    o = om.attention(qkv)
    ref = _sdpa_reference(H, w, qkv)
    assert np.abs(o - ref).max() <= 1e-6 * max(1.0, np.abs(ref).max())
    o64 = om.attention_dense_f64(qkv, math.log(2.0))        # the oracle's own dense fp64 mode
    assert np.abs(o64 - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())


@pytest.mark.parametrize("attention", ["hpsa", "casa"])
@pytest.mark.parametrize("c", [2, 4, 5])
@pytest.mark.parametrize("regime", ["overflow", "underflow", "mixed"])
def test_attention_shifted_fallback_against_fp64_sdpa(oracle_mod, regime, c, attention):
    """Rows whose unshifted weight sum leaves [2^-64, 2^64] take the max-shifted form: scores of
    a few hundred overflow 2^s, scores below -125 would all clamp to the same weight; on d_h = 4
    (BCH) and d_h = 16 (the d = 128 LDPC codes)."""
    cfg, H, G, w, y, x = build_workload(c, batch=1, attention=attention)
    om = oracle_mod.OracleModel(H, w)
    rng = np.random.default_rng(9)
    qkv = rng.standard_normal((om.L, 3 * w.d))
    d = w.d
    dh = d // w.heads
    # Scores of about 150-200 (base-2 units) for every head width: far outside the unshifted
    # range [2^-64, 2^64] of the weight sums, and of the same size at d_h = 4, 8 and 16 (fp32
    # rounding of a score grows like d_h |s|).  Random products add up like sqrt(d_h), the
    # same-sign products of the underflow rows like d_h.
    over = 20.0 * math.sqrt(4 / dh)
    if regime == "overflow":
        qkv[:, :d] *= over
    elif regime == "underflow":
        qkv[:, :d] = (np.abs(qkv[:, :d]) * 4.0 + 8.0) * (4 / dh)
        qkv[:, d:2 * d] = -np.abs(qkv[:, d:2 * d]) - 4.0
    else:                                   # a third of the tokens in each regime
        qkv[::3, :d] *= over
        qkv[1::3, :d] = (np.abs(qkv[1::3, :d]) * 4.0 + 8.0) * (4 / dh)
        qkv[1::3, d:2 * d] = -np.abs(qkv[1::3, d:2 * d]) - 4.0
    qkv = qkv.astype(np.float32)
    # share of (row, head) pairs whose unshifted weight sum sum_j 2^s_j leaves [2^-64, 2^64]
    M1, M2 = oracle_mod.masks(H)
    q64, k64 = qkv[:, :d].astype(np.float64), qkv[:, d:2 * d].astype(np.float64)
    out_of_range = []
    for hh in range(w.heads):
        sl = slice(hh * dh, (hh + 1) * dh)
        mask = (M1 | M2) if attention == "casa" else (M1 if hh < w.first_ring_heads else M2)
        sc = np.where(mask.astype(bool), q64[:, sl] @ k64[:, sl].T, -np.inf)
        S2 = np.log2(np.exp2(sc - sc.max(1, keepdims=True)).sum(1)) + sc.max(1)
        out_of_range.append((S2 > 64) | (S2 < -64))
    share = np.mean(out_of_range)
    assert share >= {"overflow": 0.3, "underflow": 1.0, "mixed": 0.15}[regime], share
    o = om.attention(qkv)
    ref = _sdpa_reference(H, w, qkv)
    assert np.isfinite(o).all()
    assert np.abs(o - ref).max() <= 1e-5 * max(1.0, np.abs(ref).max())


def test_attention_single_neighbour_rows_copy_value(oracle_mod):
    """Hamming variables 4, 5, 6 have one check each: their first-ring rows are that check's V,
    up to the three roundings of (e v) * (1 / e)."""
    cfg, H, G, w, y, x = build_workload(1, batch=1)
    om = oracle_mod.OracleModel(H, w)
    rng = np.random.default_rng(7)
    qkv = rng.standard_normal((om.L, 3 * w.d)).astype(np.float32)
    o = om.attention(qkv)
    d, dh, n = w.d, w.d // w.heads, H.shape[1]
    for v in (4, 5, 6):
        (chk,) = np.nonzero(H[:, v])[0]
        for hh in range(w.first_ring_heads):
            sl = slice(hh * dh, (hh + 1) * dh)
            ref = qkv[n + chk, 2 * d:][sl].astype(np.float64)
            assert (np.abs(o[v, sl] - ref) <= 3 * 2.0 ** -24 * np.abs(ref)).all()


# ------------------------------------------------------------------------ head
def test_head_against_fp64(oracle_mod):
    cfg, H, G, w, y, x = build_workload(2, batch=4)
    om = oracle_mod.OracleModel(H, w)
    rng = np.random.default_rng(8)
    X = rng.standard_normal((om.L, w.d)).astype(np.float32)
    f, bits, z = om.head(X, y[0])
    z64 = X.astype(np.float64) @ w.head_w1.astype(np.float64) + w.head_b1
    f64 = z64 @ w.head_wo.astype(np.float64) + w.head_bo
    assert np.abs(z - z64).max() <= 1e-5 and np.abs(f - f64).max() <= 1e-5
    assert (bits == ((y[0] * f) < 0)).all()                 # bin(y * f)


def test_casa_mask_is_ecct_mask_and_doubles_pairs(oracle_mod):
    """CASA (Section 3) lets every head see the nodes at most two Tanner steps away: its per-head
    pair count is |M1| + |M2|, twice HPSA's total over 8 heads when h_f = h_s (Section 4.2)."""
    cfg, H, G, w, y, x = build_workload(2, batch=1)
    M1, M2 = oracle_mod.masks(H)
    m, n = H.shape
    L = n + m
    # BFS distance <= 2 in the Tanner graph, self included
    A = np.zeros((L, L), bool)
    A[:n, n:] = H.T.astype(bool)
    A[n:, :n] = H.astype(bool)
    reach = np.eye(L, dtype=bool) | A | ((A.astype(int) @ A.astype(int)) > 0)
    assert ((M1.astype(bool) | M2.astype(bool)) == reach).all()
    hp = 4 * M1.sum() + 4 * M2.sum()
    ca = 8 * (M1.astype(bool) | M2.astype(bool)).sum()
    assert ca == 2 * hp
