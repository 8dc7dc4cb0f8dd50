"""AAP weight import (Section 4.1, Eq. 1): fp32 weights -> ternary matrix and scale gamma*delta.

The oracle is pinned to numpy (median / linear-method quantile of |W|, float32 division rounded
half to even) and to the invariants of RoundClip; the library entry point `aecct_aap_ternarize`
(a host step of model creation, no GPU work) must equal the oracle bit for bit.
"""
import numpy as np
import pytest

import oracle


def _matrices():
    """Seeded fp32 matrices with the shapes of the in-block maps (d x d, d x 4d, 4d x d) and
    assorted distributions: Gaussian, uniform, heavy-tailed, with exact zeros and duplicates."""
    rng = np.random.default_rng(11)
    out = []
    for d in (32, 64, 128):
        for shape in ((d, d), (d, 4 * d), (4 * d, d)):
            out.append(rng.standard_normal(shape).astype(np.float32) * 0.05)
    out.append(rng.uniform(-1, 1, (64, 64)).astype(np.float32))
    out.append((rng.standard_t(2, (128, 128)) * 0.02).astype(np.float32))
    z = rng.standard_normal((32, 32)).astype(np.float32)
    z[rng.random(z.shape) < 0.6] = 0.0
    out.append(z)
    dup = rng.choice(np.float32([-0.5, -0.25, 0.0, 0.25, 0.5, 1.0]), (33, 17)).astype(np.float32)
    out.append(dup)
    out.append(np.float32([[-0.0, 0.0, 0.0]]))
    out.append(np.float32([3.0]))
    out.append(np.float32([2.0, -1.0]))
    return out


# ------------------------------------------------------------------------ oracle pins
@pytest.mark.parametrize("i", range(16))
def test_oracle_gamma_is_numpy_median(i):
    w = _matrices()[i]
    t, s = oracle.aap_ternarize(w, p=0.5, delta=1.0, eps=0.0)
    med = np.median(np.abs(w).astype(np.float64))        # exact mean of the two middle values
    assert s == np.float32(med)


@pytest.mark.parametrize("p", [0.0, 0.1, 0.25, 0.9, 1.0])
def test_oracle_gamma_is_numpy_linear_quantile(p):
    for w in _matrices()[:12]:
        t, s = oracle.aap_ternarize(w, p=p, delta=1.0, eps=0.0)
        q = np.quantile(np.abs(w).astype(np.float64), np.float64(np.float32(p)), method="linear")
        assert abs(float(s) - q) <= float(np.spacing(np.float32(q))), (p, s, q)
    w = _matrices()[0]
    assert oracle.aap_ternarize(w, p=0.0, eps=0.0)[1] == np.abs(w).min()
    assert oracle.aap_ternarize(w, p=1.0, eps=0.0)[1] == np.abs(w).max()


@pytest.mark.parametrize("delta,eps", [(1.0, 1e-8), (1.7, 1e-8), (0.3, 0.0), (2.5, 1e-3)])
def test_oracle_ternary_is_numpy_roundclip(delta, eps):
    for w in _matrices():
        t, s = oracle.aap_ternarize(w, p=0.5, delta=delta, eps=eps)
        gamma = np.float32(np.median(np.abs(w).astype(np.float64)))
        assert s == gamma * np.float32(delta)
        den = np.float32(s + np.float32(eps))
        if den == 0:
            ref = np.sign(w)
        else:
            ref = np.clip(np.rint(w / den), -1, 1)                    # float32 division, ties to even
        assert (t == ref.astype(np.int8)).all()
        # invariants of RoundClip: values strictly inside +-den/2 vanish, beyond +-1.5 den clip
        assert set(np.unique(t)) <= {-1, 0, 1}
        if den > 0:
            assert (t[np.abs(w) < den / 2 * (1 - 1e-6)] == 0).all()
            assert (t[w > den * 0.5 * (1 + 1e-6)] == 1).all() and (t[w < -den * 0.5 * (1 + 1e-6)] == -1).all()


def test_oracle_ties_and_degenerate():
    # quotients exactly +-0.5 and +-1.5 round half to even: 0 and +-2 -> clipped to +-1
    w = np.float32([0.5, -0.5, 1.5, -1.5, 1.0, 1.0, 1.0])       # |w| median 1.0
    t, s = oracle.aap_ternarize(w, p=0.5, delta=1.0, eps=0.0)
    assert s == 1.0 and list(t) == [0, 0, 1, -1, 1, 1, 1]
    # all zeros: gamma = 0, scale 0, every entry 0 (eps > 0) or sign rule (eps = 0)
    z = np.zeros((4, 4), np.float32)
    for eps in (1e-8, 0.0):
        t, s = oracle.aap_ternarize(z, eps=eps)
        assert s == 0.0 and (t == 0).all()
    # gamma = 0 with nonzero weights and eps = 0: the sign of each weight
    w = np.float32([0.0, 0.0, 0.0, 2.0, -3.0])
    t, s = oracle.aap_ternarize(w, eps=0.0)
    assert s == 0.0 and list(t) == [0, 0, 0, 1, -1]
    # the paper's observation: a median-based scale leaves about a quarter of Gaussian weights at 0
    g = np.random.default_rng(3).standard_normal(200_000).astype(np.float32)
    t, s = oracle.aap_ternarize(g)
    from math import erf, sqrt
    p0 = erf(0.5 * 0.6744897501960817 / sqrt(2))                   # P(|z| < median|z| / 2)
    assert abs((t == 0).mean() - p0) < 0.005


# ------------------------------------------------------------------------ library parity
def _lib():
    import paper_2410_05911_amd as P
    P.lib()
    return P


@pytest.mark.parametrize("p,delta,eps", [(0.5, 1.0, 1e-8), (0.5, 1.37, 1e-8), (0.25, 0.8, 0.0),
                                         (0.9, 2.0, 1e-6), (0.0, 1.0, 1e-8), (1.0, 0.5, 0.0)])
def test_library_matches_oracle_bit_for_bit(p, delta, eps):
    P = _lib()
    for w in _matrices():
        t_o, s_o = oracle.aap_ternarize(w, p=p, delta=delta, eps=eps)
        t_l, s_l = P.aap_ternarize(w, p, delta, eps)
        assert s_l.tobytes() == s_o.tobytes()
        assert (t_l == t_o).all()
    z = np.float32([0.0, -0.0, 5.0, -2.0])
    assert (P.aap_ternarize(z, 0.25, 1.0, 0.0)[0] == oracle.aap_ternarize(z, p=0.25, eps=0.0)[0]).all()


def test_library_rejects_bad_arguments():
    P = _lib()
    w = np.ones(8, np.float32)
    for p, delta, eps in ((-0.1, 1.0, 0.0), (1.5, 1.0, 0.0), (0.5, 0.0, 0.0), (0.5, -1.0, 0.0),
                          (0.5, float("inf"), 0.0), (0.5, 1.0, -1e-8), (0.5, 1.0, float("nan"))):
        with pytest.raises(P.AecctError) as ei:
            P.aap_ternarize(w, p, delta, eps)
        assert ei.value.status == P.ERR_INVALID_ARG
    bad = w.copy()
    bad[3] = np.nan
    with pytest.raises(P.AecctError):
        P.aap_ternarize(bad)
    with pytest.raises(P.AecctError):
        P.aap_ternarize(np.zeros(0, np.float32))
