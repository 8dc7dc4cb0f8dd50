"""Pins of the float64 QAT oracle (Section 6, second phase; Section 4.1 Eq. 1-3): its hand-written
gradients against torch autograd, finite differences and the inference oracle."""
import copy

import numpy as np
import pytest
import torch

from workloads import CONFIGS, build_workload, random_qat_params
from workloads.configs import parity_check
from workloads.channel import awgn_words
from workloads.codes import generator_from_parity

KINDS = ("q", "k", "v", "o", "ff1", "ff2")


def _problem(c, batch, seed=5, layers=None, zero_codeword=True):
    cfg = CONFIGS[c]
    H = parity_check(cfg)
    m, n = H.shape
    N = cfg.n_layers if layers is None else layers
    p = random_qat_params(n, m, cfg.d, N, seed=seed)
    G = generator_from_parity(H)
    y, x, _ = awgn_words(G, batch, (3.0, 5.0, 7.0), seed=seed + 1)
    xs = None if zero_codeword else (1 - 2 * x.astype(np.int8)).astype(np.float32)
    if zero_codeword:          # the paper trains on the all-zero codeword: y = 1 + noise
        y = (np.abs(y) * np.sign(y) * (1 - 2 * x.astype(np.float32))).astype(np.float32)
    return H, p, y, xs


def _torch_forward(H, p, y, xs, heads, hf, attention, ln_eps=1e-5, aap_eps=1e-8):
    """The same QAT forward in torch float64 with stop-gradients written as detach(): every leaf
    tensor requires grad, and autograd derives the backward independently of the oracle's."""
    import oracle.qat as Q
    dt = torch.float64
    leaf = lambda a: torch.tensor(np.asarray(a, np.float64), dtype=dt, requires_grad=True)
    P = {"embed": leaf(p["embed"]), "w": {k: leaf(p["w"][k]) for k in KINDS},
         "b": {k: leaf(p["b"][k]) for k in KINDS}, "delta": leaf(p["delta"])}
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "head_w1", "head_wo", "head_bo"):
        P[k] = leaf(p[k])
    P["head_b1"] = leaf(np.float64(p["head_b1"]))
    m, n = H.shape
    L = n + m
    d = P["embed"].shape[1]
    N = P["w"]["q"].shape[0]
    dh = d // heads
    masks = [torch.tensor(M) for M in Q.head_masks(H, heads, hf, attention)]
    yt = torch.tensor(y, dtype=dt)
    syn = torch.tensor(((y < 0).astype(np.int64) @ H.astype(np.int64).T) % 2, dtype=dt)
    t = torch.cat([yt.abs(), 1 - 2 * syn], 1)
    X = t[:, :, None] * P["embed"][None]

    def quant(Z):
        a = Z.abs().amax(-1, keepdim=True).detach()
        safe = torch.where(a == 0, torch.ones_like(a), a)
        q = torch.clamp(torch.round(Z * (127.0 / safe)), -127, 127)
        Zq = torch.where(a == 0, torch.zeros_like(Z), q * safe / 127.0)
        return Z + (Zq - Z).detach()

    def lin(Z, l, i, k):
        Wl = P["w"][k][l]
        gamma = torch.quantile(Wl.detach().abs().reshape(-1), 0.5)
        s = gamma * P["delta"][l, i]
        u = Wl / (s + aap_eps)
        T = torch.clamp(torch.round(u), -1, 1)
        That = u + (T - u).detach()
        return (quant(Z) @ That) * s + P["b"][k][l]

    for l in range(N):
        Qm, Km, Vm = (lin(X, l, i, k) for i, k in enumerate(("q", "k", "v")))
        outs = []
        for h in range(heads):
            sl = slice(h * dh, (h + 1) * dh)
            S = Qm[:, :, sl] @ Km[:, :, sl].transpose(1, 2).contiguous() / dh ** 0.5
            S = S.masked_fill(~masks[h][None], float("-inf"))
            outs.append(torch.softmax(S, -1) @ Vm[:, :, sl])
        O = torch.cat(outs, -1)
        X1 = torch.nn.functional.layer_norm(X + lin(O, l, 3, "o"), (d,), P["ln1_g"][l], P["ln1_b"][l], eps=ln_eps)
        G = torch.relu(lin(X1, l, 4, "ff1"))
        X = torch.nn.functional.layer_norm(X1 + lin(G, l, 5, "ff2"), (d,), P["ln2_g"][l], P["ln2_b"][l], eps=ln_eps)
    z = X @ P["head_w1"] + P["head_b1"]
    f = z @ P["head_wo"] + P["head_bo"]
    sgn = torch.ones_like(yt) if xs is None else torch.tensor(xs, dtype=dt)
    target = ((yt * sgn) < 0).to(dt)
    loss = torch.nn.functional.binary_cross_entropy_with_logits(-f, target)
    loss.backward()
    return loss.item(), f.detach().numpy(), P


def _rel(a, b, floor=1e-15):
    """Normwise relative difference, with an absolute floor for gradients that vanish."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), floor / 1e-9))


@pytest.mark.parametrize("c,batch,attention,zero_cw", [(1, 16, "hpsa", True), (1, 16, "casa", False),
                                                        (2, 6, "hpsa", True), (2, 4, "hpsa", False)])
def test_gradients_equal_torch_autograd(c, batch, attention, zero_cw):
    import oracle.qat as Q
    H, p, y, xs = _problem(c, batch, zero_codeword=zero_cw)
    hf = 4
    loss, f, g = Q.forward_backward(H, p, y, xs, heads=8, first_ring_heads=hf, attention=attention)
    tl, tf, P = _torch_forward(H, p, y, xs, 8, hf, attention)
    assert abs(loss - tl) <= 1e-12 * max(1.0, abs(tl))
    assert np.abs(f - tf).max() <= 1e-10
    for k in KINDS:
        assert _rel(g["w"][k], P["w"][k].grad) <= 1e-9, ("w", k)
        assert _rel(g["b"][k], P["b"][k].grad) <= 1e-9, ("b", k)
    assert _rel(g["delta"], P["delta"].grad) <= 1e-9
    for k in ("embed", "ln1_g", "ln1_b", "ln2_g", "ln2_b", "head_w1", "head_wo", "head_bo"):
        assert _rel(g[k], P[k].grad) <= 1e-9, k
    assert abs(g["head_b1"] - P["head_b1"].grad.item()) <= 1e-9 * max(1.0, abs(g["head_b1"]))
    # the straight-through gradients are not trivially zero anywhere
    assert all(np.abs(g["w"][k]).max() > 0 for k in KINDS) and np.abs(g["delta"]).min() > 0
    # the key bias adds q.b_k to every score of a row: the softmax ignores it, its gradient is 0
    assert np.abs(g["b"]["k"]).max() <= 1e-15
    assert np.abs(g["b"]["q"]).max() > 1e-6


def test_finite_differences_after_the_last_quantisation():
    """Between the last quantisation point and the loss the step is smooth: the last layer's
    second bias and LayerNorm, and the head.  Central differences match the oracle's gradients."""
    import oracle.qat as Q
    H, p, y, xs = _problem(2, 5, layers=2)
    loss, f, g = Q.forward_backward(H, p, y, xs)

    def L_of(q):
        return Q.forward_backward(H, q, y, xs, with_grads=False)[0]

    checks = [("b", "ff2", (1, 3)), ("b", "ff2", (1, 17)), ("ln2_g", None, (1, 5)), ("ln2_b", None, (1, 30)),
              ("head_w1", None, (7,)), ("head_wo", None, (12, 4)), ("head_wo", None, (40, 30)), ("head_bo", None, (9,)),
              ("head_b1", None, None)]
    for name, kind, idx in checks:
        h = 1e-5
        qp, qm = copy.deepcopy(p), copy.deepcopy(p)
        if name == "head_b1":
            qp[name], qm[name] = p[name] + h, p[name] - h
            ref = g[name]
        else:
            ap = qp[name][kind] if kind else qp[name]
            am = qm[name][kind] if kind else qm[name]
            ap = ap.astype(np.float64)
            am = am.astype(np.float64)
            ap[idx] += h
            am[idx] -= h
            if kind:
                qp[name][kind], qm[name][kind] = ap, am
            else:
                qp[name], qm[name] = ap, am
            ref = (g[name][kind] if kind else g[name])[idx]
        fd = (L_of(qp) - L_of(qm)) / (2 * h)
        assert abs(fd - ref) <= 1e-6 * max(1e-3, abs(ref)), (name, idx, fd, ref)


@pytest.mark.parametrize("c", [1, 2])
def test_forward_equals_fp64_inference_on_ternary_latents(oracle_mod, c):
    """Latent weights that are exactly scale x ternary, with most entries nonzero, delta = 1 and
    eps = 0: Eq. 1 returns the same ternary matrix and the scale gamma = that scale, so the QAT
    forward is the inference model, and its noise estimate equals the oracle's fp64 decode."""
    import oracle.qat as Q
    from workloads import random_weights
    cfg, H, G, w, y, x = build_workload(c, batch=12)
    m, n = H.shape
    w = random_weights(n, m, cfg.d, cfg.n_layers, 8, p_zero=0.3, seed=17)
    p = random_qat_params(n, m, cfg.d, cfg.n_layers, seed=1)
    p.update(embed=w.embed, ln1_g=w.ln1_g, ln1_b=w.ln1_b, ln2_g=w.ln2_g, ln2_b=w.ln2_b, head_w1=w.head_w1,
             head_b1=w.head_b1, head_wo=w.head_wo, head_bo=w.head_bo)
    p["delta"] = np.ones((cfg.n_layers, 6), np.float32)
    for i, k in enumerate(KINDS):
        p["w"][k] = (w.w[k].astype(np.float32) * w.scale[:, i][:, None, None]).astype(np.float32)
        p["b"][k] = w.b[k]
        for l in range(cfg.n_layers):
            T, s, gamma = Q.aap_ternary(p["w"][k][l].astype(np.float64), 1.0, 0.0)
            assert (T == w.w[k][l]).all() and s == np.float64(w.scale[l, i])
    loss, f, _ = Q.forward_backward(H, p, y, None, aap_eps=0.0, with_grads=False)
    b64, f64 = oracle_mod.OracleModel(H, w).decode_ref64(y)
    assert np.abs(f - f64).max() <= 1e-9
