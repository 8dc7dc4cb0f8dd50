"""QAT forward and backward of AECCT in float64 -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

The second training phase of Section 6: the encoder's in-block linear maps are AAP linear layers
(Section 4.1) whose weights are latent fp32 tensors, ternarised in every forward pass (Eq. 1)
with gamma = Percentile(|W|, 0.5) of the current weights and a learnable factor delta, while
their inputs are absmax-quantised to int8 (Eq. 2) and the product is dequantised as in Eq. 3.
The loss is the cross entropy of the multiplicative noise (Section 3, Section 6).  Only the test
suite may import this module.

Plain numpy, dense (-inf)-masked attention per head, every gradient written out by hand from the
chain rule (no autograd).  Readings where the paper is silent (all stated with the functions):
  - Eq. 2 and Eq. 1 pass gradients straight through their rounding (the quantisation-aware
    training of the cited BitNet line of work): the activation scale alpha and the percentile
    gamma are treated as constants of the step; delta receives the gradient of the scale
    gamma*delta and of the division inside the rounding;
  - the noise estimate f is the logit of "the sign of y is right": bit = bin(y f), so the target
    of the multiplicative noise is z = [y x_s < 0] (x_s the transmitted +-1 word) and the loss is
    the mean over words and bits of BCE-with-logits(-f, z);
  - alpha per token (the inference default), the fixed positional table (if any) is not trained.
Pins (tests/test_qat_oracle.py): every gradient equals torch float64 autograd of the same forward
written with stop-gradients; central finite differences on the parameters between the last
quantisation point and the loss; the forward equals the oracle's fp64 inference decode when the
latent weights are exactly scale x ternary.
"""
from __future__ import annotations

import numpy as np

from . import masks as _masks

KINDS = ("q", "k", "v", "o", "ff1", "ff2")


def head_masks(H, heads, first_ring_heads, attention="hpsa"):
    """Per-head boolean (L, L) masks: HPSA (Section 4.2) gives heads below h_f the first ring and
    the others the second ring; CASA (Section 3) gives every head their union."""
    M1, M2 = _masks(H)
    M1, M2 = M1.astype(bool), M2.astype(bool)
    if attention == "casa":
        return [M1 | M2] * heads
    return [M1 if h < first_ring_heads else M2 for h in range(heads)]


def aap_ternary(W, delta, eps, margins=None):
    """Eq. 1 on latent weights: gamma = the 0.5 quantile of |W| (linear interpolation between
    order statistics), s = gamma * delta, T = RoundClip(W / (s + eps), -1, 1) (half to even).
    margins (dict or None) keeps the least distance of |W / (s + eps)| to the tie 1/2."""
    gamma = float(np.quantile(np.abs(W), 0.5))
    s = gamma * float(delta)
    u = W / (s + eps)
    if margins is not None:
        margins["ternary"] = min(margins.get("ternary", np.inf), float(np.abs(np.abs(u) - 0.5).min()))
    T = np.clip(np.rint(u), -1.0, 1.0)
    return T, s, gamma


def quant_dequant(X, margins=None):
    """Eq. 2 per token row, then back to the value it stands for: q alpha / 127 (0 for alpha 0).
    margins (dict or None) keeps the least distance of a code's x 127 / alpha to a tie k + 1/2."""
    a = np.abs(X).max(-1, keepdims=True)
    safe = np.where(a == 0, 1.0, a)
    u = X * (127.0 / safe)
    if margins is not None:
        margins["act"] = min(margins.get("act", np.inf), float(np.abs(u - (np.floor(u) + 0.5)).min()))
    q = np.clip(np.rint(u), -127, 127)
    return np.where(a == 0, 0.0, q * safe / 127.0)


def layernorm_fwd(R, g, b, eps):
    mu = R.mean(-1, keepdims=True)
    e = R - mu
    var = (e * e).mean(-1, keepdims=True)
    rho = 1.0 / np.sqrt(var + eps)
    xn = e * rho
    return xn * g + b, (xn, rho)


def layernorm_bwd(dy, g, cache):
    """dR, dg, db of out = xn g + b with xn = (R - mean) / sqrt(var + eps)."""
    xn, rho = cache
    dxn = dy * g
    dR = rho * (dxn - dxn.mean(-1, keepdims=True) - xn * (dxn * xn).mean(-1, keepdims=True))
    return dR, (dy * xn).reshape(-1, xn.shape[-1]).sum(0), dy.reshape(-1, xn.shape[-1]).sum(0)


def _linear_bwd(dY, Xh, W, T, s, gamma, eps):
    """Eq. 3 with the straight-through Eq. 1: Y = (Xh That) s + b, That = u + sg(T - u),
    u = W / (s + eps), s = sg(gamma) delta.  Returns dXh, dW, d delta, db."""
    K, nout = W.shape
    Gm = Xh.reshape(-1, K).T @ dY.reshape(-1, nout)                 # Xh^T dY, [K][out]
    dW = Gm * (s / (s + eps))
    ddelta = gamma * float((Gm * T).sum()) - s * gamma / (s + eps) ** 2 * float((Gm * W).sum())
    dXh = (dY @ T.T) * s
    return dXh, dW, ddelta, dY.reshape(-1, nout).sum(0)


def forward_backward(H, p, y, xs=None, *, heads=8, first_ring_heads=None, attention="hpsa", ln_eps=1e-5,
                     aap_eps=1e-8, with_grads=True, margins=None):
    """One QAT step's loss and gradients on a batch.

    p: dict with embed [L, d], pos [L, d] or None, w[kind] [N, in, out] latent weights, delta
    [N, 6], b[kind] [N, out], ln1_g, ln1_b, ln2_g, ln2_b [N, d], head_w1 [d], head_b1 (float),
    head_wo [L, n], head_bo [n].  y: [B, n] channel outputs; xs: [B, n] transmitted +-1 words
    (None: the all-zero codeword, x_s = +1).
    Returns (loss, f [B, n], grads dict with the keys of p except pos; None without grads).
    margins: a dict that receives the least distance of any rounding decision to its tie:
    "act" (Eq. 2, in code units) and "ternary" (Eq. 1, |W| / (s + eps) against 1/2).
    """
    f64 = np.float64
    H = np.asarray(H, np.int64)
    m, n = H.shape
    L = n + m
    E = np.asarray(p["embed"], f64)
    d = E.shape[1]
    N = np.asarray(p["w"]["q"]).shape[0]
    dh = d // heads
    hf = heads // 2 if first_ring_heads is None else first_ring_heads
    y = np.asarray(y, np.float32)
    B = y.shape[0]
    masks = head_masks(H, heads, hf, attention)
    W = {k: np.asarray(p["w"][k], f64) for k in KINDS}
    bias = {k: np.asarray(p["b"][k], f64) for k in KINDS}
    delta = np.asarray(p["delta"], f64)
    ln = {k: np.asarray(p[k], f64) for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b")}

    # pre-processing h(y) = [|y|, 1 - 2 s(y)] and the embedding (Section 3)
    syn = ((y < 0).astype(np.int64) @ H.T) % 2
    t = np.concatenate([np.abs(y).astype(f64), 1.0 - 2.0 * syn], 1)           # [B, L]
    X = t[:, :, None] * E[None]
    if p.get("pos") is not None:
        X = X + np.asarray(p["pos"], f64)[None]

    cache = []
    for l in range(N):
        c = {"X": X}
        tern = [aap_ternary(W[k][l], delta[l, i], aap_eps, margins) for i, k in enumerate(KINDS)]
        c["tern"] = tern
        Xh = quant_dequant(X, margins)
        c["Xh"] = Xh
        QKV = [(Xh @ tern[i][0]) * tern[i][1] + bias[k][l] for i, k in enumerate(("q", "k", "v"))]
        c["QKV"] = QKV
        Q, K, V = QKV
        O = np.zeros_like(Q)
        P = []
        for h in range(heads):
            sl = slice(h * dh, (h + 1) * dh)
            S = Q[:, :, sl] @ K[:, :, sl].transpose(0, 2, 1) / np.sqrt(dh)
            S = np.where(masks[h][None], S, -np.inf)
            S = S - S.max(-1, keepdims=True)
            Pe = np.exp(S)
            Ph = Pe / Pe.sum(-1, keepdims=True)
            P.append(Ph)
            O[:, :, sl] = Ph @ V[:, :, sl]
        c["P"], c["O"] = P, O
        Oh = quant_dequant(O, margins)
        c["Oh"] = Oh
        R1 = X + (Oh @ tern[3][0]) * tern[3][1] + bias["o"][l]
        X1, c["ln1"] = layernorm_fwd(R1, ln["ln1_g"][l], ln["ln1_b"][l], ln_eps)
        c["X1"] = X1
        X1h = quant_dequant(X1, margins)
        c["X1h"] = X1h
        F = (X1h @ tern[4][0]) * tern[4][1] + bias["ff1"][l]
        c["F"] = F
        G = np.maximum(F, 0.0)
        Gh = quant_dequant(G, margins)
        c["Gh"] = Gh
        R2 = X1 + (Gh @ tern[5][0]) * tern[5][1] + bias["ff2"][l]
        X, c["ln2"] = layernorm_fwd(R2, ln["ln2_g"][l], ln["ln2_b"][l], ln_eps)
        cache.append(c)

    # head (Section 3) and the loss of the multiplicative noise (Section 6)
    w1 = np.asarray(p["head_w1"], f64)
    Wo = np.asarray(p["head_wo"], f64)
    z = X @ w1 + float(p["head_b1"])                                            # [B, L]
    f = z @ Wo + np.asarray(p["head_bo"], f64)                                  # [B, n]
    sgn = np.ones_like(y) if xs is None else np.asarray(xs, np.float32)
    target = ((y * sgn) < 0).astype(f64)
    loss = float(np.mean(np.logaddexp(0.0, -f) + target * f))
    if not with_grads:
        return loss, f, None

    g = {"w": {k: np.zeros_like(W[k]) for k in KINDS}, "b": {k: np.zeros_like(bias[k]) for k in KINDS},
         "delta": np.zeros_like(delta)}
    for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        g[k] = np.zeros_like(ln[k])
    df = (target - 1.0 / (1.0 + np.exp(f))) / (B * n)                          # d/df of the mean BCE
    g["head_bo"] = df.sum(0)
    g["head_wo"] = z.T @ df
    dz = df @ Wo.T
    g["head_b1"] = float(dz.sum())
    g["head_w1"] = (dz[:, :, None] * X).reshape(-1, d).sum(0)
    dX = dz[:, :, None] * w1

    for l in reversed(range(N)):
        c = cache[l]
        tern = c["tern"]

        def lin(dY, Xh, i, kind):
            T, s, gamma = tern[i]
            dXh, dW, dd, db = _linear_bwd(dY, Xh, W[kind][l], T, s, gamma, aap_eps)
            g["w"][kind][l] = dW
            g["delta"][l, i] = dd
            g["b"][kind][l] = db
            return dXh

        dR2, g["ln2_g"][l], g["ln2_b"][l] = layernorm_bwd(dX, ln["ln2_g"][l], c["ln2"])
        dX1 = dR2.copy()
        dGh = lin(dR2, c["Gh"], 5, "ff2")
        dF = dGh * (c["F"] > 0)                                                # ReLU; Eq. 2 passes straight
        dX1 += lin(dF, c["X1h"], 4, "ff1")
        dR1, g["ln1_g"][l], g["ln1_b"][l] = layernorm_bwd(dX1, ln["ln1_g"][l], c["ln1"])
        dX = dR1.copy()
        dO = lin(dR1, c["Oh"], 3, "o")
        Q, K, V = c["QKV"]
        dQ, dK, dV = np.zeros_like(Q), np.zeros_like(K), np.zeros_like(V)
        for h in range(heads):
            sl = slice(h * dh, (h + 1) * dh)
            Ph = c["P"][h]
            dOh = dO[:, :, sl]
            dV[:, :, sl] = Ph.transpose(0, 2, 1) @ dOh
            dP = dOh @ V[:, :, sl].transpose(0, 2, 1)
            dS = Ph * (dP - (Ph * dP).sum(-1, keepdims=True)) / np.sqrt(dh)
            dQ[:, :, sl] = dS @ K[:, :, sl]
            dK[:, :, sl] = dS.transpose(0, 2, 1) @ Q[:, :, sl]
        for i, (kind, dY) in enumerate((("q", dQ), ("k", dK), ("v", dV))):
            dX += lin(dY, c["Xh"], i, kind)
    g["embed"] = (t[:, :, None] * dX).sum(0)
    return loss, f, g
